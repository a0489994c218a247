"""Parity of the last stage's LM head (final RMSNorm + logits projection,
stage_lm_head) with the oracle's lm_head, on the stored weights and inputs.
Small shapes are compared in full (both GEMM paths: <= 128 rows split-K,
more rows tiled; selected rows with repeats and the identity selection);
the Llama-3.1-70B head (vocab 128256) on every row and a sample of vocabulary
columns (the oracle restricted to those rows of W_lm)."""

from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import stage_oracle as O
from paper_2606_18600_amd import synth
from paper_2606_18600_amd.harness import (DeviceStage, device_layer_weights, model_config,
                                          pack_lm_head, torch_dtype, upload_weights)
from tests.gpu_pair import log
from tests.helpers import ocfg, rel_l2

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


def _stage(shape, dtype, seed, max_tokens):
    w = [upload_weights(synth.host_layer_weights(shape, seed, 0), dtype)]
    return DeviceStage(shape, dtype, 0, w, 8, max_tokens, 4)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n_hidden,rows", [
    (40, [39, 0, 17, 17, 5]),          # selected rows, one repeated
    (40, None),                        # rows 0..39
    (200, list(range(199, 69, -1))),   # 130 rows: the tiled GEMM in bf16
])
def test_lm_head_small(dtype, n_hidden, rows):
    seed, shape, V = 2641, synth.TINY, 1024
    rng = np.random.default_rng(seed)
    td = torch_dtype(dtype)
    x = torch.from_numpy(rng.standard_normal((n_hidden, shape.hidden))).to("cuda", td)
    g = torch.from_numpy(rng.uniform(0.5, 1.5, shape.hidden)).to("cuda", td)
    w = torch.from_numpy(rng.standard_normal((V, shape.hidden)) / 16).to("cuda", td)
    st = _stage(shape, dtype, seed, 256)
    try:
        wp = pack_lm_head(st.cfg, w)
        y = st.lm_head(g, wp, x, rows=rows)
        torch.cuda.synchronize()
        sel = list(range(n_hidden)) if rows is None else rows
        x64 = x.double().cpu().numpy()[sel]
        ref = O.lm_head(ocfg(shape), x64, g.double().cpu().numpy(), w.double().cpu().numpy())
        e = rel_l2(y.double().cpu().numpy(), ref)
        log(f"  tiny {dtype} {len(sel)} rows of {n_hidden}: rel_l2 {e:.3e}")
        assert e <= TOL[dtype]
    finally:
        st.close()


def test_lm_head_rejects_bad_rows():
    from paper_2606_18600_amd.stage import STAGE_ERR_INVALID_ARG, StageError
    shape = synth.TINY
    st = _stage(shape, "bf16", 1, 64)
    try:
        x = torch.zeros((10, shape.hidden), dtype=torch.bfloat16, device="cuda")
        g = torch.ones(shape.hidden, dtype=torch.bfloat16, device="cuda")
        w = torch.zeros((128, shape.hidden), dtype=torch.bfloat16, device="cuda")
        for bad in ([0, 10], [-1]):
            with pytest.raises(StageError) as ei:
                st.lm_head(g, w, x, rows=bad)
            assert ei.value.code == STAGE_ERR_INVALID_ARG
    finally:
        st.close()


@pytest.mark.parametrize("n_rows", [64, 8, 200])
def test_lm_head_l70_sampled_columns(n_rows):
    """64 decode rows and 8 last-of-prompt rows (split-K GEMM), 200 rows
    (tiled GEMM); every row, 2048 sampled vocabulary columns plus the first
    and last."""
    seed, shape, V = 2642, synth.LLAMA70B, 128256
    log(f"l70 LM head, {n_rows} rows, vocab {V}")
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    w = torch.empty((V, shape.hidden), dtype=torch.bfloat16, device="cuda").normal_(0, 0.02,
                                                                                   generator=g)
    gain = torch.empty(shape.hidden, device="cuda").normal_(1.0, 0.02, generator=g).to(torch.bfloat16)
    x = torch.randn((256, shape.hidden), generator=g, device="cuda").to(torch.bfloat16)
    rng = np.random.default_rng(seed)
    rows = None if n_rows == 200 else sorted(rng.choice(256, n_rows, replace=False).tolist())
    cfg = model_config(shape, "bf16")
    # the last layer of the stage that owns the workspace
    st = DeviceStage(shape, "bf16", 79, [device_layer_weights(shape, seed, 79, "bf16")], 8, 256, 4)
    try:
        wp = pack_lm_head(cfg, w)
        y = st.lm_head(gain, wp, x, rows=rows, n_rows=n_rows)
        torch.cuda.synchronize()
        cols = np.unique(np.concatenate([[0, V - 1], rng.choice(V, 2048, replace=False)]))
        sel = list(range(n_rows)) if rows is None else rows
        ref = O.lm_head(ocfg(shape), x.double().cpu().numpy()[sel], gain.double().cpu().numpy(),
                        w[torch.from_numpy(cols).cuda()].double().cpu().numpy())
        got = y[:, torch.from_numpy(cols).cuda()].double().cpu().numpy()
        e = rel_l2(got, ref)
        log(f"  {n_rows} rows x {len(cols)} sampled columns: rel_l2 {e:.3e}")
        assert e <= TOL["bf16"]
        assert torch.isfinite(y).all()
    finally:
        st.close()
