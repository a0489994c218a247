"""stage_decode_noalloc (GPU): the decode entry point that runs over the
library's static scratch array instead of a bound workspace.

Each case runs two stages over the same weights and identical KV pools: one
through stage_decode (bound workspace), one through stage_decode_noalloc.
Both paths launch the same deterministic kernels, so outputs and every byte
of the KV pools must be equal. Two calls in a row, the second with a smaller
batch; the tiny case is also checked against the oracle (relative L2 <= 2e-2
in bf16, <= 1e-4 in fp32). The noalloc stage's bound workspace is filled
with NaN bytes before its first noalloc call, so a read of it would show.
"""

from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2606_18600_amd import stage as S
from paper_2606_18600_amd import synth
from paper_2606_18600_amd.harness import (DeviceStage, device_layer_weights, model_config,
                                          pack_layer)
from tests.gpu_pair import Pair, log
from tests.helpers import rel_l2

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}
OTHER = synth.ModelShape("tiny-theta1e4", hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                         ffn=704, rms_eps=1e-5, rope_theta=1e4)


def _poison(st: DeviceStage) -> None:
    st.workspace.fill_(0xFF)      # bf16/fp32 NaN bit patterns everywhere


class _Case:
    """A reference Pair (stage_decode + oracle) and a noalloc twin stage."""

    def __init__(self, shape, dtype, seed):
        self.shape, self.dtype, self.seed = shape, dtype, seed
        self.lens = synth.uniform_lengths(seed, 0, 6, 16, 64)
        self.bt_np = synth.make_block_tables(self.lens + 4, 8, synth.BlockAllocator(64, seed))
        self.bt = torch.from_numpy(self.bt_np).cuda()
        self.pair = Pair(shape, dtype, 2, 64, 512, 8, seed)
        self.twin = DeviceStage(shape, dtype, 0, self.pair.dev_w, 64, 512, 8)
        x = synth.hidden_states(seed, 1, int(self.lens.sum()), shape.hidden)
        y, yr, _ = self.pair.prefill(self.lens, np.zeros(6, np.int32), self.bt_np, x)
        assert rel_l2(y, yr) <= TOL[dtype]
        xt = torch.from_numpy(x).to("cuda", self.pair.td)
        self.twin.prefill(self.lens, np.zeros(6, np.int32), self.bt, xt)
        torch.cuda.synchronize()
        assert torch.equal(self.twin.kv_pool, self.pair.gpu.kv_pool)
        _poison(self.twin)

    def step(self, k, rows):
        """One decode of sequences `rows` on both paths; bitwise comparison
        and the oracle check of the reference."""
        ctx = (self.lens[rows] + k).astype(np.int32)
        bt_np = self.bt_np[rows].copy()
        x = synth.hidden_states(self.seed, 10 + k, len(rows), self.shape.hidden)
        y, yr, _ = self.pair.decode(ctx, bt_np, x)
        xt = torch.from_numpy(x).to("cuda", self.pair.td)
        y_na = self.twin.decode_noalloc(ctx, torch.from_numpy(bt_np).cuda(), xt)
        torch.cuda.synchronize()
        e = rel_l2(y_na.double().cpu().numpy(), yr)
        log(f"  {self.shape.name} {self.dtype} call {k} ({len(rows)} seqs): "
            f"noalloc vs oracle rel_l2 {e:.3e}")
        assert e <= TOL[self.dtype]
        assert np.array_equal(y_na.double().cpu().numpy(), y), "outputs differ from stage_decode"
        assert torch.equal(self.twin.kv_pool, self.pair.gpu.kv_pool), "KV pools differ"

    def close(self):
        self.twin.close()
        self.pair.close()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_decode_matches_stage_decode_tiny(dtype):
    """Two tiny stages with different rotary bases alternate on the shared
    array (each call re-uploads its table); 6 sequences, then 3."""
    log(f"[test] noalloc tiny dtype={dtype}")
    a = _Case(synth.TINY, dtype, 2606)
    b = _Case(OTHER, dtype, 2607)
    try:
        a.step(0, [0, 1, 2, 3, 4, 5])
        b.step(0, [0, 1, 2, 3, 4, 5])
        a.step(1, [1, 3, 4])
        b.step(1, [5, 0, 2])
    finally:
        a.close()
        b.close()


def test_noalloc_decode_matches_stage_decode_l70_layer():
    """One Llama-3.1-70B-shaped layer at the decode batch of 64 (contexts
    512..2048), then 40 of those sequences: bitwise equal to stage_decode."""
    seed, shape, layer, B = 2611, synth.LLAMA70B, 20, 64
    log("[test] noalloc l70 layer, batch 64 then 40")
    cfg = model_config(shape, "bf16")
    w = pack_layer(cfg, device_layer_weights(shape, seed, layer, "bf16"))
    ctx = synth.uniform_lengths(seed, 1, B, 512, 2048)
    nblocks = int(((ctx + 17) // 16).sum()) + 8
    bt_np = synth.make_block_tables(ctx + 2, int((ctx.max() + 17) // 16),
                                    synth.BlockAllocator(nblocks, seed))
    ref = DeviceStage(shape, "bf16", layer, [w], nblocks, B, B, packed=True)
    na = DeviceStage(shape, "bf16", layer, [w], nblocks, B, B, packed=True)
    log(f"  workspace {S.stage_workspace_bytes(na.handle)} bytes")
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    try:
        ref.kv_pool.normal_(0.0, 1.0, generator=g)
        na.kv_pool.copy_(ref.kv_pool)
        _poison(na)
        for k, rows in enumerate([np.arange(B), np.sort(np.random.default_rng(seed).choice(
                B, 40, replace=False))]):
            bt = torch.from_numpy(bt_np[rows].copy()).cuda()
            c = (ctx[rows] + k).astype(np.int32)
            x = torch.randn((len(rows), shape.hidden), generator=g, device="cuda").to(
                torch.bfloat16)
            y = ref.decode(c, bt, x)
            y_na = na.decode_noalloc(c, bt, x)
            torch.cuda.synchronize()
            log(f"  call {k}: {len(rows)} seqs, equal={torch.equal(y, y_na)}")
            assert torch.isfinite(y_na.float()).all()
            assert torch.equal(y, y_na), f"call {k}: outputs differ"
            assert torch.equal(ref.kv_pool, na.kv_pool), f"call {k}: KV pools differ"
    finally:
        ref.close()
        na.close()


def test_noalloc_rejects_a_workspace_beyond_the_array():
    """A stage sized for 2048-token steps needs more than the static array:
    STAGE_ERR_CAPACITY, and nothing is written."""
    seed, shape = 2612, synth.LLAMA70B
    log("[test] noalloc capacity error")
    cfg = model_config(shape, "bf16")
    w = pack_layer(cfg, device_layer_weights(shape, seed, 20, "bf16"))
    st = DeviceStage(shape, "bf16", 20, [w], 16, 2048, 64, packed=True)
    try:
        assert S.stage_workspace_bytes(st.handle) > 128 << 20
        bt = torch.zeros((2, 4), dtype=torch.int32, device="cuda")
        x = torch.zeros((2, shape.hidden), dtype=torch.bfloat16, device="cuda")
        out = torch.full_like(x, 7.0)
        with pytest.raises(S.StageError) as e:
            st.decode_noalloc([3, 5], bt, x, out)
        assert e.value.code == S.STAGE_ERR_CAPACITY
        assert "static scratch" in str(e.value)
        torch.cuda.synchronize()
        assert (out == 7.0).all()
    finally:
        st.close()
