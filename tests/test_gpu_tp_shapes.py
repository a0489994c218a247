"""Parity at the shapes one tensor-parallel rank of Llama-3.1-70B holds
(TP 2, 4, 8: 32/16/8 query heads, 4/2/1 kv heads, FFN 14336/7168/3584),
in the launch configurations of the static-batch sweep: a 2048-token
prefill step of 763-token prompts (two whole and one split) and a decode
step of 32 sequences with contexts 763-994. Sampled rows against the exact
oracle, each given the stage's keys/values of its earlier positions."""

from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2606_18600_amd import synth
from paper_2606_18600_amd.estimator import tp_shard
from paper_2606_18600_amd.harness import DeviceStage, device_layer_weights, model_config, pack_layer
from tests.gpu_pair import log
from tests.test_gpu_fullsize import _check_rows_one_layer, _host64, _sample_rows

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("tp", [2, 4, 8])
def test_tp_shard_layer_sampled(tp):
    seed, layer = 2620 + tp, 7
    shape = tp_shard(synth.LLAMA70B, tp)
    log(f"{shape.name}: one layer, prefill step 763+763+522 and decode batch 32")
    cfg = model_config(shape, "bf16")
    w = device_layer_weights(shape, seed, layer, "bf16")
    w64 = _host64(w)
    pc = np.array([0, 0, 0], np.int32)
    pq = np.array([763, 763, 522], np.int32)
    dctx = synth.uniform_lengths(seed, 3, 32, 763, 994)
    alloc = synth.BlockAllocator(int(((pq + 15) // 16).sum() + ((dctx + 16) // 16).sum()) + 4,
                                 seed)
    pbt_np = synth.make_block_tables(pc + pq, 48, alloc)
    dbt_np = synth.make_block_tables(dctx + 1, 63, alloc)
    nb = int(max(pbt_np.max(), dbt_np.max())) + 1
    st = DeviceStage(shape, "bf16", layer, [pack_layer(cfg, w)], nb, 2048, 32, packed=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    rng = np.random.default_rng(seed)
    try:
        st.kv_pool.normal_(0.0, 1.0, generator=g)  # decode contexts
        x = torch.randn((2048, shape.hidden), generator=g, device="cuda").to(torch.bfloat16)
        y = st.prefill(pq, pc, torch.from_numpy(pbt_np).cuda(), x)
        torch.cuda.synchronize()
        _check_rows_one_layer(shape, st, w64, pbt_np, _sample_rows(rng, pq, pc, 6),
                              x.double().cpu().numpy(), y.double().cpu().numpy(), "prefill rows")
        xd = x[:32].contiguous()
        yd = st.decode(dctx, torch.from_numpy(dbt_np).cuda(), xd)
        torch.cuda.synchronize()
        pick = sorted({0, 31, int(np.argmax(dctx))} | set(rng.choice(32, 4, replace=False).tolist()))
        _check_rows_one_layer(shape, st, w64, dbt_np, [(j, int(dctx[j]), j) for j in pick],
                              xd.double().cpu().numpy(), yd.double().cpu().numpy(), "decode rows")
    finally:
        st.close()
