"""The 80-layer Llama-3.1-70B-shaped model as four 20-layer stages over the
same weights and KV pool (GPU): parity at the depth of the full-model
workload.

Through 20 random bf16 layers the storage floor (the oracle with bf16
rounding emulated at the stage's rounding points, against the exact oracle)
already exceeds 2e-2, and it keeps growing with depth. Stage composition
(pinned in the oracle: [l0, m) then [m, l1) equals [l0, l1)) lets each
20-layer sub-range be checked on its own, fed the GPU's own hidden state at
its boundary, which is what a pipeline stage receives anyway.

Two steps in the workload's launch configurations: a decode step of batch
128 (contexts uniform 1024..4096) and a mixed step of those 128 decodes plus
2048 prefill tokens (a continuation chunk of 1500 tokens behind 500 cached
ones, and a fresh 548-token prompt). For three sampled decode sequences,
whose contexts were written by the stages' own chunked prefill, the oracle
runs each sub-range's 20 layers from the GPU boundary state and the stages'
context KV, exactly (fp64) and with bf16 storage emulated. Bar per sub-range:
max(2e-2, 1.25 x floor) on the outputs, against both; the new K/V of each
sub-range's first layer (where the oracle and the stage see the same input)
within 2e-2. The oracle reads the stored weights: each layer is regenerated
from its seed and checked, after packing, to equal what the stage holds.
"""

from __future__ import annotations

import time

import numpy as np
import pytest
import torch

from oracle import stage_oracle as O
from paper_2606_18600_amd import synth
from paper_2606_18600_amd.harness import (DeviceStage, device_layer_weights, model_config,
                                          pack_layer)
from tests.gpu_pair import gpu_kv_to_oracle_layout, log
from tests.helpers import ocfg, rel_l2

pytestmark = pytest.mark.gpu
TOL = 2e-2
SEED = 2690
PACKED = ("w_qkv", "w_o", "w_gate_up", "w_down")


def _sample_cache(st, li, bt_row, n_tok):
    """Layer li of a stage: the blocks holding a sequence's first n_tok
    positions, in the oracle's layout (blocks renumbered 0..)."""
    nb = (n_tok + 15) // 16
    ids = torch.tensor([int(b) for b in bt_row[:nb]], dtype=torch.long, device="cuda")
    return gpu_kv_to_oracle_layout(st.kv_view()[li:li + 1, ids])[0]


@pytest.fixture(scope="module")
def depth_run():
    """The GPU part: 80 layers as four 20-layer stages, the sampled
    sequences' contexts written by the stages' chunked prefill, then a
    decode step and a mixed step through all four; the boundary hidden
    states of the sampled rows."""
    shape, nL, per, B = synth.LLAMA70B, 80, 20, 128
    H = shape.hidden
    cfg = model_config(shape, "bf16")
    t0 = time.time()
    log("[test] l70 80 layers as 4 x 20 layers: generating and packing weights")
    packed = [pack_layer(cfg, device_layer_weights(shape, SEED, l, "bf16"), free_source=True)
              for l in range(nL)]
    ctx = synth.uniform_lengths(SEED, 1, B, 1024, 4096)
    sample = [int(np.argmin(ctx)), int(np.argmax(ctx)), 37]
    pc = np.array([500, 0], np.int32)
    pq = np.array([1500, 548], np.int32)
    nblk_d = (ctx + 2 + 15) // 16
    nblk_p = (pc + pq + 15) // 16
    nblocks = int(nblk_d.sum() + nblk_p.sum()) + 4
    alloc = synth.BlockAllocator(nblocks, SEED)
    dbt_np = synth.make_block_tables(ctx + 2, int(nblk_d.max()), alloc)
    pbt_np = synth.make_block_tables(pc + pq, int(nblk_p.max()), alloc)
    dbt, pbt = torch.from_numpy(dbt_np).cuda(), torch.from_numpy(pbt_np).cuda()
    layer_numel = nblocks * shape.n_kv_heads * 2 * 16 * shape.head_dim
    log(f"  KV pool: {nblocks} blocks x {nL} layers = {nL * layer_numel * 2 / 1e9:.1f} GB")
    pool = torch.empty(nL * layer_numel, dtype=torch.bfloat16, device="cuda")
    g = torch.Generator(device="cuda")
    g.manual_seed(SEED)
    pool.normal_(0.0, 1.0, generator=g)   # contexts of the unsampled sequences
    stages = [DeviceStage(shape, "bf16", k * per, packed[k * per:(k + 1) * per], nblocks, 2176,
                          B + 2, packed=True,
                          kv_pool=pool[k * per * layer_numel:(k + 1) * per * layer_numel])
              for k in range(nL // per)]
    try:
        log(f"  context prefill of sequences {sample} ({[int(ctx[s]) for s in sample]} tokens)")
        for s in sample:
            done = 0
            while done < ctx[s]:
                q = int(min(2048, ctx[s] - done))
                x = torch.randn((q, H), generator=g, device="cuda").to(torch.bfloat16)
                for st in stages:
                    x = st.prefill([q], [done], dbt[s:s + 1].contiguous(), x)
                done += q
        log("  decode step (batch 128) and mixed step (2048 prefill + 128 decodes)")
        b1 = [torch.randn((B, H), generator=g, device="cuda").to(torch.bfloat16)]
        for st in stages:
            b1.append(st.decode(ctx, dbt, b1[-1]))
        b2 = [torch.randn((2048 + B, H), generator=g, device="cuda").to(torch.bfloat16)]
        for st in stages:
            b2.append(st.mixed(pq, pc, pbt, ctx + 1, dbt, b2[-1]))
        torch.cuda.synchronize()
        # boundary hidden states of the sampled rows: [stage boundary][row]
        rows1 = [b[sample].double().cpu().numpy() for b in b1]
        rows2 = [b[[2048 + s for s in sample]].double().cpu().numpy() for b in b2]
        del b1, b2
        log(f"  GPU part done in {time.time() - t0:.0f} s")
        yield dict(shape=shape, cfg=cfg, per=per, packed=packed, stages=stages, ctx=ctx,
                   sample=sample, dbt_np=dbt_np, rows1=rows1, rows2=rows2)
    finally:
        for st in stages:
            st.close()


# one test per sub-range, so that each runs its 20 oracle layers (about a
# minute) on its own
@pytest.mark.parametrize("k", [0, 1, 2, 3])
def test_l70_80_layers_as_four_20_layer_stages(depth_run, k):
    d = depth_run
    shape, cfg, per, packed = d["shape"], d["cfg"], d["per"], d["packed"]
    ctx, sample, dbt_np, rows1, rows2 = d["ctx"], d["sample"], d["dbt_np"], d["rows1"], d["rows2"]
    st = d["stages"][k]
    t0 = time.time()
    oc = ocfg(shape)
    nS = len(sample)
    # rows of both steps in one oracle batch: step 1 (position ctx), then
    # step 2 (position ctx + 1), each with its own cache copy
    x0 = np.concatenate([rows1[k], rows2[k]])
    x_ex, x_em = x0, x0
    pos = [int(ctx[s]) for s in sample] + [int(ctx[s]) + 1 for s in sample]
    for li in range(per):
        l = k * per + li
        rm = device_layer_weights(shape, SEED, l, "bf16")
        again = pack_layer(cfg, rm)
        for name in PACKED:
            assert torch.equal(again[name], packed[l][name]), (l, name)
        del again
        w64 = {n: v.to(torch.float64).cpu().numpy() for n, v in rm.items()}
        del rm
        parts = [_sample_cache(st, li, dbt_np[s], int(ctx[s]) + 2) for s in sample]
        seqs, base = [], 0
        kk, vv = [], []
        for j in range(2 * nS):          # step-1 copies, then step-2 copies
            c = parts[j % nS]
            kk.append(c["k"])
            vv.append(c["v"])
            nb = c["k"].shape[0]
            seqs.append(O.SeqSpec(pos[j], 1, list(range(base, base + nb))))
            base += nb
        gpu_k = [(c["k"][p // 16, p % 16].copy(), c["v"][p // 16, p % 16].copy())
                 for c, p in zip(parts + parts, pos)]
        cache_ex = {"k": np.concatenate(kk), "v": np.concatenate(vv)}
        cache_em = {"k": cache_ex["k"].copy(), "v": cache_ex["v"].copy()}
        x_ex = O.layer_forward(oc, w64, x_ex, seqs, cache_ex)
        x_em = O.layer_forward(oc, w64, x_em, seqs, cache_em, rounding=O.round_to_bf16)
        del w64
        if li == 0:
            for j, sp in enumerate(seqs):
                p = sp.ctx_len
                b, o = sp.block_table[p // 16], p % 16
                ek = rel_l2(gpu_k[j][0], cache_ex["k"][b, o])
                ev = rel_l2(gpu_k[j][1], cache_ex["v"][b, o])
                assert ek <= TOL and ev <= TOL, (k, j, ek, ev)
    for j in range(2 * nS):
        gpu = (rows1 if j < nS else rows2)[k + 1][j % nS]
        e_ex, e_em = rel_l2(gpu, x_ex[j]), rel_l2(gpu, x_em[j])
        floor = rel_l2(x_em[j], x_ex[j])
        s = sample[j % nS]
        log(f"  layers [{k * per}, {(k + 1) * per}) step {1 + j // nS} seq {s} "
            f"ctx {int(ctx[s])}: vs exact {e_ex:.3e}, vs bf16-emulated {e_em:.3e}, "
            f"floor {floor:.3e}")
        assert e_ex <= max(TOL, 1.25 * floor), (k, j, e_ex, floor)
        assert e_em <= max(TOL, 1.25 * floor), (k, j, e_em, floor)
    log(f"  sub-range {k} done in {time.time() - t0:.0f} s")
