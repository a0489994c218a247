"""Parity at the model-sized shapes (GPU), on outputs the oracle can compute
one by one.

* Llama-3.1-70B-shaped decode step, 20 layers [20, 40), batch 64, contexts
  uniform 512..2048, shuffled block tables: the launch configuration the
  bench times. For sampled sequences the oracle runs all 20 layers (fp64)
  from a snapshot of those sequences' context KV (written by the stage's own
  chunked prefill beforehand), and checks the output rows and every KV entry
  the step wrote.
* Llama-70B-shaped chunked prefill (a 2048-token chunk, then a 952-token
  continuation) and the Qwen3-32B-shaped mixed step (4 x 512 prefill chunks
  with prefixes 0/512/1024/1536 + 128 decodes, contexts 256..4096): one layer
  at a time, each sampled row checked by the oracle given the keys/values of
  its earlier positions (from the stage), together with its own new K/V.

Tolerance: relative L2 <= 2e-2 (bf16 mode) per layer. Through the 20-layer
stage the bf16 storage floor (the oracle with bf16 rounding emulated, against
the exact oracle) is itself about 2.8e-2; the end-to-end check allows 1.25x
that floor.
"""

from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import stage_oracle as O
from paper_2606_18600_amd import synth
from paper_2606_18600_amd.harness import (DeviceStage, device_layer_weights,
                                          model_config, pack_layer)
from tests.gpu_pair import gpu_kv_to_oracle_layout, kv_plane_index, log
from tests.helpers import ocfg, rel_l2

pytestmark = pytest.mark.gpu
TOL = 2e-2


def _host64(w):
    return {k: v.detach().to(torch.float64).cpu().numpy() for k, v in w.items()}


def _seq_cache(st, bt_row, n_tok):
    """Per layer, the oracle's cache for one sequence: the blocks holding its
    first n_tok positions, gathered on the device and converted, renumbered
    0.. (plus one spare block for the position the oracle writes)."""
    nb = (n_tok + 15) // 16
    ids = torch.tensor(list(bt_row[:nb]), dtype=torch.long, device="cuda")
    per_layer = gpu_kv_to_oracle_layout(st.kv_view()[:, ids])
    out = []
    for c in per_layer:
        spare = np.zeros((1,) + c["k"].shape[1:])
        out.append(({"k": np.concatenate([c["k"], spare]), "v": np.concatenate([c["v"], spare])},
                    list(range(nb + 1))))
    return out


def _kv_at(cache, table, p):
    return cache["k"][table[p // 16], p % 16], cache["v"][table[p // 16], p % 16]


def _check_all_written_kv(shape, st, w64, tables, ctx_lens, q_lens, x_in, tag, chunk=2048):
    """Every K/V entry a one-layer call wrote (all of its rows), against the
    oracle's own projection of the call's input rows (O.project_qkv: RMSNorm,
    QKV projection, q/k-norm, RoPE, from the stored weights). Checked row by
    row, so one wrong token cannot hide in a large call."""
    oc = ocfg(shape)
    nkv, d = shape.n_kv_heads, shape.head_dim
    pos = np.concatenate([np.arange(c, c + q) for c, q in zip(ctx_lens, q_lens)]).astype(np.int64)
    blk = np.concatenate([np.asarray(tables[i])[np.arange(c, c + q) // 16]
                          for i, (c, q) in enumerate(zip(ctx_lens, q_lens))]).astype(np.int64)
    assert len(pos) == x_in.shape[0]
    ki, vi = kv_plane_index(16, d)
    ki_t, vi_t = torch.from_numpy(ki).cuda(), torch.from_numpy(vi).cuda()
    planes = st.kv_view()[0].reshape(st.num_blocks, nkv, 2, 16 * d)
    worst_k = worst_v = 0.0
    for r0 in range(0, len(pos), chunk):
        r1 = min(len(pos), r0 + chunk)
        _, k_ref, v_ref = O.project_qkv(oc, w64, x_in[r0:r1], pos[r0:r1])
        b_t = torch.from_numpy(blk[r0:r1]).cuda()
        o_t = torch.from_numpy(pos[r0:r1] % 16).cuda()
        sel = planes[b_t]                                  # [n, nkv, 2, 16 d]
        gk = torch.gather(sel[:, :, 0, :], 2, ki_t[o_t][:, None, :].expand(-1, nkv, -1))
        gv = torch.gather(sel[:, :, 1, :], 2, vi_t[o_t][:, None, :].expand(-1, nkv, -1))
        gk, gv = gk.double().cpu().numpy(), gv.double().cpu().numpy()
        for g, ref, name in ((gk, k_ref, "K"), (gv, v_ref, "V")):
            err = np.linalg.norm((g - ref).reshape(len(g), -1), axis=1) / \
                np.linalg.norm(ref.reshape(len(ref), -1), axis=1)
            i = int(np.argmax(err))
            assert err[i] <= TOL, f"{tag}: {name} of row {r0 + i} (position {pos[r0 + i]}) " \
                                  f"rel_l2 {err[i]:.3e}"
            if name == "K":
                worst_k = max(worst_k, float(err.max()))
            else:
                worst_v = max(worst_v, float(err.max()))
    log(f"  {tag}: all {len(pos)} written K/V rows, worst per-row rel_l2 K {worst_k:.3e} "
        f"V {worst_v:.3e}")


def test_l70_decode_20_layers_sampled():
    seed, shape = 2606, synth.LLAMA70B
    L0, nL, B = 20, 20, 64
    log("l70 decode, 20 layers, batch 64: generating weights")
    cfg = model_config(shape, "bf16")
    rowmajor = [device_layer_weights(shape, seed, L0 + l, "bf16") for l in range(nL)]
    packed = [pack_layer(cfg, w) for w in rowmajor]
    ctx = synth.uniform_lengths(seed, 1, B, 512, 2048)
    sample = [int(np.argmin(ctx)), int(np.argmax(ctx)), 17]
    nblocks = int(((ctx + 16) // 16 + 1).sum()) + 8
    bt_np = synth.make_block_tables(ctx + 1, int((ctx.max() + 16) // 16),
                                    synth.BlockAllocator(nblocks, seed))
    bt = torch.from_numpy(bt_np).cuda()
    st = DeviceStage(shape, "bf16", L0, packed, nblocks, 2048, B, packed=True)
    try:
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        st.kv_pool.normal_(0.0, 1.0, generator=g)   # contexts of the unsampled sequences
        # contexts of the sampled sequences: chunked prefill through the stage
        log(f"  context prefill of sequences {sample} ({[int(ctx[s]) for s in sample]} tokens)")
        for s in sample:
            done = 0
            while done < ctx[s]:
                q = int(min(2048, ctx[s] - done))
                x = torch.randn((q, shape.hidden), generator=g, device="cuda").to(torch.bfloat16)
                st.prefill([q], [done], bt[s:s + 1].contiguous(), x)
                done += q
        torch.cuda.synchronize()
        before = {s: _seq_cache(st, bt_np[s], int(ctx[s])) for s in sample}
        xin = torch.randn((B, shape.hidden), generator=g, device="cuda").to(torch.bfloat16)
        log("  decode step")
        y = st.decode(ctx, bt, xin)
        torch.cuda.synchronize()
        y64 = y.double().cpu().numpy()
        after = {s: _seq_cache(st, bt_np[s], int(ctx[s]) + 1) for s in sample}
    finally:
        st.close()
    # oracle: 20 layers for the sampled sequences, from the context snapshot,
    # exact (fp64) and with bf16 storage emulated at the stage's rounding points
    oc = ocfg(shape)
    x_in = xin.double().cpu().numpy()[sample]
    x_ex, x_em = x_in, x_in
    for l in range(nL):
        w = _host64(rowmajor[l])
        rows_ex, rows_em, errs = [], [], []
        for i, s in enumerate(sample):
            p = int(ctx[s])
            gk, gv = _kv_at(*after[s][l], p)
            cache, table = before[s][l]
            c_em = {k: v.copy() for k, v in cache.items()}
            rows_ex.append(O.layer_forward(oc, w, x_ex[i:i + 1], [O.SeqSpec(p, 1, table)], cache))
            rows_em.append(O.layer_forward(oc, w, x_em[i:i + 1], [O.SeqSpec(p, 1, table)], c_em,
                                           rounding=O.round_to_bf16))
            ek = rel_l2(gk, _kv_at(cache, table, p)[0])
            ekm = rel_l2(gk, _kv_at(c_em, table, p)[0])
            errs.append((ek, ekm))
            if l == 0:
                assert ek <= TOL and rel_l2(gv, _kv_at(cache, table, p)[1]) <= TOL
        x_ex, x_em = np.concatenate(rows_ex), np.concatenate(rows_em)
        del w
        log(f"  layer {L0 + l}: new-K rel_l2 vs exact / vs bf16-emulated: "
            + ", ".join(f"{a:.2e}/{b:.2e}" for a, b in errs))
    # Through 20 random layers the bf16 storage floor itself (the oracle with
    # bf16 rounding emulated, against the exact oracle) exceeds 2e-2, so the
    # end-to-end bar is the larger of 2e-2 and 1.25x that floor; the per-layer
    # bar (2e-2) is held by test_l70_decode_one_layer_sampled.
    for i, s in enumerate(sample):
        e_ex = rel_l2(y64[s], x_ex[i])
        e_em = rel_l2(y64[s], x_em[i])
        floor = rel_l2(x_em[i], x_ex[i])
        log(f"  seq {s} ctx {int(ctx[s])}: output rel_l2 vs exact {e_ex:.3e}, vs bf16-emulated "
            f"{e_em:.3e}; emulated vs exact (bf16 floor) {floor:.3e}")
        assert e_ex <= max(TOL, 1.25 * floor), (s, e_ex, floor)
        assert e_em <= max(TOL, 1.25 * floor), (s, e_em, floor)


def test_l70_first_positions_and_one_token_prompts():
    """One L70 layer. A decode batch of 64 whose first sequences sit at
    positions 0, 1, 15 and 16 (the rest at U[512, 2048]); then one prefill
    call of 2048 rows made of prompts of 1, 1, 17 and 2029 tokens (the
    2048-row path: split query / key-value QKV, RoPE in the query product's
    epilogue). Every edge row against the oracle, and every K/V entry both
    calls wrote."""
    seed, shape, layer, B = 2613, synth.LLAMA70B, 33, 64
    log("l70 first positions and one-token prompts, one layer")
    cfg = model_config(shape, "bf16")
    w = device_layer_weights(shape, seed, layer, "bf16")
    w64 = _host64(w)
    ctx = synth.uniform_lengths(seed, 1, B, 512, 2048)
    ctx[:4] = [0, 1, 15, 16]
    pq = np.array([1, 1, 17, 2029], np.int32)
    pc = np.zeros(4, np.int32)
    alloc = synth.BlockAllocator(int(((ctx + 16) // 16).sum() + ((pq + 15) // 16).sum()) + 8, seed)
    dbt_np = synth.make_block_tables(ctx + 1, int((ctx.max() + 16) // 16), alloc)
    pbt_np = synth.make_block_tables(pq, int((pq.max() + 15) // 16), alloc)
    nb = int(max(dbt_np.max(), pbt_np.max())) + 1
    st = DeviceStage(shape, "bf16", layer, [pack_layer(cfg, w)], nb, 2048, B, packed=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    try:
        st.kv_pool.normal_(0.0, 1.0, generator=g)
        x = torch.randn((B, shape.hidden), generator=g, device="cuda").to(torch.bfloat16)
        y = st.decode(ctx, torch.from_numpy(dbt_np).cuda(), x)
        torch.cuda.synchronize()
        x64, y64 = x.double().cpu().numpy(), y.double().cpu().numpy()
        rows = [(j, int(ctx[j]), j) for j in (0, 1, 2, 3, 40)]
        _check_rows_one_layer(shape, st, w64, dbt_np, rows, x64, y64, "decode rows at 0/1/15/16")
        _check_all_written_kv(shape, st, w64, dbt_np, ctx, np.ones(B, np.int32), x64, "decode")
        x = torch.randn((2048, shape.hidden), generator=g, device="cuda").to(torch.bfloat16)
        y = st.prefill(pq, pc, torch.from_numpy(pbt_np).cuda(), x)
        torch.cuda.synchronize()
        x64, y64 = x.double().cpu().numpy(), y.double().cpu().numpy()
        rows = [(0, 0, 0), (1, 0, 1)] + [(2, p, 2 + p) for p in range(17)] + \
            _sample_rows(np.random.default_rng(seed), pq, pc, 6)
        _check_rows_one_layer(shape, st, w64, pbt_np, rows, x64, y64, "prefill rows")
        _check_all_written_kv(shape, st, w64, pbt_np, pc, pq, x64, "prefill 1+1+17+2029")
    finally:
        st.close()


def test_l70_decode_one_layer_sampled():
    """One L70 layer at the decode launch configuration (batch 64, contexts
    U[512, 2048]); sampled rows against the exact oracle, fed the same input."""
    seed, shape, layer, B = 2607, synth.LLAMA70B, 20, 64
    log("l70 decode, one layer, batch 64")
    cfg = model_config(shape, "bf16")
    w = device_layer_weights(shape, seed, layer, "bf16")
    w64 = _host64(w)
    ctx = synth.uniform_lengths(seed, 1, B, 512, 2048)
    nblocks = int(((ctx + 16) // 16).sum()) + 8
    bt_np = synth.make_block_tables(ctx + 1, int((ctx.max() + 16) // 16),
                                    synth.BlockAllocator(nblocks, seed))
    st = DeviceStage(shape, "bf16", layer, [pack_layer(cfg, w)], nblocks, 2048, B, packed=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    try:
        st.kv_pool.normal_(0.0, 1.0, generator=g)
        x = torch.randn((B, shape.hidden), generator=g, device="cuda").to(torch.bfloat16)
        y = st.decode(ctx, torch.from_numpy(bt_np).cuda(), x)
        torch.cuda.synchronize()
        rng = np.random.default_rng(seed)
        pick = sorted({0, B - 1, int(np.argmax(ctx)), int(np.argmin(ctx))} |
                      set(rng.choice(B, 4, replace=False).tolist()))
        rows = [(j, int(ctx[j]), j) for j in pick]
        _check_rows_one_layer(shape, st, w64, bt_np, rows, x.double().cpu().numpy(),
                              y.double().cpu().numpy(), "decode rows")
        _check_all_written_kv(shape, st, w64, bt_np, ctx, np.ones(B, np.int32),
                              x.double().cpu().numpy(), "decode")
    finally:
        st.close()


def _check_rows_one_layer(shape, st, w64, tables, rows, x_in, y_out, tag):
    """Each sampled (seq index, position, row) checked on its own: the oracle
    is given the keys/values of positions < p from the stage's cache, and
    computes the row's output and its own K/V."""
    oc = ocfg(shape)
    worst = 0.0
    for si, p, r in rows:
        cache, table = _seq_cache(st, tables[si], p + 1)[0]
        gk, gv = _kv_at(cache, table, p)
        gk, gv = gk.copy(), gv.copy()
        yr = O.layer_forward(oc, w64, x_in[r:r + 1], [O.SeqSpec(p, 1, table)], cache)
        ok, ov = _kv_at(cache, table, p)
        e, ek, ev = rel_l2(y_out[r], yr[0]), rel_l2(gk, ok), rel_l2(gv, ov)
        worst = max(worst, e, ek, ev)
        assert e <= TOL and ek <= TOL and ev <= TOL, (tag, si, p, e, ek, ev)
    log(f"  {tag}: {len(rows)} sampled rows, worst rel_l2 {worst:.3e}")


def _sample_rows(rng, q_lens, ctx_lens, n):
    starts = np.concatenate([[0], np.cumsum(q_lens)])
    out = []
    for si in range(len(q_lens)):
        out.append((si, int(ctx_lens[si]), int(starts[si])))                         # first row
        out.append((si, int(ctx_lens[si] + q_lens[si] - 1), int(starts[si + 1] - 1)))  # last row
    for r in rng.choice(int(starts[-1]), size=n, replace=False):
        si = int(np.searchsorted(starts, r, side="right") - 1)
        out.append((si, int(ctx_lens[si] + r - starts[si]), int(r)))
    return out


def test_l70_prefill_chunks_sampled():
    seed, shape, layer = 11, synth.LLAMA70B, 20
    log("l70 chunked prefill, one layer, 2048 + 952 + 200 + 1280 tokens")
    cfg = model_config(shape, "bf16")
    w = device_layer_weights(shape, seed, layer, "bf16")
    w64 = _host64(w)
    n = 4480
    bt_np = synth.make_block_tables([n], (n + 15) // 16, synth.BlockAllocator(300, seed))
    bt = torch.from_numpy(bt_np).cuda()
    st = DeviceStage(shape, "bf16", layer, [pack_layer(cfg, w)], 300, 2048, 4, packed=True)
    rng = np.random.default_rng(seed)
    try:
        # 2048 rows: split query / key-value QKV with RoPE in the query
        # product; 952: plain tiles; 200: one row tile, products split over K;
        # 1280: O and down on 192-row tiles (224 tiles fill a round, 160
        # 256-row tiles would not)
        for ctx0, q in ((0, 2048), (2048, 952), (3000, 200), (3200, 1280)):
            x = torch.from_numpy(synth.hidden_states(seed, ctx0, q, shape.hidden)).cuda().to(
                torch.bfloat16)
            y = st.prefill([q], [ctx0], bt, x)
            torch.cuda.synchronize()
            rows = _sample_rows(rng, [q], [ctx0], 10)
            _check_rows_one_layer(shape, st, w64, bt_np, rows, x.double().cpu().numpy(),
                                  y.double().cpu().numpy(), f"chunk ctx={ctx0} q={q}")
            _check_all_written_kv(shape, st, w64, bt_np, [ctx0], [q], x.double().cpu().numpy(),
                                  f"chunk ctx={ctx0} q={q}")
    finally:
        st.close()


def test_l70_bench_prefill_schedule_sampled():
    """The prefill bench's launch configuration on one L70 layer: its 8 prompts
    (U[1024, 4096], the bench's seed) in its 11 chunked steps of at most 2048
    tokens, among them a step of three prompts with a 3689-token prefix and
    the final 154-token step. Each step's first and last rows of every prompt
    plus 4 random rows against the oracle."""
    seed, shape, layer = 2606, synth.LLAMA70B, 20
    p_lens = synth.uniform_lengths(seed, 2, 8, 1024, 4096)
    steps = synth.chunk_schedule(p_lens, 2048)
    log(f"l70 bench prefill schedule, one layer: {len(steps)} steps, {int(p_lens.sum())} tokens")
    cfg = model_config(shape, "bf16")
    w = device_layer_weights(shape, seed, layer, "bf16")
    w64 = _host64(w)
    nblk = int(((p_lens + 15) // 16).sum()) + 1
    bt_np = synth.make_block_tables(p_lens, int(((p_lens + 15) // 16).max()),
                                    synth.BlockAllocator(nblk, seed))
    bt_all = torch.from_numpy(bt_np).cuda()
    st = DeviceStage(shape, "bf16", layer, [pack_layer(cfg, w)], nblk, 2048, 8, packed=True)
    rng = np.random.default_rng(seed)
    try:
        for k, step in enumerate(steps):
            idx = [int(i) for i, _, _ in step]
            ctx = [int(c) for _, c, _ in step]
            q = [int(n) for _, _, n in step]
            x = torch.from_numpy(synth.hidden_states(seed, 100 + k, sum(q), shape.hidden)).cuda().to(
                torch.bfloat16)
            y = st.prefill(q, ctx, bt_all[idx].contiguous(), x)
            torch.cuda.synchronize()
            rows = _sample_rows(rng, q, ctx, 4)
            _check_rows_one_layer(shape, st, w64, bt_np[idx], rows, x.double().cpu().numpy(),
                                  y.double().cpu().numpy(), f"step {k} {list(zip(ctx, q))}")
            _check_all_written_kv(shape, st, w64, bt_np[idx], ctx, q, x.double().cpu().numpy(),
                                  f"step {k}")
    finally:
        st.close()


@pytest.mark.parametrize("gain_std", [0.02, 0.5], ids=["workload-gains", "wide-gains"])
def test_q32_mixed_step_sampled(gain_std):
    """The Qwen3-32B mixed step at its launch configuration. Its 2048 prefill
    rows take the query product with q RMSNorm and RoPE in the epilogue; with
    norm gains 1 + N(0, 0.5^2) (instead of the workload's 1 + N(0, 0.02^2))
    a gain applied to the wrong columns, or not at all, moves the queries by
    tens of percent."""
    seed, shape, layer = 24, synth.QWEN32B, 24
    log(f"qwen3-32b mixed step, one layer: 4 x 512 prefill + 128 decodes, gain std {gain_std}")
    cfg = model_config(shape, "bf16")
    w = device_layer_weights(shape, seed, layer, "bf16", gain_std=gain_std)
    w64 = _host64(w)
    pc = np.array([0, 512, 1024, 1536], np.int32)
    pq = np.full(4, 512, np.int32)
    dctx = synth.uniform_lengths(seed, 3, 128, 256, 4096)
    alloc = synth.BlockAllocator(int(((pc + pq + 15) // 16).sum() + ((dctx + 16) // 16).sum()) + 4,
                                 seed)
    pbt_np = synth.make_block_tables(pc + pq, 128, alloc)
    dbt_np = synth.make_block_tables(dctx + 1, 257, alloc)
    nb = int(max(pbt_np.max(), dbt_np.max())) + 1
    st = DeviceStage(shape, "bf16", layer, [pack_layer(cfg, w)], nb, 2176, 132, packed=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    try:
        st.kv_pool.normal_(0.0, 1.0, generator=g)  # cached prefixes and decode contexts
        x = torch.randn((2176, shape.hidden), generator=g, device="cuda").to(torch.bfloat16)
        y = st.mixed(pq, pc, torch.from_numpy(pbt_np).cuda(), dctx, torch.from_numpy(dbt_np).cuda(),
                     x)
        torch.cuda.synchronize()
        rng = np.random.default_rng(seed)
        x64, y64 = x.double().cpu().numpy(), y.double().cpu().numpy()
        prow = _sample_rows(rng, pq, pc, 8)
        _check_rows_one_layer(shape, st, w64, pbt_np, prow, x64, y64, "prefill rows")
        drow = [(int(j), int(dctx[j]), 2048 + int(j))
                for j in sorted({0, 127, int(np.argmax(dctx)), int(np.argmin(dctx))} |
                                set(rng.choice(128, 6, replace=False).tolist()))]
        _check_rows_one_layer(shape, st, w64, dbt_np, drow, x64, y64, "decode rows")
        _check_all_written_kv(shape, st, w64, list(pbt_np) + list(dbt_np),
                              list(pc) + list(dctx), list(pq) + [1] * len(dctx), x64,
                              "mixed step")
    finally:
        st.close()


def test_l70_decode_batch128_one_layer_sampled():
    """The 80-layer workload's decode-only step shape: batch 128 (the split-K
    GEMMs with 8 m-tiles), contexts U[1024, 4096]."""
    seed, shape, layer, B = 2608, synth.LLAMA70B, 60, 128
    log("l70 decode, one layer, batch 128")
    cfg = model_config(shape, "bf16")
    w = device_layer_weights(shape, seed, layer, "bf16")
    w64 = _host64(w)
    ctx = synth.uniform_lengths(seed, 1, B, 1024, 4096)
    nblocks = int(((ctx + 16) // 16).sum()) + 8
    bt_np = synth.make_block_tables(ctx + 1, int((ctx.max() + 16) // 16),
                                    synth.BlockAllocator(nblocks, seed))
    st = DeviceStage(shape, "bf16", layer, [pack_layer(cfg, w)], nblocks, 2176, B, packed=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    try:
        st.kv_pool.normal_(0.0, 1.0, generator=g)
        x = torch.randn((B, shape.hidden), generator=g, device="cuda").to(torch.bfloat16)
        y = st.decode(ctx, torch.from_numpy(bt_np).cuda(), x)
        torch.cuda.synchronize()
        rng = np.random.default_rng(seed)
        pick = sorted({0, B - 1, int(np.argmax(ctx)), int(np.argmin(ctx))} |
                      set(rng.choice(B, 4, replace=False).tolist()))
        rows = [(j, int(ctx[j]), j) for j in pick]
        _check_rows_one_layer(shape, st, w64, bt_np, rows, x.double().cpu().numpy(),
                              y.double().cpu().numpy(), "decode rows (batch 128)")
        _check_all_written_kv(shape, st, w64, bt_np, ctx, np.ones(B, np.int32),
                              x.double().cpu().numpy(), "decode (batch 128)")
    finally:
        st.close()


def test_l70_mixed_step_sampled():
    """The 80-layer workload's mixed step shape: 128 decodes (contexts
    U[1024, 4096]) plus 2048 prefill tokens, one continuation chunk that
    starts mid-block and one fresh prompt."""
    seed, shape, layer = 2609, synth.LLAMA70B, 79
    log("l70 mixed step, one layer: 1500 + 548 prefill + 128 decodes")
    cfg = model_config(shape, "bf16")
    w = device_layer_weights(shape, seed, layer, "bf16")
    w64 = _host64(w)
    pc = np.array([1000, 0], np.int32)
    pq = np.array([1500, 548], np.int32)
    dctx = synth.uniform_lengths(seed, 3, 128, 1024, 4096)
    alloc = synth.BlockAllocator(int(((pc + pq + 15) // 16).sum() + ((dctx + 16) // 16).sum()) + 4,
                                 seed)
    pbt_np = synth.make_block_tables(pc + pq, int(((pc + pq + 15) // 16).max()), alloc)
    dbt_np = synth.make_block_tables(dctx + 1, int((dctx.max() + 16) // 16), alloc)
    nb = int(max(pbt_np.max(), dbt_np.max())) + 1
    st = DeviceStage(shape, "bf16", layer, [pack_layer(cfg, w)], nb, 2176, 130, packed=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    try:
        st.kv_pool.normal_(0.0, 1.0, generator=g)  # cached prefix and decode contexts
        x = torch.randn((2176, shape.hidden), generator=g, device="cuda").to(torch.bfloat16)
        y = st.mixed(pq, pc, torch.from_numpy(pbt_np).cuda(), dctx, torch.from_numpy(dbt_np).cuda(),
                     x)
        torch.cuda.synchronize()
        rng = np.random.default_rng(seed)
        x64, y64 = x.double().cpu().numpy(), y.double().cpu().numpy()
        prow = _sample_rows(rng, pq, pc, 8)
        _check_rows_one_layer(shape, st, w64, pbt_np, prow, x64, y64, "prefill rows")
        drow = [(int(j), int(dctx[j]), 2048 + int(j))
                for j in sorted({0, 127, int(np.argmax(dctx)), int(np.argmin(dctx))} |
                                set(rng.choice(128, 6, replace=False).tolist()))]
        _check_rows_one_layer(shape, st, w64, dbt_np, drow, x64, y64, "decode rows")
        _check_all_written_kv(shape, st, w64, list(pbt_np) + list(dbt_np),
                              list(pc) + list(dctx), list(pq) + [1] * len(dctx), x64,
                              "mixed step")
    finally:
        st.close()


def test_l70_one_call_prefill_of_8192_tokens_sampled():
    """The largest single call the benches never make: one L70 layer, one
    prefill call of 8192 tokens (prompts of 5000 and 3192, the second after a
    cached prefix of 700): 32 row tiles in every GEMM, 8192-query attention
    items. Sampled rows against the exact oracle."""
    seed, shape, layer = 2661, synth.LLAMA70B, 55
    log("l70 one prefill call of 8192 tokens, one layer")
    cfg = model_config(shape, "bf16")
    w = device_layer_weights(shape, seed, layer, "bf16")
    w64 = _host64(w)
    pc = np.array([0, 700], np.int32)
    pq = np.array([5000, 3192], np.int32)
    nbs = int(((pc + pq + 15) // 16).max())
    bt_np = synth.make_block_tables(pc + pq, nbs, synth.BlockAllocator(2 * nbs + 8, seed))
    st = DeviceStage(shape, "bf16", layer, [pack_layer(cfg, w)], 2 * nbs + 8, 8192, 2, packed=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    try:
        st.kv_pool.normal_(0.0, 1.0, generator=g)  # the cached prefix of the second prompt
        x = torch.randn((8192, shape.hidden), generator=g, device="cuda").to(torch.bfloat16)
        y = st.prefill(pq, pc, torch.from_numpy(bt_np).cuda(), x)
        torch.cuda.synchronize()
        rng = np.random.default_rng(seed)
        _check_rows_one_layer(shape, st, w64, bt_np, _sample_rows(rng, pq, pc, 8),
                              x.double().cpu().numpy(), y.double().cpu().numpy(), "rows")
        _check_all_written_kv(shape, st, w64, bt_np, pc, pq, x.double().cpu().numpy(),
                              "8192-token call")
    finally:
        st.close()
