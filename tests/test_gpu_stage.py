"""Parity of the HIP stage with the CPU oracle (GPU).

Every call is compared element by element with the oracle run on the same
stored weights, inputs and block tables, and the KV entries the calls wrote
are compared as well. Tolerances: relative L2 <= 1e-4 in the fp32 mode,
<= 2e-2 in the bf16 mode, and max-abs <= 5e-3 per layer on the tiny config in
the fp32 mode.
"""

from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2606_18600_amd import stage as S
from paper_2606_18600_amd import synth
from tests.gpu_pair import Pair, log
from tests.helpers import rel_l2

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}

QWEN_SMALL = synth.ModelShape("qwen-small", hidden=512, n_q_heads=8, n_kv_heads=1, head_dim=128,
                              ffn=768, rms_eps=1e-6, rope_theta=1e6, qk_norm=True,
                              qk_rms_eps=1e-6)


def _check(tag, y, yr, x, tol):
    e = rel_l2(y, yr)
    ed = rel_l2(y - x, yr - x)
    log(f"  {tag}: rel_l2={e:.3e} delta_rel_l2={ed:.3e} max_abs={np.abs(y - yr).max():.3e}")
    assert np.isfinite(y).all()
    assert e <= tol, f"{tag}: rel_l2 {e:.3e} > {tol}"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tiny_prefill_then_16_decodes(dtype):
    """The tiny config end to end: 4 prompts of 16-64 tokens, prefill, then 16
    decode steps with fresh N(0,1) inputs, shuffled block tables."""
    seed = 2606
    shape = synth.TINY
    log(f"tiny-stage flow dtype={dtype} seed={seed}")
    lens = synth.uniform_lengths(seed, 0, 4, 16, 64)
    alloc = synth.BlockAllocator(64, seed)
    bt = synth.make_block_tables(lens + 16, 8, alloc)
    pair = Pair(shape, dtype, 2, 64, 256, 8, seed)
    try:
        y, yr, x = pair.prefill(lens, np.zeros(4, np.int32), bt,
                                synth.hidden_states(seed, 1, int(lens.sum()), shape.hidden))
        _check("prefill", y, yr, x, TOL[dtype])
        ctx = lens.copy()
        for step in range(16):
            y, yr, x = pair.decode(ctx, bt, synth.hidden_states(seed, 100 + step, 4, shape.hidden))
            _check(f"decode {step}", y, yr, x, TOL[dtype])
            ctx += 1
        kv = pair.kv_errors()
        log(f"  kv rel_l2={kv:.3e}")
        assert kv <= TOL[dtype]
    finally:
        pair.close()


@pytest.mark.parametrize("layer", [0, 1])
def test_tiny_per_layer_max_abs_fp32(layer):
    seed = 2606
    shape = synth.TINY
    log(f"tiny per-layer max-abs layer={layer}")
    w = [synth.host_layer_weights(shape, seed, layer)]
    lens = synth.uniform_lengths(seed, 0, 4, 16, 64)
    bt = synth.make_block_tables(lens + 4, 8, synth.BlockAllocator(64, seed))
    pair = Pair(shape, "f32", 1, 64, 256, 8, seed, layer_begin=layer, host_weights=w)
    try:
        y, yr, _ = pair.prefill(lens, np.zeros(4, np.int32), bt,
                                synth.hidden_states(seed, 1, int(lens.sum()), shape.hidden))
        worst = np.abs(y - yr).max()
        ctx = lens.copy()
        for step in range(4):
            y, yr, _ = pair.decode(ctx, bt, synth.hidden_states(seed, 100 + step, 4, shape.hidden))
            worst = max(worst, np.abs(y - yr).max())
            ctx += 1
        log(f"  max_abs={worst:.3e}")
        assert worst <= 5e-3
    finally:
        pair.close()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("T", [100, 128, 129, 300])
def test_prefill_token_counts_cover_both_gemm_paths(dtype, T):
    """T <= 128 runs the split-K GEMMs, T > 128 the LDS-tiled GEMMs."""
    seed = 7 + T
    shape = synth.TINY
    log(f"prefill T={T} dtype={dtype}")
    r = np.random.default_rng(seed)
    cuts = np.sort(r.choice(np.arange(1, T), size=2, replace=False))
    lens = np.diff(np.concatenate([[0], cuts, [T]])).astype(np.int32)
    bt = synth.make_block_tables(lens, 32, synth.BlockAllocator(96, seed))
    pair = Pair(shape, dtype, 2, 96, 512, 8, seed)
    try:
        y, yr, x = pair.prefill(lens, np.zeros(3, np.int32), bt,
                                synth.hidden_states(seed, 1, T, shape.hidden))
        _check("prefill", y, yr, x, TOL[dtype])
        assert pair.kv_errors() <= TOL[dtype]
    finally:
        pair.close()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_ragged_lengths_and_block_boundaries(dtype):
    seed = 31
    shape = synth.TINY
    log(f"ragged dtype={dtype}")
    lens = np.array([1, 15, 16, 17, 33], np.int32)
    bt = synth.make_block_tables(lens + 20, 8, synth.BlockAllocator(64, seed))
    pair = Pair(shape, dtype, 2, 64, 256, 8, seed)
    try:
        y, yr, x = pair.prefill(lens, np.zeros(5, np.int32), bt,
                                synth.hidden_states(seed, 1, int(lens.sum()), shape.hidden))
        _check("prefill", y, yr, x, TOL[dtype])
        # continuation chunks that start mid-block
        q2 = np.array([3, 1, 16, 15, 2], np.int32)
        y, yr, x = pair.prefill(q2, lens, bt, synth.hidden_states(seed, 2, int(q2.sum()),
                                                                  shape.hidden))
        _check("chunk", y, yr, x, TOL[dtype])
        ctx = lens + q2
        for step in range(3):
            y, yr, x = pair.decode(ctx, bt, synth.hidden_states(seed, 10 + step, 5, shape.hidden))
            _check(f"decode {step}", y, yr, x, TOL[dtype])
            ctx += 1
        assert pair.kv_errors() <= TOL[dtype]
    finally:
        pair.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tables_and_buffers_filled_to_capacity(dtype):
    """Every limit at its maximum in one flow: a prompt of exactly
    max_blocks_per_seq * 16 tokens (its table row full), a decode that
    writes the last slot of its sequence's last block, a prefill of exactly
    max_tokens rows from max_seqs sequences, and every block of the pool in
    use by the end."""
    seed = 53
    shape = synth.TINY
    mb = 4                                        # 64 tokens per table row
    lens = np.array([63, 64, 48], np.int32)
    final = lens + np.array([1, 0, 1], np.int32)  # sequences 0 and 2 decode once
    n_blocks = int(((final + 15) // 16).sum())    # 12: all of them used
    bt = synth.make_block_tables(final, mb, synth.BlockAllocator(n_blocks, seed))
    T = int(lens.sum())
    log(f"capacity dtype={dtype}: prompts {lens.tolist()} in rows of {mb} blocks, "
        f"{n_blocks} blocks, max_tokens {T}")
    pair = Pair(shape, dtype, 2, n_blocks, T, 3, seed)
    try:
        y, yr, x = pair.prefill(lens, np.zeros(3, np.int32), bt,
                                synth.hidden_states(seed, 1, T, shape.hidden))
        _check("prefill", y, yr, x, TOL[dtype])
        y, yr, x = pair.decode(np.array([63, 48], np.int32), bt[[0, 2]],
                               synth.hidden_states(seed, 2, 2, shape.hidden))
        _check("decode", y, yr, x, TOL[dtype])
        assert len(pair.written) == n_blocks * 16 - 15  # all slots but the last block's tail of seq 2
        kv = pair.kv_errors()
        log(f"  kv rel_l2={kv:.3e}")
        assert kv <= TOL[dtype]
    finally:
        pair.close()


def test_decode_of_a_first_token():
    """A decode token with no context (position 0) attends only to itself."""
    seed = 41
    shape = synth.TINY
    bt = synth.make_block_tables([5, 5], 2, synth.BlockAllocator(8, seed))
    pair = Pair(shape, "bf16", 2, 8, 16, 4, seed)
    try:
        y, yr, x = pair.decode(np.array([0, 0], np.int32), bt,
                               synth.hidden_states(seed, 1, 2, shape.hidden))
        _check("decode@0", y, yr, x, TOL["bf16"])
    finally:
        pair.close()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", [synth.TINY, QWEN_SMALL], ids=["tiny", "qwen-small"])
def test_mixed_step(dtype, shape):
    """Prefill chunks (fresh and continuation) and decodes in one call."""
    seed = 53
    log(f"mixed {shape.name} dtype={dtype}")
    d_ctx0 = np.array([40, 3, 100, 17], np.int32)
    p_total = np.array([70, 48], np.int32)
    alloc = synth.BlockAllocator(128, seed)
    dbt = synth.make_block_tables(d_ctx0 + 4, 16, alloc)
    pbt = synth.make_block_tables(p_total, 16, alloc)
    pair = Pair(shape, dtype, 2, 128, 256, 8, seed)
    try:
        y, yr, x = pair.prefill(d_ctx0, np.zeros(4, np.int32), dbt,
                                synth.hidden_states(seed, 1, int(d_ctx0.sum()), shape.hidden))
        _check("context prefill", y, yr, x, TOL[dtype])
        # step 1: first chunks of two prompts + 4 decodes
        pq, pc = np.array([30, 48], np.int32), np.array([0, 0], np.int32)
        y, yr, x = pair.mixed(pq, pc, pbt, d_ctx0, dbt,
                              synth.hidden_states(seed, 2, int(pq.sum()) + 4, shape.hidden))
        _check("mixed 1", y, yr, x, TOL[dtype])
        # step 2: continuation chunk of prompt 0 + decodes
        pq2, pc2 = np.array([40], np.int32), np.array([30], np.int32)
        y, yr, x = pair.mixed(pq2, pc2, pbt[:1], d_ctx0 + 1, dbt,
                              synth.hidden_states(seed, 3, 44, shape.hidden))
        _check("mixed 2", y, yr, x, TOL[dtype])
        assert pair.kv_errors() <= TOL[dtype]
    finally:
        pair.close()


@pytest.mark.parametrize("shape", [synth.TINY, QWEN_SMALL], ids=["tiny", "qwen-small"])
def test_last_rows_of_large_steps_on_split_k(shape):
    """Steps of 256 k + r rows (k >= 5, 0 < r <= 128): the first 256 k rows run
    on whole 256-row tiles and the last r on the split-K kernels, whose
    partial planes RoPE, the RMSNorms and the output cast add to those rows
    only. Covers a prefill-only step with r = 128, a mixed step whose last
    rows are all decodes (r = 40), and r = 129 (no split) for contrast."""
    seed = 61
    dtype = "bf16"
    log(f"row tail {shape.name}")
    d_ctx0 = synth.uniform_lengths(seed, 1, 40, 5, 60).astype(np.int32)
    # four prompts: a first prefill of [500, 480, 300, 128] tokens, then
    # continuations of [600, 680] and [1280, 129] tokens
    totals = np.array([1100, 1160, 1580, 257], np.int32)
    alloc = synth.BlockAllocator(512, seed)
    dbt = synth.make_block_tables(d_ctx0 + 4, 8, alloc)
    pbt = synth.make_block_tables(totals, 100, alloc)
    pair = Pair(shape, dtype, 2, 512, 1536, 48, seed)
    try:
        # decode contexts (T = sum of 40 lengths: small, split-K or mid-split)
        y, yr, x = pair.prefill(d_ctx0, np.zeros(40, np.int32), dbt,
                                synth.hidden_states(seed, 2, int(d_ctx0.sum()), shape.hidden))
        _check("context prefill", y, yr, x, TOL[dtype])
        # prefill-only step of 1408 = 5 * 256 + 128 rows
        q1 = np.array([500, 480, 300, 128], np.int32)
        y, yr, x = pair.prefill(q1, np.zeros(4, np.int32), pbt,
                                synth.hidden_states(seed, 3, int(q1.sum()), shape.hidden))
        _check("prefill 1408", y, yr, x, TOL[dtype])
        # mixed step: 1280 prefill rows (continuations) + 40 decodes = 1320 rows
        pq = np.array([600, 680], np.int32)
        y, yr, x = pair.mixed(pq, q1[:2], pbt[:2].copy(), d_ctx0, dbt,
                              synth.hidden_states(seed, 4, 1320, shape.hidden))
        _check("mixed 1320", y, yr, x, TOL[dtype])
        # 1409 = 5 * 256 + 129 rows: no split
        q3 = np.array([1280, 129], np.int32)
        y, yr, x = pair.prefill(q3, q1[2:], pbt[2:].copy(),
                                synth.hidden_states(seed, 5, 1409, shape.hidden))
        _check("prefill 1409", y, yr, x, TOL[dtype])
        assert pair.kv_errors() <= TOL[dtype]
    finally:
        pair.close()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_qwen_small_long_context_decode(dtype):
    """head_dim 128, GQA group 8, q/k-norm, contexts long enough for many
    decode key splits (uneven last split)."""
    seed = 67
    shape = QWEN_SMALL
    log(f"qwen-small long-context dtype={dtype}")
    ctx = np.array([2500, 700, 129], np.int32)
    alloc = synth.BlockAllocator(300, seed)
    bt = synth.make_block_tables(ctx + 3, 160, alloc)
    pair = Pair(shape, dtype, 1, 300, 1024, 4, seed)
    try:
        done = np.zeros(3, np.int32)
        i = 0
        while (done < ctx).any():
            q = np.minimum(ctx - done, 400).astype(np.int32)
            live = q > 0
            y, yr, x = pair.prefill(q[live], done[live], bt[live],
                                    synth.hidden_states(seed, 10 + i, int(q.sum()), shape.hidden))
            _check(f"chunk {i}", y, yr, x, TOL[dtype])
            done += q
            i += 1
        for step in range(3):
            y, yr, x = pair.decode(ctx + step, bt,
                                   synth.hidden_states(seed, 100 + step, 3, shape.hidden))
            _check(f"decode {step}", y, yr, x, TOL[dtype])
        assert pair.kv_errors() <= TOL[dtype]
    finally:
        pair.close()


@pytest.mark.parametrize("lens", [[20, 9], [150, 61]], ids=["split-k", "tiled"])
def test_hidden_out_may_alias_hidden_in(lens):
    """Writing the output over the input gives the same result, bitwise: the
    input is read (by the first RMSNorm) before anything is written to the
    output, and every kernel is deterministic (the split-K GEMMs write
    partial planes that the next kernel sums in a fixed order; no atomics)."""
    seed = 71
    shape = synth.TINY
    lens = np.array(lens, np.int32)
    T = int(lens.sum())
    bt = synth.make_block_tables(lens, 16, synth.BlockAllocator(32, seed))
    pair = Pair(shape, "bf16", 2, 32, 256, 4, seed)
    try:
        x = synth.hidden_states(seed, 1, T, shape.hidden)
        xin = torch.from_numpy(x).to("cuda", torch.bfloat16)
        ref = pair.gpu.prefill(lens, [0, 0], torch.from_numpy(bt).cuda(), xin.clone())
        # the same slots are rewritten with the same values, so the call repeats exactly
        out = pair.gpu.prefill(lens, [0, 0], torch.from_numpy(bt).cuda(), xin, hidden_out=xin)
        torch.cuda.synchronize()
        assert out.data_ptr() == xin.data_ptr()
        assert torch.equal(out, ref)
    finally:
        pair.close()


def test_debug_mode_checks_block_ids_on_the_host(monkeypatch):
    """With STAGE_DEBUG=1 a call whose block table sends a read past the pool
    (or below 0) is rejected before anything is enqueued; entries past a
    sequence's length are not read and not checked."""
    monkeypatch.setenv("STAGE_DEBUG", "1")
    seed = 71
    shape = synth.TINY
    lens = np.array([20, 9], np.int32)
    zeros = np.zeros(2, np.int32)
    bt = synth.make_block_tables(lens, 4, synth.BlockAllocator(16, seed))
    pair = Pair(shape, "bf16", 2, 16, 64, 4, seed)
    try:
        y, yr, x = pair.prefill(lens, zeros, bt, synth.hidden_states(seed, 1, 29, shape.hidden))
        _check("prefill", y, yr, x, TOL["bf16"])
        xin = torch.zeros((29, shape.hidden), dtype=torch.bfloat16, device="cuda")
        for row, col, bad_id in [(1, 0, 16), (0, 1, -1)]:
            bad = bt.copy()
            bad[row, col] = bad_id
            with pytest.raises(S.StageError) as e:
                pair.gpu.prefill(lens, zeros, torch.from_numpy(bad).cuda(), xin)
            assert e.value.code == S.STAGE_ERR_INVALID_ARG
            assert f"block_tables[{row}][{col}]" in str(e.value)
        unused = bt.copy()
        unused[1, 3] = 999  # sequence 1 (9 tokens) reads only entry 0
        torch.cuda.synchronize()
        pair.gpu.decode(lens, torch.from_numpy(unused).cuda(), xin[:2])
        torch.cuda.synchronize()
    finally:
        pair.close()


def test_forward_calls_return_validation_codes():
    shape = synth.TINY
    bt = torch.zeros((2, 4), dtype=torch.int32, device="cuda")
    pair = Pair(shape, "bf16", 1, 16, 64, 2, 5)
    try:
        x = torch.zeros((70, shape.hidden), dtype=torch.bfloat16, device="cuda")
        with pytest.raises(S.StageError) as e:
            pair.gpu.prefill([3, 0], [0, 0], bt, x)
        assert e.value.code == S.STAGE_ERR_INVALID_ARG
        with pytest.raises(S.StageError) as e:
            pair.gpu.prefill([70], [0], bt[:1], x)             # 70 tokens > 4 blocks
        assert e.value.code == S.STAGE_ERR_CAPACITY
        with pytest.raises(S.StageError) as e:
            pair.gpu.decode([1, 2, 3], torch.zeros((3, 4), dtype=torch.int32, device="cuda"),
                            x[:3])                              # 3 seqs > max_seqs 2
        assert e.value.code == S.STAGE_ERR_CAPACITY
    finally:
        pair.close()


def test_op_timing_hook():
    """The op-timing hook: with timing on, every op class of a decode step is
    timed (the four products once per layer) and the outputs are bitwise
    those of the same step with timing off."""
    seed, n_layers = 61, 2
    shape = QWEN_SMALL
    ctx = np.array([30, 5, 17, 64], np.int32)
    bt_np = synth.make_block_tables(ctx + 1, 5, synth.BlockAllocator(24, seed))
    pair = Pair(shape, "bf16", n_layers, 24, 64, 4, seed)
    try:
        h = pair.gpu.handle
        bt = torch.from_numpy(bt_np).cuda()
        x = torch.from_numpy(synth.hidden_states(seed, 1, 4, shape.hidden)).to("cuda",
                                                                              torch.bfloat16)
        y0 = pair.gpu.decode(ctx, bt, x).clone()
        S.stage_set_op_timing(h, True)
        y1 = pair.gpu.decode(ctx, bt, x).clone()
        ms, n = S.stage_read_op_times(h)
        S.stage_set_op_timing(h, False)
        y2 = pair.gpu.decode(ctx, bt, x).clone()
        ms2, n2 = S.stage_read_op_times(h)
        log(f"  op ms: {dict(zip(S.OP_NAMES, np.round(ms, 4)))}")
        for j, name in enumerate(S.OP_NAMES):
            if name == "lm_head":
                assert n[j] == 0
            else:
                assert n[j] >= n_layers and ms[j] > 0.0, name
            if name in ("qkv", "o_proj", "gate_up", "down"):
                assert n[j] == n_layers, name
        assert sum(n2) == 0 and sum(ms2) == 0.0  # counters reset by the read; timing off
        assert torch.equal(y0, y1) and torch.equal(y0, y2)
    finally:
        pair.close()


@pytest.mark.parametrize("kind,shape_fn", [
    ("w_qkv", lambda s: (s.qkv_width, s.hidden)), ("w_o", lambda s: (s.hidden, s.q_width)),
    ("w_gate_up", lambda s: (2 * s.ffn, s.hidden)), ("w_down", lambda s: (s.hidden, s.ffn))])
def test_pack_weight_layout(kind, shape_fn):
    """stage_pack_weight places element (n, k) of the row-major matrix where
    the documented layout says: fragment ((n/64)*(K/32) + k/32)*4 + (n/16)%4,
    lane (n%16) + 16*((k%32)/8), element k%8 (gate-up rows interleaved per 64)."""
    from paper_2606_18600_amd.harness import PACK_KINDS, model_config
    shape = QWEN_SMALL
    N, K = shape_fn(shape)
    cfg = model_config(shape, "bf16")
    src = torch.arange(N * K, dtype=torch.float32).remainder_(251).sub_(125).to(
        torch.bfloat16).reshape(N, K).cuda()
    dst = torch.empty_like(src)
    S.stage_pack_weight(cfg, PACK_KINDS[kind], src.data_ptr(), dst.data_ptr(), 0)
    torch.cuda.synchronize()
    a, p = src.cpu().float().numpy(), dst.cpu().float().numpy().reshape(-1)
    n = np.arange(N)[:, None]
    k = np.arange(K)[None, :]
    frag = ((n // 64) * (K // 32) + k // 32) * 4 + (n // 16) % 4
    lane = n % 16 + 16 * ((k % 32) // 8)
    pos = frag * 512 + lane * 8 + k % 8
    if kind == "w_gate_up":
        F = shape.ffn
        g, r = n // 64, n % 64
        rows = np.where(r < 32, 32 * g + r, F + 32 * g + r - 32)
        expect = a[rows[:, 0]]
    else:
        expect = a
    np.testing.assert_array_equal(p[pos], np.broadcast_to(expect, (N, K)))


@pytest.mark.parametrize("nbytes", [16, 4096, 3 * 1024 * 1024 + 48, 64 << 20])
def test_copy_probe_copies_exactly(nbytes):
    """The calibration copy moves every byte (grid-stride tail included)."""
    log(f"[test] copy probe {nbytes} bytes")
    g = torch.Generator(device="cuda")
    g.manual_seed(nbytes)
    src = torch.randint(0, 1 << 30, (nbytes // 4,), dtype=torch.int32, device="cuda",
                        generator=g)
    dst = torch.full((nbytes // 4 + 4,), -7, dtype=torch.int32, device="cuda")
    S.stage_copy_probe(src.data_ptr(), dst.data_ptr(), nbytes)
    torch.cuda.synchronize()
    assert torch.equal(dst[: nbytes // 4], src)
    assert (dst[nbytes // 4:] == -7).all()      # nothing written past the end


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_stage_composition(dtype):
    """Pipeline partitioning: stage [0, 1) followed by stage [1, 2) equals
    stage [0, 2) over a prefill and three decode steps. fp32 mode: bitwise
    (the fp32 stage output is the residual stream itself and every kernel
    is deterministic). bf16: within tolerance, since the hidden state that
    crosses the stage boundary is rounded to bf16 there."""
    from paper_2606_18600_amd.harness import DeviceStage, torch_dtype, upload_weights
    seed, shape = 2610, synth.TINY
    log(f"stage composition dtype={dtype}")
    td = torch_dtype(dtype)
    w = [upload_weights(synth.host_layer_weights(shape, seed, l), dtype) for l in range(2)]
    lens = synth.uniform_lengths(seed, 0, 4, 16, 64)
    bt = torch.from_numpy(synth.make_block_tables(lens + 4, 8, synth.BlockAllocator(48, seed)))
    bt = bt.cuda()
    whole = DeviceStage(shape, dtype, 0, w, 48, 256, 8)
    first = DeviceStage(shape, dtype, 0, w[:1], 48, 256, 8)
    second = DeviceStage(shape, dtype, 1, w[1:], 48, 256, 8)
    try:
        steps = [(lens, np.zeros(4, np.int32), int(lens.sum()))]
        steps += [(np.ones(4, np.int32), lens + i, 4) for i in range(3)]
        for k, (q, c, T) in enumerate(steps):
            x = torch.from_numpy(synth.hidden_states(seed, 10 + k, T, shape.hidden)).cuda().to(td)
            if k == 0:
                y = whole.prefill(q, c, bt, x)
                y2 = second.prefill(q, c, bt, first.prefill(q, c, bt, x))
            else:
                y = whole.decode(c, bt, x)
                y2 = second.decode(c, bt, first.decode(c, bt, x))
            torch.cuda.synchronize()
            a, b = y.double().cpu().numpy(), y2.double().cpu().numpy()
            e = rel_l2(b, a)
            log(f"  step {k}: rel_l2 {e:.3e}")
            if dtype == "f32":
                assert torch.equal(y, y2), f"step {k}: not bitwise equal ({e:.3e})"
            else:
                assert e <= TOL[dtype], (k, e)
    finally:
        whole.close()
        first.close()
        second.close()


@pytest.mark.parametrize("shape", [synth.TINY, QWEN_SMALL], ids=["tiny", "qwen-small"])
def test_two_stages_on_two_streams(shape):
    """Two stages over the same weights (each with its own KV pool and
    workspace) driven step by step on two streams of default priority with
    no synchronisation between them give, bit for bit, what one of them
    gives alone: a stage keeps no state that another stage's calls touch."""
    from paper_2606_18600_amd.harness import DeviceStage, upload_weights
    seed, dtype = 2720, "bf16"
    log(f"two stages on two streams: {shape.name}")
    w = [upload_weights(synth.host_layer_weights(shape, seed, l), dtype) for l in range(2)]
    lens = np.array([37, 150, 5, 64], np.int32)
    bt = torch.from_numpy(synth.make_block_tables(lens + 8, 16, synth.BlockAllocator(64, seed)))
    bt = bt.cuda()
    steps = [(lens, np.zeros(4, np.int32), int(lens.sum()))]
    steps += [(np.ones(4, np.int32), lens + i, 4) for i in range(6)]
    xs = [torch.from_numpy(synth.hidden_states(seed, 10 + k, T, shape.hidden)).cuda()
          .to(torch.bfloat16) for k, (_, _, T) in enumerate(steps)]

    def step(st, k, s):
        q, c, _ = steps[k]
        with torch.cuda.stream(s):
            if k == 0:
                return st.prefill(q, c, bt, xs[k], stream=s.cuda_stream)
            return st.decode(c, bt, xs[k], stream=s.cuda_stream)

    alone = DeviceStage(shape, dtype, 0, w, 64, 256, 4)
    a = DeviceStage(shape, dtype, 0, w, 64, 256, 4)
    b = DeviceStage(shape, dtype, 0, w, 64, 256, 4)
    try:
        main = torch.cuda.current_stream()
        ref = [step(alone, k, main) for k in range(len(steps))]
        torch.cuda.synchronize()
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
        s1.wait_stream(main)
        s2.wait_stream(main)
        ya, yb = [], []
        for k in range(len(steps)):  # enqueued alternately, step by step
            ya.append(step(a, k, s1))
            yb.append(step(b, k, s2))
        torch.cuda.synchronize()
        for k in range(len(steps)):
            assert torch.equal(ya[k], ref[k]), f"stream 1, step {k}"
            assert torch.equal(yb[k], ref[k]), f"stream 2, step {k}"
        log(f"  {len(steps)} steps bitwise equal on both streams")
    finally:
        alone.close()
        a.close()
        b.close()
