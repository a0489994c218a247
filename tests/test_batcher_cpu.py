"""Continuous-batching host logic (the driver of the 80-layer workload):
admission on the KV pool, the per-step plan and the block accounting. CPU
only; no stage is run."""

import numpy as np
import pytest

from paper_2606_18600_amd.batcher import Batcher, Request


def _held(b):
    return [blk for r in b.running for blk in r.blocks]


def _check_blocks(b, num_blocks):
    held = _held(b)
    assert len(held) == len(set(held)), "a block is held twice"
    assert not set(held) & set(b.alloc.free), "a held block is also free"
    assert len(held) + len(b.alloc.free) == num_blocks


def test_admission_reserves_the_whole_lifetime_and_keeps_fifo_order():
    b = Batcher(num_blocks=10, max_blocks_per_seq=8, max_decodes=4, prefill_budget=64)
    b.submit(Request(0, prompt=40, out=24, arrival=0.0))   # 4 blocks
    b.submit(Request(1, prompt=80, out=20, arrival=0.0))   # 7 blocks: does not fit after #0
    b.submit(Request(2, prompt=10, out=5, arrival=0.0))    # 1 block, but behind #1
    b.admit(0.0)
    assert [r.rid for r in b.running] == [0]
    assert len(b.running[0].blocks) == 4
    assert [r.rid for r in b.queue] == [1, 2]               # no overtaking
    _check_blocks(b, 10)


def test_requests_wait_for_their_arrival_time():
    b = Batcher(num_blocks=100, max_blocks_per_seq=16)
    b.submit(Request(0, 16, 4, arrival=1.0))
    b.admit(0.5)
    assert not b.running
    b.admit(1.0)
    assert [r.rid for r in b.running] == [0]


def test_plan_respects_the_prefill_budget_and_the_decode_cap():
    b = Batcher(num_blocks=1000, max_blocks_per_seq=64, max_decodes=3, prefill_budget=100)
    for i in range(5):                                      # 5 in decode phase
        r = Request(i, prompt=32, out=8, arrival=0.0)
        r.prefilled = 32
        r.blocks = b.alloc.take(r.need_blocks(16))
        b.running.append(r)
    for i in range(5, 8):                                   # 3 waiting for prefill
        b.submit(Request(i, prompt=70, out=8, arrival=0.0))
    b.admit(0.0)
    prefill, decodes = b.plan()
    assert len(decodes) == 3
    assert sum(q for _, _, q in prefill) == 100
    # first come first served: request 5 whole, then 30 tokens of request 6
    assert [(r.rid, c, q) for r, c, q in prefill] == [(5, 0, 70), (6, 0, 30)]
    b.commit(prefill, decodes)
    prefill, _ = b.plan()
    assert [(r.rid, c, q) for r, c, q in prefill] == [(6, 30, 40), (7, 0, 60)]


def test_block_tables_hold_each_requests_blocks():
    b = Batcher(num_blocks=50, max_blocks_per_seq=8)
    for i in range(3):
        b.submit(Request(i, prompt=20 + 10 * i, out=10, arrival=0.0))
    b.admit(0.0)
    bt = b.tables(b.running)
    for row, r in zip(bt, b.running):
        assert list(row[: len(r.blocks)]) == list(r.blocks)
        assert (row[len(r.blocks):] == 0).all()


@pytest.mark.parametrize("seed", [0, 1])
def test_simulation_runs_every_request_to_completion(seed):
    rng = np.random.default_rng(seed)
    nb = 120
    b = Batcher(num_blocks=nb, max_blocks_per_seq=40, max_decodes=6, prefill_budget=96,
                seed=seed)
    reqs = [Request(i, int(rng.integers(1, 300)), int(rng.integers(1, 60)), 0.0)
            for i in range(40)]
    for r in reqs:
        b.submit(r)
    steps = 0
    while b.queue or b.running:
        b.admit(0.0)
        prefill, decodes = b.plan()
        assert prefill or decodes, "stalled with work left"
        for r, c, q in prefill:                             # chunks continue where they stopped
            assert c == r.prefilled and 1 <= q <= r.prompt - r.prefilled
        for r in decodes:
            assert r.in_decode and not r.done
            # the token decoded this step fits in the reserved blocks
            assert r.prompt + r.decoded + 1 <= 16 * len(r.blocks)
        b.commit(prefill, decodes)
        _check_blocks(b, nb)
        steps += 1
        assert steps < 10000
    assert b.finished == len(reqs)
    assert all(r.prefilled == r.prompt and r.decoded == r.out for r in reqs)
    assert sorted(b.alloc.free) == list(range(nb))


def test_sustainable_rate_balances_prefill_with_decode():
    """At the roofline-sustainable rate the prefill tokens of a step keep pace
    with its decodes: P / mean_prompt requests start per step while
    max_decodes / mean_out finish, and the rate is that count over the
    step's Eq. 1 time."""
    from paper_2606_18600_amd import synth
    from paper_2606_18600_amd.batcher import lognormal_mean, sustainable_rate
    from paper_2606_18600_amd.roofline import step_roofline_ms
    mean_out = lognormal_mean(256, 0.8)
    assert mean_out == pytest.approx(256 * np.exp(0.32))
    rate, ms, P = sustainable_rate(synth.LLAMA70B, 80, 2560.0, mean_out)
    assert P == round(128 * 2560.0 / mean_out)
    assert P / 2560.0 == pytest.approx(128 / mean_out, rel=1e-3)
    expect = step_roofline_ms(synth.LLAMA70B, 80, [((2560.0 - P) / 2, P)],
                              np.full(128, 2560.0 + mean_out / 2))
    assert ms == pytest.approx(expect)
    assert rate == pytest.approx(128 / mean_out / (ms / 1e3), rel=1e-3)
    # prompts so long that the budget binds: prefill-limited
    rate2, _, P2 = sustainable_rate(synth.LLAMA70B, 80, 40000.0, 100.0)
    assert P2 == 2048
    assert rate2 < 128 / 100.0 / (ms / 1e3)
