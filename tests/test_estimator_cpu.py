"""The static latency estimator (host math, no GPU): its operation counts
against Table 2 wherever Table 2 is right, the corrections where it is not,
Eq. 1's max, chunking invariance, and the Eq. 3/4 and communication terms."""

from __future__ import annotations

import math

import pytest

from paper_2606_18600_amd import estimator as E
from paper_2606_18600_amd import synth

L70 = synth.LLAMA70B


def _by_name(ops):
    return {o.name: o for o in ops}


@pytest.mark.parametrize("tp", [1, 2, 4, 8])
def test_prefill_counts_match_table2(tp):
    """Table 2, prefill rows, Llama-3.1-70B (H = n_q * d, so Table 2's H^2
    terms hold), one TP rank of `tp`; E = 2."""
    B, S = 3, 763
    H, F, Hkv = 8192, 28672, 8 * 128
    ops = _by_name(E.prefill_ops(E.tp_shard(L70, tp), [(0, S)] * B))
    T = B * S
    assert ops["qkv"].flops == B * (2 * S * H * H + 4 * S * H * Hkv) / tp
    assert ops["o_proj"].flops == 2 * B * S * H * H / tp
    assert ops["gate_up"].flops == 4 * B * S * H * F / tp
    assert ops["down"].flops == 2 * B * S * H * F / tp
    # Table 2 prices the full S x S score matrix; only causal pairs are computed
    assert math.isclose(ops["attention"].flops, 4 * B * S * S * H / tp * (S + 1) / (2 * S))
    # memory scans: Table 2's terms plus each op's output
    assert ops["qkv"].bytes / 2 - T * (H + 2 * Hkv) / tp == B * S * H + (H * H + 2 * H * Hkv) / tp
    assert ops["o_proj"].bytes / 2 - T * H == (B * S * H + H * H) / tp
    assert ops["gate_up"].bytes / 2 - T * F / tp == B * S * H + 2 * H * F / tp
    assert ops["down"].bytes / 2 - T * H == (B * S * F + H * F) / tp
    # attention reads the queries and every visible key/value once
    assert ops["attention"].bytes / 2 - T * H / tp == (B * S * H + 2 * B * S * Hkv) / tp


@pytest.mark.parametrize("tp", [1, 8])
def test_decode_counts_match_table2(tp):
    """Table 2, decode rows, for one step t (S_out = 1 in its sums)."""
    B, s_in, t = 5, 763, 17
    H, F, Hkv = 8192, 28672, 8 * 128
    ops = _by_name(E.decode_ops(E.tp_shard(L70, tp), [s_in + t - 1] * B))
    assert ops["qkv"].flops == B * (2 * H * H + 4 * H * Hkv) / tp
    assert ops["o_proj"].flops == 2 * B * H * H / tp
    assert ops["gate_up"].flops == 4 * B * H * F / tp
    assert ops["down"].flops == 2 * B * H * F / tp
    # Table 2's decode attention term omits the batch
    assert ops["attention"].flops == B * 4 * (s_in + t) * H / tp
    assert ops["qkv"].bytes / 2 - B * (H + 2 * Hkv) / tp == B * H + (H * H + 2 * H * Hkv) / tp
    assert ops["attention"].bytes / 2 - B * H / tp == (B * H + 2 * B * (s_in + t) * Hkv) / tp
    assert ops["gate_up"].bytes / 2 - B * F / tp == B * H + 2 * H * F / tp
    assert ops["down"].bytes / 2 - B * H == (B * F + H * F) / tp


def test_qwen3_query_width_differs_from_hidden():
    q = synth.QWEN32B   # H 5120, 64 x 128 = 8192 query width
    ops = _by_name(E.decode_ops(q, [100]))
    assert ops["o_proj"].flops == 2 * 8192 * 5120
    assert ops["qkv"].flops == 2 * 5120 * (8192 + 2 * 8 * 128)


def test_eq1_takes_the_larger_term():
    cal = E.Calibration(tflops=1000.0, gbs=5000.0)
    # memory-bound: 1 GFLOP, 1 GB -> 1 us compute vs 200 us memory
    assert math.isclose(E.op_ms(E.Op("x", 1e9, 1e9), cal), 0.2)
    # compute-bound: 1 TFLOP, 1 MB
    assert math.isclose(E.op_ms(E.Op("y", 1e12, 1e6), cal), 1.0)
    dec = _by_name(E.decode_ops(L70, [1000]))
    pre = _by_name(E.prefill_ops(L70, [(0, 2048)]))
    g = dec["gate_up"]
    assert E.op_ms(g, E.DATASHEET) == g.bytes / (E.DATASHEET.gbs * 1e9) * 1e3
    p = pre["gate_up"]
    assert E.op_ms(p, E.DATASHEET) == p.flops / (E.DATASHEET.tflops * 1e12) * 1e3


def test_chunked_prefill_has_the_same_flops():
    """Splitting prompts into steps leaves the projection FLOPs and the causal
    pair count unchanged; a compute-bound prefill is priced the same."""
    cal = E.Calibration(tflops=1.0, gbs=1e12)  # everything compute-bound
    for B in (1, 3, 32):
        one, _ = E.static_batch_ms(L70, 2, B, 763, 0, cal)
        chunked, _ = E.static_batch_ms(L70, 2, B, 763, 0, cal, prefill_chunk=2048)
        assert math.isclose(one, chunked, rel_tol=1e-12)


def test_static_batch_decode_sum():
    cal = E.Calibration(tflops=1e9, gbs=1.0)  # memory-bound
    _, dc = E.static_batch_ms(L70, 1, 2, 10, 3, cal)
    by = sum(sum(o.bytes for o in E.decode_ops(L70, [10 + t - 1] * 2)) for t in (1, 2, 3))
    assert math.isclose(dc, by / 1e9 * 1e3)


def test_tp_shard_shapes():
    s8 = E.tp_shard(L70, 8)
    assert (s8.n_q_heads, s8.n_kv_heads, s8.ffn, s8.hidden) == (8, 1, 3584, 8192)
    assert E.tp_shard(L70, 1) is L70
    with pytest.raises(ValueError):
        E.tp_shard(L70, 16)
    with pytest.raises(ValueError):
        E.tp_shard(L70, 3)


def test_throughput_and_communication_terms():
    assert E.pipeline_latency_ms([3.0, 5.0, 4.0], [20.0, 10.0, 30.0]) == 35.0
    assert E.requests_per_second(32, 2000.0) == 16.0
    # L_PP: alpha + B*S*H*E / beta
    assert math.isclose(E.comm_pp_ms(1e-5, 10.0, 4, 1, 8192), (1e-5 + 4 * 8192 * 2 / 1e10) * 1e3)
    assert E.comm_tp_ms(1e-5, 100.0, 4, 1, 8192, 1, 80) == 0.0
    # ring all-reduce: reduce-scatter + all-gather, each tp-1 steps of n/tp
    # bytes; two all-reduces per layer
    a, b, tp, layers, n = 2e-6, 50.0, 4, 10, 64 * 8192 * 2
    steps = 2 * 2 * (tp - 1) * layers
    assert math.isclose(E.comm_tp_ms(a, b, 64, 1, 8192, tp, layers),
                        steps * (a + n / tp / (b * 1e9)) * 1e3)


def test_mape():
    assert E.mape([110, 90], [100, 100]) == pytest.approx(10.0)
    assert E.mape([1.0], [1.0]) == 0.0


def test_launch_cost_adds_per_kernel_of_each_step():
    base = E.Calibration(tflops=1000.0, gbs=5000.0)
    lat = E.Calibration(tflops=1000.0, gbs=5000.0, launch_us=4.0)
    n_layers, B, s_in, s_out = 10, 3, 763, 5
    pf0, dc0 = E.static_batch_ms(L70, n_layers, B, s_in, s_out, base, prefill_chunk=2048)
    pf1, dc1 = E.static_batch_ms(L70, n_layers, B, s_in, s_out, lat, prefill_chunk=2048)
    steps = len(synth.chunk_schedule([s_in] * B, 2048))  # 2 steps: 2048 + 241 tokens
    assert steps == 2
    assert math.isclose(pf1 - pf0, steps * (n_layers * 8 + 2) * 4.0e-3)
    assert math.isclose(dc1 - dc0, s_out * (n_layers * 10 + 2) * 4.0e-3)
