"""The step roofline (the paper's Eq. 1 with corrected Table 2 counts) against
hand-computed values (CPU only)."""

import numpy as np
import pytest

from paper_2606_18600_amd import roofline as R
from paper_2606_18600_amd import synth


def test_linear_weights_of_the_llama70b_layer():
    # q 64*128 + k,v 2*8*128 = 10240 rows of 8192; O 8192x8192; gate-up 2*28672x8192; down 8192x28672
    n = sum(N * K for N, K in R.linear_shapes(synth.LLAMA70B))
    assert n == 10240 * 8192 + 8192 * 8192 + 57344 * 8192 + 8192 * 28672 == 855_638_016
    assert synth.LLAMA70B.params_per_layer() == n + 2 * 8192


def test_qwen3_q_width_differs_from_hidden():
    shapes = R.linear_shapes(synth.QWEN32B)
    assert shapes[0] == ((64 + 16) * 128, 5120)     # QKV: q width 8192 + k,v 2048
    assert shapes[1] == (5120, 8192)                # O reads the 8192-wide attention output


def test_decode_step_bytes_of_the_l70_stage():
    # 20 layers, 64 sequences of 1242 cached tokens: weights once + valid KV once
    ctx = np.full(64, 1242)
    w = 20 * synth.LLAMA70B.params_per_layer() * 2
    kv = 20 * 64 * 1243 * (2 * 8 * 128 * 2)
    io = 2 * 64 * 8192 * 2
    assert R.decode_step_bytes(synth.LLAMA70B, 20, ctx) == pytest.approx(w + kv + io, rel=1e-12)
    assert w / 1e9 == pytest.approx(34.23, abs=0.01)


def test_causal_pairs():
    # a fresh chunk of q tokens sees q(q+1)/2 pairs; a chunk after ctx cached tokens adds q*ctx
    assert R.attention_pairs([(0, 4)]) == 10
    assert R.attention_pairs([(100, 3)]) == 300 + 6
    assert R.attention_pairs([(0, 2), (5, 1)]) == 3 + 6


def test_step_roofline_decode_is_bytes_over_bandwidth():
    # B=64 decode is memory bound on every op: time = bytes / 8 TB/s (plus the small
    # activation terms the per-op form counts)
    shape = synth.LLAMA70B
    ctx = np.full(64, 1242)
    t = R.step_roofline_ms(shape, 20, [], ctx)
    lin = sum(N * K * 2 + 64 * K * 2 + 64 * N * 2 for N, K in R.linear_shapes(shape))
    kv = 64 * 1243 * R.kv_bytes_per_token(shape)
    assert t == pytest.approx(20 * (lin + kv) / 8e12 * 1e3, rel=1e-12)
    assert 5.0 < t < 5.3


def test_step_roofline_prefill_is_flops_over_peak():
    shape = synth.LLAMA70B
    chunks = [(0, 2048)]
    t = R.step_roofline_ms(shape, 20, chunks, [])
    lin = 2.0 * 2048 * 855_638_016
    attn = 4.0 * 128 * 64 * (2048 * 2049 / 2)
    assert t == pytest.approx(20 * (lin + attn) / 2.5e15 * 1e3, rel=1e-9)


def test_gate_up_swiglu_bytes_of_the_llama70b_decode_launch():
    # [57344, 8192] bf16 weight + [64, 8192] bf16 input + [64, 28672] bf16 product
    assert R.gate_up_swiglu_bytes(synth.LLAMA70B, 64) == 939524096 + 1048576 + 3670016

