"""The FLOP/byte roofline of a stage step (the paper's Eq. 1, Sec. 4.1.1,
with the per-op counts of Table 2 corrected).

Eq. 1 prices each operation as max(FLOPs / peak FLOPS, bytes / peak HBM
bandwidth) and sums over operations. Corrections to Table 2 used here:
the K/V projection width is n_kv * d (Table 2's H_kv is the total KV width),
q width n_q * d may differ from H (Qwen3), attention counts only causal
(query, key) pairs, decode attention is summed over the batch, and outputs
are counted in the memory terms.
"""

from __future__ import annotations

from typing import Iterable, Sequence, Tuple

import numpy as np

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA


def gemm_bytes(M: int, N: int, K: int, out_bytes: int) -> int:
    """Algorithmic HBM bytes of one GEMM launch: W and A (bf16) read once,
    the output written once."""
    return N * K * 2 + M * K * 2 + M * N * out_bytes


def gate_up_swiglu_bytes(shape, M: int) -> int:
    """Algorithmic HBM bytes of one fused gate-up + SwiGLU launch over M rows:
    the [2F, H] bf16 weight and the [M, H] bf16 input read once, the [M, F]
    bf16 product m written once."""
    F, H = shape.ffn, shape.hidden
    return 2 * F * H * 2 + M * H * 2 + M * F * 2


def linear_shapes(shape) -> Sequence[Tuple[int, int]]:
    """(N, K) of the four projections of a layer."""
    H, d, F = shape.hidden, shape.head_dim, shape.ffn
    qkvw = (shape.n_q_heads + 2 * shape.n_kv_heads) * d
    return ((qkvw, H), (H, shape.n_q_heads * d), (2 * F, H), (H, F))


def kv_bytes_per_token(shape) -> int:
    return 2 * shape.n_kv_heads * shape.head_dim * 2


def decode_step_bytes(shape, n_layers: int, ctx_lens) -> float:
    """Algorithmic bytes of one decode step: every weight once, the valid KV
    of every sequence once per layer (its own new token included), and the
    hidden rows in and out."""
    B = len(ctx_lens)
    per_layer = shape.params_per_layer() * 2 + float(np.sum(np.asarray(ctx_lens) + 1)) * \
        kv_bytes_per_token(shape)
    return n_layers * per_layer + 2 * B * shape.hidden * 2


def attention_pairs(chunks: Iterable[Tuple[int, int]]) -> float:
    """Causal (query, key) pairs of prefill chunks given as (ctx, q)."""
    return sum(float(q) * ctx + q * (q + 1) / 2.0 for ctx, q in chunks)


def prefill_flops(shape, n_layers: int, chunks) -> float:
    """Algorithmic FLOPs of prefill chunks: 2 * (linear weights) per token
    plus 4 * d * n_q per causal (query, key) pair."""
    lin = 2.0 * sum(N * K for N, K in linear_shapes(shape))
    toks = float(sum(q for _, q in chunks))
    return n_layers * (toks * lin +
                       4.0 * shape.head_dim * shape.n_q_heads * attention_pairs(chunks))


def step_roofline_ms(shape, n_layers: int, chunks, dec_ctx,
                     peak_tflops: float = BF16_PEAK_TFLOPS, peak_gbs: float = HBM_PEAK_GBS):
    """Eq. 1 for one step: sum over ops of max(F / peak, B / bandwidth).
    chunks: prefill chunks (ctx, q); dec_ctx: contexts of the decode tokens."""
    d, nq = shape.head_dim, shape.n_q_heads
    T = sum(q for _, q in chunks) + len(dec_ctx)
    t = 0.0
    for N, K in linear_shapes(shape):
        t += max(2.0 * T * N * K / (peak_tflops * 1e12),
                 (N * K * 2 + T * K * 2 + T * N * 2) / (peak_gbs * 1e9))
    kvt = kv_bytes_per_token(shape)
    if chunks:
        fl = 4.0 * d * nq * attention_pairs(chunks)
        by = sum(float(c + q) for c, q in chunks) * kvt + 2.0 * sum(q for _, q in chunks) * nq * d * 2
        t += max(fl / (peak_tflops * 1e12), by / (peak_gbs * 1e9))
    if len(dec_ctx):
        keys = float(np.sum(np.asarray(dec_ctx) + 1))
        t += max(4.0 * d * nq * keys / (peak_tflops * 1e12), keys * kvt / (peak_gbs * 1e9))
    return n_layers * t * 1e3
