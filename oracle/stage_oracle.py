"""CPU oracle for one pipeline stage's forward pass (TEST INFRASTRUCTURE).

This module is the parity checker for the HIP stage library, nothing more.
Only code under ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it. The product path never
calls it, and it shares no code, tables or helpers with the HIP path.

What it computes
----------------
ShuntServe partitions a decoder-only LLM into *stages*: contiguous ranges of
transformer layers, each assigned to one device (paper Sec. 2.3, "Uneven
Layer Partitioning in PP"; Algorithm 1 grows a placement one stage of
``l - l'`` consecutive layers at a time). Consecutive stages exchange only the
hidden-state tensor, B*S*H*E bytes (Sec. 4.1.2, Eq. 2). The per-layer work
the paper's estimator prices is attention followed by a gated FFN: the QKV
projection, attention, output projection, up-and-gate projection and down
projection rows of Table 2 (Sec. 4.1.1). The models the paper serves are
Llama-3.1-70B and Qwen3-32B in BF16 (Sec. 7, "Model and Cluster Setup"), so a
layer is the pre-norm Llama/Qwen3 block: RMSNorm, grouped-query attention with
rotary position embedding (plus per-head RMSNorm of q and k for Qwen3), a
residual add, RMSNorm, a SwiGLU FFN and a second residual add.

Paging, chunked prefill and continuous batching do not change the result in
real arithmetic; they only change where keys live and which rows share a
call. The oracle therefore evaluates the textbook definition directly: each
sequence's keys and values are gathered from the paged cache into contiguous
arrays and attention is a dense masked softmax over them.

Conventions where the paper is silent (each is listed, with its reason, in the
design notes of the repository):

* RMSNorm: ``x / sqrt(mean(x^2) + eps) * g`` over the last axis.
* RoPE: "rotate-half" pairing of element ``j`` with ``j + d/2``, angle
  ``p * theta^(-2j/d)``, 0-based positions, no frequency scaling.
* GQA: query head ``h`` reads kv head ``h // (n_q / n_kv)``.
* Attention scale ``1/sqrt(d)``, inclusive causal mask (a query sees itself),
  no bias, soft-cap or window.
* SwiGLU: ``silu(h W_g^T) * (h W_u^T)`` with ``silu(z) = z / (1 + e^-z)``.
* Weights are row-major ``[N, K]`` and applied as ``y = x W^T``. ``w_qkv``
  stacks the q rows, then k, then v; ``w_gate_up`` stacks gate rows then up.
* KV cache (the oracle's own layout): per layer ``k`` and ``v`` arrays of
  shape ``[num_blocks, block_size, n_kv, d]``. Token ``p`` of a sequence with
  block table ``bt`` lives at ``(bt[p // block_size], p % block_size)``.

Precision: float64 by default; ``dtype=np.float32`` runs the same code in
float32 (used only to time a CPU baseline). A diagnostic sub-mode
(``rounding=round_to_bf16``) rounds to bfloat16 at the points where a bf16
stage stores values (norm outputs, q, k, v, attention probabilities before
they weight v, the attention output, the SwiGLU output). It is never the
parity reference; it measures how far bf16 storage alone moves the result
(the floor any bf16 implementation shares).

Parity status: every function here is pinned by ``tests/test_oracle_*.py``
(closed forms, invariants, brute force and an independent library
implementation of the decoder layer).
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Sequence

import numpy as np

__all__ = [
    "OracleConfig",
    "SeqSpec",
    "new_kv_cache",
    "rms_norm",
    "silu",
    "rope",
    "round_to_bf16",
    "slot_of",
    "attention_one_sequence",
    "project_qkv",
    "layer_forward",
    "stage_forward",
]


@dataclass(frozen=True)
class OracleConfig:
    """Shape and constants of one decoder layer.

    ``qk_norm`` selects the Qwen3 variant with per-head RMSNorm on q and k.
    """

    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    rms_eps: float
    rope_theta: float
    qk_norm: bool = False
    qk_rms_eps: float = 1e-6
    block_size: int = 16

    @property
    def q_width(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_width(self) -> int:
        return self.n_kv_heads * self.head_dim


@dataclass
class SeqSpec:
    """One sequence of a step: ``ctx_len`` tokens already cached, ``q_len``
    new tokens in this call (a decode step has ``q_len == 1``), and its block
    table (a list of block ids, long enough for ``ctx_len + q_len``)."""

    ctx_len: int
    q_len: int
    block_table: Sequence[int]


def new_kv_cache(cfg: OracleConfig, n_layers: int, num_blocks: int,
                 dtype=np.float64) -> List[Dict[str, np.ndarray]]:
    """A zeroed paged KV cache: one ``{'k','v'}`` pair of
    ``[num_blocks, block_size, n_kv, d]`` arrays per layer of the stage."""
    shape = (num_blocks, cfg.block_size, cfg.n_kv_heads, cfg.head_dim)
    return [{"k": np.zeros(shape, dtype), "v": np.zeros(shape, dtype)}
            for _ in range(n_layers)]


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """Root-mean-square normalisation over the last axis, times gain ``g``."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def silu(z: np.ndarray) -> np.ndarray:
    """SiLU / swish: ``z * sigmoid(z)``."""
    return z / (1.0 + np.exp(-z))


def rope(u: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotary position embedding, rotate-half pairing.

    ``u``: ``[n, heads, d]``; ``pos``: ``[n]`` integer positions. Element
    ``j < d/2`` is paired with ``j + d/2`` and the pair is rotated by the angle
    ``pos * theta**(-2j/d)``. Angles are formed in float64 whatever the dtype
    of ``u``.
    """
    d = u.shape[-1]
    half = d // 2
    j = np.arange(half, dtype=np.float64)
    omega = theta ** (-2.0 * j / d)                       # [d/2]
    ang = pos.astype(np.float64)[:, None] * omega[None]   # [n, d/2]
    c = np.cos(ang)[:, None, :].astype(u.dtype)
    s = np.sin(ang)[:, None, :].astype(u.dtype)
    a, b = u[..., :half], u[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 value (ties to even), returned in the
    input dtype: keep the top 16 bits of the float32 representation after
    adding half an ulp of bfloat16 (plus the tie-breaking bit)."""
    f = np.asarray(a, np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.asarray(a).dtype)


def slot_of(block_table: Sequence[int], p: int, block_size: int):
    """(block id, offset) holding position ``p`` of a sequence."""
    return int(block_table[p // block_size]), p % block_size


def attention_one_sequence(q: np.ndarray, k_all: np.ndarray, v_all: np.ndarray,
                           q_pos: np.ndarray, rounding=None) -> np.ndarray:
    """Causal grouped-query attention for one sequence.

    ``q``: ``[n, n_q, d]`` queries at positions ``q_pos``; ``k_all``,
    ``v_all``: ``[C, n_kv, d]`` keys/values of positions ``0..C-1``.
    Query at position ``p`` attends to keys ``t <= p``. Returns
    ``[n, n_q, d]``.
    """
    n, n_q, d = q.shape
    n_kv = k_all.shape[1]
    group = n_q // n_kv
    C = k_all.shape[0]
    out = np.empty_like(q)
    t = np.arange(C)
    visible = t[None, :] <= q_pos[:, None]                # [n, C]
    scale = 1.0 / np.sqrt(d)
    for h in range(n_q):
        kvh = h // group
        s = (q[:, h, :] @ k_all[:, kvh, :].T) * scale     # [n, C]
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        if rounding is None:
            p = p / p.sum(axis=1, keepdims=True)
        else:
            p = rounding(p) / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v_all[:, kvh, :]
    return out


def project_qkv(cfg: OracleConfig, w: Dict[str, np.ndarray], x: np.ndarray,
                pos: np.ndarray, rounding=None):
    """The attention inputs of a layer for rows ``x`` ``[T, H]`` at positions
    ``pos`` ``[T]``: RMSNorm, the QKV projection, (Qwen3) per-head RMSNorm of
    q and k, and RoPE of q and k. Returns ``q`` ``[T, n_q, d]`` and the keys
    and values the layer writes to its cache, ``k``, ``v`` ``[T, n_kv, d]``."""
    rnd = rounding if rounding is not None else (lambda a: a)
    nq, nkv, d = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    T = x.shape[0]
    h = rnd(rms_norm(x, w["attn_norm"], cfg.rms_eps))
    qkv = h @ w["w_qkv"].T                                 # [T, (nq+2nkv)d]
    q = qkv[:, :nq * d].reshape(T, nq, d)
    k = qkv[:, nq * d:(nq + nkv) * d].reshape(T, nkv, d)
    v = qkv[:, (nq + nkv) * d:].reshape(T, nkv, d)
    if cfg.qk_norm:
        q = rms_norm(q, w["q_norm"], cfg.qk_rms_eps)
        k = rms_norm(k, w["k_norm"], cfg.qk_rms_eps)
    q = rnd(rope(q, pos, cfg.rope_theta))
    k = rnd(rope(k, pos, cfg.rope_theta))
    v = rnd(v)
    return q, k, v


def layer_forward(cfg: OracleConfig, w: Dict[str, np.ndarray], x: np.ndarray,
                  seqs: Sequence[SeqSpec], kv: Dict[str, np.ndarray],
                  rounding=None) -> np.ndarray:
    """One pre-norm decoder layer over a packed batch.

    ``x``: ``[T, H]`` rows of all sequences packed in order (``q_len`` rows
    each). The new keys and values are written into ``kv`` (this layer's
    cache) at their slots before attention reads the sequence back. Returns
    the updated residual stream ``[T, H]``.
    """
    dt = x.dtype
    rnd = rounding if rounding is not None else (lambda a: a)
    H, nq, nkv, d = cfg.hidden, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    T = x.shape[0]
    assert T == sum(s.q_len for s in seqs)

    # attention branch
    pos = np.concatenate([np.arange(s.ctx_len, s.ctx_len + s.q_len) for s in seqs]) \
        if T else np.zeros(0, np.int64)
    q, k, v = project_qkv(cfg, w, x, pos, rounding)

    attn = np.empty((T, nq, d), dt)
    row = 0
    for s in seqs:
        rows = slice(row, row + s.q_len)
        for i in range(s.q_len):
            b, o = slot_of(s.block_table, s.ctx_len + i, cfg.block_size)
            kv["k"][b, o] = k[row + i]
            kv["v"][b, o] = v[row + i]
        C = s.ctx_len + s.q_len
        k_all = np.stack([kv["k"][slot_of(s.block_table, t, cfg.block_size)] for t in range(C)])
        v_all = np.stack([kv["v"][slot_of(s.block_table, t, cfg.block_size)] for t in range(C)])
        attn[rows] = attention_one_sequence(q[rows], k_all, v_all, pos[rows], rounding)
        row += s.q_len

    x = x + rnd(attn.reshape(T, nq * d)) @ w["w_o"].T

    # FFN branch
    h2 = rnd(rms_norm(x, w["ffn_norm"], cfg.rms_eps))
    gu = h2 @ w["w_gate_up"].T                              # [T, 2F]
    m = rnd(silu(gu[:, :cfg.ffn]) * gu[:, cfg.ffn:])
    x = x + m @ w["w_down"].T
    return x


def lm_head(cfg: OracleConfig, x: np.ndarray, final_norm: np.ndarray,
            w_lm: np.ndarray) -> np.ndarray:
    """Logits of the last pipeline stage (Table 2, "Logits Calculation"):
    the model's final RMSNorm of each selected output row ``x`` ``[n, H]``,
    then the vocabulary projection ``w_lm`` ``[V, H]``. Returns ``[n, V]``."""
    return rms_norm(x, final_norm, cfg.rms_eps) @ w_lm.T


def stage_forward(cfg: OracleConfig, layers: Sequence[Dict[str, np.ndarray]],
                  x: np.ndarray, seqs: Sequence[SeqSpec],
                  kv_cache: Sequence[Dict[str, np.ndarray]], dtype=np.float64,
                  rounding=None) -> np.ndarray:
    """Forward pass of one stage: the layers of ``layers`` applied in order.

    ``layers[i]`` and ``kv_cache[i]`` belong to the i-th layer of the stage's
    contiguous range. ``x`` is the stage input ``[T, H]`` (the previous
    stage's hidden states); the return value is the stage output, which the
    next stage would receive. Weights are cast to ``dtype`` on use; the KV
    cache is updated in place.
    """
    x = np.asarray(x, dtype)
    for w, kv in zip(layers, kv_cache):
        wd = {name: np.asarray(a, dtype) for name, a in w.items()}
        x = layer_forward(cfg, wd, x, seqs, kv, rounding)
    return x
