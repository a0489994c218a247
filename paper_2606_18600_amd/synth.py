"""Seeded synthetic workloads for the stage: model shapes, weights, batches.

This module only draws random numbers and lays out batches; it holds none of
the stage's arithmetic. Tests feed the same draws to the HIP stage and to the
CPU oracle; the bench uses it to build its workloads.

Model shapes follow the two models the paper serves, Llama-3.1-70B and
Qwen3-32B in BF16 (Sec. 7, "Model and Cluster Setup"), plus a tiny
Llama-style shape for parity at sizes a CPU finishes in seconds. The paper
publishes no weights or traces usable here, so every tensor is random:
projection weights are N(0, 0.02^2); norm gains are 1 + N(0, 0.02^2) so that
each layer is not close to the identity; stage inputs are N(0, 1).
"""

from __future__ import annotations

from dataclasses import dataclass, replace
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

BLOCK = 16

# Tensor ids keep every weight's random stream distinct and independent of
# which other tensors are drawn.
_TENSOR_IDS = {"attn_norm": 0, "w_qkv": 1, "q_norm": 2, "k_norm": 3, "w_o": 4,
               "ffn_norm": 5, "w_gate_up": 6, "w_down": 7}
GAIN_NAMES = ("attn_norm", "q_norm", "k_norm", "ffn_norm")


@dataclass(frozen=True)
class ModelShape:
    name: str
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    rms_eps: float
    rope_theta: float
    qk_norm: bool = False
    qk_rms_eps: float = 1e-6
    block_size: int = BLOCK

    @property
    def q_width(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_width(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def qkv_width(self) -> int:
        return self.q_width + 2 * self.kv_width

    def weight_shapes(self) -> Dict[str, Tuple[int, ...]]:
        H, d, F = self.hidden, self.head_dim, self.ffn
        shapes = {"attn_norm": (H,), "w_qkv": (self.qkv_width, H),
                  "w_o": (H, self.q_width), "ffn_norm": (H,),
                  "w_gate_up": (2 * F, H), "w_down": (H, F)}
        if self.qk_norm:
            shapes["q_norm"] = (d,)
            shapes["k_norm"] = (d,)
        return shapes

    def params_per_layer(self) -> int:
        return int(sum(np.prod(s) for s in self.weight_shapes().values()))


TINY = ModelShape("tiny-llama", hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                  ffn=704, rms_eps=1e-5, rope_theta=5e5)
LLAMA70B = ModelShape("llama-3.1-70b", hidden=8192, n_q_heads=64, n_kv_heads=8,
                      head_dim=128, ffn=28672, rms_eps=1e-5, rope_theta=5e5)
QWEN32B = ModelShape("qwen3-32b", hidden=5120, n_q_heads=64, n_kv_heads=8, head_dim=128,
                     ffn=25600, rms_eps=1e-6, rope_theta=1e6, qk_norm=True, qk_rms_eps=1e-6)
SHAPES = {s.name: s for s in (TINY, LLAMA70B, QWEN32B)}


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng([int(k) & 0xFFFFFFFF for k in key])


def host_layer_weights(shape: ModelShape, seed: int, global_layer: int,
                       std: float = 0.02, gain_std: float = 0.02,
                       dtype=np.float32) -> Dict[str, np.ndarray]:
    """Random weights of one layer, drawn on the host in float64 and stored
    in ``dtype``. The stream of each tensor is keyed by
    (seed, global layer index, tensor id)."""
    out = {}
    for name, shp in shape.weight_shapes().items():
        r = _rng(seed, global_layer, _TENSOR_IDS[name])
        if name in GAIN_NAMES:
            a = 1.0 + gain_std * r.standard_normal(shp)
        else:
            a = std * r.standard_normal(shp)
        out[name] = a.astype(dtype)
    return out


def hidden_states(seed: int, stream: int, T: int, H: int, dtype=np.float32) -> np.ndarray:
    """Stage input rows, N(0, 1)."""
    return _rng(seed, 0x5EED, stream).standard_normal((T, H)).astype(dtype)


@dataclass
class Batch:
    """A step's request batch as the stage sees it."""
    ctx_lens: np.ndarray     # int32 [S] tokens cached before the step
    q_lens: np.ndarray       # int32 [S] new tokens in the step
    block_tables: np.ndarray  # int32 [S, max_blocks]

    @property
    def num_seqs(self) -> int:
        return int(len(self.q_lens))

    @property
    def num_tokens(self) -> int:
        return int(self.q_lens.sum())


class BlockAllocator:
    """Hands out KV-block ids from a shuffled free list, so block tables are
    scattered across the pool as in a long-running paged cache."""

    def __init__(self, num_blocks: int, seed: int, reserve_zero: bool = False):
        r = _rng(seed, 0xB10C)
        ids = np.arange(num_blocks, dtype=np.int32)
        if reserve_zero:
            ids = ids[1:]
        self.free: List[int] = list(r.permutation(ids))

    def take(self, n: int) -> List[int]:
        if n > len(self.free):
            raise MemoryError(f"KV pool exhausted: need {n} blocks, {len(self.free)} free")
        out, self.free = self.free[:n], self.free[n:]
        return out

    def give_back(self, ids: Sequence[int]) -> None:
        self.free.extend(int(i) for i in ids)


def make_block_tables(total_lens: Sequence[int], max_blocks: int,
                      alloc: BlockAllocator, block: int = BLOCK) -> np.ndarray:
    """Block table rows long enough for each sequence's final length; unused
    entries are 0 (never read, since reads stop at the sequence length)."""
    bt = np.zeros((len(total_lens), max_blocks), np.int32)
    for i, n in enumerate(total_lens):
        nb = (int(n) + block - 1) // block
        if nb > max_blocks:
            raise ValueError(f"sequence of {n} tokens needs {nb} > {max_blocks} blocks")
        bt[i, :nb] = alloc.take(nb)
    return bt


def uniform_lengths(seed: int, stream: int, n: int, lo: int, hi: int) -> np.ndarray:
    """``n`` integers uniform on ``[lo, hi]`` inclusive."""
    return _rng(seed, 0x1E4, stream).integers(lo, hi + 1, size=n).astype(np.int32)


def lognormal_lengths(seed: int, stream: int, n: int, median: float, sigma: float,
                      cap: int) -> np.ndarray:
    r = _rng(seed, 0x106, stream)
    v = np.rint(np.exp(np.log(median) + sigma * r.standard_normal(n)))
    return np.clip(v, 1, cap).astype(np.int32)


def poisson_arrivals(seed: int, stream: int, n: int, rate: float) -> np.ndarray:
    """Arrival times (seconds) of a Poisson process of ``rate`` per second."""
    r = _rng(seed, 0xA11, stream)
    return np.cumsum(r.exponential(1.0 / rate, size=n))


def chunk_schedule(prompt_lens: Sequence[int], budget: int) -> List[List[Tuple[int, int, int]]]:
    """Chunked-prefill schedule: steps of at most ``budget`` tokens, filled
    first come first served; a prompt may span several steps and a step may
    hold several prompts. Each step is a list of (prompt index, ctx_len,
    q_len)."""
    steps: List[List[Tuple[int, int, int]]] = []
    cur: List[Tuple[int, int, int]] = []
    room = budget
    for i, n in enumerate(prompt_lens):
        done = 0
        while done < n:
            take = min(room, n - done)
            cur.append((i, done, take))
            done += take
            room -= take
            if room == 0:
                steps.append(cur)
                cur, room = [], budget
    if cur:
        steps.append(cur)
    return steps


# ---------------------------------------------------------------------------
# Named workloads, with their sizes.
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class Workload:
    key: str
    shape: ModelShape
    layer_begin: int
    layer_end: int
    description: str

    @property
    def n_layers(self) -> int:
        return self.layer_end - self.layer_begin


WORKLOADS = {
    "tiny": Workload("tiny", TINY, 0, 2,
                     "tiny Llama-style stage, 2 layers; 4 prompts of 16-64 tokens, "
                     "prefill then 16 decode steps"),
    "l70-decode": Workload("l70-decode", LLAMA70B, 20, 40,
                           "Llama-3.1-70B-shaped stage, layers [20,40), bf16; decode batch 64, "
                           "contexts uniform 512-2048"),
    "l70-prefill": Workload("l70-prefill", LLAMA70B, 20, 40,
                            "Llama-3.1-70B-shaped stage, layers [20,40), bf16; 8 prompts of "
                            "1024-4096 tokens, chunked prefill with a 2048-token budget"),
    "q32-mixed": Workload("q32-mixed", QWEN32B, 24, 40,
                          "Qwen3-32B-shaped stage, layers [24,40), bf16; each step 4 prefill "
                          "chunks of 512 (prefixes 0/512/1024/1536) + 128 decodes, contexts "
                          "uniform 256-4096"),
    "l70-full": Workload("l70-full", LLAMA70B, 0, 80,
                         "Llama-3.1-70B-shaped model as one 80-layer stage, bf16; continuous "
                         "batching, <=128 decodes, contexts 1024-4096, lognormal outputs"),
}


def shrink(shape: ModelShape, **kw) -> ModelShape:
    return replace(shape, **kw)
