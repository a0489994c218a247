"""Request migration by recomputation (the paper's alternative to copying a
request's KV cache to another instance, Sec. 5.1): the receiving stage
rebuilds the KV of a request by running its stage_prefill over the hidden
states of every token the request has so far (prompt and generated tokens),
in chunks, into blocks of its own pool. The stage's outputs for those rows
are what its successor stage needs to recompute its own layers.

Host orchestration only: each chunk is one stage_prefill call through the
C ABI; every step of the computation runs in the stage's kernels.
"""

from __future__ import annotations

from typing import List, Tuple

import torch


def recompute_kv(stage, hidden: torch.Tensor, block_table: torch.Tensor, chunk: int = 2048,
                 out: torch.Tensor = None, stream: int = 0) -> torch.Tensor:
    """Rebuild one request's KV in `stage` from the hidden states of all of
    its tokens, `hidden` [L, H] (positions 0..L-1), into the blocks of
    `block_table` [1, max_blocks] (int32, device). Chunks of at most `chunk`
    tokens (at most the stage's max_tokens) are prefilled in order, each
    attending to the keys the previous chunks wrote. Returns the stage's
    output rows [L, H] (written into `out` when given)."""
    L = hidden.shape[0]
    if out is None:
        out = torch.empty_like(hidden)
    for c0 in range(0, L, chunk):
        q = min(chunk, L - c0)
        stage.prefill([q], [c0], block_table, hidden[c0:c0 + q], out[c0:c0 + q], stream=stream)
    return out


def transfer_bytes(shape, n_layers: int, tokens: int) -> int:
    """Bytes a KV transfer of `tokens` tokens moves for `n_layers` layers:
    K and V of every kv head, in bf16 (the amount recomputation avoids)."""
    return tokens * n_layers * 2 * shape.n_kv_heads * shape.head_dim * 2


def migration_points(shape, n_layers: int, lengths, recompute_ms, links_gbs) -> List[Tuple]:
    """(tokens, KV bytes, recompute ms, {link: transfer ms}) per context
    length: the comparison the paper's migration choice rests on."""
    rows = []
    for L, ms in zip(lengths, recompute_ms):
        b = transfer_bytes(shape, n_layers, L)
        rows.append((L, b, ms, {k: b / (g * 1e9) * 1e3 for k, g in links_gbs.items()}))
    return rows
