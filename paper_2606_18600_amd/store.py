"""The shared tensor store and the engine side of it (Sec. 5.2, "Shared
Tensor Store").

The paper's store is a process that loads a model's weights and owns the
KV-cache space once; serving engines in other processes reference that
memory zero-copy, so an engine can start (or restart) without loading
anything. Here the store is ``TensorStore``: every tensor is one device
allocation of the C ABI (``stage_store_alloc``, below 2 GiB, exported as an
IPC handle). An engine process calls ``attach`` with the published handles
and builds its stage over the mapped pointers (``PointerStage``).

Handles travel as hex strings in a small JSON request (``TensorStore.export``), which
``paper_2606_18600_amd.engine`` reads on stdin.
"""

from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import torch

from . import stage as S
from .harness import PACK_KINDS, WEIGHT_FIELDS

MAX_BYTES = S.STAGE_STORE_MAX_BYTES


class TensorStore:
    """Store side: named device allocations, each exported by handle."""

    def __init__(self):
        self.ptr: Dict[str, int] = {}
        self.nbytes: Dict[str, int] = {}
        self.handle: Dict[str, bytes] = {}

    def alloc(self, name: str, nbytes: int) -> int:
        """A zero-filled allocation of ``nbytes`` (< 2 GiB) named ``name``."""
        assert name not in self.ptr, name
        ptr, h = S.stage_store_alloc(nbytes)
        self.ptr[name], self.nbytes[name], self.handle[name] = ptr, nbytes, h
        return ptr

    def put(self, name: str, src: torch.Tensor, stream: int = 0) -> int:
        """A new allocation holding a copy of ``src`` (device or host)."""
        src = src.contiguous()
        n = src.numel() * src.element_size()
        ptr = self.alloc(name, n)
        S.stage_store_write(ptr, src.data_ptr(), n, stream)
        return ptr

    def put_packed(self, name: str, cfg: S.stage_model_config, kind: str, src: torch.Tensor,
                   stream: int = 0) -> int:
        """A new allocation holding a row-major projection matrix in the
        layout the stage reads (packed by stage_pack_weight straight into
        the store)."""
        n = src.numel() * src.element_size()
        ptr = self.alloc(name, n)
        S.stage_pack_weight(cfg, PACK_KINDS[kind], src.data_ptr(), ptr, stream)
        return ptr

    def put_layer(self, prefix: str, cfg: S.stage_model_config, w: Dict[str, torch.Tensor],
                  stream: int = 0) -> Dict[str, int]:
        """One layer's row-major weights: projections packed, gains copied.
        Returns the layer's pointers by weight field."""
        out = {}
        for f in WEIGHT_FIELDS:
            if f not in w:
                continue
            key = f"{prefix}.{f}"
            out[f] = (self.put_packed(key, cfg, f, w[f], stream) if f in PACK_KINDS
                      else self.put(key, w[f], stream))
        return out

    def export(self, names: Optional[Sequence[str]] = None) -> Dict[str, Dict]:
        """Handles (hex) and sizes of the named allocations (default: all)."""
        names = list(self.ptr) if names is None else list(names)
        return {n: {"handle": self.handle[n].hex(), "bytes": self.nbytes[n]} for n in names}

    def read(self, name: str, dtype: torch.dtype, stream: int = 0) -> torch.Tensor:
        """A device copy of a store allocation as a flat torch tensor."""
        esize = torch.tensor([], dtype=dtype).element_size()
        out = torch.empty(self.nbytes[name] // esize, dtype=dtype, device="cuda")
        S.stage_store_write(out.data_ptr(), self.ptr[name], out.numel() * esize, stream)
        return out

    def close(self) -> None:
        for name in list(self.ptr):
            S.stage_store_free(self.ptr.pop(name))
        self.nbytes.clear()
        self.handle.clear()


def attach(exported: Dict[str, Dict]) -> Dict[str, int]:
    """Engine side: map every exported allocation; returns pointers by name."""
    out = {}
    try:
        for name, e in exported.items():
            out[name] = S.stage_store_attach(bytes.fromhex(e["handle"]))
    except Exception:
        detach(out)
        raise
    return out


def detach(ptrs: Dict[str, int]) -> None:
    for name in list(ptrs):
        S.stage_store_detach(ptrs.pop(name))


def layer_pointers(ptrs: Dict[str, int], prefixes: Sequence[str]) -> List[Dict[str, int]]:
    """Per layer, the pointers of its weight fields (names ``prefix.field``)."""
    return [{f: ptrs[f"{p}.{f}"] for f in WEIGHT_FIELDS if f"{p}.{f}" in ptrs} for p in prefixes]


__all__ = ["TensorStore", "attach", "detach", "layer_pointers", "MAX_BYTES"]
