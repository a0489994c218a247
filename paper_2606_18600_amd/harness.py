"""Device-memory plumbing around the stage ABI (PyTorch for memory and
streams only; every step of the forward pass runs in the HIP library).

``DeviceStage`` owns the caller side of the ABI contract: it allocates the
weights' device copies, the KV pool, block tables and the workspace as torch
tensors, creates the stage over them and forwards calls.
"""

from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import stage as S
from .synth import GAIN_NAMES, ModelShape, _TENSOR_IDS

WEIGHT_FIELDS = ("attn_norm", "w_qkv", "q_norm", "k_norm", "w_o", "ffn_norm", "w_gate_up",
                 "w_down")


def torch_dtype(dtype: str) -> torch.dtype:
    return {"bf16": torch.bfloat16, "f32": torch.float32}[dtype]


def model_config(shape: ModelShape, dtype: str, max_position: int = 8192) -> S.stage_model_config:
    return S.stage_model_config(
        hidden=shape.hidden, n_q_heads=shape.n_q_heads, n_kv_heads=shape.n_kv_heads,
        head_dim=shape.head_dim, ffn=shape.ffn, qk_norm=1 if shape.qk_norm else 0,
        block_size=shape.block_size, rms_eps=shape.rms_eps, qk_rms_eps=shape.qk_rms_eps,
        rope_theta=shape.rope_theta, max_position=max_position,
        dtype=S.STAGE_BF16 if dtype == "bf16" else S.STAGE_F32)


def upload_weights(host: Dict[str, np.ndarray], dtype: str, device="cuda") -> Dict[str, torch.Tensor]:
    """Copy host weights to the device in the mode dtype (fp32 -> bf16 is
    round-to-nearest-even)."""
    td = torch_dtype(dtype)
    return {k: torch.from_numpy(np.ascontiguousarray(v, np.float32)).to(device=device, dtype=td)
            for k, v in host.items()}


def device_layer_weights(shape: ModelShape, seed: int, global_layer: int, dtype: str,
                         std: float = 0.02, gain_std: float = 0.02,
                         device="cuda") -> Dict[str, torch.Tensor]:
    """Random weights generated on the device (for model-sized stages where a
    host draw would take too long): N(0, std^2) projections, 1 + N(0,
    gain_std^2) gains, each tensor from its own seeded device generator."""
    td = torch_dtype(dtype)
    out = {}
    for name, shp in shape.weight_shapes().items():
        g = torch.Generator(device=device)
        g.manual_seed((seed * 1_000_003 + global_layer * 1009 + _TENSOR_IDS[name]) & 0x7FFFFFFF)
        if name in GAIN_NAMES:
            t = torch.empty(shp, dtype=torch.float32, device=device).normal_(1.0, gain_std,
                                                                            generator=g)
            out[name] = t.to(td)
        else:
            out[name] = torch.empty(shp, dtype=td, device=device).normal_(0.0, std, generator=g)
    return out


def to_host64(weights: Dict[str, torch.Tensor]) -> Dict[str, np.ndarray]:
    """The stored values, as float64 host arrays."""
    return {k: v.detach().to(torch.float64).cpu().numpy() for k, v in weights.items()}


PACK_KINDS = {"w_qkv": S.STAGE_W_QKV, "w_o": S.STAGE_W_O, "w_gate_up": S.STAGE_W_GATE_UP,
              "w_down": S.STAGE_W_DOWN}


def pack_layer(cfg: S.stage_model_config, w: Dict[str, torch.Tensor],
               free_source: bool = False) -> Dict[str, torch.Tensor]:
    """Row-major layer weights -> the layout the stage reads (stage_pack_weight)."""
    out = {}
    for k, v in list(w.items()):
        if k in PACK_KINDS:
            dst = torch.empty_like(v)
            S.stage_pack_weight(cfg, PACK_KINDS[k], v.data_ptr(), dst.data_ptr(),
                                torch.cuda.current_stream().cuda_stream)
            out[k] = dst
            if free_source:
                torch.cuda.current_stream().synchronize()
                del w[k]
        else:
            out[k] = v
    return out


def pack_lm_head(cfg: S.stage_model_config, w_lm: torch.Tensor) -> torch.Tensor:
    """Row-major [vocab, hidden] LM-head matrix -> the layout stage_lm_head reads."""
    dst = torch.empty_like(w_lm)
    S.stage_pack_lm_head(cfg, w_lm.shape[0], w_lm.data_ptr(), dst.data_ptr(),
                         torch.cuda.current_stream().cuda_stream)
    return dst


class DeviceStage:
    """A stage over row-major weights (packed here through the ABI) or over
    weights already packed (``packed=True``)."""

    def __init__(self, shape: ModelShape, dtype: str, layer_begin: int,
                 weights: Sequence[Dict[str, torch.Tensor]], num_blocks: int, max_tokens: int,
                 max_seqs: int, max_position: int = 8192, device="cuda",
                 kv_pool: Optional[torch.Tensor] = None, packed: bool = False):
        self.shape, self.dtype = shape, dtype
        self.n_layers = len(weights)
        self.num_blocks = num_blocks
        self.cfg = model_config(shape, dtype, max_position)
        if not packed:
            weights = [pack_layer(self.cfg, w) for w in weights]
        td = torch_dtype(dtype)
        numel = self.n_layers * num_blocks * shape.n_kv_heads * 2 * shape.block_size * shape.head_dim
        if kv_pool is None:
            kv_pool = torch.zeros(numel, dtype=td, device=device)
        assert kv_pool.numel() >= numel and kv_pool.dtype == td
        self.kv_pool = kv_pool
        self.weights = list(weights)
        for w in self.weights:
            for k, v in w.items():
                assert v.is_contiguous() and v.dtype == td, k
        ptrs = [{f: w[f].data_ptr() for f in WEIGHT_FIELDS if f in w} for w in self.weights]
        self._create(layer_begin, ptrs, kv_pool.data_ptr(), max_tokens, max_seqs, device)

    def _create(self, layer_begin: int, layer_ptrs: Sequence[Dict[str, int]], kv_ptr: int,
                max_tokens: int, max_seqs: int, device) -> None:
        """stage_create over device pointers, then a workspace of the size
        the stage asks for."""
        layers = [S.stage_layer_weights(*[w.get(f) for f in WEIGHT_FIELDS]) for w in layer_ptrs]
        self.handle = S.stage_create(self.cfg, layer_begin, layer_begin + len(layers), layers,
                                     kv_ptr, self.num_blocks, max_tokens, max_seqs)
        nbytes = S.stage_workspace_bytes(self.handle)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
        S.stage_bind_workspace(self.handle, self.workspace.data_ptr(), nbytes)

    # --- calls -------------------------------------------------------------
    @staticmethod
    def batch(q_lens, ctx_lens, block_tables: torch.Tensor) -> S.stage_batch:
        assert block_tables.dtype == torch.int32 and block_tables.is_contiguous()
        return S.make_batch(q_lens, ctx_lens, block_tables.data_ptr(), block_tables.shape[1])

    def _out(self, hidden_in, hidden_out):
        return torch.empty_like(hidden_in) if hidden_out is None else hidden_out

    def prefill(self, q_lens, ctx_lens, bt, hidden_in, hidden_out=None, stream=0):
        out = self._out(hidden_in, hidden_out)
        S.stage_prefill(self.handle, self.batch(q_lens, ctx_lens, bt), hidden_in.data_ptr(),
                        out.data_ptr(), stream)
        return out

    def decode(self, ctx_lens, bt, hidden_in, hidden_out=None, stream=0):
        out = self._out(hidden_in, hidden_out)
        S.stage_decode(self.handle, self.batch(np.ones(len(ctx_lens), np.int32), ctx_lens, bt),
                       hidden_in.data_ptr(), out.data_ptr(), stream)
        return out

    def decode_noalloc(self, ctx_lens, bt, hidden_in, hidden_out=None, stream=0):
        """stage_decode_noalloc: the decode over the library's static scratch."""
        out = self._out(hidden_in, hidden_out)
        S.stage_decode_noalloc(self.handle,
                               self.batch(np.ones(len(ctx_lens), np.int32), ctx_lens, bt),
                               hidden_in.data_ptr(), out.data_ptr(), stream)
        return out

    def mixed(self, p_q_lens, p_ctx_lens, p_bt, d_ctx_lens, d_bt, hidden_in, hidden_out=None,
              stream=0):
        out = self._out(hidden_in, hidden_out)
        pb = self.batch(p_q_lens, p_ctx_lens, p_bt) if len(p_q_lens) else None
        db = self.batch(np.ones(len(d_ctx_lens), np.int32), d_ctx_lens, d_bt) \
            if len(d_ctx_lens) else None
        S.stage_step_mixed(self.handle, pb, db, hidden_in.data_ptr(), out.data_ptr(), stream)
        return out

    def lm_head(self, final_norm: torch.Tensor, w_lm_packed: torch.Tensor, hidden: torch.Tensor,
                rows=None, n_rows: Optional[int] = None, logits: Optional[torch.Tensor] = None,
                stream=0) -> torch.Tensor:
        """Logits [n_rows, vocab] (fp32) of the selected rows of `hidden`."""
        vocab = w_lm_packed.shape[0]
        n = len(rows) if rows is not None else (hidden.shape[0] if n_rows is None else n_rows)
        if logits is None:
            logits = torch.empty((n, vocab), dtype=torch.float32, device=hidden.device)
        S.stage_lm_head(self.handle, final_norm.data_ptr(), w_lm_packed.data_ptr(), vocab,
                        hidden.data_ptr(), hidden.shape[0], rows, n, logits.data_ptr(), stream)
        return logits

    def kv_view(self) -> torch.Tensor:
        s = self.shape
        n = self.n_layers * self.num_blocks * s.n_kv_heads * 2 * s.block_size * s.head_dim
        return self.kv_pool[:n].view(self.n_layers, self.num_blocks, s.n_kv_heads, 2,
                                     s.block_size, s.head_dim)

    def close(self):
        if self.handle:
            S.stage_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class PointerStage(DeviceStage):
    """A stage over packed weights and a KV pool given as raw device
    pointers (e.g. memory mapped from a tensor store); only the workspace is
    allocated here."""

    def __init__(self, shape: ModelShape, dtype: str, layer_begin: int,
                 layer_ptrs: Sequence[Dict[str, int]], kv_ptr: int, num_blocks: int,
                 max_tokens: int, max_seqs: int, max_position: int = 8192, device="cuda"):
        self.shape, self.dtype = shape, dtype
        self.n_layers = len(layer_ptrs)
        self.num_blocks = num_blocks
        self.cfg = model_config(shape, dtype, max_position)
        self.kv_pool = None
        self.weights = []
        self._create(layer_begin, layer_ptrs, kv_ptr, max_tokens, max_seqs, device)

    def kv_view(self) -> torch.Tensor:
        raise RuntimeError("a stage over raw pointers has no KV tensor to view")
