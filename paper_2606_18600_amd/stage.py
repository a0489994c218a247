"""ctypes binding of the stage C ABI (``include/stage.h``).

The functions carry the C names and only marshal arguments: pointers are
passed as integers (``tensor.data_ptr()``), host length arrays as numpy
int32 arrays. A non-zero ``stage_status`` is raised as :class:`StageError`
with the library's message. The library is the only implementation: if
``libstage.so`` is missing, loading raises instead of falling back to
anything else.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libstage.so")

STAGE_OK = 0
STAGE_ERR_INVALID_ARG = 1
STAGE_ERR_UNSUPPORTED = 2
STAGE_ERR_OUT_OF_MEMORY = 3
STAGE_ERR_DEVICE = 4
STAGE_ERR_CAPACITY = 5

STAGE_F32 = 0
STAGE_BF16 = 1

OP_NAMES = ("norm", "qkv", "rope_kv", "attn", "o_proj", "gate_up", "down", "lm_head")
STAGE_OP_COUNT = len(OP_NAMES)

EXPORTED = ("stage_create", "stage_workspace_bytes", "stage_bind_workspace", "stage_prefill",
            "stage_decode", "stage_step_mixed", "stage_destroy", "stage_last_error",
            "stage_validate_step", "stage_set_op_timing", "stage_read_op_times",
            "stage_pack_weight", "stage_copy_probe", "stage_lm_head", "stage_pack_lm_head",
            "stage_decode_noalloc", "stage_store_alloc", "stage_store_free", "stage_store_write",
            "stage_store_attach", "stage_store_detach")

STAGE_STORE_MAX_BYTES = 1 << 31

STAGE_W_QKV = 0
STAGE_W_O = 1
STAGE_W_GATE_UP = 2
STAGE_W_DOWN = 3


class StageError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"stage error {code}: {msg}")
        self.code = code
        self.msg = msg


class stage_model_config(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("ffn", ctypes.c_int32), ("qk_norm", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("qk_rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_double),
                ("max_position", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class stage_layer_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("attn_norm", "w_qkv", "q_norm", "k_norm", "w_o", "ffn_norm", "w_gate_up",
                 "w_down")]


class stage_ipc_handle(ctypes.Structure):
    _fields_ = [("bytes", ctypes.c_ubyte * 64)]


class stage_batch(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("q_lens", ctypes.POINTER(ctypes.c_int32)),
                ("ctx_lens", ctypes.POINTER(ctypes.c_int32)),
                ("block_tables", ctypes.c_void_p), ("max_blocks_per_seq", ctypes.c_int32)]


_lib: Optional[ctypes.CDLL] = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load ``libstage.so`` (once). Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise StageError(STAGE_ERR_DEVICE, f"{path} not found: build it with "
                         "`python -m paper_2606_18600_amd.build`")
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32 = ctypes.c_int32
    lib.stage_create.argtypes = [ctypes.POINTER(stage_model_config), i32, i32,
                                 ctypes.POINTER(stage_layer_weights), P, i32, i32, i32,
                                 ctypes.POINTER(P)]
    lib.stage_workspace_bytes.argtypes = [P]
    lib.stage_workspace_bytes.restype = ctypes.c_size_t
    lib.stage_bind_workspace.argtypes = [P, P, ctypes.c_size_t]
    lib.stage_prefill.argtypes = [P, ctypes.POINTER(stage_batch), P, P, P]
    lib.stage_decode.argtypes = [P, ctypes.POINTER(stage_batch), P, P, P]
    lib.stage_decode_noalloc.argtypes = [P, ctypes.POINTER(stage_batch), P, P, P]
    lib.stage_step_mixed.argtypes = [P, ctypes.POINTER(stage_batch),
                                     ctypes.POINTER(stage_batch), P, P, P]
    lib.stage_destroy.argtypes = [P]
    lib.stage_last_error.restype = ctypes.c_char_p
    lib.stage_validate_step.argtypes = [ctypes.POINTER(stage_model_config), i32, i32,
                                        ctypes.POINTER(stage_batch), ctypes.POINTER(stage_batch)]
    lib.stage_pack_weight.argtypes = [ctypes.POINTER(stage_model_config), i32, P, P, P]
    lib.stage_copy_probe.argtypes = [P, P, ctypes.c_size_t, P]
    lib.stage_lm_head.argtypes = [P, P, P, i32, P, i32, ctypes.POINTER(ctypes.c_int32), i32, P, P]
    lib.stage_pack_lm_head.argtypes = [ctypes.POINTER(stage_model_config), i32, P, P, P]
    lib.stage_store_alloc.argtypes = [ctypes.c_size_t, ctypes.POINTER(P),
                                      ctypes.POINTER(stage_ipc_handle)]
    lib.stage_store_free.argtypes = [P]
    lib.stage_store_write.argtypes = [P, P, ctypes.c_size_t, P]
    lib.stage_store_attach.argtypes = [ctypes.POINTER(stage_ipc_handle), ctypes.POINTER(P)]
    lib.stage_store_detach.argtypes = [P]
    lib.stage_set_op_timing.argtypes = [P, i32]
    lib.stage_read_op_times.argtypes = [P, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_int64)]
    for name in ("stage_create", "stage_bind_workspace", "stage_prefill", "stage_decode",
                 "stage_decode_noalloc",
                 "stage_step_mixed", "stage_destroy", "stage_validate_step",
                 "stage_set_op_timing", "stage_read_op_times", "stage_pack_weight",
                 "stage_copy_probe", "stage_lm_head", "stage_pack_lm_head", "stage_store_alloc",
                 "stage_store_free", "stage_store_write", "stage_store_attach",
                 "stage_store_detach"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def stage_last_error() -> str:
    return load_library().stage_last_error().decode()


def _check(code: int) -> None:
    if code != STAGE_OK:
        raise StageError(code, stage_last_error())


def make_batch(q_lens, ctx_lens, block_tables_ptr: int, max_blocks_per_seq: int) -> stage_batch:
    """Marshal host length arrays (kept alive on the returned struct) and a
    device block-table pointer into a ``stage_batch``."""
    q = np.ascontiguousarray(q_lens, dtype=np.int32)
    c = np.ascontiguousarray(ctx_lens, dtype=np.int32)
    b = stage_batch(len(q), q.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                    c.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), block_tables_ptr,
                    max_blocks_per_seq)
    b._keep = (q, c)
    return b


def stage_create(cfg: stage_model_config, layer_begin: int, layer_end: int,
                 layers: Sequence[stage_layer_weights], kv_pool: int, num_blocks: int,
                 max_tokens: int, max_seqs: int) -> int:
    lib = load_library()
    arr = (stage_layer_weights * max(1, len(layers)))(*layers)
    out = ctypes.c_void_p()
    _check(lib.stage_create(ctypes.byref(cfg), layer_begin, layer_end,
                            arr if len(layers) else None, kv_pool, num_blocks, max_tokens,
                            max_seqs, ctypes.byref(out)))
    return out.value


def stage_workspace_bytes(st: int) -> int:
    return int(load_library().stage_workspace_bytes(st))


def stage_bind_workspace(st: int, dev: int, nbytes: int) -> None:
    _check(load_library().stage_bind_workspace(st, dev, nbytes))


def _bp(b: Optional[stage_batch]):
    return ctypes.byref(b) if b is not None else None


def stage_prefill(st: int, batch: stage_batch, hidden_in: int, hidden_out: int,
                  stream: int = 0) -> None:
    _check(load_library().stage_prefill(st, _bp(batch), hidden_in, hidden_out, stream))


def stage_decode(st: int, batch: stage_batch, hidden_in: int, hidden_out: int,
                 stream: int = 0) -> None:
    _check(load_library().stage_decode(st, _bp(batch), hidden_in, hidden_out, stream))


def stage_decode_noalloc(st: int, batch: stage_batch, hidden_in: int, hidden_out: int,
                         stream: int = 0) -> None:
    _check(load_library().stage_decode_noalloc(st, _bp(batch), hidden_in, hidden_out, stream))


def stage_step_mixed(st: int, prefill: Optional[stage_batch], decode: Optional[stage_batch],
                     hidden_in: int, hidden_out: int, stream: int = 0) -> None:
    _check(load_library().stage_step_mixed(st, _bp(prefill), _bp(decode), hidden_in,
                                           hidden_out, stream))


def stage_destroy(st: int) -> None:
    _check(load_library().stage_destroy(st))


def stage_validate_step(cfg: stage_model_config, max_tokens: int, max_seqs: int,
                        prefill: Optional[stage_batch], decode: Optional[stage_batch]) -> int:
    """Returns the status code (does not raise)."""
    return int(load_library().stage_validate_step(ctypes.byref(cfg), max_tokens, max_seqs,
                                                  _bp(prefill), _bp(decode)))


def stage_pack_weight(cfg: stage_model_config, kind: int, src: int, dst: int,
                      stream: int = 0) -> None:
    _check(load_library().stage_pack_weight(ctypes.byref(cfg), kind, src, dst, stream))


def stage_copy_probe(src: int, dst: int, nbytes: int, stream: int = 0) -> None:
    _check(load_library().stage_copy_probe(src, dst, nbytes, stream))


def stage_lm_head(st: int, final_norm: int, w_lm: int, vocab: int, hidden: int,
                  hidden_rows: int, rows, n_rows: int, logits: int, stream: int = 0) -> None:
    """``rows``: host int32 indices into ``hidden`` (or None for 0..n_rows-1)."""
    if rows is None:
        rp = None
    else:
        r = np.ascontiguousarray(rows, dtype=np.int32)
        if len(r) != n_rows:
            raise StageError(STAGE_ERR_INVALID_ARG, f"{len(r)} row indices for n_rows={n_rows}")
        rp = r.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    _check(load_library().stage_lm_head(st, final_norm, w_lm, vocab, hidden, hidden_rows, rp,
                                        n_rows, logits, stream))


def stage_pack_lm_head(cfg: stage_model_config, vocab: int, src: int, dst: int,
                       stream: int = 0) -> None:
    _check(load_library().stage_pack_lm_head(ctypes.byref(cfg), vocab, src, dst, stream))


def stage_set_op_timing(st: int, enable: bool) -> None:
    _check(load_library().stage_set_op_timing(st, 1 if enable else 0))


def stage_read_op_times(st: int) -> Tuple[list, list]:
    ms = (ctypes.c_double * STAGE_OP_COUNT)()
    n = (ctypes.c_int64 * STAGE_OP_COUNT)()
    _check(load_library().stage_read_op_times(st, ms, n))
    return list(ms), list(n)


def stage_store_alloc(nbytes: int) -> Tuple[int, bytes]:
    """(device pointer, 64-byte IPC handle) of a new zero-filled store
    allocation."""
    p = ctypes.c_void_p()
    h = stage_ipc_handle()
    _check(load_library().stage_store_alloc(nbytes, ctypes.byref(p), ctypes.byref(h)))
    return p.value, bytes(h.bytes)


def stage_store_free(ptr: int) -> None:
    _check(load_library().stage_store_free(ptr))


def stage_store_write(dst: int, src: int, nbytes: int, stream: int = 0) -> None:
    _check(load_library().stage_store_write(dst, src, nbytes, stream))


def stage_store_attach(handle: bytes) -> int:
    if len(handle) != 64:
        raise StageError(STAGE_ERR_INVALID_ARG, f"an IPC handle has 64 bytes, got {len(handle)}")
    h = stage_ipc_handle()
    ctypes.memmove(h.bytes, handle, 64)
    p = ctypes.c_void_p()
    _check(load_library().stage_store_attach(ctypes.byref(h), ctypes.byref(p)))
    return p.value


def stage_store_detach(ptr: int) -> None:
    _check(load_library().stage_store_detach(ptr))
