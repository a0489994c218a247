"""Drive the HIP stage and the CPU oracle side by side on identical inputs
(test code only). The oracle always consumes the values the device stores
(weights and inputs copied back after conversion to the mode dtype)."""

from __future__ import annotations

import sys
from typing import Dict, List, Optional

import numpy as np
import torch

from oracle import stage_oracle as O
from paper_2606_18600_amd import synth
from paper_2606_18600_amd.harness import DeviceStage, to_host64, torch_dtype, upload_weights
from tests.helpers import ocfg, rel_l2, seqs_from


def kv_plane_index(block: int, d: int):
    """Index arrays (o, dd) -> flat position of K[o][dd] and V[o][dd] inside
    one (block, kv head) plane (the fragment layouts of the KV pool)."""
    o = np.arange(block)[:, None]
    dd = np.arange(d)[None, :]
    k = (dd // 32) * 512 + (o + 16 * ((dd % 32) // 8)) * 8 + dd % 8
    v = (dd // 32) * 512 + (dd % 16 + 16 * (o // 4)) * 8 + ((dd // 16) % 2) * 4 + o % 4
    return k, v


def gpu_kv_to_oracle_layout(kv6: torch.Tensor) -> List[Dict[str, np.ndarray]]:
    """Convert the GPU pool [L][nb][nkv][2][16][d] (planes in fragment order)
    into per-layer {'k','v'} arrays [nb][16][nkv][d] in float64."""
    a = kv6.detach().to(torch.float64).cpu().numpy()
    L, nb, nkv, _, blk, d = a.shape
    ki, vi = kv_plane_index(blk, d)
    out = []
    for l in range(L):
        flat = a[l].reshape(nb, nkv, 2, blk * d)
        k = flat[:, :, 0, :][:, :, ki]          # [nb][nkv][16][d]
        v = flat[:, :, 1, :][:, :, vi]
        out.append({"k": np.ascontiguousarray(k.transpose(0, 2, 1, 3)),
                    "v": np.ascontiguousarray(v.transpose(0, 2, 1, 3))})
    return out


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


class Pair:
    def __init__(self, shape: synth.ModelShape, dtype: str, n_layers: int, num_blocks: int,
                 max_tokens: int, max_seqs: int, seed: int, layer_begin: int = 0,
                 host_weights: Optional[List[Dict[str, np.ndarray]]] = None,
                 max_position: int = 8192):
        self.shape, self.dtype = shape, dtype
        self.td = torch_dtype(dtype)
        if host_weights is None:
            host_weights = [synth.host_layer_weights(shape, seed, layer_begin + l)
                            for l in range(n_layers)]
        self.dev_w = [upload_weights(h, dtype) for h in host_weights]
        self.w64 = [to_host64(d) for d in self.dev_w]
        self.gpu = DeviceStage(shape, dtype, layer_begin, self.dev_w, num_blocks, max_tokens,
                               max_seqs, max_position=max_position)
        self.cfg = ocfg(shape)
        self.okv = O.new_kv_cache(self.cfg, n_layers, num_blocks)
        self.written = set()  # (block, offset) slots written so far

    def _in(self, x: np.ndarray):
        xin = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to("cuda", self.td)
        return xin, xin.to(torch.float64).cpu().numpy()

    def _note(self, ctx_lens, q_lens, bt):
        for c, q, row in zip(ctx_lens, q_lens, bt):
            for p in range(int(c), int(c) + int(q)):
                self.written.add((int(row[p // 16]), p % 16))

    def prefill(self, q_lens, ctx_lens, bt: np.ndarray, x: np.ndarray):
        xin, x64 = self._in(x)
        y = self.gpu.prefill(q_lens, ctx_lens, torch.from_numpy(bt).cuda(), xin)
        yr = O.stage_forward(self.cfg, self.w64, x64, seqs_from(ctx_lens, q_lens, bt), self.okv)
        self._note(ctx_lens, q_lens, bt)
        return y.to(torch.float64).cpu().numpy(), yr, x64

    def decode(self, ctx_lens, bt: np.ndarray, x: np.ndarray):
        xin, x64 = self._in(x)
        y = self.gpu.decode(ctx_lens, torch.from_numpy(bt).cuda(), xin)
        ones = [1] * len(ctx_lens)
        yr = O.stage_forward(self.cfg, self.w64, x64, seqs_from(ctx_lens, ones, bt), self.okv)
        self._note(ctx_lens, ones, bt)
        return y.to(torch.float64).cpu().numpy(), yr, x64

    def mixed(self, pq, pc, pbt, dc, dbt, x: np.ndarray):
        xin, x64 = self._in(x)
        y = self.gpu.mixed(pq, pc, torch.from_numpy(pbt).cuda(), dc, torch.from_numpy(dbt).cuda(),
                           xin)
        seqs = seqs_from(pc, pq, pbt) + seqs_from(dc, [1] * len(dc), dbt)
        yr = O.stage_forward(self.cfg, self.w64, x64, seqs, self.okv)
        self._note(pc, pq, pbt)
        self._note(dc, [1] * len(dc), dbt)
        return y.to(torch.float64).cpu().numpy(), yr, x64

    def kv_errors(self):
        """Max relative error of the written KV slots (GPU vs oracle), K and V."""
        torch.cuda.synchronize()
        g = gpu_kv_to_oracle_layout(self.gpu.kv_view())
        worst = 0.0
        for l, (gl, ol) in enumerate(zip(g, self.okv)):
            for t in ("k", "v"):
                a = np.stack([gl[t][b, o] for b, o in sorted(self.written)])
                r = np.stack([ol[t][b, o] for b, o in sorted(self.written)])
                worst = max(worst, rel_l2(a, r))
        return worst

    def close(self):
        self.gpu.close()


def bf16_round(a: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
