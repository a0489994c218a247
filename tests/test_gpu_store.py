"""The shared tensor store across processes (GPU).

A store (this process) loads a model's weights once into device allocations
of its own, each below 2 GiB and exported by IPC handle, together with a KV
pool and an output buffer. Its own stage serves a reference sequence of
calls. Then a fresh engine process (``python -m paper_2606_18600_amd.engine``)
maps the handles, builds a stage over the store's memory without loading
anything, and serves the same calls over other blocks of the same pool,
writing its outputs into the store's output buffer; meanwhile the store's
stage keeps serving decode steps of other sequences. The engine's outputs and
every KV block it wrote must equal the reference's bitwise (same kernels,
same inputs), and the time the engine took to attach and create its stage is
reported.
"""

from __future__ import annotations

import json
import os
import subprocess
import sys
import tempfile
import time

import numpy as np
import pytest
import torch

from paper_2606_18600_amd import synth
from paper_2606_18600_amd.harness import (PointerStage, device_layer_weights, model_config,
                                          torch_dtype, upload_weights)
from paper_2606_18600_amd.store import TensorStore, layer_pointers
from tests.gpu_pair import log

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _calls(lens, seed):
    """A prefill of the prompts, then three decode steps."""
    n = len(lens)
    calls = [("prefill", list(map(int, lens)), [0] * n, (seed, 1))]
    for k in range(3):
        calls.append(("decode", [1] * n, [int(c) + k for c in lens], (seed, 10 + k)))
    return calls


def _run(st, calls, bt, shape, td, out=None):
    ys = []
    for op, q, c, inp in calls:
        x = torch.from_numpy(synth.hidden_states(*inp, sum(q), shape.hidden)).to("cuda", td)
        if op == "prefill":
            ys.append(st.prefill(q, c, bt, x))
        else:
            ys.append(st.decode(c, bt, x))
    return ys


@pytest.mark.parametrize("case", ["tiny-bf16", "tiny-f32", "l70-layer-bf16"])
def test_engine_process_attaches_to_the_store(case):
    seed = 2700
    if case.startswith("tiny"):
        shape, dtype, n_layers, L0 = synth.TINY, case.split("-")[1], 2, 0
        host = [synth.host_layer_weights(shape, seed, l) for l in range(n_layers)]
        rowmajor = [upload_weights(h, dtype) for h in host]
        lens = synth.uniform_lengths(seed, 0, 4, 16, 64)
    else:
        shape, dtype, n_layers, L0 = synth.LLAMA70B, "bf16", 1, 47
        rowmajor = [device_layer_weights(shape, seed, L0, dtype)]
        lens = np.array([300, 700], np.int32)
    log(f"[test] store + engine process, {case}")
    td = torch_dtype(dtype)
    esize = torch.tensor([], dtype=td).element_size()
    cfg = model_config(shape, dtype)
    n = len(lens)
    need = (lens + 3 + 15) // 16                     # blocks per sequence for prompt + 3 decodes
    per_set = int(need.sum())
    serve_len = 4096 if shape is synth.TINY else 256
    serve_blocks = n * ((64 + serve_len + 15) // 16)
    num_blocks = 2 * per_set + serve_blocks
    alloc = synth.BlockAllocator(num_blocks, seed)
    bt_a = synth.make_block_tables(lens + 3, int(need.max()), alloc)     # the store's stage
    bt_b = synth.make_block_tables(lens + 3, int(need.max()), alloc)     # the engine's
    bt_c = synth.make_block_tables(np.full(n, 64 + serve_len), (64 + serve_len + 15) // 16,
                                   alloc)                                # served meanwhile
    block_elems = shape.n_kv_heads * 2 * 16 * shape.head_dim
    calls = _calls(lens, seed)
    rows = [sum(q) for _, q, _, _ in calls]
    store = TensorStore()
    st = proc = None
    try:
        prefixes = [f"L{L0 + i}" for i in range(n_layers)]
        layer_ptrs = [store.put_layer(p, cfg, w) for p, w in zip(prefixes, rowmajor)]
        kv = store.alloc("kv", n_layers * num_blocks * block_elems * esize)
        store.alloc("out", sum(rows) * shape.hidden * esize)
        torch.cuda.synchronize()
        del rowmajor
        log(f"  store: {len(store.ptr)} allocations, largest "
            f"{max(store.nbytes.values()) / 2**20:.0f} MiB")
        assert max(store.nbytes.values()) < 2 ** 31

        t0 = time.perf_counter()
        st = PointerStage(shape, dtype, L0, layer_ptrs, kv, num_blocks, 2048, 8)
        torch.cuda.synchronize()
        create_ms = (time.perf_counter() - t0) * 1e3
        ref = _run(st, calls, torch.from_numpy(bt_a).cuda(), shape, td)
        # the served-meanwhile sequences: a 64-token prompt each
        btc = torch.from_numpy(bt_c).cuda()
        st.prefill([64] * n, [0] * n, btc, torch.zeros((64 * n, shape.hidden), dtype=td,
                                                        device="cuda"))
        torch.cuda.synchronize()

        offs = np.concatenate([[0], np.cumsum(rows)]) * shape.hidden * esize
        req = {"shape": {f: getattr(shape, f) for f in shape.__dataclass_fields__},
               "dtype": dtype, "layer_begin": L0, "layers": prefixes, "kv_pool": "kv",
               "out": "out", "handles": store.export(), "num_blocks": num_blocks,
               "max_tokens": 2048, "max_seqs": 8,
               "calls": [{"op": op, "q_lens": q, "ctx_lens": c,
                          "block_tables": bt_b.tolist(), "input": list(inp),
                          "out_offset": int(o)}
                         for (op, q, c, inp), o in zip(calls, offs)]}
        fo, fe = tempfile.TemporaryFile("w+"), tempfile.TemporaryFile("w+")
        proc = subprocess.Popen([sys.executable, "-m", "paper_2606_18600_amd.engine"],
                                cwd=ROOT, stdin=subprocess.PIPE, stdout=fo, stderr=fe,
                                text=True)
        proc.stdin.write(json.dumps(req))
        proc.stdin.close()
        served, t_spawn = 0, time.perf_counter()
        x = torch.zeros((n, shape.hidden), dtype=td, device="cuda")
        while proc.poll() is None and served < serve_len:
            st.decode(np.full(n, 64 + served, np.int32), btc, x)
            torch.cuda.synchronize()
            served += 1
            if time.perf_counter() - t_spawn > 240:
                break
        proc.wait(timeout=240)
        fo.seek(0)
        fe.seek(0)
        stdout, stderr = fo.read(), fe.read()
        lines = [l for l in stdout.splitlines() if l.startswith("{")]
        assert proc.returncode == 0 and lines, f"engine failed: {stdout}\n{stderr[-2000:]}"
        res = json.loads(lines[-1])
        log(f"  engine: attach {res['attach_ms']:.1f} ms ({res['handles']} handles), stage "
            f"create {res['create_ms']:.1f} ms, start-up {res['startup_ms']:.0f} ms, serve "
            f"{res['serve_ms']:.1f} ms; in-process stage create {create_ms:.1f} ms; the store "
            f"served {served} decode steps meanwhile")
        assert served >= 1

        out = store.read("out", td)
        pool = store.read("kv", td).view(n_layers, num_blocks, block_elems)
        for k, y in enumerate(ref):
            a = offs[k] // esize
            got = out[a:a + y.numel()].view_as(y)
            assert torch.equal(got, y), f"call {k}: engine output differs from the store's stage"
        for s in range(n):
            ia = torch.from_numpy(bt_a[s, :need[s]].astype(np.int64)).cuda()
            ib = torch.from_numpy(bt_b[s, :need[s]].astype(np.int64)).cuda()
            assert torch.equal(pool[:, ib], pool[:, ia]), f"sequence {s}: KV blocks differ"
        assert torch.count_nonzero(pool[:, torch.from_numpy(
            bt_b[:, :1].reshape(-1).astype(np.int64)).cuda()]) > 0
    finally:
        if proc is not None and proc.poll() is None:
            proc.kill()
            proc.wait()
        if st is not None:
            st.close()
        torch.cuda.synchronize()
        store.close()
