"""An engine process over a shared tensor store (Sec. 5.2, "Shared Tensor
Store"): it maps the store's weights and KV space by IPC handle, builds its
stage over them without loading anything, serves the calls it is given and
reports how long the attach took.

Run as ``python -m paper_2606_18600_amd.engine`` with a JSON request on
stdin::

    {"shape": {ModelShape fields}, "dtype": "bf16" | "f32",
     "layer_begin": 0, "layers": ["L0", ...],        # name prefixes in the store
     "kv_pool": "kv", "out": "out",                   # store names
     "handles": {name: {"handle": hex, "bytes": n}},  # TensorStore.export()
     "num_blocks": N, "max_tokens": T, "max_seqs": S, "max_position": P,
     "calls": [{"op": "prefill" | "decode", "q_lens": [...], "ctx_lens": [...],
                "block_tables": [[...], ...], "input": [seed, stream],
                "out_offset": bytes}, ...]}

Each call's input rows are the seeded N(0, 1) hidden states
``synth.hidden_states(seed, stream, T, hidden)`` in the mode dtype, and its
output rows are written straight into the store's ``out`` allocation at
``out_offset``. One JSON line goes to stdout: the attach, stage-creation and
serving times in milliseconds.
"""

from __future__ import annotations

import json
import sys
import time


def serve(req: dict) -> dict:
    t_start = time.perf_counter()
    import numpy as np
    import torch

    from . import stage as S
    from . import store
    from . import synth
    from .harness import PointerStage, torch_dtype

    torch.cuda.set_device(0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ptrs = store.attach(req["handles"])
    t1 = time.perf_counter()
    shape = synth.ModelShape(**req["shape"])
    st = PointerStage(shape, req["dtype"], req["layer_begin"],
                      store.layer_pointers(ptrs, req["layers"]), ptrs[req["kv_pool"]],
                      req["num_blocks"], req["max_tokens"], req["max_seqs"],
                      max_position=req.get("max_position", 8192))
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    td = torch_dtype(req["dtype"])
    esize = torch.tensor([], dtype=td).element_size()
    out_ptr = ptrs[req["out"]]
    out_bytes = req["handles"][req["out"]]["bytes"]
    try:
        for c in req["calls"]:
            q = np.asarray(c["q_lens"], np.int32)
            ctx = np.asarray(c["ctx_lens"], np.int32)
            bt = torch.tensor(c["block_tables"], dtype=torch.int32, device="cuda")
            T = int(q.sum())
            if c["out_offset"] + T * shape.hidden * esize > out_bytes:
                raise ValueError("call output does not fit the store's output allocation")
            x = torch.from_numpy(synth.hidden_states(*c["input"], T, shape.hidden)).to(
                "cuda", td)
            batch = st.batch(q, ctx, bt)
            hout = out_ptr + int(c["out_offset"])
            if c["op"] == "prefill":
                S.stage_prefill(st.handle, batch, x.data_ptr(), hout, 0)
            elif c["op"] == "decode":
                S.stage_decode(st.handle, batch, x.data_ptr(), hout, 0)
            else:
                raise ValueError(f"unknown op {c['op']!r}")
        torch.cuda.synchronize()
        t3 = time.perf_counter()
    finally:
        st.close()
        torch.cuda.synchronize()
        store.detach(ptrs)
    return {"ok": True, "attach_ms": (t1 - t0) * 1e3, "create_ms": (t2 - t1) * 1e3,
            "serve_ms": (t3 - t2) * 1e3, "startup_ms": (t0 - t_start) * 1e3,
            "calls": len(req["calls"]), "handles": len(req["handles"])}


def main() -> int:
    req = json.loads(sys.stdin.read())
    try:
        res = serve(req)
    except Exception as e:  # reported to the store, which decides
        print(json.dumps({"ok": False, "error": f"{type(e).__name__}: {e}"}), flush=True)
        return 1
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
