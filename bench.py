"""Benchmark of the stage forward pass on one MI355X.

Workload (the metric's configuration): a Llama-3.1-70B-shaped stage of 20
consecutive layers, [20, 40), bf16 random-init weights N(0, 0.02^2); decode
batch of 64 sequences with contexts uniform on 512..2048 tokens, paged KV in
16-token blocks with shuffled block tables. One step = one stage_decode call
(every layer: RMSNorm, QKV, q/k-RoPE + KV write, split-K paged attention,
O-proj, RMSNorm, gate-up + SwiGLU, down). The same stage then runs a chunked
prefill of 8 prompts of 1024..4096 tokens with a 2048-token budget per step.

Prints one JSON line: decode tok/s as `value`, the roofline of the dominant
kernel (timed with HIP events on the launch stream), the prefill figures,
and the CPU oracle timed on a bounded sample on the host.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2606_18600_amd.roofline import (BF16_PEAK_TFLOPS, HBM_PEAK_GBS,  # noqa: E402
                                           decode_step_bytes, gemm_bytes, prefill_flops,
                                           step_roofline_ms)

METRIC = "stage decode tok/s + prefill tok/s on 1 GPU; % of HBM / MFMA roofline"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def bench_q32_mixed(args):
    """Qwen3-32B-shaped mixed step, 16 layers [24, 40): every step carries 4
    prefill chunks of 512 tokens (cached prefixes 0/512/1024/1536) and 128
    decode tokens with contexts uniform 256..4096."""
    import torch
    from paper_2606_18600_amd import stage as S
    from paper_2606_18600_amd import synth
    from paper_2606_18600_amd.harness import (DeviceStage, device_layer_weights, model_config,
                                              pack_layer)
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    shape, seed = synth.QWEN32B, args.seed
    wl = synth.WORKLOADS["q32-mixed"]
    L0, nL = wl.layer_begin, wl.n_layers
    K, W = args.steps, args.warmup
    cfg = model_config(shape, "bf16")
    log(f"[bench] generating {nL} layers of {shape.name} weights on the device")
    weights = [pack_layer(cfg, device_layer_weights(shape, seed, l, "bf16"), free_source=True)
               for l in range(L0, wl.layer_end)]
    pc = np.array([0, 512, 1024, 1536], np.int32)
    pq = np.full(4, 512, np.int32)
    dctx0 = synth.uniform_lengths(seed, 3, 128, 256, 4096)
    steps_total = W + 2 * K
    dfinal = dctx0 + steps_total + 1
    alloc_n = int(((pc + pq + 15) // 16).sum() + ((dfinal + 15) // 16).sum()) + 1
    alloc = synth.BlockAllocator(alloc_n, seed)
    pbt = torch.from_numpy(synth.make_block_tables(pc + pq, 128, alloc)).to(dev)
    dbt = torch.from_numpy(synth.make_block_tables(dfinal, int(((dfinal + 15) // 16).max()),
                                                   alloc)).to(dev)
    st = DeviceStage(shape, "bf16", L0, weights, alloc_n, max_tokens=2176, max_seqs=132,
                     packed=True)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    st.kv_pool.normal_(0.0, 1.0, generator=g)
    x = torch.empty((2176, shape.hidden), dtype=torch.bfloat16, device=dev).normal_(generator=g)
    out = torch.empty_like(x)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    i = 0
    for _ in range(W):
        st.mixed(pq, pc, pbt, dctx0 + i, dbt, x, out, stream=sp)
        i += 1
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ctx_timed = []
    e0.record(stream)
    for _ in range(K):
        st.mixed(pq, pc, pbt, dctx0 + i, dbt, x, out, stream=sp)
        ctx_timed.append(dctx0 + i)
        i += 1
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / K
    S.stage_set_op_timing(st.handle, True)
    for _ in range(K):
        st.mixed(pq, pc, pbt, dctx0 + i, dbt, x, out, stream=sp)
        i += 1
    op_ms, op_n = S.stage_read_op_times(st.handle)
    st.close()
    chunks = list(zip(pc.tolist(), pq.tolist()))
    roof = float(np.mean([step_roofline_ms(shape, nL, chunks, c) for c in ctx_timed]))
    res = {"workload": "q32-mixed: Qwen3-32B-shaped stage, layers [24,40); per step 4 x 512 "
                       "prefill chunks (prefixes 0/512/1024/1536) + 128 decodes, contexts "
                       "uniform 256-4096",
           "ms_per_step": round(ms, 3), "prefill_tok_s": round(2048 / (ms / 1e3), 1),
           "decode_tok_s": round(128 / (ms / 1e3), 1),
           "roofline_ms": round(roof, 3), "roofline_frac": round(roof / ms, 4),
           "ops_ms_per_step": {S.OP_NAMES[j]: round(op_ms[j] / K, 4) for j in range(len(op_ms))}}
    log(f"[bench] q32-mixed {ms:.3f} ms/step (roofline {roof:.3f} ms, {roof / ms:.1%}); "
        f"{2048 / (ms / 1e3):.0f} prefill + {128 / (ms / 1e3):.0f} decode tok/s")
    return res


def cpu_baseline(shape, ctx_lens, seed):
    """The oracle (float32) on the host: one decode step of one layer for the
    whole batch, scaled by the stage's 20 layers (every layer costs the same)."""
    import torch
    from oracle import stage_oracle as O
    from paper_2606_18600_amd import synth
    cfg = O.OracleConfig(shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                         shape.ffn, shape.rms_eps, shape.rope_theta)
    w = synth.host_layer_weights(shape, seed, 20, dtype=np.float32)
    B = len(ctx_lens)
    nbps = (ctx_lens + 1 + 15) // 16
    nb = int(nbps.sum())
    kv = O.new_kv_cache(cfg, 1, nb, np.float32)
    r = np.random.default_rng(seed)
    kv[0]["k"][:] = r.standard_normal(kv[0]["k"].shape, dtype=np.float32)
    kv[0]["v"][:] = r.standard_normal(kv[0]["v"].shape, dtype=np.float32)
    starts = np.concatenate([[0], np.cumsum(nbps)])
    seqs = [O.SeqSpec(int(c), 1, list(range(starts[i], starts[i + 1])))
            for i, c in enumerate(ctx_lens)]
    x = synth.hidden_states(seed, 9, B, shape.hidden)
    O.stage_forward(cfg, [w], x[:2], seqs[:2], kv, dtype=np.float32)  # warm caches
    t0 = time.perf_counter()
    O.stage_forward(cfg, [w], x, seqs, kv, dtype=np.float32)
    dt = time.perf_counter() - t0
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count()
    step_s = dt * 20
    return {"value": B / step_s, "unit": "tok/s", "cores": int(cores), "kind": "oracle",
            "sample": f"one decode step of one layer, batch {B} (contexts as the workload), "
                      f"float32, {dt:.2f} s, scaled x20 layers"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--seed", type=int, default=2606)
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--requests", type=int, default=512,
                    help="l70-full: new requests queued behind the 128 running ones")
    ap.add_argument("--arrival-rate", type=float, default=0.0,
                    help="l70-full: Poisson arrivals per second (0: all at t=0)")
    ap.add_argument("--workload", default="l70-decode",
                    choices=["l70-decode", "q32-mixed", "l70-full"],
                    help="l70-decode (default: the metric's workload, plus the chunked prefill "
                         "of the same stage); q32-mixed and l70-full print their own line")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the stage runs on a single MI355X and this build "
              f"has no multi-GPU path (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    if args.workload == "q32-mixed":
        print(json.dumps({"metric": METRIC, "n_gpus": 1, "steps": args.steps,
                          "warmup": args.warmup, "dtype": "bf16", "data": "synthetic",
                          **bench_q32_mixed(args)}), flush=True)
        return
    if args.workload == "l70-full":
        from paper_2606_18600_amd.batcher import bench_l70_full
        print(json.dumps({"metric": METRIC, "n_gpus": 1, "dtype": "bf16", "data": "synthetic",
                          **bench_l70_full(args, log)}), flush=True)
        return

    import torch
    from paper_2606_18600_amd import stage as S
    from paper_2606_18600_amd import synth
    from paper_2606_18600_amd.harness import (DeviceStage, device_layer_weights, model_config,
                                              pack_layer)

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    shape = synth.LLAMA70B
    wl = synth.WORKLOADS["l70-decode"]
    L0, L1 = wl.layer_begin, wl.layer_end
    nL = L1 - L0
    seed = args.seed
    B, K, W = 64, args.steps, args.warmup

    log(f"[bench] generating {nL} layers of {shape.name} weights on the device")
    cfg = model_config(shape, "bf16")
    weights = [pack_layer(cfg, device_layer_weights(shape, seed, l, "bf16"), free_source=True)
               for l in range(L0, L1)]
    ctx0 = synth.uniform_lengths(seed, 1, B, 512, 2048)
    steps_total = W + 2 * K
    dec_final = ctx0 + steps_total + 1
    dec_blocks = int(((dec_final + 15) // 16).sum())
    p_lens = synth.uniform_lengths(seed, 2, 8, 1024, 4096)
    pf_blocks = int(((p_lens + 15) // 16).sum())
    num_blocks = dec_blocks + pf_blocks + 1
    alloc = synth.BlockAllocator(num_blocks, seed)
    dec_bt_np = synth.make_block_tables(dec_final, int(((dec_final + 15) // 16).max()), alloc)
    pf_bt_np = synth.make_block_tables(p_lens, int(((p_lens + 15) // 16).max()), alloc)

    st = DeviceStage(shape, "bf16", L0, weights, num_blocks, max_tokens=2048, max_seqs=B,
                     packed=True)
    # Context KV: random N(0,1) values (decode cost does not depend on them).
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    st.kv_pool.normal_(0.0, 1.0, generator=g)
    dec_bt = torch.from_numpy(dec_bt_np).to(dev)
    xs = torch.empty((steps_total, B, shape.hidden), dtype=torch.bfloat16, device=dev)
    xs.normal_(0.0, 1.0, generator=g)
    out = torch.empty((B, shape.hidden), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream

    log(f"[bench] decode: B={B} ctx U[512,2048] mean {ctx0.mean():.0f}, warmup {W}, steps {K}")
    i = 0
    for _ in range(W):
        st.decode(ctx0 + i, dec_bt, xs[i], out, stream=sp)
        i += 1
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    ctx_timed = []
    e0.record(stream)
    for _ in range(K):
        st.decode(ctx0 + i, dec_bt, xs[i], out, stream=sp)
        ctx_timed.append(ctx0 + i)
        i += 1
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / K
    assert torch.isfinite(out.float()).all(), "non-finite stage output"
    dec_tok_s = B / (ms / 1e3)
    step_bytes = float(np.mean([decode_step_bytes(shape, nL, c) for c in ctx_timed]))
    log(f"[bench] decode {ms:.3f} ms/step, {dec_tok_s:.0f} tok/s, "
        f"{step_bytes / (ms / 1e3) / 1e9:.0f} GB/s algorithmic")

    # per-op timing pass (HIP events on the launch stream, inside the library)
    S.stage_set_op_timing(st.handle, True)
    for _ in range(K):
        st.decode(ctx0 + i, dec_bt, xs[i], out, stream=sp)
        i += 1
    op_ms, op_n = S.stage_read_op_times(st.handle)
    S.stage_set_op_timing(st.handle, False)
    ops = {S.OP_NAMES[j]: {"ms_per_step": op_ms[j] / K, "launches_per_step": op_n[j] / K}
           for j in range(len(op_ms))}
    gu_avg_ms = op_ms[S.OP_NAMES.index("gate_up")] / op_n[S.OP_NAMES.index("gate_up")]
    gu_bytes = gemm_bytes(B, 2 * shape.ffn, shape.hidden, 4)
    gu_gbs = gu_bytes / (gu_avg_ms / 1e3) / 1e9
    log(f"[bench] ops ms/step: " + ", ".join(f"{k}={v['ms_per_step']:.3f}" for k, v in ops.items()))
    log(f"[bench] gate_up split-K GEMM: {gu_avg_ms * 1e3:.1f} us/launch, {gu_gbs:.0f} GB/s")

    result = {
        "metric": METRIC, "value": round(dec_tok_s, 1), "unit": "tok/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: random-init weights N(0,0.02^2) (gains 1+N(0,0.02^2)), "
                "N(0,1) hidden inputs, random context KV, shuffled block tables",
        "config": {"workload": "l70-decode: Llama-3.1-70B-shaped stage, layers [20,40), "
                               "decode batch 64, contexts uniform 512-2048, KV block 16",
                   "layers": nL, "batch": B, "hidden": shape.hidden, "block": 16},
        "roofline": {"bound": "hbm", "kernel": "gemm_skinny_bf16 (gate-up, split-K)",
                     "achieved": round(gu_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gu_gbs / HBM_PEAK_GBS, 4), "traffic": None,
                     "bytes_per_launch": gu_bytes, "us_per_launch": round(gu_avg_ms * 1e3, 2)},
        "step_roofline": {"bound": "hbm", "algorithmic_bytes": step_bytes,
                          "roofline_ms": round(step_bytes / (HBM_PEAK_GBS * 1e9) * 1e3, 4),
                          "measured_ms": round(ms, 4),
                          "frac": round(step_bytes / (HBM_PEAK_GBS * 1e9) / (ms / 1e3), 4)},
        "ops_ms_per_step": {k: round(v["ms_per_step"], 4) for k, v in ops.items()},
    }

    if not args.no_prefill:
        pf_bt = torch.from_numpy(pf_bt_np).to(dev)
        steps = synth.chunk_schedule(p_lens, 2048)
        xin = torch.empty((2048, shape.hidden), dtype=torch.bfloat16, device=dev)
        xin.normal_(0.0, 1.0, generator=g)
        pout = torch.empty_like(xin)

        def run_prefill():
            for stp in steps:
                idx = [s[0] for s in stp]
                T = sum(s[2] for s in stp)
                st.prefill([s[2] for s in stp], [s[1] for s in stp], pf_bt[idx].contiguous(),
                           xin[:T], pout[:T], stream=sp)

        log(f"[bench] prefill: 8 prompts, {int(p_lens.sum())} tokens, {len(steps)} chunks")
        run_prefill()
        torch.cuda.synchronize()
        e0.record(stream)
        run_prefill()
        e1.record(stream)
        torch.cuda.synchronize()
        pms = e0.elapsed_time(e1)
        ptok = float(p_lens.sum())
        chunks = [(s[1], s[2]) for stp in steps for s in stp]
        pfl = prefill_flops(shape, nL, chunks)
        S.stage_set_op_timing(st.handle, True)
        run_prefill()
        op_ms, op_n = S.stage_read_op_times(st.handle)
        S.stage_set_op_timing(st.handle, False)
        j = S.OP_NAMES.index("gate_up")
        # full 2048-token chunks dominate; FLOPs per launch from the mean chunk size
        mean_T = ptok / len(steps)
        gu_fl = 2.0 * mean_T * 2 * shape.ffn * shape.hidden
        gu_tfs = gu_fl / (op_ms[j] / op_n[j] / 1e3) / 1e12
        result["prefill"] = {
            "workload": "l70-prefill: same stage, 8 prompts uniform 1024-4096, chunked prefill, "
                        "2048-token budget",
            "tok_s": round(ptok / (pms / 1e3), 1), "ms_total": round(pms, 3),
            "algorithmic_tflop": round(pfl / 1e12, 2),
            "tflops": round(pfl / (pms / 1e3) / 1e12, 1),
            "frac_mfma_peak": round(pfl / (pms / 1e3) / 1e12 / BF16_PEAK_TFLOPS, 4),
            "ops_ms": {S.OP_NAMES[k]: round(op_ms[k], 3) for k in range(len(op_ms))},
            "gate_up_tflops": round(gu_tfs, 1),
        }
        log(f"[bench] prefill {pms:.1f} ms, {ptok / (pms / 1e3):.0f} tok/s, "
            f"{pfl / (pms / 1e3) / 1e12:.0f} TFLOP/s; gate_up {gu_tfs:.0f} TFLOP/s")

    st.close()
    del weights
    torch.cuda.empty_cache()

    if not args.no_cpu:
        log("[bench] timing the CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(shape, ctx0, seed)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
