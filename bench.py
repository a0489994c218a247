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
                                           decode_step_bytes, gate_up_swiglu_bytes, prefill_flops,
                                           step_roofline_ms)

METRIC = "stage decode tok/s + prefill tok/s on 1 GPU; % of HBM / MFMA roofline"
# The gate-up + SwiGLU operation of a 2176-row mixed step: two launches, the
# first 2048 rows on 256 x 256 tiles and the last 128 on the split-K kernel
# (one K range, SwiGLU in its epilogue); its time is that of both.
GATE_UP_MIXED_OP = ("gemm_tiled_bf16 + gemm_skinny8_bf16 (gate-up + SwiGLU op of a 2176-row step: "
                    "2048 rows on 256x256 tiles, the last 128 on the split-K kernel)")


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
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    ctx_timed = []
    ev[0].record(stream)
    for k in range(K):
        st.mixed(pq, pc, pbt, dctx0 + i, dbt, x, out, stream=sp)
        ev[k + 1].record(stream)
        ctx_timed.append(dctx0 + i)
        i += 1
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[K]) / K
    step_ms = [ev[k].elapsed_time(ev[k + 1]) for k in range(K)]
    assert torch.isfinite(out.float()).all(), "non-finite stage output"
    S.stage_set_op_timing(st.handle, True)
    for _ in range(K):
        st.mixed(pq, pc, pbt, dctx0 + i, dbt, x, out, stream=sp)
        i += 1
    op_ms, op_n = S.stage_read_op_times(st.handle)
    st.close()
    del weights, st
    torch.cuda.empty_cache()
    chunks = list(zip(pc.tolist(), pq.tolist()))
    roof = float(np.mean([step_roofline_ms(shape, nL, chunks, c) for c in ctx_timed]))
    est_in = {"shape": shape, "n_layers": nL, "chunks": chunks, "dec_ctx": ctx_timed}
    # dominant kernel: the gate-up + SwiGLU product of the 2176-row step
    j = S.OP_NAMES.index("gate_up")
    gu_us = op_ms[j] / op_n[j] * 1e3
    gu_fl = 2.0 * 2176 * 2 * shape.ffn * shape.hidden
    gu_tfs = gu_fl / (gu_us / 1e6) / 1e12
    res = {"workload": "q32-mixed: Qwen3-32B-shaped stage, layers [24,40); per step 4 x 512 "
                       "prefill chunks (prefixes 0/512/1024/1536) + 128 decodes, contexts "
                       "uniform 256-4096",
           "steps": K, "warmup": W,
           "ms_per_step": round(ms, 3),
           "step_ms_p50": round(float(np.percentile(step_ms, 50)), 3),
           "step_ms_p90": round(float(np.percentile(step_ms, 90)), 3),
           "prefill_tok_s": round(2048 / (ms / 1e3), 1),
           "decode_tok_s": round(128 / (ms / 1e3), 1),
           "roofline_ms": round(roof, 3), "roofline_frac": round(roof / ms, 4),
           "roofline": {"bound": "mfma", "kernel": GATE_UP_MIXED_OP,
                        "achieved": round(gu_tfs, 1), "peak": BF16_PEAK_TFLOPS,
                        "unit": "TFLOP/s", "frac": round(gu_tfs / BF16_PEAK_TFLOPS, 4),
                        "traffic": None, "flop_per_op": gu_fl,
                        "us_per_op": round(gu_us, 1)},
           "ops_ms_per_step": {S.OP_NAMES[j]: round(op_ms[j] / K, 4) for j in range(len(op_ms))}}
    log(f"[bench] q32-mixed {ms:.3f} ms/step (roofline {roof:.3f} ms, {roof / ms:.1%}); "
        f"{2048 / (ms / 1e3):.0f} prefill + {128 / (ms / 1e3):.0f} decode tok/s; "
        f"gate-up {gu_tfs:.0f} TFLOP/s")
    if not getattr(args, "no_cpu", False):
        log("[bench] timing the CPU oracle: one mixed step of one Qwen3-32B-shaped layer")
        sec, reps, spent = oracle_layer_step(shape, chunks + [(int(c), 1) for c in dctx0], seed)
        res["cpu_baseline"] = cpu_block(2048 + 128, nL, sec, reps, spent,
                                        "one mixed step (4 x 512 prefill + 128 decode tokens; "
                                        "value counts both)")
    res["_est"] = est_in
    return res


def bench_tiny(args):
    """The tiny configuration end to end: 2 layers (hidden 256, 4/2 heads,
    head_dim 64, ffn 704), fp32 weights N(0, 0.02^2) from the seed, 4 prompts
    of 16..64 tokens prefilled in one call, then 16 decode steps; whole-run
    times in the fp32 and bf16 modes (launch-bound: neither roofline
    applies), and the oracle over the same run on the host."""
    import torch
    from paper_2606_18600_amd import synth
    from paper_2606_18600_amd.harness import DeviceStage, upload_weights
    dev = torch.device("cuda:0")
    shape, seed = synth.TINY, args.seed
    host = [synth.host_layer_weights(shape, seed, l) for l in range(2)]
    lens = synth.uniform_lengths(seed, 0, 4, 16, 64)
    bt_np = synth.make_block_tables(lens + 16, 8, synth.BlockAllocator(64, seed))
    bt = torch.from_numpy(bt_np).to(dev)
    xp = synth.hidden_states(seed, 1, int(lens.sum()), shape.hidden)
    xd = [synth.hidden_states(seed, 100 + k, 4, shape.hidden) for k in range(16)]
    n_tok = int(lens.sum()) + 64
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    res = {"workload": "tiny: 2 layers, hidden 256, 4 q / 2 kv heads, head_dim 64, ffn 704; "
                       "4 prompts uniform 16-64 prefilled, then 16 decode steps",
           "prompt_tokens": int(lens.sum()), "decode_tokens": 64}
    for dt in ("f32", "bf16"):
        td = torch.float32 if dt == "f32" else torch.bfloat16
        st = DeviceStage(shape, dt, 0, [upload_weights(h, dt) for h in host], 64, 256, 8)
        xpt = torch.from_numpy(xp).to(dev, td)
        xdt = [torch.from_numpy(a).to(dev, td) for a in xd]
        out = torch.empty_like(xpt)

        def run():
            st.prefill(lens, np.zeros(4, np.int32), bt, xpt, out, stream=sp)
            for k in range(16):
                st.decode(lens + k, bt, xdt[k], out[:4], stream=sp)

        for _ in range(3):
            run()
        torch.cuda.synchronize()
        reps = max(5, args.steps)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            run()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        st.close()
        res[dt] = {"ms_per_run": round(ms, 4), "tok_s": round(n_tok / (ms / 1e3), 1),
                   "runs": reps}
        log(f"[bench] tiny {dt}: {ms:.3f} ms per run (prefill + 16 decodes), "
            f"{n_tok / (ms / 1e3):.0f} tok/s")
    if not getattr(args, "no_cpu", False):
        from oracle import stage_oracle as O
        cfg = O.OracleConfig(shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                             shape.ffn, shape.rms_eps, shape.rope_theta)

        def oracle_run():
            kv = O.new_kv_cache(cfg, 2, 64, np.float32)
            O.stage_forward(cfg, host, xp, [O.SeqSpec(0, int(q), list(r))
                                            for q, r in zip(lens, bt_np)], kv, dtype=np.float32)
            for k in range(16):
                O.stage_forward(cfg, host, xd[k], [O.SeqSpec(int(c) + k, 1, list(r))
                                                   for c, r in zip(lens, bt_np)], kv,
                                dtype=np.float32)

        sec, reps, spent = time_oracle(oracle_run, 5.0)
        res["cpu_baseline"] = {"value": round(n_tok / sec, 1), "unit": "tok/s",
                               "cores": blas_threads(), "kind": "oracle",
                               "sample": f"the whole run (prefill + 16 decode steps, 2 layers) "
                                         f"in float32, {reps} run(s) in {spent:.1f} s"}
    return res


def bench_full_model(args):
    """The 80-layer model as one stage under continuous batching, with the
    roofline of its dominant kernels and the oracle baseline."""
    import torch
    from paper_2606_18600_amd import stage as S
    from paper_2606_18600_amd import synth
    from paper_2606_18600_amd.batcher import bench_l70_full
    shape, nL = synth.LLAMA70B, 80
    res = bench_l70_full(args, log)
    j = S.OP_NAMES.index("gate_up")
    for name in ("decode_only", "offline", "poisson"):
        r = res[name]
        op_ms, op_n = r.pop("_op_ms", None), r.pop("_op_n", None)
        if op_ms is not None and op_n[j]:
            r["ops_ms_per_step"] = {S.OP_NAMES[k]: round(op_ms[k] / 3, 3)
                                    for k in range(len(op_ms))}
    # dominant kernels: the decode-only step's gate-up (HBM) and the mixed
    # step's gate-up (MFMA), from the per-op timing of the steps after the
    # timed ones
    d = res["decode_only"]
    if "ops_ms_per_step" in d:
        gu_us = d["ops_ms_per_step"]["gate_up"] / nL * 1e3
        B = 128
        byts = 2 * shape.ffn * shape.hidden * 2 + B * shape.hidden * 2 + B * shape.ffn * 2
        gbs = byts / (gu_us / 1e6) / 1e9
        res["roofline"] = {"bound": "hbm", "kernel": "gemm_skinny8_bf16 (gate-up + SwiGLU of "
                                                     "decode-only steps: 65-128 rows; "
                                                     "gemm_skinny_bf16 below)",
                           "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                           "bytes_per_launch": byts, "us_per_launch": round(gu_us, 1),
                           "note": "bytes at batch 128; the batch shrinks as requests finish"}
    m = res["offline"]
    if "ops_ms_per_step" in m:
        gu_us = m["ops_ms_per_step"]["gate_up"] / nL * 1e3
        fl = 2.0 * 2176 * 2 * shape.ffn * shape.hidden
        res["roofline_mixed"] = {"bound": "mfma", "kernel": GATE_UP_MIXED_OP,
                                 "achieved": round(fl / (gu_us / 1e6) / 1e12, 1),
                                 "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                 "frac": round(fl / (gu_us / 1e6) / 1e12 / BF16_PEAK_TFLOPS, 4),
                                 "traffic": None, "us_per_op": round(gu_us, 1),
                                 "note": "FLOPs at 2176 rows (2048 prefill + 128 decode)"}
    if not getattr(args, "no_cpu", False):
        log("[bench] timing the CPU oracle: one decode step (batch 128) of one layer")
        ctx = synth.uniform_lengths(args.seed, 10, 128, 1024, 4096)
        sec, reps, spent = oracle_layer_step(shape, [(int(c), 1) for c in ctx], args.seed)
        res["cpu_baseline"] = cpu_block(128, nL, sec, reps, spent,
                                        "one decode step, batch 128, contexts uniform 1024-4096")
    return res


def estimator_check(args, result, configs, est_blocks):
    """The static latency estimator (Sec. 4.1.1: Eq. 1 with a one-time
    calibration, plus the per-launch cost) against the steps this run just
    measured: the Llama-70B-shaped decode step and chunked prefill run, and
    the Qwen3-32B-shaped mixed step. The calibration is measured here, on
    the same GPU, with the gate-up projection of a one-layer stage."""
    from paper_2606_18600_amd import estimator as E
    from paper_2606_18600_amd import synth
    t0 = time.time()
    cal = E.calibrate(synth.LLAMA70B, args.seed, log=log)
    out = {"calibration": {"tflops": round(cal.tflops, 1), "gbs": round(cal.gbs, 1),
                           "launch_us": round(cal.launch_us, 2),
                           "seconds": round(time.time() - t0, 1)}}
    rows = []

    def row(name, pred, meas):
        rows.append((pred, meas))
        out[name] = {"predicted_ms": round(pred, 3), "measured_ms": round(meas, 3),
                     "error_pct": round(100.0 * (pred - meas) / meas, 2)}

    l70, q32 = est_blocks
    if l70 is not None:
        sh, nL = l70["shape"], l70["n_layers"]
        launches = E.step_launches(nL, "decode") * cal.launch_us * 1e-3
        pred = float(np.mean([step_roofline_ms(sh, nL, [], c, cal.tflops, cal.gbs)
                              for c in l70["dec_ctx"]])) + launches
        row("l70_decode_step", pred, result["ms_per_step"])
        if "prefill_steps" in l70 and "prefill" in result:
            pred = sum(step_roofline_ms(sh, nL, stp, [], cal.tflops, cal.gbs)
                       + E.step_launches(nL, "prefill") * cal.launch_us * 1e-3
                       for stp in l70["prefill_steps"])
            row("l70_prefill_run", pred, result["prefill"]["ms_total"])
    if q32 is not None:
        sh, nL = q32["shape"], q32["n_layers"]
        launches = E.step_launches(nL, "prefill") * cal.launch_us * 1e-3
        pred = float(np.mean([step_roofline_ms(sh, nL, q32["chunks"], c, cal.tflops, cal.gbs)
                              for c in q32["dec_ctx"]])) + launches
        row("q32_mixed_step", pred, configs["q32_mixed"]["ms_per_step"])
    if rows:
        out["mape_pct"] = round(E.mape([p for p, _ in rows], [m for _, m in rows]), 2)
    log(f"[bench] estimator: {out}")
    return out


def bench_default(args):
    """One line for all five configurations: the metric's workload (the
    20-layer Llama-3.1-70B-shaped decode, batch 64) as `value`, the chunked
    prefill of the same stage, the tiny stage, the Qwen3-32B-shaped mixed step
    and the 80-layer model under continuous batching, each with its roofline
    and the oracle's time on the host."""
    import torch
    from paper_2606_18600_amd import stage as S
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    parts = ("tiny", "l70-decode", "q32-mixed", "l70-full")
    only = set(args.only.split(",")) if args.only else set(parts)
    if not only <= set(parts):
        raise SystemExit(f"--only takes a comma-separated subset of {', '.join(parts)}")
    configs = {}
    result = None
    if "tiny" in only:
        configs["tiny"] = bench_tiny(args)
    if "l70-decode" in only:
        result, ms, step_bytes, gu_gbs = bench_l70_stage(args)
    if "q32-mixed" in only:
        configs["q32_mixed"] = bench_q32_mixed(args)
    if "l70-full" in only:
        configs["l70_full"] = bench_full_model(args)
    if result is None:
        result = {"metric": METRIC, "value": None, "unit": "tok/s", "n_gpus": 1,
                  "steps": args.steps, "warmup": args.warmup, "higher_is_better": True,
                  "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
                  "config": {"workload": "partial run (--only)"}}
    if not args.no_estimator and ("l70-decode" in only or "q32-mixed" in only):
        est_blocks = [result.pop("_est", None)] + [configs.get("q32_mixed", {}).pop("_est", None)]
        result["estimator"] = estimator_check(args, result, configs, est_blocks)
    for c in configs.values():
        c.pop("_est", None)
    result.pop("_est", None)
    cal = calibrate(torch, S, stream)
    if "l70-decode" in only:
        cal["gate_up_frac_of_copy"] = round(gu_gbs / cal["copy_GBs"], 4)
        cal["decode_step_frac_of_copy"] = round(step_bytes / (ms / 1e3) / 1e9 / cal["copy_GBs"],
                                                4)
        if "prefill" in result:
            cal["prefill_frac_of_gemm_probe"] = round(
                result["prefill"]["tflops"] / cal["gemm_TFLOPs"], 4)
    result["calibrated"] = cal
    log(f"[bench] calibration: {cal}")
    result["host"] = host_info()
    result["configs"] = configs
    return result


# Context lengths of the migration sweep, and the links a migrated
# request's KV would otherwise cross: data-centre NICs between instances and,
# for scale, one xGMI link inside a node.
MIGRATE_LENGTHS = (1024, 2048, 4096, 8192, 16384, 32768, 65536)
MIGRATE_LINKS_GBS = {"25GbE": 3.125, "100GbE": 12.5, "400GbE": 50.0, "xGMI_link": 153.0}


def bench_migrate(args):
    """Migration by recomputation on the Llama-3.1-70B-shaped 20-layer stage:
    for each context length, the time to rebuild one request's KV by chunked
    prefill (2048-token chunks) over the hidden states of all its tokens,
    next to the bytes a KV transfer of the same request would move."""
    import torch
    from paper_2606_18600_amd import stage as S
    from paper_2606_18600_amd import synth
    from paper_2606_18600_amd.harness import (DeviceStage, device_layer_weights, model_config,
                                              pack_layer)
    from paper_2606_18600_amd.migrate import migration_points, recompute_kv
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    shape, seed = synth.LLAMA70B, args.seed
    wl = synth.WORKLOADS["l70-decode"]
    L0, nL = wl.layer_begin, wl.n_layers
    Lmax = max(MIGRATE_LENGTHS)
    nb = Lmax // 16
    cfg = model_config(shape, "bf16", max_position=Lmax)
    log(f"[bench] generating {nL} layers of {shape.name} weights on the device")
    weights = [pack_layer(cfg, device_layer_weights(shape, seed, l, "bf16"), free_source=True)
               for l in range(L0, wl.layer_end)]
    bt = torch.from_numpy(synth.make_block_tables([Lmax], nb, synth.BlockAllocator(nb + 1, seed)))
    bt = bt.to(dev)
    st = DeviceStage(shape, "bf16", L0, weights, nb + 1, max_tokens=2048, max_seqs=1, packed=True,
                     max_position=Lmax)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    hidden = torch.empty((Lmax, shape.hidden), dtype=torch.bfloat16, device=dev)
    hidden.normal_(0.0, 1.0, generator=g)
    out = torch.empty_like(hidden)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    recompute_kv(st, hidden[:4096], bt, 2048, out[:4096], stream=sp)  # warm-up
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ms_list, extra = [], []
    for L in MIGRATE_LENGTHS:
        reps = max(1, min(args.steps, 8192 // L))
        e0.record(stream)
        for _ in range(reps):
            recompute_kv(st, hidden[:L], bt, 2048, out[:L], stream=sp)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        S.stage_set_op_timing(st.handle, True)
        recompute_kv(st, hidden[:L], bt, 2048, out[:L], stream=sp)
        op_ms, _ = S.stage_read_op_times(st.handle)
        S.stage_set_op_timing(st.handle, False)
        assert torch.isfinite(out[:L].float()).all(), "non-finite stage output"
        chunks = [(c0, min(2048, L - c0)) for c0 in range(0, L, 2048)]
        fl = prefill_flops(shape, nL, chunks)
        ms_list.append(ms)
        extra.append({"tflops": round(fl / (ms / 1e3) / 1e12, 1),
                      "frac_mfma_peak": round(fl / (ms / 1e3) / 1e12 / BF16_PEAK_TFLOPS, 4),
                      "attn_share": round(op_ms[S.OP_NAMES.index("attn")] / sum(op_ms), 4)})
        log(f"[bench] recompute {L} tokens: {ms:.1f} ms ({reps} reps), "
            f"{fl / (ms / 1e3) / 1e12:.0f} TFLOP/s, attention {extra[-1]['attn_share']:.0%}")
    st.close()
    pts = []
    for (L, b, ms, link_ms), ex in zip(migration_points(shape, nL, MIGRATE_LENGTHS, ms_list,
                                                        MIGRATE_LINKS_GBS), extra):
        pts.append({"tokens": L, "recompute_ms": round(ms, 2),
                    "recompute_ms_per_layer": round(ms / nL, 3),
                    "kv_transfer_bytes": b, "kv_transfer_ms": {k: round(v, 2)
                                                               for k, v in link_ms.items()},
                    "breakeven_link_GBs": round(b / (ms / 1e3) / 1e9, 2), **ex})
    return {"workload": "migrate: Llama-3.1-70B-shaped stage, layers [20,40); one request's KV "
                        "rebuilt by chunked prefill (2048-token chunks) at 1K-64K tokens",
            "points": pts}


# The estimator sweep: the 80-layer Llama-3.1-70B cut into PP stages of TP
# ranks (PP x TP = 8), one rank's stage measured at its own shape; static
# batches of B requests with the mean prompt/output lengths of the paper's
# trace (763 / 232).
EST_CONFIGS = ((8, 1), (4, 2), (2, 4), (1, 8))
EST_BATCHES = (1, 2, 4, 8, 16, 32)
EST_S_IN, EST_S_OUT = 763, 232


def bench_estimator(args):
    """Static latency estimator against the measured stage (Sec. 4.1.1 and
    the accuracy experiment of Sec. 7): one-time calibration, then for each
    (PP, TP) and batch size the measured prefill + decode latency of one
    rank's stage next to Eq. 1's prediction; MAPE over all configurations."""
    import torch
    from paper_2606_18600_amd import estimator as E
    from paper_2606_18600_amd import synth
    from paper_2606_18600_amd.harness import (DeviceStage, device_layer_weights, model_config,
                                              pack_layer)
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    base, seed = synth.LLAMA70B, args.seed
    t0 = time.time()
    cal_l = E.calibrate(base, seed, log=log)
    cal_s = time.time() - t0
    # the paper's Eq. 1 alone, and with the per-launch cost
    cal = E.Calibration(cal_l.tflops, cal_l.gbs, 0.0, cal_l.gemm_samples, cal_l.gemv_samples)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    Bmax, nbs = max(EST_BATCHES), (EST_S_IN + EST_S_OUT + 15) // 16
    rows = []
    for pp, tp in EST_CONFIGS:
        shape, nL = E.tp_shard(base, tp), 80 // pp
        log(f"[bench] PP{pp}/TP{tp}: {nL} layers of {shape.name}")
        cfg = model_config(shape, "bf16")
        weights = [pack_layer(cfg, device_layer_weights(shape, seed, l, "bf16"), free_source=True)
                   for l in range(nL)]
        bt = torch.from_numpy(synth.make_block_tables(
            [EST_S_IN + EST_S_OUT] * Bmax, nbs, synth.BlockAllocator(Bmax * nbs + 1, seed))).to(dev)
        st = DeviceStage(shape, "bf16", 0, weights, Bmax * nbs + 1, max_tokens=2048,
                         max_seqs=Bmax, packed=True)
        x = torch.empty((2048, shape.hidden), dtype=torch.bfloat16, device=dev).normal_()
        out = torch.empty_like(x)

        def run(B):
            steps = synth.chunk_schedule([EST_S_IN] * B, 2048)
            tabs = [bt[[i for i, _, _ in stp]].contiguous() for stp in steps]
            ev[0].record(stream)
            for stp, tb in zip(steps, tabs):
                T = sum(q for _, _, q in stp)
                st.prefill([q for _, _, q in stp], [c for _, c, _ in stp], tb, x[:T], out[:T],
                           stream=sp)
            ev[1].record(stream)
            for t in range(1, EST_S_OUT + 1):
                st.decode(np.full(B, EST_S_IN + t - 1, np.int32), bt[:B], x[:B], out[:B],
                          stream=sp)
            ev[2].record(stream)
            torch.cuda.synchronize()
            return ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2])

        run(EST_BATCHES[0])  # warm-up
        for B in EST_BATCHES:
            pf, dc = run(B)
            ppf, pdc = E.static_batch_ms(shape, nL, B, EST_S_IN, EST_S_OUT, cal, prefill_chunk=2048)
            dpf, ddc = E.static_batch_ms(shape, nL, B, EST_S_IN, EST_S_OUT, E.DATASHEET,
                                         prefill_chunk=2048)
            lpf, ldc = E.static_batch_ms(shape, nL, B, EST_S_IN, EST_S_OUT, cal_l,
                                         prefill_chunk=2048)
            rows.append({"pp": pp, "tp": tp, "layers": nL, "batch": B,
                         "measured_ms": {"prefill": round(pf, 2), "decode": round(dc, 2)},
                         "predicted_ms": {"prefill": round(ppf, 2), "decode": round(pdc, 2)},
                         "datasheet_ms": {"prefill": round(dpf, 2), "decode": round(ddc, 2)},
                         "with_launch_ms": {"prefill": round(lpf, 2), "decode": round(ldc, 2)}})
            log(f"[bench]   B={B:2d}: measured {pf:8.1f} + {dc:8.1f} ms, predicted {ppf:8.1f} + "
                f"{pdc:8.1f} ms ({(ppf + pdc) / (pf + dc) - 1:+.1%})")
        st.close()
        del weights, st
        torch.cuda.empty_cache()

    def err(key, part=None):
        get = (lambda r, k: r[k]["prefill"] + r[k]["decode"]) if part is None else \
            (lambda r, k: r[k][part])
        return round(E.mape([get(r, key) for r in rows], [get(r, "measured_ms") for r in rows]), 2)

    res = {"workload": "estimator: Llama-3.1-70B, PP x TP in {8x1, 4x2, 2x4, 1x8}, one rank's "
                       "stage at its shard shape; static batches B = 1..32 of 763-token prompts "
                       "(2048-token prefill steps) and 232 decode steps",
           "calibration": {"tflops": round(cal.tflops, 1), "gbs": round(cal.gbs, 1),
                           "launch_us": round(cal_l.launch_us, 2),
                           "gemm_tflops": {k: round(v, 1) for k, v in cal.gemm_samples.items()},
                           "gemv_gbs": {k: round(v, 1) for k, v in cal.gemv_samples.items()},
                           "seconds": round(cal_s, 1)},
           "mape_pct": {"calibrated": err("predicted_ms"), "datasheet": err("datasheet_ms"),
                        "calibrated_with_launch": err("with_launch_ms"),
                        "calibrated_prefill": err("predicted_ms", "prefill"),
                        "calibrated_decode": err("predicted_ms", "decode")},
           "points": rows}
    log(f"[bench] MAPE calibrated {res['mape_pct']['calibrated']}%, "
        f"with launch cost {res['mape_pct']['calibrated_with_launch']}%, "
        f"datasheet {res['mape_pct']['datasheet']}%")
    return res


def bench_lm_head(args):
    """The last stage's LM head on the Llama-3.1-70B shape (vocab 128256):
    final RMSNorm + logits of 64 decode rows, of the last rows of 8 prompts,
    and of 256 rows (the tiled GEMM); HBM roofline of the weight read."""
    import torch
    from paper_2606_18600_amd import stage as S
    from paper_2606_18600_amd import synth
    from paper_2606_18600_amd.harness import (DeviceStage, device_layer_weights, model_config,
                                              pack_lm_head)
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    shape, seed, V = synth.LLAMA70B, args.seed, 128256
    cfg = model_config(shape, "bf16")
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    w = torch.empty((V, shape.hidden), dtype=torch.bfloat16, device=dev).normal_(0, 0.02,
                                                                                generator=g)
    wp = pack_lm_head(cfg, w)
    del w
    gain = torch.empty(shape.hidden, device=dev).normal_(1.0, 0.02, generator=g).to(torch.bfloat16)
    st = DeviceStage(shape, "bf16", 79, [device_layer_weights(shape, seed, 79, "bf16")], 8, 256, 4)
    x = torch.empty((256, shape.hidden), dtype=torch.bfloat16, device=dev).normal_(generator=g)
    logits = torch.empty((256, V), dtype=torch.float32, device=dev)
    sp = torch.cuda.current_stream().cuda_stream
    K = max(args.steps, 10)
    res = {"workload": "lm-head: Llama-3.1-70B final RMSNorm + logits, vocab 128256, hidden 8192",
           "cases": []}
    for label, n, rows in (("decode batch 64", 64, None), ("last rows of 8 prompts", 8,
                                                           list(range(255, 0, -32))),
                           ("256 rows", 256, None)):
        call = lambda: st.lm_head(gain, wp, x, rows=rows, n_rows=n, logits=logits[:n], stream=sp)
        call()
        torch.cuda.synchronize()
        S.stage_set_op_timing(st.handle, True)
        for _ in range(K):
            call()
        op_ms, op_n = S.stage_read_op_times(st.handle)
        S.stage_set_op_timing(st.handle, False)
        ms = op_ms[S.OP_NAMES.index("lm_head")] / K
        byts = V * shape.hidden * 2 + n * shape.hidden * 2 + n * V * 4
        fl = 2.0 * n * V * shape.hidden
        res["cases"].append({"rows": n, "label": label, "us_per_call": round(ms * 1e3, 1),
                             "algorithmic_bytes": byts, "GBs": round(byts / (ms / 1e3) / 1e9, 1),
                             "frac_hbm_peak": round(byts / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                             "tflops": round(fl / (ms / 1e3) / 1e12, 1)})
        log(f"[bench] lm-head {label}: {ms * 1e3:.1f} us, {byts / (ms / 1e3) / 1e9:.0f} GB/s, "
            f"{fl / (ms / 1e3) / 1e12:.0f} TFLOP/s")
    assert torch.isfinite(logits).all(), "non-finite logits"
    st.close()
    return res


# The decode gate-up projection is the split-K GEMM instantiated with the
# fused SwiGLU epilogue (template arguments <m-tiles, 1>).
GATE_UP_DECODE_KERNEL = r"gemm_skinny_bf16<\d+, ?1>"
KERNEL_SOURCES = ("paper_2606_18600_amd/csrc/k_gemm.hip", "paper_2606_18600_amd/csrc/common.hpp",
                  "paper_2606_18600_amd/csrc/packed.hpp", "paper_2606_18600_amd/csrc/kernels.hpp")
TRAFFIC_FILE = "profiles/gate_up_l70_decode_traffic.txt"


def kernel_source_sha():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def committed_traffic(kernel_re):
    """HBM bytes per launch of the kernel, from the committed counter summary
    (FETCH_SIZE and WRITE_SIZE runs scaled by the copy probe), or None when
    the summary is missing or the kernel sources changed since it was made."""
    import re
    path = os.path.join(ROOT, TRAFFIC_FILE)
    if not os.path.exists(path):
        return None, "no counter summary"
    sha, rows = None, {}
    for line in open(path):
        if line.startswith("source_sha256:"):
            sha = line.split(":", 1)[1].strip()
        elif line.startswith("TRAFFIC "):
            kv = dict(t.split("=", 1) for t in line.split()[1:])
            rows[kv["kernel"]] = kv
    if sha != kernel_source_sha():
        return None, "counters predate the current kernel sources"
    for name, kv in rows.items():
        if re.fullmatch(kernel_re, name):
            return (int(float(kv["fetch_bytes"]) + float(kv["write_bytes"])),
                    f"{TRAFFIC_FILE}: {name} grid {kv['grid']}, fetch {kv['fetch_bytes']} + "
                    f"write {kv['write_bytes']} bytes per launch")
    return None, "kernel not in the counter summary"


def calibrate(torch, S, stream):
    """Secondary denominators measured on this GPU: the library's plain
    streaming copy (read + write bytes) and a large bf16 library GEMM."""
    nbytes = 4 << 30
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1.0)
    sp = stream.cuda_stream
    ts = []
    for r in range(6):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        S.stage_copy_probe(src.data_ptr(), dst.data_ptr(), nbytes, sp)
        b.record(stream)
        b.synchronize()
        if r:
            ts.append(a.elapsed_time(b))
    copy_gbs = 2 * nbytes / (float(np.median(ts)) / 1e3) / 1e9
    del src, dst
    n = 8192
    x = torch.randn((n, n), dtype=torch.bfloat16, device="cuda")
    y = torch.randn((n, n), dtype=torch.bfloat16, device="cuda")
    ts = []
    for r in range(6):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        torch.mm(x, y)
        b.record(stream)
        b.synchronize()
        if r:
            ts.append(a.elapsed_time(b))
    gemm_tfs = 2.0 * n ** 3 / (float(np.median(ts)) / 1e3) / 1e12
    return {"copy_GBs": round(copy_gbs, 1), "copy_bytes": 2 * nbytes,
            "gemm_TFLOPs": round(gemm_tfs, 1), "gemm_probe": f"torch.mm bf16 {n}^3"}


def _short_kernel(name):
    for junk in ("void ", "stage_k::(anonymous namespace)::", "(anonymous namespace)::",
                 "stage_k::"):
        name = name.replace(junk, "")
    i = name.find("(")
    return name[:i] if i > 0 else name


def _csv_rows(d, suffix):
    import csv
    import glob
    files = sorted(glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True))
    if not files:
        raise SystemExit(f"no *{suffix} under {d}")
    rows = []
    for f in files:
        with open(f, newline="") as fh:
            rows += list(csv.DictReader(fh))
    return rows


def _grid(r):
    if "Grid_Size_X" in r:
        wg = max(1, int(r["Workgroup_Size_X"]))
        return f"{int(r['Grid_Size_X']) // wg},{int(r.get('Grid_Size_Y', 1))}"
    wg = max(1, int(r.get("Workgroup_Size", 1)))
    return f"{int(r['Grid_Size']) // wg}"


def summarize_trace(d, title, cmd, top=24):
    """Per (kernel, grid) launch statistics of a rocprofv3 kernel trace."""
    import collections
    g = collections.defaultdict(list)
    for r in _csv_rows(d, "kernel_trace.csv"):
        g[(_short_kernel(r["Kernel_Name"]), _grid(r))].append(
            (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    tot = sum(sum(v) for v in g.values())
    out = [f"# {title}", "", f"command: {cmd}", "",
           "Per (kernel, grid) launch statistics from the kernel trace (durations in us):", "",
           f"{'kernel':56s} {'grid':>10s} {'calls':>6s} {'avg_us':>9s} {'min_us':>9s} "
           f"{'max_us':>9s} {'pct':>6s}"]
    for (k, grid), v in sorted(g.items(), key=lambda kv: -sum(kv[1]))[:top]:
        out.append(f"{k[:56]:56s} {grid:>10s} {len(v):6d} {sum(v) / len(v):9.1f} "
                   f"{min(v):9.1f} {max(v):9.1f} {100 * sum(v) / tot:6.2f}")
    return "\n".join(out)


def summarize_pmc(fetch_dir, write_dir, title, cmds, algorithmic, top=12):
    """HBM traffic per launch from a FETCH_SIZE run and a WRITE_SIZE run, each
    scaled by what the counter reads for the copy probe of known size."""
    import collections
    per = {}
    for cname, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        g = collections.defaultdict(list)
        for r in _csv_rows(d, "counter_collection.csv"):
            if r["Counter_Name"] != cname:
                continue
            g[(_short_kernel(r["Kernel_Name"]), _grid(r))].append(float(r["Counter_Value"]))
        per[cname] = {k: float(np.mean(v)) for k, v in g.items()}
    copy_key = [k for k in per["FETCH_SIZE"] if k[0].startswith("copy_probe_kernel")]
    if not copy_key:
        raise SystemExit("the copy probe is missing from the counter run")
    ck = copy_key[0]
    copy_bytes = 4 << 30
    f_scale = copy_bytes / (per["FETCH_SIZE"][ck] * 1024)
    w_scale = copy_bytes / (per["WRITE_SIZE"][ck] * 1024)
    out = [f"# {title}", ""] + [f"command: {c}" for c in cmds] + [
        "",
        f"Copy probe ({ck[0]}, grid {ck[1]}): {copy_bytes} bytes read and written per launch;",
        f"FETCH_SIZE reads {per['FETCH_SIZE'][ck]:.0f} KiB, WRITE_SIZE "
        f"{per['WRITE_SIZE'][ck]:.0f} KiB -> scale factors {f_scale:.4f} (fetch), "
        f"{w_scale:.4f} (write).",
        "",
        "Scaled HBM bytes per launch (mean over launches), largest fetchers first:",
        "",
        f"{'kernel':44s} {'grid':>10s} {'fetch_KiB':>12s} {'write_KiB':>11s} "
        f"{'fetch_bytes':>13s} {'write_bytes':>12s}"]
    keys = sorted(per["FETCH_SIZE"], key=lambda k: -per["FETCH_SIZE"][k])[:top]
    lines = []
    for k in keys:
        fk, wk = per["FETCH_SIZE"][k], per["WRITE_SIZE"].get(k, 0.0)
        fb, wb = fk * 1024 * f_scale, wk * 1024 * w_scale
        out.append(f"{k[0][:44]:44s} {k[1]:>10s} {fk:12.0f} {wk:11.0f} {fb:13.0f} {wb:12.0f}")
        lines.append(f"TRAFFIC kernel={k[0].replace(' ', '')} grid={k[1]} fetch_bytes={fb:.0f} "
                     f"write_bytes={wb:.0f}")
    out += ["", f"Algorithmic bytes per launch: {algorithmic}", "",
            f"source_sha256: {kernel_source_sha()}",
            "(sha256 over " + ", ".join(KERNEL_SOURCES) + "; bench.py reports the traffic",
            "only while these sources are unchanged)", ""] + lines
    return "\n".join(out)


def host_info():
    """The host the oracle baselines run on."""
    model = ""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "nproc": os.cpu_count(), "oracle_threads": blas_threads()}


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return int(max([i.get("num_threads", 1) for i in threadpool_info()] + [1]))
    except Exception:
        return int(os.cpu_count() or 1)


def time_oracle(fn, budget_s=10.0, max_reps=40):
    """Seconds per call of fn: calls repeated until about budget_s have
    passed (at least once; the first call is dropped when there are more)."""
    ts = []
    t_start = time.perf_counter()
    while len(ts) < max_reps and (not ts or time.perf_counter() - t_start < budget_s):
        t0 = time.perf_counter()
        fn()
        ts.append(time.perf_counter() - t0)
    body = ts[1:] if len(ts) > 2 else ts
    return float(np.mean(body)), len(ts), time.perf_counter() - t_start


def oracle_layer_step(shape, seqs, seed, budget_s=10.0):
    """The oracle (float32) for one step of one layer: sequences given as
    (ctx, q) pairs, their context KV present in a paged cache (values do not
    change the cost), random weights of the layer's shape. Returns (seconds
    per step and layer, repetitions, seconds spent)."""
    from oracle import stage_oracle as O
    from paper_2606_18600_amd.synth import GAIN_NAMES
    cfg = O.OracleConfig(shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                         shape.ffn, shape.rms_eps, shape.rope_theta, shape.qk_norm,
                         shape.qk_rms_eps)
    r = np.random.default_rng(seed)
    w = {}
    for name, shp in shape.weight_shapes().items():
        a = r.standard_normal(shp, dtype=np.float32)
        w[name] = (1.0 + 0.02 * a) if name in GAIN_NAMES else 0.02 * a
    nbps = [(int(c) + int(q) + 15) // 16 for c, q in seqs]
    kv = O.new_kv_cache(cfg, 1, int(sum(nbps)), np.float32)
    kv[0]["k"].fill(0.01)
    kv[0]["v"].fill(0.01)
    starts = np.concatenate([[0], np.cumsum(nbps)]).astype(int)
    specs = [O.SeqSpec(int(c), int(q), list(range(starts[i], starts[i + 1])))
             for i, (c, q) in enumerate(seqs)]
    x = r.standard_normal((int(sum(q for _, q in seqs)), shape.hidden), dtype=np.float32)
    return time_oracle(lambda: O.stage_forward(cfg, [w], x, specs, kv, dtype=np.float32),
                       budget_s)


def cpu_block(tokens_per_step, n_layers, sec_layer, reps, spent, what, unit="tok/s"):
    """A cpu_baseline entry: one step of one layer timed, scaled by the
    stage's layers (every layer of a stage costs the same)."""
    step_s = sec_layer * n_layers
    return {"value": round(tokens_per_step / step_s, 3), "unit": unit, "cores": blas_threads(),
            "kind": "oracle",
            "sample": f"{what}; one layer in float32, {reps} run(s) in {spent:.1f} s, "
                      f"{sec_layer:.3f} s each, scaled x{n_layers} layers"}


def bench_l70_stage(args):
    """The metric's workload: the 20-layer Llama-3.1-70B-shaped stage, decode
    batch 64, then the chunked prefill of 8 prompts on the same stage."""
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
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    ctx_timed = []
    ev[0].record(stream)
    for k in range(K):
        st.decode(ctx0 + i, dec_bt, xs[i], out, stream=sp)
        ev[k + 1].record(stream)
        ctx_timed.append(ctx0 + i)
        i += 1
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[K]) / K
    step_ms = [ev[k].elapsed_time(ev[k + 1]) for k in range(K)]
    e0, e1 = ev[0], ev[K]
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
    gu_bytes = gate_up_swiglu_bytes(shape, B)
    gu_gbs = gu_bytes / (gu_avg_ms / 1e3) / 1e9
    log(f"[bench] ops ms/step: " + ", ".join(f"{k}={v['ms_per_step']:.3f}" for k, v in ops.items()))
    log(f"[bench] gate_up split-K GEMM: {gu_avg_ms * 1e3:.1f} us/launch, {gu_gbs:.0f} GB/s")

    gu_traffic, traffic_note = committed_traffic(GATE_UP_DECODE_KERNEL)
    result = {
        "metric": METRIC, "value": round(dec_tok_s, 1), "unit": "tok/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: random-init weights N(0,0.02^2) (gains 1+N(0,0.02^2)), "
                "N(0,1) hidden inputs, random context KV, shuffled block tables",
        "config": {"workload": "l70-decode: Llama-3.1-70B-shaped stage, layers [20,40), "
                               "decode batch 64, contexts uniform 512-2048, KV block 16",
                   "layers": nL, "batch": B, "hidden": shape.hidden, "block": 16},
        "roofline": {"bound": "hbm", "kernel": "gemm_skinny_bf16 (gate-up + SwiGLU, one K range)",
                     "achieved": round(gu_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gu_gbs / HBM_PEAK_GBS, 4), "traffic": gu_traffic,
                     "bytes_per_launch": gu_bytes, "us_per_launch": round(gu_avg_ms * 1e3, 2)},
        "step_ms_p50": round(float(np.percentile(step_ms, 50)), 4),
        "step_ms_p90": round(float(np.percentile(step_ms, 90)), 4),
        "step_roofline": {"bound": "hbm", "algorithmic_bytes": step_bytes,
                          "roofline_ms": round(step_bytes / (HBM_PEAK_GBS * 1e9) * 1e3, 4),
                          "measured_ms": round(ms, 4),
                          "frac": round(step_bytes / (HBM_PEAK_GBS * 1e9) / (ms / 1e3), 4)},
        "ops_ms_per_step": {k: round(v["ms_per_step"], 4) for k, v in ops.items()},
    }
    result["roofline"]["traffic_note"] = traffic_note
    result["_est"] = {"shape": shape, "n_layers": nL, "dec_ctx": ctx_timed}

    steps = []
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
        result["_est"]["prefill_steps"] = [[(c, q) for _, c, q in stp] for stp in steps]
        log(f"[bench] prefill {pms:.1f} ms, {ptok / (pms / 1e3):.0f} tok/s, "
            f"{pfl / (pms / 1e3) / 1e12:.0f} TFLOP/s; gate_up {gu_tfs:.0f} TFLOP/s")

    st.close()
    del weights, st
    torch.cuda.empty_cache()
    if not args.no_cpu:
        log("[bench] timing the CPU oracle: one decode step and one 2048-token chunk of one layer")
        sec, reps, spent = oracle_layer_step(shape, [(int(c), 1) for c in ctx0], seed)
        result["cpu_baseline"] = cpu_block(B, nL, sec, reps, spent,
                                           f"one decode step, batch {B} (contexts as the workload)")
        if "prefill" in result:
            first = steps[0]
            sec, reps, spent = oracle_layer_step(shape, [(c, q) for _, c, q in first], seed)
            result["prefill"]["cpu_baseline"] = cpu_block(
                sum(q for _, _, q in first), nL, sec, reps, spent,
                f"one 2048-token prefill step (the schedule's first: {len(first)} prompt chunk(s))")
    return result, ms, step_bytes, gu_gbs


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--seed", type=int, default=2606)
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-estimator", action="store_true",
                    help="default run: skip the estimator's check against the measured steps")
    ap.add_argument("--only", default="",
                    help="default run: comma-separated subset of tiny, l70-decode (with the "
                         "chunked prefill of the same stage), q32-mixed, l70-full")
    ap.add_argument("--requests", type=int, default=512,
                    help="l70-full: new requests queued behind the 128 running ones")
    ap.add_argument("--arrival-rate", type=float, default=0.0,
                    help="l70-full: Poisson arrivals per second (0: all at t=0)")
    ap.add_argument("--workload", default="l70-decode",
                    choices=["l70-decode", "q32-mixed", "l70-full", "migrate", "estimator",
                             "lm-head"],
                    help="l70-decode (default: the metric's workload, plus the chunked prefill "
                         "of the same stage); the others print their own line")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="print a summary of a rocprofv3 kernel trace under DIR and exit")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print HBM traffic per launch from FETCH_SIZE / WRITE_SIZE runs and exit")
    ap.add_argument("--summary-title", default="")
    ap.add_argument("--summary-cmd", action="append", default=[])
    ap.add_argument("--summary-algorithmic", default="",
                    help="with --summarize-pmc: the algorithmic-bytes line (default: the "
                         "decode gate-up's)")
    args = ap.parse_args()
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace, args.summary_title,
                              " ; ".join(args.summary_cmd)))
        return
    if args.summarize_pmc:
        from paper_2606_18600_amd import synth
        sh = synth.LLAMA70B
        alg = args.summary_algorithmic or (
            f"decode gate-up + SwiGLU (M=64, N={2 * sh.ffn}, K={sh.hidden}) "
            f"{gate_up_swiglu_bytes(sh, 64)} bytes")
        print(summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.summary_title,
                            args.summary_cmd, alg))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the stage runs on a single MI355X and the library "
              f"has no multi-GPU path (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    if args.workload == "q32-mixed":
        res = bench_q32_mixed(args)
        res.pop("_est", None)
        print(json.dumps({"metric": METRIC, "n_gpus": 1, "steps": args.steps,
                          "warmup": args.warmup, "dtype": "bf16", "data": "synthetic",
                          **res}), flush=True)
        return
    if args.workload == "lm-head":
        print(json.dumps({"metric": METRIC, "n_gpus": 1, "dtype": "bf16", "data": "synthetic",
                          **bench_lm_head(args)}), flush=True)
        return
    if args.workload == "estimator":
        print(json.dumps({"metric": METRIC, "n_gpus": 1, "dtype": "bf16", "data": "synthetic",
                          **bench_estimator(args)}), flush=True)
        return
    if args.workload == "migrate":
        print(json.dumps({"metric": METRIC, "n_gpus": 1, "dtype": "bf16", "data": "synthetic",
                          **bench_migrate(args)}), flush=True)
        return
    if args.workload == "l70-full":
        from paper_2606_18600_amd.batcher import bench_l70_full
        print(json.dumps({"metric": METRIC, "n_gpus": 1, "dtype": "bf16", "data": "synthetic",
                          **bench_l70_full(args, log)}), flush=True)
        return

    result = bench_default(args)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
