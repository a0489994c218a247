"""Continuous batching over one stage: the workload driver for the full
80-layer Llama-3.1-70B-shaped model run as a single stage.

Requests carry a prompt (context) length and an output length. A request is
admitted only when the KV pool can hold its whole lifetime, ceil((prompt +
output) / 16) blocks, so no admitted request is ever preempted. Every step
decodes one token for up to ``max_decodes`` requests whose prompts are in the
cache, and prefills up to ``prefill_budget`` prompt tokens of admitted
requests, first come first served (a prompt may span steps). The step is one
stage_step_mixed call; the stage has no LM head, so decode inputs are fresh
N(0, 1) rows and a request finishes after its output length in decode steps.
"""

from __future__ import annotations

import time
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

from . import synth
from .roofline import step_roofline_ms


@dataclass
class Request:
    rid: int
    prompt: int
    out: int
    arrival: float
    blocks: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int32))
    prefilled: int = 0   # prompt tokens already in the cache
    decoded: int = 0     # decode steps done

    @property
    def in_decode(self) -> bool:
        return self.prefilled == self.prompt

    @property
    def done(self) -> bool:
        return self.decoded >= self.out

    def need_blocks(self, block: int) -> int:
        return (self.prompt + self.out + block - 1) // block


class Batcher:
    def __init__(self, num_blocks: int, max_blocks_per_seq: int, max_decodes: int = 128,
                 prefill_budget: int = 2048, block: int = synth.BLOCK, seed: int = 0):
        self.alloc = synth.BlockAllocator(num_blocks, seed)
        self.block = block
        self.max_blocks = max_blocks_per_seq
        self.max_decodes = max_decodes
        self.prefill_budget = prefill_budget
        self.queue: List[Request] = []
        self.running: List[Request] = []
        self.finished = 0

    def submit(self, r: Request) -> None:
        self.queue.append(r)

    def admit(self, now: float) -> None:
        while self.queue and self.queue[0].arrival <= now:
            r = self.queue[0]
            need = r.need_blocks(self.block)
            if need > len(self.alloc.free) or need > self.max_blocks:
                break
            r.blocks = self.take_blocks(need)
            self.running.append(self.queue.pop(0))

    def plan(self):
        """(prefill entries [(request, ctx, q)], decode requests) for one step."""
        decodes = [r for r in self.running if r.in_decode and not r.done][: self.max_decodes]
        room = self.prefill_budget
        prefill = []
        for r in self.running:
            if room == 0:
                break
            if not r.in_decode:
                q = min(room, r.prompt - r.prefilled)
                prefill.append((r, r.prefilled, q))
                room -= q
        return prefill, decodes

    def commit(self, prefill, decodes) -> None:
        for r, _, q in prefill:
            r.prefilled += q
        for r in decodes:
            r.decoded += 1
        keep = []
        for r in self.running:
            if r.done:
                self.alloc.give_back(r.blocks)
                self.finished += 1
            else:
                keep.append(r)
        self.running = keep

    def take_blocks(self, n: int) -> np.ndarray:
        # int32 arrays, so that building a step's block tables is one row
        # copy per request (a list of ids converts element by element: ~1 ms
        # per step at 128 requests)
        return np.asarray(self.alloc.take(n), np.int32)

    def tables(self, reqs) -> np.ndarray:
        bt = np.zeros((max(1, len(reqs)), self.max_blocks), np.int32)
        for i, r in enumerate(reqs):
            bt[i, : len(r.blocks)] = r.blocks
        return bt


def lognormal_mean(median: float, sigma: float) -> float:
    return float(median * np.exp(sigma * sigma / 2.0))


def sustainable_rate(shape, n_layers: int, mean_prompt: float, mean_out: float,
                     max_decodes: int = 128, budget: int = 2048) -> Tuple[float, float, int]:
    """Request rate that the Eq. 1 roofline sustains with the batch full: every
    step decodes ``max_decodes`` tokens and prefills the prompt tokens that
    keep pace with them (``mean_prompt / mean_out`` per decode token, at most
    ``budget``); live decode contexts average ``mean_prompt + mean_out / 2``
    and a prefill chunk sits behind half of what is left of its prompt.
    Returns (requests per second, roofline ms of such a step, prefill tokens
    per step)."""
    P = int(min(budget, round(max_decodes * mean_prompt / mean_out)))
    ctx = np.full(max_decodes, mean_prompt + mean_out / 2.0)
    prefix = max(0.0, (mean_prompt - P) / 2.0)
    ms = step_roofline_ms(shape, n_layers, [(prefix, P)], ctx)
    per_step = min(max_decodes / mean_out, P / mean_prompt)
    return per_step / (ms / 1e3), ms, P


def run_continuous(st, shape, n_layers: int, seed: int, steps: int, warm: int, n_new: int,
                   rate: float, num_blocks: int, max_blocks: int, xin, out, stream, log,
                   op_steps: int = 0, max_decodes: int = 128, budget: int = 2048,
                   stream_base: int = 10) -> Dict:
    """One continuous-batching run on a stage. 128 requests are running at
    the start, in their decode phase: contexts uniform 1024..4096 (already
    cached; the pool holds random values there) and remaining outputs
    lognormal (median 256, sigma 0.8, capped at 4096). ``n_new`` more
    requests (prompts uniform 1024..4096, the same outputs) arrive as a
    Poisson process of ``rate`` per second, or all at t = 0 when ``rate`` is
    0. The clock is the GPU's: after each step is enqueued the host waits for
    the step before it and reads its end event, so admission sees arrivals
    one step late at most; when nothing can run, the clock moves to the next
    arrival (idle time). Timed: ``steps`` steps after ``warm``; then
    ``op_steps`` more with per-op timing."""
    import torch
    from . import stage as S
    dev = xin.device
    b = Batcher(num_blocks, max_blocks, max_decodes, budget, seed=seed)
    n_init = max_decodes
    ctx0 = synth.uniform_lengths(seed, stream_base, n_init, 1024, 4096)
    prompts = synth.uniform_lengths(seed, stream_base + 1, max(1, n_new), 1024, 4096)
    outs = synth.lognormal_lengths(seed, stream_base + 2, n_init + n_new, 256, 0.8, 4096)
    arr = (synth.poisson_arrivals(seed, stream_base + 3, n_new, rate) if rate > 0
           else np.zeros(n_new))
    for i in range(n_init):
        r = Request(i, int(ctx0[i]), int(outs[i]), 0.0)
        r.prefilled = r.prompt
        r.blocks = b.take_blocks(r.need_blocks(synth.BLOCK))
        b.running.append(r)
    for j in range(n_new):
        b.submit(Request(n_init + j, int(prompts[j]), int(outs[n_init + j]), float(arr[j])))

    sp = stream.cuda_stream
    total = warm + steps + op_steps
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(total)]
    clock, idle = 0.0, 0.0
    rec, host_ms = [], []
    op_ms = op_n = None
    for k in range(total):
        if k == warm + steps and op_steps:
            torch.cuda.synchronize()
            S.stage_set_op_timing(st.handle, True)
        t0 = time.perf_counter()
        b.admit(clock)
        prefill, decodes = b.plan()
        while not prefill and not decodes and b.queue:
            nxt = b.queue[0].arrival
            if nxt <= clock:
                raise RuntimeError("request does not fit the KV pool")
            idle += nxt - clock
            clock = nxt
            b.admit(clock)
            prefill, decodes = b.plan()
        if not prefill and not decodes:
            break
        pq = [q for _, _, q in prefill]
        pc = [c for _, c, _ in prefill]
        dc = [r.prompt + r.decoded for r in decodes]
        pbt = torch.from_numpy(b.tables([r for r, _, _ in prefill])).to(dev, non_blocking=True)
        dbt = torch.from_numpy(b.tables(decodes)).to(dev, non_blocking=True)
        T = sum(pq) + len(dc)
        host_ms.append((time.perf_counter() - t0) * 1e3)
        ev[k][0].record(stream)
        st.mixed(pq, pc, pbt, dc, dbt, xin[:T], out[:T], stream=sp)
        ev[k][1].record(stream)
        rec.append((k, sum(pq), len(dc), [(c, q) for c, q in zip(pc, pq)], dc))
        b.commit(prefill, decodes)
        if k >= 1:
            ev[k - 1][1].synchronize()
            clock = ev[0][0].elapsed_time(ev[k - 1][1]) / 1e3 + idle
        if k % 8 == 7:
            log(f"[bench]   step {k + 1}: running {len(b.running)}, queued {len(b.queue)}, "
                f"finished {b.finished}, clock {clock:.2f} s")
    torch.cuda.synchronize()
    if op_steps:
        op_ms, op_n = S.stage_read_op_times(st.handle)
        S.stage_set_op_timing(st.handle, False)
    times = [ev[k][0].elapsed_time(ev[k][1]) for k, *_ in rec]
    timed = [(t, r) for t, r in zip(times, rec) if warm <= r[0] < warm + steps]
    tot_ms = sum(t for t, _ in timed)
    p_tok = sum(r[1] for _, r in timed)
    d_tok = sum(r[2] for _, r in timed)
    roof = [step_roofline_ms(shape, n_layers, r[3], r[4]) for _, r in timed]
    step_ms = [t for t, _ in timed]
    res = {"steps": len(timed), "warmup": warm,
           "ms_per_step": round(tot_ms / max(1, len(timed)), 3),
           "step_ms_p50": round(float(np.percentile(step_ms, 50)), 3) if step_ms else None,
           "step_ms_p90": round(float(np.percentile(step_ms, 90)), 3) if step_ms else None,
           "decode_tok_s": round(d_tok / (tot_ms / 1e3), 1) if tot_ms else 0.0,
           "prefill_tok_s": round(p_tok / (tot_ms / 1e3), 1) if tot_ms else 0.0,
           "decode_tokens": d_tok, "prefill_tokens": p_tok,
           "roofline_ms_per_step": round(float(np.mean(roof)), 3) if roof else None,
           "roofline_frac": round(float(np.sum(roof)) / tot_ms, 4) if tot_ms else None,
           "host_ms_per_step": round(float(np.mean(host_ms)), 3) if host_ms else None,
           "idle_s": round(idle, 3), "arrival_rate_per_s": rate,
           "new_requests": n_new, "admitted_new": n_new - len(b.queue),
           "finished_requests": b.finished, "queued_at_end": len(b.queue)}
    if op_ms is not None:
        res["_op_ms"], res["_op_n"] = op_ms, op_n
    return res


def setup_l70_full(seed: int, log, reserve_bytes: int = 4 << 30):
    """The 80-layer stage, its weights (plus the embedding and LM head of the
    full model, which occupy HBM though a stage never runs them) and a KV
    pool sized from the HBM that is left."""
    import torch
    from .harness import DeviceStage, device_layer_weights, model_config, pack_layer
    dev = torch.device("cuda:0")
    shape, nL = synth.LLAMA70B, 80
    cfg = model_config(shape, "bf16")
    log(f"[bench] generating {nL} layers of {shape.name} weights on the device")
    weights = [pack_layer(cfg, device_layer_weights(shape, seed, l, "bf16"), free_source=True)
               for l in range(nL)]
    emb = torch.empty((2, 128256, shape.hidden), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    free, _ = torch.cuda.mem_get_info()
    block_bytes = nL * shape.n_kv_heads * 2 * 16 * shape.head_dim * 2
    ws_guess = 3 << 30
    num_blocks = int((free - ws_guess - reserve_bytes) // block_bytes)
    log(f"[bench] KV pool: {num_blocks} blocks x {block_bytes >> 10} KiB = "
        f"{num_blocks * block_bytes / 1e9:.1f} GB ({num_blocks * 16} tokens)")
    max_ctx = 4096 + 4096
    kv_pool = torch.empty(num_blocks * block_bytes // 2, dtype=torch.bfloat16, device=dev)
    st = DeviceStage(shape, "bf16", 0, weights, num_blocks, max_tokens=2048 + 128, max_seqs=160,
                     max_position=max_ctx, kv_pool=kv_pool, packed=True)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    st.kv_pool.normal_(0.0, 1.0, generator=g)
    xin = torch.empty((2048 + 128, shape.hidden), dtype=torch.bfloat16, device=dev)
    xin.normal_(generator=g)
    return st, weights, emb, num_blocks, max_ctx // 16, xin


def bench_l70_full(args, log):
    """80 layers of the Llama-3.1-70B shape as one stage under continuous
    batching, in three runs over the same stage: decode-only (the 128 running
    requests, no arrivals), offline (``--requests`` new requests all queued
    at t = 0) and online (the same requests arriving as a Poisson process at
    1.25 x the rate the Eq. 1 roofline sustains, or ``--arrival-rate``)."""
    import torch
    shape, seed, nL = synth.LLAMA70B, args.seed, 80
    st, weights, emb, num_blocks, max_blocks, xin = setup_l70_full(seed, log)
    out = torch.empty_like(xin)
    stream = torch.cuda.current_stream()
    mean_prompt, mean_out = (1024 + 4096) / 2.0, lognormal_mean(256, 0.8)
    lam_star, lam_ms, lam_P = sustainable_rate(shape, nL, mean_prompt, mean_out)
    lam = getattr(args, "arrival_rate", 0.0) or 1.25 * lam_star
    n_new = int(getattr(args, "requests", 512))
    log(f"[bench] roofline-sustainable rate {lam_star:.2f} req/s (steps of 128 decodes + "
        f"{lam_P} prefill tokens, {lam_ms:.1f} ms each); Poisson arrivals at {lam:.2f} req/s")
    res = {"workload": "l70-full: Llama-3.1-70B-shaped 80-layer model as one stage, bf16; "
                       "continuous batching, <=128 decodes + <=2048 prefill tokens per step, "
                       "contexts uniform 1024-4096, outputs lognormal(median 256, sigma 0.8), "
                       "admission on the KV pool",
           "kv_pool_blocks": num_blocks,
           "sustainable_rate_per_s": round(lam_star, 3),
           "sustainable_step": {"roofline_ms": round(lam_ms, 3), "decodes": 128,
                                "prefill_tokens": lam_P},
           "arrival_rate_per_s": round(lam, 3)}
    runs = (("decode_only", 0, 0.0), ("offline", n_new, 0.0), ("poisson", n_new, lam))
    for name, nn, rate in runs:
        log(f"[bench] l70-full {name}: {nn} new requests, rate {rate:.2f}/s")
        r = run_continuous(st, shape, nL, seed, args.steps, args.warmup, nn, rate, num_blocks,
                           max_blocks, xin, out, stream, log, op_steps=3)
        res[name] = r
        log(f"[bench] l70-full {name}: {r['ms_per_step']:.1f} ms/step, "
            f"{r['decode_tok_s']:.0f} decode + {r['prefill_tok_s']:.0f} prefill tok/s, "
            f"{r['roofline_frac']:.1%} of the Eq. 1 roofline")
    st.close()
    del emb, weights
    torch.cuda.empty_cache()
    return res
