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
from typing import List, Optional

import numpy as np

from . import synth
from .roofline import step_roofline_ms


@dataclass
class Request:
    rid: int
    prompt: int
    out: int
    arrival: float
    blocks: List[int] = field(default_factory=list)
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
            r.blocks = self.alloc.take(need)
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

    def tables(self, reqs) -> np.ndarray:
        bt = np.zeros((max(1, len(reqs)), self.max_blocks), np.int32)
        for i, r in enumerate(reqs):
            bt[i, : len(r.blocks)] = r.blocks
        return bt


def bench_l70_full(args, log):
    """80 layers of the Llama-3.1-70B shape as one stage under continuous
    batching. Starts from 128 requests in their decode phase (contexts
    uniform 1024..4096, outputs lognormal median 256 sigma 0.8, progress
    uniform over the output) whose cached KV holds random values, plus a
    stream of new requests (all arriving at t = 0 unless --arrival-rate is
    given) that go through chunked prefill as blocks free up."""
    import torch
    from . import stage as S
    from .harness import DeviceStage, device_layer_weights, model_config, pack_layer

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    shape, seed = synth.LLAMA70B, args.seed
    nL = 80
    cfg = model_config(shape, "bf16")
    log(f"[bench] generating {nL} layers of {shape.name} weights on the device")
    weights = []
    for l in range(nL):
        weights.append(pack_layer(cfg, device_layer_weights(shape, seed, l, "bf16"),
                                  free_source=True))
    # the embedding and LM head of the full model occupy HBM though a stage
    # never runs them (hidden states in, hidden states out)
    emb = torch.empty((2, 128256, shape.hidden), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    free, _ = torch.cuda.mem_get_info()
    block_bytes = nL * shape.n_kv_heads * 2 * 16 * shape.head_dim * 2
    ws_guess = 3 << 30
    num_blocks = int((free - ws_guess - (4 << 30)) // block_bytes)
    log(f"[bench] KV pool: {num_blocks} blocks x {block_bytes >> 10} KiB = "
        f"{num_blocks * block_bytes / 1e9:.1f} GB ({num_blocks * 16} tokens)")
    max_ctx = 4096 + 4096
    max_blocks = max_ctx // 16
    kv_pool = torch.empty(num_blocks * block_bytes // 2, dtype=torch.bfloat16, device=dev)
    st = DeviceStage(shape, "bf16", 0, weights, num_blocks, max_tokens=2048 + 128, max_seqs=160,
                     max_position=max_ctx, kv_pool=kv_pool, packed=True)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    st.kv_pool.normal_(0.0, 1.0, generator=g)

    rng = np.random.default_rng(seed)
    b = Batcher(num_blocks, max_blocks, 128, 2048, seed=seed)
    n_init, n_new = 128, int(getattr(args, "requests", 512))
    prompts = synth.uniform_lengths(seed, 10, n_init + n_new, 1024, 4096)
    outs = synth.lognormal_lengths(seed, 11, n_init + n_new, 256, 0.8, 4096)
    rate = getattr(args, "arrival_rate", 0.0) or 0.0
    arr = synth.poisson_arrivals(seed, 12, n_new, rate) if rate > 0 else np.zeros(n_new)
    for i in range(n_init):
        r = Request(i, int(prompts[i]), int(outs[i]), 0.0)
        r.prefilled = r.prompt
        r.decoded = int(rng.integers(0, r.out))
        r.blocks = b.alloc.take(r.need_blocks(16))
        b.running.append(r)
    for j in range(n_new):
        b.submit(Request(n_init + j, int(prompts[n_init + j]), int(outs[n_init + j]),
                         float(arr[j])))

    xin = torch.empty((2048 + 128, shape.hidden), dtype=torch.bfloat16, device=dev)
    xin.normal_(generator=g)
    out = torch.empty_like(xin)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    steps, warm = args.steps, args.warmup
    gpu_clock = 0.0
    rec = []
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(warm + steps)]
    host_ms = []
    for k in range(warm + steps):
        t0 = time.perf_counter()
        b.admit(gpu_clock)
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
        if k % 16 == 15:
            ev[k][1].synchronize()
            gpu_clock = sum(ev[i][0].elapsed_time(ev[i][1]) for i in range(k + 1)) / 1e3
            log(f"[bench]   step {k + 1}: running {len(b.running)}, queued {len(b.queue)}, "
                f"finished {b.finished}")
    torch.cuda.synchronize()
    times = [ev[k][0].elapsed_time(ev[k][1]) for k, *_ in rec]
    timed = [(t, r) for t, r in zip(times, rec) if r[0] >= warm]
    tot_ms = sum(t for t, _ in timed)
    p_tok = sum(r[1] for _, r in timed)
    d_tok = sum(r[2] for _, r in timed)
    dec_only = [(t, r) for t, r in timed if r[1] == 0]
    roof = [step_roofline_ms(shape, nL, r[3], r[4]) for _, r in timed]
    res = {"workload": "l70-full: Llama-3.1-70B-shaped 80-layer model as one stage, bf16; "
                       "continuous batching, <=128 decodes + <=2048 prefill tokens per step, "
                       "contexts uniform 1024-4096, outputs lognormal(median 256, sigma 0.8), "
                       "admission on the KV pool",
           "steps": len(timed), "warmup": warm, "kv_pool_blocks": num_blocks,
           "decode_tok_s": round(d_tok / (tot_ms / 1e3), 1),
           "prefill_tok_s": round(p_tok / (tot_ms / 1e3), 1),
           "ms_per_step": round(tot_ms / max(1, len(timed)), 3),
           "roofline_ms_per_step": round(float(np.mean(roof)), 3),
           "roofline_frac": round(float(np.sum(roof)) / tot_ms, 4),
           "host_ms_per_step": round(float(np.mean(host_ms)), 3),
           "finished_requests": b.finished}
    if dec_only:
        dm = float(np.mean([t for t, _ in dec_only]))
        res["decode_only_ms_per_step"] = round(dm, 3)
        res["decode_only_tok_s"] = round(float(np.mean([r[2] for _, r in dec_only])) / (dm / 1e3), 1)
    log(f"[bench] l70-full: {res}")
    st.close()
    del emb
    return res


