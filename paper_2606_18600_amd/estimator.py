"""Static latency estimator of a pipeline stage and its one-time calibration
(Sec. 4.1.1).

Each operation of a layer is priced by Eq. 1, the roofline: the larger of
its FLOPs over the effective FLOP rate and its memory-scan bytes over the
effective memory bandwidth. A stage's latency is the sum over the operations
of Table 2 times its layer count. Under static batching (the paper's
accuracy experiment, Sec. 7 "Serving Performance Estimation Accuracy"), a
batch of B requests with S_in prompt tokens and S_out output tokens costs one
prefill of all prompts plus S_out decode steps. Decode step t (1-based)
attends S_in + t keys per sequence.

The operation counts are those of Table 2 with these corrections (the same
ones the stage's roofline uses):
- the K/V projection width is n_kv * d (Table 2's H_kv stands for that width);
- the query / attention-output width n_q * d may differ from H (Qwen3);
- prefill attention counts causal (query, key) pairs only;
- decode attention is summed over the B sequences of the batch;
- each operation's output is counted in its memory term.
Tensor parallelism enters through the shard shape: one rank holds n_q/TP
query heads, n_kv/TP kv heads and F/TP of the FFN. This reproduces Table 2's
division by D_TP for every projection.

The denominators come from a one-time calibration on the device. The
effective FLOP rate is taken from a compute-bound GEMM and the effective
bandwidth from a memory-bound GEMV. Each is measured at several batch sizes
and summarised by the median (Sec. 4.1.1; Sec. 7 "One-time Calibration
Overhead").

One refinement goes beyond the paper's formulation. Its Discussion (Sec. 8)
names kernel-launch overhead as a non-linear cost that Eq. 1 leaves out. On
MI355X every kernel boundary costs a few microseconds, whatever the kernel
does. A stage step launches a fixed number of kernels per layer. So the
calibration also measures one scalar, the mean cost per launch beyond Eq. 1,
on a one-layer decode step. With `launch_us` > 0, each step adds that much
per kernel it launches. With `launch_us` = 0 the estimator is Eq. 1 alone. Eq. 3 (requests per second), Eq. 4 (pipeline latency as the
slowest stage's prefill plus the slowest stage's decode) and the alpha-beta
communication terms L_PP and L_TP of Sec. 4.1.2 are given for the placement
optimizer's cost curve. The communication terms take link figures as
arguments; nothing here measures a network.
"""

from __future__ import annotations

import dataclasses
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np

from .roofline import BF16_PEAK_TFLOPS, HBM_PEAK_GBS
from .synth import chunk_schedule


@dataclass(frozen=True)
class Op:
    """One operation of a layer: FLOPs and memory-scan bytes."""
    name: str
    flops: float
    bytes: float


@dataclass(frozen=True)
class Calibration:
    """Effective compute rate (TFLOP/s) and memory bandwidth (GB/s), with the
    per-batch-size samples they were taken from."""
    tflops: float
    gbs: float
    launch_us: float = 0.0
    gemm_samples: Dict[int, float] = dataclasses.field(default_factory=dict)
    gemv_samples: Dict[int, float] = dataclasses.field(default_factory=dict)


DATASHEET = Calibration(BF16_PEAK_TFLOPS, HBM_PEAK_GBS)


def tp_shard(shape, tp: int):
    """The layer shape one tensor-parallel rank of `tp` holds: query and kv
    heads and the FFN width divided by `tp` (column split of QKV and gate-up,
    row split of O and down; Sec. 2.3, Sec. 4.1.2)."""
    if tp < 1 or shape.n_kv_heads % tp or shape.n_q_heads % tp or shape.ffn % tp:
        raise ValueError(f"{shape.name}: heads {shape.n_q_heads}/{shape.n_kv_heads} and ffn "
                         f"{shape.ffn} must divide by tp={tp}")
    if tp == 1:
        return shape
    return dataclasses.replace(shape, name=f"{shape.name}-tp{tp}",
                               n_q_heads=shape.n_q_heads // tp,
                               n_kv_heads=shape.n_kv_heads // tp, ffn=shape.ffn // tp)


def _proj_ops(shape, T: int, E: int) -> List[Op]:
    """The four projections over T rows (Table 2: QKV, Output, Up and Gate,
    Down): 2 * rows * N * K FLOPs; weight, input and output bytes."""
    H, F = shape.hidden, shape.ffn
    qw = shape.n_q_heads * shape.head_dim
    qkvw = qw + 2 * shape.n_kv_heads * shape.head_dim
    return [
        Op("qkv", 2.0 * T * H * qkvw, E * (T * H + qkvw * H + T * qkvw)),
        Op("o_proj", 2.0 * T * qw * H, E * (T * qw + H * qw + T * H)),
        # gate and up are one [2F, H] product whose SwiGLU output is [T, F]
        Op("gate_up", 2.0 * T * H * 2 * F, E * (T * H + 2 * F * H + T * F)),
        Op("down", 2.0 * T * F * H, E * (T * F + H * F + T * H)),
    ]


def prefill_ops(shape, chunks, E: int = 2) -> List[Op]:
    """One layer's operations for prefill chunks given as (ctx, q): q new
    tokens after ctx cached ones. Attention: 4 * d * n_q FLOPs per causal
    (query, key) pair; reads every visible key/value once per sequence and
    the queries, writes the outputs."""
    d, nq, nkv = shape.head_dim, shape.n_q_heads, shape.n_kv_heads
    T = sum(q for _, q in chunks)
    pairs = sum(q * c + q * (q + 1) / 2.0 for c, q in chunks)
    keys = sum(c + q for c, q in chunks)
    ops = _proj_ops(shape, T, E)
    ops.insert(1, Op("attention", 4.0 * d * nq * pairs,
                     E * (keys * 2 * nkv * d + 2.0 * T * nq * d)))
    return ops


def decode_ops(shape, ctx_lens, E: int = 2) -> List[Op]:
    """One layer's operations for one decode step of len(ctx_lens) sequences
    (sequence i attends ctx_lens[i] + 1 keys, its own included)."""
    d, nq, nkv = shape.head_dim, shape.n_q_heads, shape.n_kv_heads
    B = len(ctx_lens)
    keys = float(np.sum(np.asarray(ctx_lens, np.float64) + 1))
    ops = _proj_ops(shape, B, E)
    ops.insert(1, Op("attention", 4.0 * d * nq * keys, E * (keys * 2 * nkv * d + 2.0 * B * nq * d)))
    return ops


def op_ms(op: Op, cal: Calibration) -> float:
    """Eq. 1: max(FLOPs / FLOP rate, bytes / bandwidth), in milliseconds."""
    return max(op.flops / (cal.tflops * 1e12), op.bytes / (cal.gbs * 1e9)) * 1e3


def layer_ms(ops: Sequence[Op], cal: Calibration) -> float:
    return sum(op_ms(o, cal) for o in ops)


# Kernels a stage step launches: per layer (prefill: norm, QKV, RoPE/KV
# write, attention, O, norm, gate-up, down; decode adds the split merge and
# the SwiGLU reduction of the split-K gate-up), plus the input norm and the
# output cast of the step.
KERNELS_PER_LAYER = {"prefill": 8, "decode": 10}
KERNELS_PER_STEP = 2


def step_launches(n_layers: int, phase: str) -> int:
    return n_layers * KERNELS_PER_LAYER[phase] + KERNELS_PER_STEP


def static_batch_ms(shape, n_layers: int, B: int, s_in: int, s_out: int, cal: Calibration,
                    prefill_chunk: Optional[int] = None):
    """(prefill ms, decode ms) of a static batch on a stage of `n_layers`
    layers of `shape`: B prompts of s_in tokens, then s_out decode steps.
    With `prefill_chunk`, the prompts are prefilled in steps of at most that
    many tokens (packed in request order, a prompt split across steps where
    it does not fit), each step priced on its own; without it, in one step."""
    if prefill_chunk is None:
        steps = [[(0, s_in)] * B]
    else:
        steps = [[(c, q) for _, c, q in st] for st in chunk_schedule([s_in] * B, prefill_chunk)]
    pf = n_layers * sum(layer_ms(prefill_ops(shape, st), cal) for st in steps)
    dc = n_layers * sum(layer_ms(decode_ops(shape, [s_in + t - 1] * B), cal)
                        for t in range(1, s_out + 1))
    pf += len(steps) * step_launches(n_layers, "prefill") * cal.launch_us * 1e-3
    dc += s_out * step_launches(n_layers, "decode") * cal.launch_us * 1e-3
    return pf, dc


def pipeline_latency_ms(stage_prefill_ms: Sequence[float], stage_decode_ms: Sequence[float]):
    """Eq. 4: the slowest stage's prefill plus the slowest stage's decode."""
    return max(stage_prefill_ms) + max(stage_decode_ms)


def requests_per_second(B: int, latency_ms: float) -> float:
    """Eq. 3: B requests complete per batch latency."""
    return B / (latency_ms / 1e3)


def comm_pp_ms(alpha_s: float, beta_gbs: float, B: int, S: int, H: int, E: int = 2) -> float:
    """L_PP (Sec. 4.1.2): one hidden-state transfer of B*S*H*E bytes between
    stages, alpha-beta model."""
    return (alpha_s + B * S * H * E / (beta_gbs * 1e9)) * 1e3


def comm_tp_ms(alpha_s: float, beta_gbs: float, B: int, S: int, H: int, tp: int, n_layers: int,
               E: int = 2) -> float:
    """L_TP (Sec. 4.1.2): two ring all-reduces of B*S*H*E bytes per layer,
    each a reduce-scatter plus an all-gather of tp-1 steps that move 1/tp of
    the data."""
    n = B * S * H * E
    return 4.0 * (alpha_s + n / (tp * beta_gbs * 1e9)) * (tp - 1) * n_layers * 1e3


def mape(pred: Sequence[float], meas: Sequence[float]) -> float:
    """Mean absolute percentage error, in percent."""
    p, m = np.asarray(pred, np.float64), np.asarray(meas, np.float64)
    return float(np.mean(np.abs(p - m) / m) * 100.0)


# --- one-time calibration on the device --------------------------------------

GEMM_TOKENS = (512, 1024, 2048, 4096)
GEMV_BATCHES = (1, 2, 4, 8, 16, 32, 64, 128)


def calibrate(shape, seed: int = 2606, reps: int = 10, log=None) -> Calibration:
    """Measure the effective FLOP rate and bandwidth with the stage's own
    gate-up projection (a [2F, H] weight) on a one-layer stage of `shape`.
    The compute-bound GEMM is that projection in prefill steps of
    GEMM_TOKENS rows. The memory-bound GEMV is the same projection in decode
    steps of GEMV_BATCHES rows. Each sample is FLOPs (or weight + activation
    bytes) over the projection's mean time from the stage's HIP-event op
    timers. Each scalar is the median of its samples. The launch cost is the
    median over the same decode steps of (measured step time - Eq. 1 for
    the layer) / kernels launched."""
    import torch
    from . import stage as S
    from . import synth
    from .harness import DeviceStage, device_layer_weights, model_config, pack_layer

    dev = torch.device("cuda:0")
    cfg = model_config(shape, "bf16")
    w = [pack_layer(cfg, device_layer_weights(shape, seed, 0, "bf16"), free_source=True)]
    Tmax, Bmax = max(GEMM_TOKENS), max(GEMV_BATCHES)
    ctx = 256
    nb_seq = (max(Tmax, ctx + 1) + 15) // 16
    alloc = synth.BlockAllocator(Bmax * nb_seq + 1, seed)
    bt = torch.from_numpy(synth.make_block_tables([nb_seq * 16] * Bmax, nb_seq, alloc)).to(dev)
    st = DeviceStage(shape, "bf16", 0, w, Bmax * nb_seq + 1, max_tokens=Tmax, max_seqs=Bmax,
                     packed=True)
    x = torch.empty((Tmax, shape.hidden), dtype=torch.bfloat16, device=dev).normal_()
    out = torch.empty_like(x)
    sp = torch.cuda.current_stream().cuda_stream
    j = S.OP_NAMES.index("gate_up")
    H, F = shape.hidden, shape.ffn

    def timed(call):
        call()  # warm-up
        torch.cuda.synchronize()
        S.stage_set_op_timing(st.handle, True)
        for _ in range(reps):
            call()
        ms, n = S.stage_read_op_times(st.handle)
        S.stage_set_op_timing(st.handle, False)
        return ms[j] / n[j]

    def step_ms(call):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        call()
        e0.record()
        for _ in range(reps):
            call()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    gemm, gemv, dec_ms = {}, {}, {}
    try:
        for T in GEMM_TOKENS:
            ms = timed(lambda: st.prefill([T], [0], bt[:1], x[:T], out[:T], stream=sp))
            gemm[T] = 2.0 * T * H * 2 * F / (ms / 1e3) / 1e12
        for B in GEMV_BATCHES:
            call = lambda: st.decode(np.full(B, ctx, np.int32), bt[:B], x[:B], out[:B], stream=sp)
            ms = timed(call)
            gemv[B] = 2.0 * (2 * F * H + B * H + B * F) / (ms / 1e3) / 1e9
            dec_ms[B] = step_ms(call)
    finally:
        st.close()
    base = Calibration(float(np.median(list(gemm.values()))), float(np.median(list(gemv.values()))))
    launch = float(np.median([(dec_ms[B] - layer_ms(decode_ops(shape, [ctx] * B), base)) * 1e3 /
                              step_launches(1, "decode") for B in GEMV_BATCHES]))
    cal = Calibration(base.tflops, base.gbs, max(0.0, launch), gemm, gemv)
    if log:
        log(f"[calibrate] GEMM TFLOP/s {', '.join(f'{k}:{v:.0f}' for k, v in gemm.items())} "
            f"-> {cal.tflops:.0f}; GEMV GB/s {', '.join(f'{k}:{v:.0f}' for k, v in gemv.items())} "
            f"-> {cal.gbs:.0f}; launch {cal.launch_us:.2f} us")
    return cal
