"""Shared test helpers: build oracle inputs from the seeded generators and
compare results. Test code only."""

from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np

from oracle.stage_oracle import OracleConfig, SeqSpec
from paper_2606_18600_amd import synth


def ocfg(shape: synth.ModelShape) -> OracleConfig:
    return OracleConfig(hidden=shape.hidden, n_q_heads=shape.n_q_heads,
                        n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim,
                        ffn=shape.ffn, rms_eps=shape.rms_eps, rope_theta=shape.rope_theta,
                        qk_norm=shape.qk_norm, qk_rms_eps=shape.qk_rms_eps,
                        block_size=shape.block_size)


def strong_weights(shape: synth.ModelShape, seed: int, layer: int) -> Dict[str, np.ndarray]:
    """Weights scaled so every branch contributes O(1) to the residual
    (std 1/sqrt(fan-in), gains U[0.5, 1.5]); pins then see any wiring error."""
    r = np.random.default_rng([seed, layer, 77])
    out = {}
    for name, shp in shape.weight_shapes().items():
        if name in synth.GAIN_NAMES:
            out[name] = r.uniform(0.5, 1.5, shp)
        else:
            out[name] = r.standard_normal(shp) / np.sqrt(shp[1])
    return out


def seqs_from(ctx_lens, q_lens, block_tables) -> List[SeqSpec]:
    return [SeqSpec(int(c), int(q), list(map(int, bt)))
            for c, q, bt in zip(ctx_lens, q_lens, block_tables)]


def rel_l2(y, ref) -> float:
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    n = np.linalg.norm(ref)
    return float(np.linalg.norm(y - ref) / (n if n > 0 else 1.0))


SMALL = synth.ModelShape("pin-small", hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=16,
                         ffn=96, rms_eps=1e-5, rope_theta=1e4)
SMALL_QK = synth.ModelShape("pin-small-qk", hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=16,
                            ffn=96, rms_eps=1e-6, rope_theta=1e6, qk_norm=True, qk_rms_eps=1e-6)
