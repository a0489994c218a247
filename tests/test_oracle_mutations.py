"""The oracle's pins catch plausible mistakes (CPU only).

Each mutant is a copy of the oracle's source with one planted mistake (a
dropped term, a flipped sign, a wrong index, a transposed operand). The test
runs the pins of ``test_oracle_pins.py`` against the mutant and requires at
least one of them to fail. The planted mistakes live only in these in-memory
copies; the real oracle is untouched.
"""

from __future__ import annotations

import inspect
import sys
import types

import pytest

import oracle.stage_oracle as real_oracle
from tests import test_oracle_pins as pins

MUTANTS = {
    "rope-sign": ("a * c - b * s, a * s + b * c", "a * c + b * s, a * s + b * c"),
    "rope-interleaved": ("a, b = u[..., :half], u[..., half:]", "a, b = u[..., 0::2], u[..., 1::2]"),
    "rope-freq": ("omega = theta ** (-2.0 * j / d)", "omega = theta ** (-1.0 * j / d)"),
    "gqa-modulo": ("kvh = h // group", "kvh = h % n_kv"),
    "causal-exclusive": ("visible = t[None, :] <= q_pos[:, None]",
                         "visible = t[None, :] <= q_pos[:, None] - 1"),
    "scale-1-over-d": ("scale = 1.0 / np.sqrt(d)", "scale = 1.0 / d"),
    "no-attn-residual": ("x = x + rnd(attn.reshape(T, nq * d)) @ w[\"w_o\"].T",
                         "x = rnd(attn.reshape(T, nq * d)) @ w[\"w_o\"].T"),
    "wo-transposed": ("rnd(attn.reshape(T, nq * d)) @ w[\"w_o\"].T",
                      "rnd(attn.reshape(T, nq * d)) @ w[\"w_o\"]"),
    "gate-up-swapped": ("m = rnd(silu(gu[:, :cfg.ffn]) * gu[:, cfg.ffn:])",
                        "m = rnd(silu(gu[:, cfg.ffn:]) * gu[:, :cfg.ffn])"),
    "silu-is-sigmoid": ("return z / (1.0 + np.exp(-z))", "return 1.0 / (1.0 + np.exp(-z))"),
    "norm-no-mean": ("ms = np.mean(x * x, axis=-1, keepdims=True)",
                     "ms = np.sum(x * x, axis=-1, keepdims=True)"),
    "norm-no-gain": ("return x / np.sqrt(ms + eps) * g", "return x / np.sqrt(ms + eps)"),
    "ffn-norm-reuses-attn-gain": ("h2 = rnd(rms_norm(x, w[\"ffn_norm\"], cfg.rms_eps))",
                                  "h2 = rnd(rms_norm(x, w[\"attn_norm\"], cfg.rms_eps))"),
    "k-v-swapped": ("v = qkv[:, (nq + nkv) * d:].reshape(T, nkv, d)",
                    "v = qkv[:, nq * d:(nq + nkv) * d].reshape(T, nkv, d)"),
    "qk-norm-skipped-on-k": ("k = rms_norm(k, w[\"k_norm\"], cfg.qk_rms_eps)", "pass"),
    "no-rope-on-k": ("k = rnd(rope(k, pos, cfg.rope_theta))", "k = rnd(k)"),
    "positions-ignore-context": ("np.arange(s.ctx_len, s.ctx_len + s.q_len)", "np.arange(0, s.q_len)"),
    "lm-head-no-final-norm": ("return rms_norm(x, final_norm, cfg.rms_eps) @ w_lm.T",
                              "return x @ w_lm.T"),
    "lm-head-gain-ignored": ("return rms_norm(x, final_norm, cfg.rms_eps) @ w_lm.T",
                             "return rms_norm(x, 1.0, cfg.rms_eps) @ w_lm.T"),
    "slot-wrong-block": ("return int(block_table[p // block_size]), p % block_size",
                         "return int(block_table[p % len(block_table)]), p % block_size"),
}

PIN_TESTS = [(name, fn) for name, fn in inspect.getmembers(pins, inspect.isfunction)
             if name.startswith("test_")]


def _mutant(old: str, new: str, monkeypatch) -> types.ModuleType:
    src = inspect.getsource(real_oracle)
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    mod = types.ModuleType("oracle_mutant")
    monkeypatch.setitem(sys.modules, "oracle_mutant", mod)
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), mod.__dict__)
    return mod


def _params(fn):
    sig = inspect.signature(fn)
    marks = getattr(fn, "pytestmark", [])
    grids = [m.args for m in marks if m.name == "parametrize"]
    if not sig.parameters:
        return [dict()]
    combos = [dict()]
    for names, values in grids:
        names = [n.strip() for n in names.split(",")] if isinstance(names, str) else list(names)
        new = []
        for c in combos:
            for v in values:
                vals = v if len(names) > 1 else (v,)
                new.append({**c, **dict(zip(names, vals))})
        combos = new
    return combos


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_some_pin_fails_on_mutant(mutant, monkeypatch):
    mod = _mutant(*MUTANTS[mutant], monkeypatch)
    monkeypatch.setattr(pins, "O", mod)
    for name, fn in PIN_TESTS:
        for kw in _params(fn):
            try:
                fn(**kw)
            except Exception:
                return  # caught by this pin
    pytest.fail(f"no oracle pin detects mutant {mutant!r}")
