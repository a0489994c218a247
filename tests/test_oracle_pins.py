"""Pins of the CPU oracle to things other than itself (CPU only).

Each test ties a part of ``oracle/stage_oracle.py`` to a closed form, an
invariant the method relies on, a brute-force evaluation, or an independent
library implementation (PyTorch's attention and RMSNorm, and the Llama /
Qwen3 decoder layers of ``transformers``). Together they are chosen so that a
dropped term, a wrong sign, a wrong index or a transposed operand anywhere in
the oracle fails at least one of them.
"""

from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import stage_oracle as O
from paper_2606_18600_amd import synth
from tests.helpers import SMALL, SMALL_QK, ocfg, rel_l2, seqs_from, strong_weights

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def _setup(shape, seed, ctx_lens, q_lens, n_layers=1, num_blocks=None, shuffle=True):
    cfg = ocfg(shape)
    totals = [c + q for c, q in zip(ctx_lens, q_lens)]
    max_blocks = max(1, max((t + 15) // 16 for t in totals))
    need = sum((t + 15) // 16 for t in totals)
    num_blocks = num_blocks or need + 3
    if shuffle:
        alloc = synth.BlockAllocator(num_blocks, seed)
    else:
        alloc = synth.BlockAllocator(num_blocks, seed)
        alloc.free = list(range(num_blocks))
    bt = synth.make_block_tables(totals, max_blocks, alloc)
    layers = [strong_weights(shape, seed, l) for l in range(n_layers)]
    return cfg, layers, bt, num_blocks


def _prefill_ctx(cfg, layers, bt, num_blocks, ctx_lens, seed):
    """Fill each sequence's first ctx_len tokens by a prefill; returns the cache."""
    kv = O.new_kv_cache(cfg, len(layers), num_blocks)
    if sum(ctx_lens):
        x = synth.hidden_states(seed, 1, int(sum(ctx_lens)), cfg.hidden, np.float64)
        seqs = seqs_from([0] * len(ctx_lens), ctx_lens, bt)
        seqs = [s for s in seqs if s.q_len > 0]
        O.stage_forward(cfg, layers, x, seqs, kv)
    return kv


def _copy_kv(kv):
    return [{k: v.copy() for k, v in d.items()} for d in kv]


# --------------------------------------------------------------------------
# P10 RMSNorm, P11 silu: closed forms and a library routine
# --------------------------------------------------------------------------

def test_rmsnorm_constant_vector_closed_form():
    for c in (0.0, 0.3, -2.5, 17.0):
        x = np.full((1, 32), c)
        g = np.linspace(0.5, 1.5, 32)
        y = O.rms_norm(x, g, 1e-5)
        np.testing.assert_allclose(y[0], g * c / np.sqrt(c * c + 1e-5), rtol=1e-14, atol=0)


def test_rmsnorm_matches_torch_and_scale_invariance():
    r = np.random.default_rng(1)
    x = r.standard_normal((5, 48)) * 3
    g = r.uniform(0.5, 1.5, 48)
    ref = torch.nn.functional.rms_norm(torch.tensor(x), (48,), torch.tensor(g), eps=1e-6).numpy()
    np.testing.assert_allclose(O.rms_norm(x, g, 1e-6), ref, rtol=1e-12, atol=1e-14)
    # with eps -> 0 the norm is invariant to a positive rescale of the row
    np.testing.assert_allclose(O.rms_norm(7.0 * x, g, 0.0), O.rms_norm(x, g, 0.0), rtol=1e-12)


def test_silu_closed_forms_and_torch():
    z = np.array([0.0, 1.0, -1.0, 40.0, -40.0, 3.5])
    y = O.silu(z)
    assert y[0] == 0.0
    np.testing.assert_allclose(y[1], 1.0 / (1.0 + np.exp(-1.0)), rtol=1e-15)
    np.testing.assert_allclose(y[1] - y[2], 1.0, rtol=1e-14)       # silu(x) - silu(-x) = x
    np.testing.assert_allclose(y[3], 40.0, rtol=1e-15)
    assert abs(y[4]) < 1e-15
    np.testing.assert_allclose(y, torch.nn.functional.silu(torch.tensor(z)).numpy(), rtol=1e-14)


# --------------------------------------------------------------------------
# P6 RoPE
# --------------------------------------------------------------------------

def test_rope_position_zero_is_identity():
    u = np.random.default_rng(2).standard_normal((3, 2, 16))
    np.testing.assert_array_equal(O.rope(u, np.zeros(3, np.int64), 1e4), u)


def test_rope_d2_closed_form():
    # d = 2: the only frequency is theta^0 = 1, so position p rotates by p radians.
    u = np.array([[[1.0, 0.0]], [[0.3, -0.7]]])
    pos = np.array([1, 5])
    y = O.rope(u, pos, 1e4)
    for i, p in enumerate(pos):
        c, s = np.cos(p), np.sin(p)
        a, b = u[i, 0]
        np.testing.assert_allclose(y[i, 0], [a * c - b * s, a * s + b * c], rtol=1e-14, atol=1e-15)


def test_rope_equals_complex_rotation_and_preserves_pair_norms():
    r = np.random.default_rng(3)
    d, theta = 16, 5e5
    u = r.standard_normal((6, 3, d))
    pos = np.array([0, 1, 2, 100, 4095, 70000])
    y = O.rope(u, pos, theta)
    # independent formulation: pair (j, j+d/2) as the complex number a + ib times e^{i p w_j}
    w = theta ** (-np.arange(d // 2) * 2.0 / d)
    zc = (u[..., : d // 2] + 1j * u[..., d // 2:]) * np.exp(1j * pos[:, None, None] * w[None, None, :])
    np.testing.assert_allclose(y[..., : d // 2], zc.real, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y[..., d // 2:], zc.imag, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y[..., : d // 2] ** 2 + y[..., d // 2:] ** 2,
                               u[..., : d // 2] ** 2 + u[..., d // 2:] ** 2, rtol=1e-12)


@pytest.mark.parametrize("delta", [1, 100, 4096])
def test_rope_relative_offset_invariance(delta):
    r = np.random.default_rng(4)
    q = r.standard_normal((5, 1, 32))
    k = r.standard_normal((5, 1, 32))
    pq = np.array([3, 9, 17, 40, 41])
    pk = np.array([0, 2, 17, 33, 41])
    s0 = np.einsum("id,jd->ij", O.rope(q, pq, 5e5)[:, 0], O.rope(k, pk, 5e5)[:, 0])
    s1 = np.einsum("id,jd->ij", O.rope(q, pq + delta, 5e5)[:, 0], O.rope(k, pk + delta, 5e5)[:, 0])
    np.testing.assert_allclose(s1, s0, rtol=1e-9, atol=1e-10)


# --------------------------------------------------------------------------
# P1, P7, P8 attention
# --------------------------------------------------------------------------

def test_attention_matches_naive_dense_and_torch_sdpa():
    r = np.random.default_rng(5)
    n_q, n_kv, d, C, n = 8, 2, 16, 37, 11
    k = r.standard_normal((C, n_kv, d))
    v = r.standard_normal((C, n_kv, d))
    q = r.standard_normal((n, n_q, d))
    pos = np.arange(C - n, C)
    out = O.attention_one_sequence(q, k, v, pos)
    # naive: explicit double loop over queries and keys
    naive = np.zeros_like(q)
    for i in range(n):
        for h in range(n_q):
            kvh = h // (n_q // n_kv)
            s = np.array([q[i, h] @ k[t, kvh] / np.sqrt(d) for t in range(pos[i] + 1)])
            p = np.exp(s - s.max())
            p /= p.sum()
            naive[i, h] = sum(p[t] * v[t, kvh] for t in range(pos[i] + 1))
    assert rel_l2(out, naive) < 1e-13
    # library: torch SDPA with GQA and an explicit causal-with-prefix mask
    mask = torch.tensor(np.arange(C)[None, :] <= pos[:, None])
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q).transpose(0, 1)[None], torch.tensor(k).transpose(0, 1)[None],
        torch.tensor(v).transpose(0, 1)[None], attn_mask=mask, enable_gqa=True)
    assert rel_l2(out, ref[0].transpose(0, 1).numpy()) < 1e-13


def test_gqa_equals_mha_with_repeated_kv():
    r = np.random.default_rng(6)
    n_q, n_kv, d, C = 6, 3, 8, 20
    k = r.standard_normal((C, n_kv, d))
    v = r.standard_normal((C, n_kv, d))
    q = r.standard_normal((C, n_q, d))
    pos = np.arange(C)
    gqa = O.attention_one_sequence(q, k, v, pos)
    mha = O.attention_one_sequence(q, np.repeat(k, 2, axis=1), np.repeat(v, 2, axis=1), pos)
    np.testing.assert_array_equal(gqa, mha)
    # consecutive grouping: heads 0,1 use kv 0; a kv-head permutation must change heads
    kp = k[:, [1, 0, 2]]
    vp = v[:, [1, 0, 2]]
    swapped = O.attention_one_sequence(q, kp, vp, pos)
    assert np.abs(swapped[:, :2] - gqa[:, :2]).max() > 1e-3
    np.testing.assert_array_equal(swapped[:, 4:], gqa[:, 4:])


def test_attention_single_key_and_identical_keys():
    r = np.random.default_rng(7)
    d = 16
    v = r.standard_normal((9, 1, d))
    q = r.standard_normal((1, 2, d))
    k1 = r.standard_normal((1, 1, d))
    np.testing.assert_array_equal(O.attention_one_sequence(q, k1, v[:1], np.array([0]))[0, 0], v[0, 0])
    k = np.repeat(k1, 9, axis=0)
    out = O.attention_one_sequence(q, k, v, np.array([8]))
    np.testing.assert_allclose(out[0, 0], v[:, 0].mean(axis=0), rtol=1e-13, atol=1e-15)


# --------------------------------------------------------------------------
# P14 library pin of a whole decoder layer: transformers' Llama and Qwen3
# --------------------------------------------------------------------------

def _hf_layer_output(shape, w, x):
    from transformers import LlamaConfig, Qwen3Config
    from transformers.models.llama.modeling_llama import LlamaDecoderLayer, LlamaRotaryEmbedding
    from transformers.models.qwen3.modeling_qwen3 import Qwen3DecoderLayer, Qwen3RotaryEmbedding
    C, L, R = ((Qwen3Config, Qwen3DecoderLayer, Qwen3RotaryEmbedding) if shape.qk_norm
               else (LlamaConfig, LlamaDecoderLayer, LlamaRotaryEmbedding))
    cfg = C(hidden_size=shape.hidden, intermediate_size=shape.ffn,
            num_attention_heads=shape.n_q_heads, num_key_value_heads=shape.n_kv_heads,
            head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
            rope_parameters={"rope_type": "default", "rope_theta": shape.rope_theta},
            max_position_embeddings=8192, attention_bias=False)
    cfg._attn_implementation = "eager"
    layer = L(cfg, layer_idx=0).to(torch.float64)
    nq, nkv, d, F = shape.q_width, shape.kv_width, shape.head_dim, shape.ffn
    sd = {"self_attn.q_proj.weight": w["w_qkv"][:nq],
          "self_attn.k_proj.weight": w["w_qkv"][nq:nq + nkv],
          "self_attn.v_proj.weight": w["w_qkv"][nq + nkv:],
          "self_attn.o_proj.weight": w["w_o"],
          "mlp.gate_proj.weight": w["w_gate_up"][:F],
          "mlp.up_proj.weight": w["w_gate_up"][F:],
          "mlp.down_proj.weight": w["w_down"],
          "input_layernorm.weight": w["attn_norm"],
          "post_attention_layernorm.weight": w["ffn_norm"]}
    if shape.qk_norm:
        sd["self_attn.q_norm.weight"] = w["q_norm"]
        sd["self_attn.k_norm.weight"] = w["k_norm"]
    layer.load_state_dict({k: torch.tensor(v) for k, v in sd.items()})
    rot = R(cfg)
    n = x.shape[0]
    xt = torch.tensor(x)[None]
    pos = torch.arange(n)[None]
    cos, sin = rot(xt, pos)
    mask = torch.full((n, n), float("-inf"), dtype=torch.float64).triu(1)[None, None]
    with torch.no_grad():
        y = layer(xt, attention_mask=mask, position_ids=pos, position_embeddings=(cos, sin))
    return y[0].numpy()


@pytest.mark.parametrize("shape", [SMALL, SMALL_QK], ids=["llama", "qwen3"])
def test_layer_matches_transformers_decoder_layer(shape):
    # transformers evaluates the norms, softmax and RoPE angles in float32 internally,
    # so agreement is ~1e-6; any wiring error is O(1).
    cfg, layers, bt, nb = _setup(shape, 11, [0], [45])
    x = synth.hidden_states(11, 2, 45, shape.hidden, np.float64)
    kv = O.new_kv_cache(cfg, 1, nb)
    y = O.stage_forward(cfg, layers, x, seqs_from([0], [45], bt), kv)
    ref = _hf_layer_output(shape, layers[0], x)
    assert rel_l2(y - x, ref - x) < 2e-5


# --------------------------------------------------------------------------
# P2-P5, P9, P12, P13: invariants of paging, chunking, decode and composition
# --------------------------------------------------------------------------

@pytest.mark.parametrize("shape", [SMALL, SMALL_QK], ids=["llama", "qwen3"])
def test_paged_shuffled_equals_contiguous_bitwise(shape):
    ctx, ql = [0, 0, 0], [23, 40, 9]
    cfg, layers, bt_s, nb = _setup(shape, 12, ctx, ql, n_layers=2, shuffle=True)
    _, _, bt_c, _ = _setup(shape, 12, ctx, ql, n_layers=2, shuffle=False)
    assert not np.array_equal(bt_s, bt_c)
    x = synth.hidden_states(12, 3, sum(ql), shape.hidden, np.float64)
    y_s = O.stage_forward(cfg, layers, x, seqs_from(ctx, ql, bt_s), O.new_kv_cache(cfg, 2, nb))
    y_c = O.stage_forward(cfg, layers, x, seqs_from(ctx, ql, bt_c), O.new_kv_cache(cfg, 2, nb))
    np.testing.assert_array_equal(y_s, y_c)


@pytest.mark.parametrize("chunk", [1, 3, 16, 17, 50])
def test_chunked_prefill_equals_one_shot(chunk):
    shape = SMALL_QK if chunk in (3, 17) else SMALL
    n = 50
    cfg, layers, bt, nb = _setup(shape, 13, [0], [n], n_layers=2)
    x = synth.hidden_states(13, 4, n, shape.hidden, np.float64)
    kv1 = O.new_kv_cache(cfg, 2, nb)
    y1 = O.stage_forward(cfg, layers, x, seqs_from([0], [n], bt), kv1)
    kv2 = O.new_kv_cache(cfg, 2, nb)
    parts = []
    for s in range(0, n, chunk):
        q = min(chunk, n - s)
        parts.append(O.stage_forward(cfg, layers, x[s:s + q], seqs_from([s], [q], bt), kv2))
    y2 = np.concatenate(parts)
    assert rel_l2(y2, y1) < 1e-12
    for l in range(2):
        for t in ("k", "v"):
            np.testing.assert_allclose(kv2[l][t], kv1[l][t], rtol=1e-12, atol=1e-13)


def test_decode_equals_last_row_of_extended_prefill():
    shape = SMALL_QK
    ctx = [21, 32, 5]
    cfg, layers, bt, nb = _setup(shape, 14, ctx, [1, 1, 1], n_layers=2)
    xs = [synth.hidden_states(14, 10 + i, c + 1, shape.hidden, np.float64) for i, c in enumerate(ctx)]
    # decode path: prefill each context, then one decode row per sequence in one batch
    kv = O.new_kv_cache(cfg, 2, nb)
    O.stage_forward(cfg, layers, np.concatenate([a[:-1] for a in xs]),
                    seqs_from([0] * 3, ctx, bt), kv)
    yd = O.stage_forward(cfg, layers, np.stack([a[-1] for a in xs]),
                         seqs_from(ctx, [1, 1, 1], bt), kv)
    # extended prefill of each whole sequence
    kv2 = O.new_kv_cache(cfg, 2, nb)
    yp = O.stage_forward(cfg, layers, np.concatenate(xs),
                         seqs_from([0] * 3, [c + 1 for c in ctx], bt), kv2)
    ends = np.cumsum([c + 1 for c in ctx]) - 1
    assert rel_l2(yd, yp[ends]) < 1e-12
    for l in range(2):
        for t in ("k", "v"):
            np.testing.assert_allclose(kv[l][t], kv2[l][t], rtol=1e-12, atol=1e-13)


def test_causal_prefix_invariance_bitwise():
    shape = SMALL
    n, p = 40, 23
    cfg, layers, bt, nb = _setup(shape, 15, [0], [n + 8], n_layers=2)
    x = synth.hidden_states(15, 5, n, shape.hidden, np.float64)
    y = O.stage_forward(cfg, layers, x, seqs_from([0], [n], bt), O.new_kv_cache(cfg, 2, nb))
    x2 = x.copy()
    x2[p:] = synth.hidden_states(15, 6, n - p, shape.hidden, np.float64)
    x3 = np.concatenate([x, synth.hidden_states(15, 7, 8, shape.hidden, np.float64)])
    y2 = O.stage_forward(cfg, layers, x2, seqs_from([0], [n], bt), O.new_kv_cache(cfg, 2, nb))
    y3 = O.stage_forward(cfg, layers, x3, seqs_from([0], [n + 8], bt), O.new_kv_cache(cfg, 2, nb))
    np.testing.assert_array_equal(y2[:p], y[:p])
    assert np.abs(y2[p:] - y[p:]).max() > 1e-3
    np.testing.assert_array_equal(y3[:n], y)


def test_zero_output_projections_give_identity_bitwise():
    shape = SMALL_QK
    cfg, layers, bt, nb = _setup(shape, 16, [0, 0], [7, 19], n_layers=2)
    for w in layers:
        w["w_o"][:] = 0.0
        w["w_down"][:] = 0.0
    x = synth.hidden_states(16, 8, 26, shape.hidden, np.float64)
    y = O.stage_forward(cfg, layers, x, seqs_from([0, 0], [7, 19], bt), O.new_kv_cache(cfg, 2, nb))
    np.testing.assert_array_equal(y, x)


def test_zero_gate_kills_ffn_branch():
    shape = SMALL
    cfg, layers, bt, nb = _setup(shape, 17, [0], [12], n_layers=1)
    x = synth.hidden_states(17, 9, 12, shape.hidden, np.float64)
    w = layers[0]
    ref = O.stage_forward(cfg, [dict(w, w_down=np.zeros_like(w["w_down"]))], x,
                          seqs_from([0], [12], bt), O.new_kv_cache(cfg, 1, nb))
    wg = dict(w, w_gate_up=w["w_gate_up"].copy())
    wg["w_gate_up"][: shape.ffn] = 0.0
    y = O.stage_forward(cfg, [wg], x, seqs_from([0], [12], bt), O.new_kv_cache(cfg, 1, nb))
    np.testing.assert_array_equal(y, ref)


def test_stage_composition_bitwise():
    shape = SMALL_QK
    ctx, ql = [0, 0], [30, 17]
    cfg, layers, bt, nb = _setup(shape, 18, ctx, ql, n_layers=3)
    x = synth.hidden_states(18, 11, 47, shape.hidden, np.float64)
    kv_a = O.new_kv_cache(cfg, 3, nb)
    y = O.stage_forward(cfg, layers, x, seqs_from(ctx, ql, bt), kv_a)
    kv_b = O.new_kv_cache(cfg, 3, nb)
    mid = O.stage_forward(cfg, layers[:2], x, seqs_from(ctx, ql, bt), kv_b[:2])
    y2 = O.stage_forward(cfg, layers[2:], mid, seqs_from(ctx, ql, bt), kv_b[2:])
    np.testing.assert_array_equal(y2, y)


def test_batch_permutation_invariance_bitwise():
    shape = SMALL
    ctx, ql = [0, 0, 0], [5, 21, 13]
    cfg, layers, bt, nb = _setup(shape, 19, ctx, ql, n_layers=2)
    x = synth.hidden_states(19, 12, 39, shape.hidden, np.float64)
    y = O.stage_forward(cfg, layers, x, seqs_from(ctx, ql, bt), O.new_kv_cache(cfg, 2, nb))
    order = [2, 0, 1]
    starts = np.concatenate([[0], np.cumsum(ql)])
    xp = np.concatenate([x[starts[i]:starts[i + 1]] for i in order])
    yp = O.stage_forward(cfg, layers, xp, seqs_from([ctx[i] for i in order], [ql[i] for i in order],
                                                    bt[order]), O.new_kv_cache(cfg, 2, nb))
    yb = np.concatenate([y[starts[i]:starts[i + 1]] for i in order])
    np.testing.assert_array_equal(yp, yb)
    # a sequence alone gives the same rows as inside the batch
    y1 = O.stage_forward(cfg, layers, x[5:26], seqs_from([0], [21], bt[1:2]), O.new_kv_cache(cfg, 2, nb))
    np.testing.assert_array_equal(y1, y[5:26])


def test_float32_oracle_close_to_float64():
    shape = synth.TINY
    cfg = ocfg(shape)
    ql = [20, 33]
    alloc = synth.BlockAllocator(12, 20)
    bt = synth.make_block_tables(ql, 4, alloc)
    layers = [synth.host_layer_weights(shape, 20, l) for l in range(2)]
    x = synth.hidden_states(20, 13, 53, shape.hidden)
    y64 = O.stage_forward(cfg, layers, x, seqs_from([0, 0], ql, bt), O.new_kv_cache(cfg, 2, 12))
    y32 = O.stage_forward(cfg, layers, x, seqs_from([0, 0], ql, bt),
                          O.new_kv_cache(cfg, 2, 12, np.float32), dtype=np.float32)
    assert y32.dtype == np.float32
    assert rel_l2(y32, y64) < 1e-6


def test_round_to_bf16_matches_torch_and_the_bf16_grid():
    r = np.random.default_rng(21)
    a = np.concatenate([r.standard_normal(5000) * 10.0 ** r.integers(-6, 6, 5000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.0078125, 3.0e38, -2.5e-39]])
    ref = torch.tensor(a, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.round_to_bf16(a), ref)
    # ties go to even: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7
    assert O.round_to_bf16(np.array([1.0 + 2.0 ** -8]))[0] == 1.0
    assert O.round_to_bf16(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6


def test_bf16_emulation_stays_close_and_default_is_exact():
    shape = SMALL_QK
    cfg, layers, bt, nb = _setup(shape, 22, [0], [30], n_layers=2)
    x = synth.hidden_states(22, 1, 30, shape.hidden, np.float64)
    y = O.stage_forward(cfg, layers, x, seqs_from([0], [30], bt), O.new_kv_cache(cfg, 2, nb))
    y0 = O.stage_forward(cfg, layers, x, seqs_from([0], [30], bt), O.new_kv_cache(cfg, 2, nb),
                         rounding=None)
    np.testing.assert_array_equal(y, y0)
    ye = O.stage_forward(cfg, layers, x, seqs_from([0], [30], bt), O.new_kv_cache(cfg, 2, nb),
                         rounding=O.round_to_bf16)
    e = rel_l2(ye, y)
    assert 1e-4 < e < 2e-2


# --------------------------------------------------------------------------
# LM head of the last stage: final RMSNorm + vocabulary projection
# --------------------------------------------------------------------------

def test_lm_head_hand_example():
    """H = 2, x = (3, 4): rms = sqrt(12.5); gain (1, 2); three vocabulary
    rows (1, 0), (0, 1), (1, 1)."""
    cfg = O.OracleConfig(hidden=2, n_q_heads=1, n_kv_heads=1, head_dim=2, ffn=2, rms_eps=0.0,
                         rope_theta=1e4)
    r = np.sqrt(12.5)
    y = O.lm_head(cfg, np.array([[3.0, 4.0]]), np.array([1.0, 2.0]),
                  np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0]]))
    np.testing.assert_allclose(y, [[3 / r, 8 / r, 11 / r]], rtol=1e-15)


def test_lm_head_constant_row_gives_row_sums_of_scaled_weight():
    """A constant row normalises to all ones (eps = 0), so logits = W g,
    whatever the constant; and the logits do not depend on the row's scale."""
    rng = np.random.default_rng(5)
    H, V = 64, 40
    cfg = O.OracleConfig(hidden=H, n_q_heads=1, n_kv_heads=1, head_dim=64, ffn=64, rms_eps=0.0,
                         rope_theta=1e4)
    g = rng.uniform(0.5, 1.5, H)
    w = rng.standard_normal((V, H))
    for c in (-3.0, 0.25, 7.0):
        y = O.lm_head(cfg, np.full((1, H), c), g, w)
        np.testing.assert_allclose(y[0], np.sign(c) * (w @ g), rtol=1e-12)
    x = rng.standard_normal((3, H))
    np.testing.assert_allclose(O.lm_head(cfg, 5.0 * x, g, w), O.lm_head(cfg, x, g, w), rtol=1e-12)


def test_lm_head_matches_transformers_norm_and_linear():
    """transformers' Llama final norm and LM head (random init, float64 weights;
    its RMSNorm computes in float32 internally, so agreement is ~1e-7 while a
    wiring error is O(1))."""
    from transformers.models.llama.modeling_llama import LlamaRMSNorm
    rng = np.random.default_rng(6)
    H, V, n = 96, 200, 5
    cfg = O.OracleConfig(hidden=H, n_q_heads=1, n_kv_heads=1, head_dim=96, ffn=96, rms_eps=1e-5,
                         rope_theta=1e4)
    g = rng.uniform(0.5, 1.5, H)
    w = rng.standard_normal((V, H)) / np.sqrt(H)
    x = rng.standard_normal((n, H))
    norm = LlamaRMSNorm(H, eps=1e-5).double()
    head = torch.nn.Linear(H, V, bias=False).double()
    with torch.no_grad():
        norm.weight.copy_(torch.tensor(g))
        head.weight.copy_(torch.tensor(w))
        ref = head(norm(torch.tensor(x))).numpy()
    assert rel_l2(O.lm_head(cfg, x, g, w), ref) < 1e-6
