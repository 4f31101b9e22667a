"""Pins of the CPU oracle against closed forms, library routines, invariants and brute force.

The paper prints no worked numerical example for the rollout, so every pin
here is a textbook value, a special case with a closed form, an invariant the
method must satisfy, or a brute-force enumeration on tiny inputs.  Each test
names the kind of mistake in the oracle that it would expose.
"""
import cmath
import dataclasses
import itertools
import math

import numpy as np
import pytest

import oracle as O
from paper_2609_38795_amd import workloads as W


def tiny_shape(**kw):
    base = dict(n_layers=2, d_model=16, n_heads=4, n_kv_heads=2, head_dim=4, d_ffn=24, vocab=11,
                rms_eps=1e-6, rope_base=10000.0, dtype="f32", feat_layers=(0, 1))
    base.update(kw)
    return W.ModelShape(**base)


def f64_weights(shape, seed, scale=0.3, gain="random"):
    w = W.random_weights(shape, seed, norm_gain=gain, scale=scale)
    return w


# ---------------------------------------------------------------- bf16 rounding
def test_bf16_round_hand_values():
    # 1 + 2^-8 is exactly half-way between 1 and 1 + 2^-7: ties to the even mantissa (1.0).
    # 1 + 3*2^-8 is half-way between 1 + 2^-7 (odd) and 1 + 2^-6 (even): goes to 1 + 2^-6.
    cases = {1.0: 1.0, 1 + 2 ** -8: 1.0, 1 + 3 * 2 ** -8: 1 + 2 ** -6,
             1 + 2 ** -8 + 2 ** -20: 1 + 2 ** -7, -(1 + 3 * 2 ** -8): -(1 + 2 ** -6),
             math.pi: 3.140625, 0.0: 0.0, 65504.0: 65536.0}
    for dt in (np.float64, np.float32):
        x = np.array(list(cases), dtype=dt)
        y = O.bf16_round(x)
        assert y.dtype == dt
        np.testing.assert_array_equal(y, np.array(list(cases.values()), dtype=dt))


def test_bf16_round_matches_torch_library():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    x32 = (rng.standard_normal(200000) * np.exp(rng.uniform(-20, 20, 200000))).astype(np.float32)
    ref = torch.from_numpy(x32).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(O.bf16_round(x32), ref)
    # float32-exact values: the direct float64 rounding equals the float32 one
    np.testing.assert_array_equal(O.bf16_round(x32.astype(np.float64)), ref.astype(np.float64))


# ---------------------------------------------------------------- RMSNorm / SiLU / softmax
def test_rmsnorm_hand_values():
    x = np.array([[1.0, 2.0, 3.0, 4.0]])
    # mean of squares = 30/4 = 7.5
    np.testing.assert_allclose(O.rmsnorm(x, np.ones(4), 0.0),
                               [[1 / math.sqrt(7.5), 2 / math.sqrt(7.5), 3 / math.sqrt(7.5),
                                 4 / math.sqrt(7.5)]], rtol=1e-15)
    # eps sits inside the root: sqrt(7.5 + 0.5) = sqrt(8); the gain multiplies afterwards
    g = np.array([2.0, 1.0, 1.0, 0.5])
    np.testing.assert_allclose(O.rmsnorm(x, g, 0.5),
                               [[2 / math.sqrt(8), 2 / math.sqrt(8), 3 / math.sqrt(8),
                                 2 / math.sqrt(8)]], rtol=1e-15)


def test_silu_hand_values():
    np.testing.assert_allclose(O.silu(np.array([0.0, 1.0, -1.0, 30.0])),
                               [0.0, 1 / (1 + math.e ** -1), -1 / (1 + math.e), 30.0], rtol=1e-12)


def test_log_softmax_values():
    lp = O.log_softmax(np.array([[0.0, math.log(3.0)]]))
    np.testing.assert_allclose(lp, [[math.log(0.25), math.log(0.75)]], rtol=1e-14)
    z = np.random.default_rng(1).standard_normal((7, 1000)) * 8
    lp = O.log_softmax(z)
    np.testing.assert_allclose(np.exp(lp).sum(-1), 1.0, atol=1e-12)
    np.testing.assert_allclose(O.log_softmax(np.zeros((1, 64))), -math.log(64), rtol=1e-15)
    np.testing.assert_allclose(O.log_softmax(z + 123.0), lp, atol=1e-12)  # shift invariance


def test_greedy_ties_go_to_lower_id():
    assert int(O.greedy_argmax(np.array([1.0, 3.0, 3.0, 2.0]))) == 1
    z = np.zeros(10)
    assert int(O.greedy_argmax(z)) == 0
    z[[7, 9]] = 5.0
    assert int(O.greedy_argmax(z)) == 7


# ---------------------------------------------------------------- RoPE
def test_rope_matches_complex_rotation_hand_case():
    # head_dim 4, base 100: theta_0 = 1, theta_1 = 100^(-1/2) = 0.1; rotate-half pairs (0,2), (1,3)
    x = np.array([[[1.0, 2.0, 3.0, 4.0]]])
    y = O.rope(x, np.array([2]), 100.0)[0, 0]
    z0 = complex(1, 3) * cmath.exp(2j * 1.0)
    z1 = complex(2, 4) * cmath.exp(2j * 0.1)
    np.testing.assert_allclose(y, [z0.real, z1.real, z0.imag, z1.imag], rtol=1e-14)


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((5, 3, 16))
    k = rng.standard_normal((5, 3, 16))
    np.testing.assert_allclose(O.rope(q, np.zeros(5), 1e4), q, rtol=0, atol=0)
    pos = np.array([0, 7, 100, 4095, 8191])
    rq = O.rope(q, pos, 5e5)
    np.testing.assert_allclose(np.linalg.norm(rq, axis=-1), np.linalg.norm(q, axis=-1), rtol=1e-13)
    # <R(p) q, R(p') k> depends only on p - p'
    a = np.einsum("thd,thd->th", O.rope(q, pos, 1e4), O.rope(k, pos + 3, 1e4))
    b = np.einsum("thd,thd->th", O.rope(q, pos + 50, 1e4), O.rope(k, pos + 53, 1e4))
    np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-11)


# ---------------------------------------------------------------- attention
def _scalar_attention(q, k, v):
    """Brute-force causal GQA attention with explicit loops (tiny inputs only)."""
    T, H, hd = q.shape
    G = k.shape[1]
    out = np.zeros_like(q)
    for t in range(T):
        for j in range(H):
            g = j // (H // G)
            sc = [sum(q[t, j, c] * k[u, g, c] for c in range(hd)) / math.sqrt(hd) for u in range(t + 1)]
            m = max(sc)
            e = [math.exp(s - m) for s in sc]
            tot = sum(e)
            for c in range(hd):
                out[t, j, c] = sum(e[u] / tot * v[u, g, c] for u in range(t + 1))
    return out


def test_attention_brute_force_gqa():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((6, 4, 3))
    k = rng.standard_normal((6, 2, 3))
    v = rng.standard_normal((6, 2, 3))
    np.testing.assert_allclose(O.causal_gqa_attention(q, k, v), _scalar_attention(q, k, v), rtol=1e-12)


def test_attention_hand_case_scale_and_mask():
    # hd = 4 -> scale 1/2.  Position 0 sees only itself; position 1 has scores [2*1/2, 0] = [1, 0].
    q = np.zeros((2, 1, 4)); k = np.zeros((2, 1, 4)); v = np.zeros((2, 1, 4))
    q[1, 0, 0] = 2.0; k[0, 0, 0] = 1.0
    v[0, 0] = [1, 2, 3, 4]; v[1, 0] = [5, 6, 7, 8]
    out = O.causal_gqa_attention(q, k, v)
    p0 = math.e / (math.e + 1)
    np.testing.assert_allclose(out[0, 0], [1, 2, 3, 4], rtol=1e-15)
    np.testing.assert_allclose(out[1, 0], p0 * np.array([1, 2, 3, 4]) + (1 - p0) * np.array([5, 6, 7, 8]),
                               rtol=1e-14)


def test_attention_rounded_probabilities_hand_case():
    """round_probs rounds exp(s - max) where it weights the values; the normaliser keeps
    the exact sum.  Position 1: scores [1, 0] -> p = [1, e^-1]; bf16(e^-1) = 188/512."""
    q = np.zeros((2, 1, 4)); k = np.zeros((2, 1, 4)); v = np.zeros((2, 1, 4))
    q[1, 0, 0] = 2.0; k[0, 0, 0] = 1.0
    v[0, 0] = [1, 2, 3, 4]; v[1, 0] = [5, 6, 7, 8]
    out = O.causal_gqa_attention(q, k, v, round_probs=O.bf16_round)
    e1 = math.exp(-1.0)
    want = (np.array([1, 2, 3, 4]) + (188 / 512) * np.array([5, 6, 7, 8])) / (1 + e1)
    np.testing.assert_allclose(out[1, 0], want, rtol=1e-14)
    np.testing.assert_allclose(out[0, 0], [1, 2, 3, 4], rtol=1e-15)
    # probabilities that bf16 holds exactly (equal scores: all ones) are unchanged
    rng = np.random.default_rng(5)
    vv = rng.standard_normal((7, 2, 5))
    kk = rng.standard_normal((7, 2, 5))
    np.testing.assert_allclose(
        O.causal_gqa_attention(np.zeros((7, 4, 5)), kk, vv, round_probs=O.bf16_round),
        O.causal_gqa_attention(np.zeros((7, 4, 5)), kk, vv), rtol=1e-14, atol=1e-15)


def test_attention_uniform_is_running_mean():
    rng = np.random.default_rng(4)
    v = rng.standard_normal((9, 2, 5))
    out = O.causal_gqa_attention(np.zeros((9, 4, 5)), rng.standard_normal((9, 2, 5)), v)
    cm = np.cumsum(v, 0) / np.arange(1, 10)[:, None, None]
    np.testing.assert_allclose(out, np.repeat(cm, 2, axis=1), rtol=1e-12)


def test_attention_matches_torch_sdpa():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(6)
    T, H, G, hd = 37, 8, 2, 16
    q, k, v = (rng.standard_normal((T, n, hd)) for n in (H, G, G))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).permute(1, 0, 2),
        torch.from_numpy(np.repeat(k, H // G, axis=1)).permute(1, 0, 2),
        torch.from_numpy(np.repeat(v, H // G, axis=1)).permute(1, 0, 2), is_causal=True)
    np.testing.assert_allclose(O.causal_gqa_attention(q, k, v), ref.permute(1, 0, 2).numpy(),
                               rtol=1e-10, atol=1e-12)


def test_attention_query_positions_select_rows():
    """q_pos places a subset of query rows among the keys: each row equals the full causal
    attention's row at that position (the scalar brute force decides both)."""
    rng = np.random.default_rng(8)
    q = rng.standard_normal((9, 4, 3))
    k = rng.standard_normal((9, 2, 3))
    v = rng.standard_normal((9, 2, 3))
    rows = np.array([0, 4, 8])
    ref = _scalar_attention(q, k, v)[rows]
    np.testing.assert_allclose(O.causal_gqa_attention(q[rows], k, v, q_pos=rows), ref, rtol=1e-12)
    # a query at position 4 ignores keys 5..8 entirely
    k2 = k.copy(); k2[5:] = 1e3 * rng.standard_normal(k2[5:].shape)
    np.testing.assert_allclose(O.causal_gqa_attention(q[[4]], k2, v, q_pos=[4]), ref[[1]],
                               rtol=1e-12)


@pytest.mark.parametrize("sections", [None, (1, 0, 1)])
@pytest.mark.parametrize("emulate", [False, True])
def test_layer_at_rows_equals_full_forward(sections, emulate):
    """One decoder layer evaluated at chosen rows equals that layer of the full forward at
    those rows (any slip in the restriction -- a query from the wrong row, keys past the row,
    a residual from another row -- fails it).  Layer 1's input is layer 0's output."""
    shape = tiny_shape(n_layers=2, head_dim=4, mrope_sections=sections or (0, 0, 0))
    w = f64_weights(shape, 21)
    P = O.Params(w)
    T = 13
    toks = W.random_tokens(shape.vocab, (1, T), 5)[0]
    x0 = O.embed_rows(P, toks)
    pos = np.arange(T) if sections is None else np.stack(
        [np.arange(T), np.arange(T) // 3, np.arange(T) % 3 + 2], axis=1)
    for probs in ([False, True] if emulate else [False]):
        outs, _ = O.decoder_forward(P, shape, x0, pos, emulate_bf16=emulate, bf16_probs=probs)
        for layer, x in ((0, x0), (1, outs[0])):
            for rows in ([T - 1], [0, 5, 6, 12], list(range(T))):
                got = O.decoder_layer_at(P, shape, layer, x, pos, rows, emulate_bf16=emulate,
                                         bf16_probs=probs)
                np.testing.assert_allclose(got, outs[layer][rows], rtol=1e-12, atol=1e-12)
    # rows past the last asked-for one do not matter
    x_mod = x0.copy()
    x_mod[7:] += 5.0
    np.testing.assert_allclose(O.decoder_layer_at(P, shape, 0, x_mod, pos, [2, 6]),
                               O.decoder_layer_at(P, shape, 0, x0, pos, [2, 6]), rtol=0, atol=0)


# ---------------------------------------------------------------- decoder layer closed forms
def _hand_model():
    """d=2, one head of dim 2, F=1, V=3: every layer output computable by hand at T=1."""
    shape = W.ModelShape(1, 2, 1, 1, 2, 1, 3, 0.0, 10000.0, "f32", (0,))
    w = {
        "tok_embed": np.array([[3.0, 4.0], [1.0, -1.0], [0.5, 2.0]], np.float32),
        "lm_head": np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0]], np.float32),
        "final_norm": np.array([1.0, 2.0], np.float32),
        "dtype": "f32",
        "layers": [{
            "attn_norm": np.array([1.0, 0.5], np.float32),
            "ffn_norm": np.array([2.0, 1.0], np.float32),
            "wq": np.array([[0.3, 0.1], [0.2, -0.4]], np.float32),
            "wk": np.array([[0.5, 0.25], [-0.5, 1.0]], np.float32),
            "wv": np.array([[1.0, 2.0], [0.0, 1.0]], np.float32),   # not symmetric
            "wo": np.array([[0.0, 1.0], [0.5, 0.0]], np.float32),   # not symmetric
            "w_gate": np.array([[1.0, 0.0]], np.float32),
            "w_up": np.array([[0.0, 1.0]], np.float32),
            "w_down": np.array([[1.0], [-2.0]], np.float32),
        }],
    }
    return shape, w


def test_decoder_single_position_closed_form():
    """At one position the softmax has one key: attention output = v.  Catches transposes,
    a swapped gate/up, a missing residual and a misplaced norm gain."""
    shape, w = _hand_model()
    P = O.Params(w)
    x = np.array([3.0, 4.0])  # token 0
    r1 = math.sqrt((9 + 16) / 2)               # rms of x = 5/sqrt(2)
    n1 = np.array([3 / r1 * 1.0, 4 / r1 * 0.5])
    v = np.array([n1[0] + 2 * n1[1], n1[1]])   # Wv n1
    h = x + np.array([v[1], 0.5 * v[0]])       # + Wo v
    r2 = math.sqrt((h[0] ** 2 + h[1] ** 2) / 2)
    n2 = np.array([h[0] / r2 * 2.0, h[1] / r2 * 1.0])
    act = n2[0] / (1 + math.exp(-n2[0])) * n2[1]   # silu(gate) * up
    h = h + np.array([act, -2 * act])
    rf = math.sqrt((h[0] ** 2 + h[1] ** 2) / 2)
    hf = np.array([h[0] / rf * 1.0, h[1] / rf * 2.0])
    z = np.array([hf[0], hf[1], hf[0] + hf[1]])
    outs, hf_o = O.decoder_forward(P, shape, x[None, :], np.array([0]))
    np.testing.assert_allclose(outs[0][0], h, rtol=1e-14)
    np.testing.assert_allclose(hf_o[0], hf, rtol=1e-14)
    np.testing.assert_allclose(O.head_logits(P, hf_o)[0], z, rtol=1e-14)


def test_decoder_two_positions_uniform_attention():
    """Wq = 0: position 1 averages v_0, v_1; position 0 sees only v_0 (causal mask)."""
    shape, w = _hand_model()
    w["layers"][0]["wq"] = np.zeros((2, 2), np.float32)
    w["layers"][0]["w_down"] = np.zeros((2, 1), np.float32)
    P = O.Params(w)
    x = np.array([[3.0, 4.0], [1.0, -1.0]])
    g = np.array([1.0, 0.5])
    n1 = x / np.sqrt((x ** 2).mean(1, keepdims=True)) * g
    v = n1 @ np.array([[1.0, 2.0], [0.0, 1.0]]).T
    o = np.stack([v[0], (v[0] + v[1]) / 2])
    expect = x + o @ np.array([[0.0, 1.0], [0.5, 0.0]]).T
    outs, _ = O.decoder_forward(P, shape, x, np.arange(2))
    np.testing.assert_allclose(outs[0], expect, rtol=1e-14)


def test_feature_is_output_of_layer():
    """feat_layers index decoder layers (0-based) by their *output* residual stream."""
    shape = tiny_shape(n_layers=2, feat_layers=(0, 1))
    w = f64_weights(shape, 11)
    w["layers"][1]["wo"][:] = 0
    w["layers"][1]["w_down"][:] = 0  # layer 1 is the identity map
    P = O.Params(w)
    toks = W.random_tokens(shape.vocab, (1, 9), 1)
    feats, _ = O.prefill_outputs(P, shape, toks[0])
    np.testing.assert_array_equal(feats[:, 0], feats[:, 1])
    x0 = O.embed_rows(P, toks[0])
    assert np.abs(feats[:, 0] - x0).max() > 1e-3  # layer 0's output is not its input
    w["layers"][0]["wo"][:] = 0
    w["layers"][0]["w_down"][:] = 0
    feats, _ = O.prefill_outputs(O.Params(w), shape, toks[0])
    np.testing.assert_allclose(feats[:, 0], x0, rtol=0, atol=0)


def test_gqa_equals_mha_with_duplicated_kv_heads():
    shape = tiny_shape(n_heads=4, n_kv_heads=2)
    w = f64_weights(shape, 12)
    mha = dataclasses.replace(shape, n_kv_heads=4)
    w2 = {**w, "layers": [dict(ld) for ld in w["layers"]]}
    for ld in w2["layers"]:
        for n in ("wk", "wv"):
            blocks = ld[n].reshape(2, shape.head_dim, shape.d_model)
            ld[n] = np.repeat(blocks, 2, axis=0).reshape(4 * shape.head_dim, shape.d_model)
    toks = W.random_tokens(shape.vocab, (1, 12), 2)
    f1, z1 = O.prefill_outputs(O.Params(w), shape, toks[0])
    f2, z2 = O.prefill_outputs(O.Params(w2), mha, toks[0])
    np.testing.assert_allclose(f1, f2, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(z1, z2, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------- whole-model closed forms
def test_zero_layer_model_is_iterated_map():
    """n_layers = 0: slot s+1's input is the greedy token of slot s, through norm -> head only."""
    shape = tiny_shape(n_layers=0, feat_layers=(), vocab=13, d_model=6)
    w = f64_weights(shape, 13, scale=1.0)
    P = O.Params(w)
    E = w["tok_embed"].astype(np.float64)
    Wl = w["lm_head"].astype(np.float64)
    g = w["final_norm"].astype(np.float64)

    def step(t):
        r = math.sqrt(sum(e * e for e in E[t]) / 6 + shape.rms_eps)
        hf = [E[t][c] / r * g[c] for c in range(6)]
        z = [sum(Wl[v][c] * hf[c] for c in range(6)) for v in range(13)]
        m = max(z)
        lse = m + math.log(sum(math.exp(q - m) for q in z))
        best = min(v for v in range(13) if z[v] == m)
        return best, [q - lse for q in z]

    toks = W.random_tokens(shape.vocab, (1, 20), 3)
    a_seq, a_pos = np.zeros(3, np.int32), np.array([0, 5, 19], np.int32)
    tk, lp, ft = O.rollout_naive(P, shape, toks, a_seq, a_pos, 6)
    for i, a in enumerate(a_pos):
        t = int(toks[0, a])
        for s in range(6):
            best, lps = step(t)
            assert tk[i, s] == best
            np.testing.assert_allclose(lp[i, s], lps, rtol=1e-12, atol=1e-12)
            t = best


def test_residual_only_model_reduces_to_zero_layer_map():
    """Wo = Wd = 0 in every layer: the residual stream keeps the input row."""
    shape = tiny_shape()
    w = f64_weights(shape, 14, scale=1.0)
    for ld in w["layers"]:
        ld["wo"][:] = 0
        ld["w_down"][:] = 0
    P = O.Params(w)
    toks = W.random_tokens(shape.vocab, (1, 10), 4)
    feats, z = O.prefill_outputs(P, shape, toks[0])
    x0 = O.embed_rows(P, toks[0])
    np.testing.assert_array_equal(feats[:, 0], x0)
    hf = O.rmsnorm(x0, P.get("final_norm"), shape.rms_eps)
    np.testing.assert_allclose(z, hf @ P.get("lm_head").T, rtol=1e-13)


def test_value_free_model_output_depends_on_token_only():
    """Wv = 0: attention contributes nothing, so a slot's output is a function of its input token."""
    shape = tiny_shape(vocab=7)
    w = f64_weights(shape, 15, scale=0.8)
    for ld in w["layers"]:
        ld["wv"][:] = 0
    P = O.Params(w)
    toks = W.random_tokens(shape.vocab, (1, 40), 5)
    feats, z = O.prefill_outputs(P, shape, toks[0])
    by_tok = {}
    for p, t in enumerate(toks[0]):
        by_tok.setdefault(int(t), p)
    a_seq, a_pos = np.zeros(4, np.int32), np.array([3, 10, 22, 39], np.int32)
    tk, lp, ft = O.rollout_naive(P, shape, toks, a_seq, a_pos, 5)
    for i, a in enumerate(a_pos):
        inp = int(toks[0, a])
        for s in range(5):
            if inp in by_tok:
                p = by_tok[inp]
                np.testing.assert_allclose(lp[i, s], O.log_softmax(z[p]), rtol=1e-12, atol=1e-12)
                np.testing.assert_allclose(ft[i, s], feats[p], rtol=1e-12, atol=1e-13)
            inp = int(tk[i, s])


# ---------------------------------------------------------------- rollout invariants
@pytest.fixture(scope="module")
def small_case():
    shape = tiny_shape(n_layers=2, d_model=16, vocab=23)
    w = f64_weights(shape, 21, scale=0.4)
    toks = W.random_tokens(shape.vocab, (2, 30), 6)
    a_seq = np.array([0, 1, 0, 1, 1, 0], np.int32)
    a_pos = np.array([4, 0, 29, 17, 9, 12], np.int32)
    return shape, O.Params(w), toks, a_seq, a_pos


def test_slot0_equals_prefill_at_anchor(small_case):
    shape, P, toks, a_seq, a_pos = small_case
    tk, lp, ft = O.rollout_naive(P, shape, toks, a_seq, a_pos, 4)
    for sq in (0, 1):
        feats, z = O.prefill_outputs(P, shape, toks[sq])
        for i in np.nonzero(a_seq == sq)[0]:
            a = a_pos[i]
            np.testing.assert_allclose(lp[i, 0], O.log_softmax(z[a]), rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(ft[i, 0], feats[a], rtol=1e-12, atol=1e-13)
            assert tk[i, 0] == int(np.argmax(z[a]))


def test_naive_equals_teacher_forced_and_kv_shared(small_case):
    shape, P, toks, a_seq, a_pos = small_case
    tk, lp, ft = O.rollout_naive(P, shape, toks, a_seq, a_pos, 5)
    tk2, lp2, ft2, margin = O.rollout_teacher_forced(P, shape, toks, a_seq, a_pos, 5, tk)
    np.testing.assert_array_equal(tk, tk2)
    np.testing.assert_allclose(lp, lp2, rtol=0, atol=1e-12)
    np.testing.assert_allclose(ft, ft2, rtol=0, atol=1e-12)
    assert (margin >= 0).all()
    tk3, lp3, ft3 = O.rollout_kv_shared(P, shape, toks, a_seq, a_pos, 5)
    np.testing.assert_array_equal(tk, tk3)
    np.testing.assert_allclose(lp, lp3, rtol=0, atol=1e-12)
    np.testing.assert_allclose(ft, ft3, rtol=0, atol=1e-12)


def test_batched_equals_sequential_and_permutation(small_case):
    shape, P, toks, a_seq, a_pos = small_case
    tk, lp, ft = O.rollout_kv_shared(P, shape, toks, a_seq, a_pos, 4)
    for i in range(len(a_seq)):
        t1, l1, f1 = O.rollout_kv_shared(P, shape, toks, a_seq[i:i + 1], a_pos[i:i + 1], 4)
        np.testing.assert_array_equal(t1[0], tk[i])
        np.testing.assert_allclose(l1[0], lp[i], rtol=0, atol=1e-12)
        np.testing.assert_allclose(f1[0], ft[i], rtol=0, atol=1e-12)
    perm = np.array([3, 0, 5, 1, 4, 2])
    tp, lpp, fp = O.rollout_kv_shared(P, shape, toks, a_seq[perm], a_pos[perm], 4)
    np.testing.assert_array_equal(tp, tk[perm])
    np.testing.assert_allclose(lpp, lp[perm], rtol=0, atol=1e-12)


def test_forced_tokens_equal_teacher_forcing(small_case):
    shape, P, toks, a_seq, a_pos = small_case
    rng = np.random.default_rng(8)
    forced = rng.integers(-1, shape.vocab, size=(len(a_seq), 4))
    tk, lp, ft = O.rollout_naive(P, shape, toks, a_seq, a_pos, 4, forced=forced)
    feed = np.where(forced >= 0, forced, tk)
    tk2, lp2, ft2, _ = O.rollout_teacher_forced(P, shape, toks, a_seq, a_pos, 4, feed)
    np.testing.assert_array_equal(tk, tk2)
    np.testing.assert_allclose(lp, lp2, rtol=0, atol=1e-12)
    tk3, lp3, ft3 = O.rollout_kv_shared(P, shape, toks, a_seq, a_pos, 4, forced=forced)
    np.testing.assert_array_equal(tk, tk3)
    np.testing.assert_allclose(lp, lp3, rtol=0, atol=1e-12)


def test_causality_future_corpus_tokens_do_not_matter(small_case):
    shape, P, toks, a_seq, a_pos = small_case
    tk, lp, ft = O.rollout_naive(P, shape, toks, a_seq, a_pos, 3)
    t2 = toks.copy()
    for i in range(len(a_seq)):
        pass
    # perturb every token after the smallest anchor of each sequence
    rng = np.random.default_rng(9)
    for sq in (0, 1):
        amin = a_pos[a_seq == sq].min()
        t2[sq, amin + 1:] = rng.integers(0, shape.vocab, size=t2.shape[1] - amin - 1)
        sel = (a_seq == sq) & (a_pos == amin)
        tkb, lpb, ftb = O.rollout_naive(P, shape, t2, a_seq[sel], a_pos[sel], 3)
        np.testing.assert_array_equal(tkb, tk[sel])
        np.testing.assert_array_equal(lpb, lp[sel])


def test_self_consistent_corpus_reproduced_and_positions_continue():
    """A corpus written greedily by the oracle itself: every rollout must continue it, and
    slot s of anchor a must equal the prefill output at a+s (positions continue the anchor)."""
    shape = tiny_shape(n_layers=2, vocab=31)
    w = f64_weights(shape, 31, scale=0.5)
    P = O.Params(w)
    seq = list(W.random_tokens(shape.vocab, (5,), 7))
    while len(seq) < 26:
        _, z = O.prefill_outputs(P, shape, np.array(seq))
        seq.append(int(np.argmax(z[-1])))
    toks = np.array([seq], np.int32)
    feats, z = O.prefill_outputs(P, shape, toks[0])
    B = 4
    a_pos = np.array([4, 9, 15, 21], np.int32)
    a_seq = np.zeros(4, np.int32)
    tk, lp, ft = O.rollout_naive(P, shape, toks, a_seq, a_pos, B)
    for i, a in enumerate(a_pos):
        np.testing.assert_array_equal(tk[i], toks[0, a + 1:a + 1 + B])
        for s in range(B):
            np.testing.assert_allclose(lp[i, s], O.log_softmax(z[a + s]), rtol=0, atol=1e-12)
            np.testing.assert_allclose(ft[i, s], feats[a + s], rtol=0, atol=1e-12)


def test_brute_force_tiny_vocab_chain_rule():
    """V = 8, B = 3: every continuation's conditionals come from independent whole-sequence
    forwards; the rollout must follow their argmax chain and report their distributions."""
    shape = tiny_shape(n_layers=1, vocab=8, d_model=8, n_heads=2, n_kv_heads=1, head_dim=4,
                       d_ffn=12, feat_layers=(0,))
    w = f64_weights(shape, 41, scale=0.7)
    P = O.Params(w)
    toks = W.random_tokens(8, (1, 12), 8)
    a = 6
    tk, lp, ft = O.rollout_naive(P, shape, toks, np.zeros(1, np.int32), np.array([a], np.int32), 3)
    prefix = list(toks[0, :a + 1])
    cond = {}
    for depth in range(3):
        for cont in itertools.product(range(8), repeat=depth):
            _, z = O.prefill_outputs(P, shape, np.array(prefix + list(cont)))
            cond[cont] = O.log_softmax(z[-1])
    # chain rule: probabilities of all length-2 continuations sum to 1
    tot = sum(math.exp(cond[()][c1] + cond[(c1,)][c2]) for c1 in range(8) for c2 in range(8))
    assert abs(tot - 1.0) < 1e-12
    path = ()
    for s in range(3):
        np.testing.assert_allclose(lp[0, s], cond[path], rtol=0, atol=1e-12)
        assert tk[0, s] == int(np.argmax(cond[path]))
        path = path + (int(tk[0, s]),)


def test_given_rows_replace_embeddings():
    shape = tiny_shape()
    w = f64_weights(shape, 51)
    P = O.Params(w)
    toks = W.random_tokens(shape.vocab, (1, 10), 9)
    rows = np.random.default_rng(3).standard_normal((10, shape.d_model)).astype(np.float32)
    mask = np.zeros(10, np.uint8); mask[:4] = 1
    x = O.embed_rows(P, toks[0], rows, mask)
    np.testing.assert_array_equal(x[:4], rows[:4].astype(np.float64))
    np.testing.assert_array_equal(x[4:], w["tok_embed"][toks[0, 4:]].astype(np.float64))


def test_bf16_emulation_close_to_exact_and_rounds():
    shape = dataclasses.replace(tiny_shape(d_model=32, head_dim=8, d_ffn=48, vocab=50), dtype="bf16")
    w = W.random_weights(shape, 61, scale=0.2)
    P = O.Params(w)
    toks = W.random_tokens(shape.vocab, (1, 16), 10)
    x0 = O.embed_rows(P, toks[0])
    outs_e, hf_e = O.decoder_forward(P, shape, x0, np.arange(16), emulate_bf16=True)
    outs_x, hf_x = O.decoder_forward(P, shape, x0, np.arange(16), emulate_bf16=False)
    np.testing.assert_array_equal(O.bf16_round(hf_e), hf_e)  # final-norm output is bf16
    assert np.abs(hf_e - hf_x).max() <= 0.05 * np.abs(hf_x).max()  # a few bf16 ulps of the row scale
    assert np.abs(hf_e - hf_x).max() > 0
