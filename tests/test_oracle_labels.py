"""Pins of the label oracle (top-8 + tail, corpus labels and erase gates, in-rollout anchors).

The paper prints no worked numeric example of these products, so the pins are
hand-computed cases, properties the paper states for them (the gate is 1 at
slot 1 and never grows; on a greedy continuation the hard gate is 1 on every
active slot and the corpus labels equal the rollout labels; a secondary block
at offset j supervises K - j slots), and invariants of the definitions.  Each
test names the mistake it would expose.
"""
import math

import numpy as np
import pytest

import oracle as O
from oracle import labels as LB
from paper_2609_38795_amd import workloads as W


def _tiny_shape(**kw):
    base = dict(n_layers=2, d_model=16, n_heads=4, n_kv_heads=2, head_dim=4, d_ffn=24, vocab=31,
                rms_eps=1e-6, rope_base=10000.0, dtype="f32", feat_layers=(0, 1))
    base.update(kw)
    return W.ModelShape(**base)


# ---------------------------------------------------------------- top-8 + tail
def test_topk_hand_case_order_ties_and_tail():
    # probabilities over 12 tokens, written by hand; two pairs of exact ties
    p = np.array([0.02, 0.20, 0.05, 0.20, 0.01, 0.10, 0.10, 0.04, 0.03, 0.15, 0.06, 0.04])
    assert abs(p.sum() - 1.0) < 1e-15
    ids, vals, tail = LB.topk_tail(np.log(p), k=8)
    # descending probability; 0.20 at ids 1 and 3 -> 1 first; 0.10 at 5, 6 -> 5 first;
    # 0.04 at ids 7 and 11: only id 7 makes the top 8
    np.testing.assert_array_equal(ids, [1, 3, 9, 5, 6, 10, 2, 7])
    np.testing.assert_allclose(np.exp(vals), p[[1, 3, 9, 5, 6, 10, 2, 7]], rtol=1e-14)
    # tail = tokens 0 (0.02), 4 (0.01), 8 (0.03), 11 (0.04)
    assert abs(tail - 0.10) < 1e-14


def test_topk_invariants_random_rows():
    # a dropped term, wrong sort direction or a tail taken over the wrong set fails one of these
    rng = np.random.default_rng(3)
    z = rng.standard_normal((50, 200)) * 3
    z[:, 17] = z[:, 40]  # ties
    lp = O.log_softmax(z)
    ids, vals, tail = LB.topk_tail(lp)
    for r in range(50):
        assert len(set(ids[r])) == 8
        assert np.all(np.diff(vals[r]) <= 0)
        np.testing.assert_array_equal(vals[r], lp[r, ids[r]])
        rest = np.setdiff1d(np.arange(200), ids[r])
        assert lp[r, rest].max() <= vals[r, -1]
        assert abs(tail[r] + np.exp(vals[r]).sum() - 1.0) < 1e-12
        for a, b in zip(ids[r][:-1], ids[r][1:]):  # equal values keep increasing ids
            if lp[r, a] == lp[r, b]:
                assert a < b


def test_topk_first_entry_is_greedy_token():
    rng = np.random.default_rng(4)
    z = rng.integers(0, 4, size=(40, 30)).astype(np.float64)  # many exact ties
    ids, _, _ = LB.topk_tail(O.log_softmax(z))
    np.testing.assert_array_equal(ids[:, 0], O.greedy_argmax(z))


def test_topk_small_vocab_has_no_tail():
    lp = O.log_softmax(np.array([[0.3, -1.0, 2.0, 0.3, 0.0]]))
    ids, vals, tail = LB.topk_tail(lp, k=8)
    np.testing.assert_array_equal(ids[0], [2, 0, 3, 4, 1, -1, -1, -1])
    assert np.all(np.isneginf(vals[0, 5:]))
    assert tail[0] == 0.0


# ---------------------------------------------------------------- envelope
def test_slot_envelope_values():
    w = LB.slot_envelope(5, gamma=2.0)
    np.testing.assert_allclose(w, [1.0, math.exp(-0.5), math.exp(-1.0), math.exp(-1.5),
                                   math.exp(-2.0)], rtol=1e-15)
    np.testing.assert_allclose(LB.slot_envelope(4, gamma=0.5)[1], math.exp(-2.0), rtol=1e-15)


# ---------------------------------------------------------------- corpus labels and gates
def test_corpus_labels_hand_case():
    # L = 5 positions, V = 3, hand log-distributions; anchor 1, block 4
    P = np.array([[0.5, 0.25, 0.25],
                  [0.125, 0.5, 0.375],    # row 1 predicts position 2
                  [0.25, 0.25, 0.5],      # row 2 predicts position 3
                  [0.6, 0.3, 0.1],        # row 3 predicts position 4
                  [0.2, 0.2, 0.6]])
    toks = np.array([0, 2, 1, 0, 1])
    valid, lab, am, clp, gs, gh = LB.corpus_labels(np.log(P), toks, [1], 4)
    np.testing.assert_array_equal(valid[0], [True, True, True, True])
    np.testing.assert_allclose(np.exp(lab[0]), P[1:5], rtol=1e-15)
    np.testing.assert_array_equal(am[0], [1, 2, 0, 2])
    # corpus continuation: x2 = 1 under row 1 (0.5), x3 = 0 under row 2 (0.25),
    # x4 = 1 under row 3 (0.3); row 4 has no next token
    np.testing.assert_allclose(np.exp(clp[0, :3]), [0.5, 0.25, 0.3], rtol=1e-15)
    assert np.isnan(clp[0, 3])
    np.testing.assert_allclose(gs[0], [1.0, 0.5, 0.125, 0.0375], rtol=1e-14)
    # hard: x2 = argmax row 1 (1) -> 1; x3 = 0 vs argmax row 2 (2) -> 0 afterwards
    np.testing.assert_array_equal(gh[0], [1.0, 1.0, 0.0, 0.0])


def test_corpus_labels_end_of_sequence_and_given_rows():
    P = np.full((4, 2), 0.5)
    toks = np.array([0, 1, 0, 1])
    valid, lab, am, clp, gs, gh = LB.corpus_labels(np.log(P), toks, [2], 4)
    np.testing.assert_array_equal(valid[0], [True, True, False, False])
    assert np.isneginf(lab[0, 2:]).all() and (am[0, 2:] == -1).all()
    np.testing.assert_allclose(gs[0], [1.0, 0.5, 0.0, 0.0])
    # a given input row is not a corpus token: the factor that needs it is 0
    is_tok = np.array([True, True, True, False])
    _, _, _, clp2, gs2, gh2 = LB.corpus_labels(np.log(P), toks, [2], 2, is_token=is_tok)
    assert np.isnan(clp2[0, 0])
    np.testing.assert_array_equal(gs2[0], [1.0, 0.0])


def test_gates_start_at_one_and_never_grow():
    rng = np.random.default_rng(11)
    lp = O.log_softmax(rng.standard_normal((40, 7)) * 2)
    toks = rng.integers(0, 7, size=40)
    valid, _, _, _, gs, gh = LB.corpus_labels(lp, toks, [0, 5, 20, 33], 8)
    for i in range(4):
        v = valid[i]
        assert gs[i, 0] == 1.0 and gh[i, 0] == 1.0
        assert np.all(np.diff(gs[i, v]) <= 0) and np.all(np.diff(gh[i, v]) <= 0)
        assert np.all(gh[i, v] <= 1) and set(np.unique(gh[i])) <= {0.0, 1.0}


def test_greedy_corpus_hard_gate_is_one_and_kd_equals_rollout():
    """Sec. 3.2: on a greedy target continuation the hard gate is 1 on every active slot,
    and the corpus-conditioned labels coincide with the rollout's."""
    shape = _tiny_shape()
    P = O.Params(W.random_weights(shape, 31, norm_gain="random", scale=0.5))
    seq = list(W.random_tokens(shape.vocab, (5,), 7))
    while len(seq) < 24:
        _, z = O.prefill_outputs(P, shape, np.array(seq))
        seq.append(int(np.argmax(z[-1])))
    toks = np.array([seq], np.int32)
    _, z = O.prefill_outputs(P, shape, toks[0])
    lp = O.log_softmax(z)
    a_pos = np.array([4, 11, 17], np.int32)
    B = 5
    valid, lab, am, clp, gs, gh = LB.corpus_labels(lp, toks[0], a_pos, B)
    assert valid.all()
    np.testing.assert_array_equal(gh, 1.0)
    tk, lpr, _ = O.rollout_naive(P, shape, toks, np.zeros(3, np.int32), a_pos, B)
    np.testing.assert_allclose(lab, lpr, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(am, tk)
    # the soft gate is the product of the greedy tokens' probabilities
    for i, a in enumerate(a_pos):
        prod = 1.0
        for s in range(B):
            assert abs(gs[i, s] - prod) <= 1e-12 * max(1.0, prod)
            prod *= float(np.exp(lp[a + s, toks[0, a + s + 1]]))


def test_corpus_slot0_equals_rollout_slot0():
    """Sec. 3.2: the first draft slot's label is the same under corpus KD and ALR (both read
    the target at the anchor itself, before any rollout token)."""
    shape = _tiny_shape(vocab=19)
    P = O.Params(W.random_weights(shape, 5, norm_gain="random", scale=0.4))
    toks = W.random_tokens(shape.vocab, (1, 20), 3)
    _, z = O.prefill_outputs(P, shape, toks[0])
    a_pos = np.array([2, 9, 19], np.int32)
    valid, lab, am, _, _, _ = LB.corpus_labels(O.log_softmax(z), toks[0], a_pos, 3)
    tk, lpr, _ = O.rollout_naive(P, shape, toks, np.zeros(3, np.int32), a_pos, 3)
    np.testing.assert_allclose(lab[:, 0], lpr[:, 0], rtol=0, atol=1e-12)
    np.testing.assert_array_equal(am[:, 0], tk[:, 0])


# ---------------------------------------------------------------- in-rollout anchors
def test_ira_hand_case():
    # B = 5 -> K = 4; primary 0 tokens y*_1..y*_5 = 10..14; labels tagged by slot index
    tokens = np.array([[10, 11, 12, 13, 14], [20, 21, 22, 23, 24]])
    lab = np.arange(2 * 5).reshape(2, 5).astype(np.float64)  # label of primary p slot s = 5p+s
    t0, ls, w, shift = LB.ira_secondary(tokens, lab, primary=[1, 0], offset=[2, 3], gamma=2.0)
    # secondary 0: primary 1, j = 2: slot 0 token y*_2 = 21; slot k <- primary slot 2+k
    assert t0[0] == 21 and t0[1] == 12  # y*_2 of primary 1, y*_3 of primary 0
    np.testing.assert_array_equal(ls[0, :3], [7, 8, 9])
    assert np.all(np.isneginf(ls[0, 3:]))
    env = LB.slot_envelope(5)
    # weights: k with j + k <= K = 4 -> k = 1, 2 for j = 2; k = 1 for j = 3
    np.testing.assert_allclose(w[0], [env[0], env[1], 0, 0, 0])
    np.testing.assert_allclose(w[1], [env[0], 0, 0, 0, 0])
    np.testing.assert_array_equal(shift, [2, 3])


def test_ira_supervises_k_minus_j_slots_and_integer_labels():
    rng = np.random.default_rng(2)
    B = 16
    tokens = rng.integers(0, 100, size=(6, B))
    ids = rng.integers(0, 100, size=(6, B, 8))
    offs = np.array([2, 5, 9, 14, 3, 7])
    t0, li, w, _ = LB.ira_secondary(tokens, ids, primary=np.arange(6), offset=offs)
    for q, j in enumerate(offs):
        assert (w[q] > 0).sum() == (B - 1) - j
        assert t0[q] == tokens[q, j - 1]
        np.testing.assert_array_equal(li[q, :B - j], ids[q, j:])
        assert (li[q, B - j:] == -1).all()


# ---------------------------------------------------------------- multimodal RoPE
def test_mrope_with_equal_axes_is_plain_rope():
    rng = np.random.default_rng(31)
    x = rng.standard_normal((9, 3, 16))
    p = rng.integers(0, 500, size=9)
    plain = O.rope(x, p, 10000.0)
    for sec in [(2, 3, 3), (8, 0, 0), (0, 4, 4)]:
        np.testing.assert_allclose(O.rope(x, np.stack([p, p, p], 1), 10000.0, sec), plain,
                                   rtol=0, atol=1e-13)


def test_mrope_sections_select_axes_hand_case():
    # head_dim 8: frequencies 0..3, theta_i = base^(-2i/8); sections (1, 1, 2):
    # frequency 0 follows t, 1 follows h, 2 and 3 follow w
    base = 16.0
    theta = [base ** (-2 * i / 8) for i in range(4)]
    pos = np.array([[3, 5, 7]])
    for i, axis in enumerate([0, 1, 1 + 1, 2]):
        x = np.zeros((1, 1, 8))
        x[0, 0, i], x[0, 0, i + 4] = 1.0, 0.5  # the pair (i, i+4)
        y = O.rope(x, pos, base, (1, 1, 2))
        ang = pos[0, axis] * theta[i]
        np.testing.assert_allclose(y[0, 0, i], math.cos(ang) - 0.5 * math.sin(ang), atol=1e-14)
        np.testing.assert_allclose(y[0, 0, i + 4], 0.5 * math.cos(ang) + math.sin(ang), atol=1e-14)
        others = [j for j in range(8) if j not in (i, i + 4)]
        assert np.abs(y[0, 0, others]).max() == 0.0


def test_mrope_scores_depend_on_per_axis_offsets_only():
    rng = np.random.default_rng(5)
    q, k = rng.standard_normal((1, 1, 16)), rng.standard_normal((1, 1, 16))
    sec = (2, 3, 3)
    P, Pk = np.array([[4, 9, 1]]), np.array([[2, 3, 8]])
    ref = float(np.sum(O.rope(q, P, 1e4, sec) * O.rope(k, Pk, 1e4, sec)))
    for shift in ([10, 0, 0], [0, 7, 0], [3, 2, 11]):
        sh = np.array([shift])
        got = float(np.sum(O.rope(q, P + sh, 1e4, sec) * O.rope(k, Pk + sh, 1e4, sec)))
        assert abs(got - ref) < 1e-12
    # a shift of one axis alone does change the score
    got = float(np.sum(O.rope(q, P + np.array([[0, 5, 0]]), 1e4, sec) * O.rope(k, Pk, 1e4, sec)))
    assert abs(got - ref) > 1e-6


def test_mrope_rollout_forms_agree_and_continue_positions():
    """Image-grid positions, text after it: naive = teacher-forced = KV-shared, slot 0 = prefill,
    and forced corpus tokens make slot s equal the prefill output at a+s (all axes advance)."""
    shape = _tiny_shape(head_dim=8, n_heads=2, n_kv_heads=1, d_model=16, mrope_sections=(1, 1, 2))
    P = O.Params(W.random_weights(shape, 13, norm_gain="random", scale=0.4))
    L, side = 30, 3
    pos = W.grid_positions(L, side)[None]
    toks = W.random_tokens(shape.vocab, (1, L), 4)
    a_seq, a_pos = np.zeros(3, np.int32), np.array([9, 15, 22], np.int32)
    tk, lp, ft = O.rollout_naive(P, shape, toks, a_seq, a_pos, 4, positions=pos)
    tk2, lp2, ft2, _ = O.rollout_teacher_forced(P, shape, toks, a_seq, a_pos, 4, tk, positions=pos)
    tk3, lp3, ft3 = O.rollout_kv_shared(P, shape, toks, a_seq, a_pos, 4, positions=pos)
    np.testing.assert_array_equal(tk, tk2)
    np.testing.assert_array_equal(tk, tk3)
    np.testing.assert_allclose(lp, lp2, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lp, lp3, rtol=0, atol=1e-12)
    feats, z = O.prefill_outputs(P, shape, toks[0], positions=pos[0])
    forced = np.stack([toks[0, a + 1:a + 5] for a in a_pos]).astype(np.int64)
    tkf, lpf, ftf = O.rollout_naive(P, shape, toks, a_seq, a_pos, 4, forced=forced, positions=pos)
    for i, a in enumerate(a_pos):
        for s in range(4):
            np.testing.assert_allclose(lpf[i, s], O.log_softmax(z[a + s]), rtol=0, atol=1e-12)
    # the grid positions matter: with index positions the outputs differ
    tk4, lp4, _ = O.rollout_naive(P, shape, toks, a_seq, a_pos, 4)
    assert np.abs(lp4 - lp).max() > 1e-6


# ---------------------------------------------------------------- early end (EOS)
def test_active_slots_and_weights_hand_case():
    toks = np.array([[5, 9, 2, 9], [1, 2, 3, 4], [9, 9, 9, 9]])
    act = LB.active_slots(toks, 9)
    np.testing.assert_array_equal(act, [[1, 1, 0, 0], [1, 1, 1, 1], [1, 0, 0, 0]])
    w = LB.slot_weights(toks, 9, gamma=2.0)
    env = LB.slot_envelope(4)
    np.testing.assert_allclose(w[0], [env[0], env[1], 0, 0])
    np.testing.assert_allclose(w[1], env)
    np.testing.assert_allclose(LB.slot_weights(toks, None), np.tile(env, (3, 1)))


def test_ira_weights_stop_at_primary_end():
    B = 8
    toks = np.array([[3, 4, 5, 7, 1, 1, 1, 1]])  # EOS = 7 fed after index 3
    lab = np.zeros((1, B))
    _, _, w, _ = LB.ira_secondary(toks, lab, [0], [2], eos_id=7)
    # the EOS is produced at primary index 3 (fed before index 4): indices 0..3 are active.
    # j = 2: index s' inherits primary index 2 + s' -> s' = 0, 1 active
    env = LB.slot_envelope(B)
    np.testing.assert_allclose(w[0], [env[0], env[1], 0, 0, 0, 0, 0, 0])
    _, _, w2, _ = LB.ira_secondary(toks, lab, [0], [2])
    assert (w2[0] > 0).sum() == (B - 1) - 2
