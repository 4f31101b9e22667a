"""GPU parity of the label products through the C ABI: top-8 + tail labels of the
rollout (alr_rollout_topk), corpus labels and erase gates (alr_corpus_labels)
and the secondary blocks of in-rollout anchors (alr_ira_assemble)."""
import numpy as np
import pytest

import oracle as O
from oracle import labels as LB
from paper_2609_38795_amd import binding, workloads as W
from gpu_util import make_engine, prefill

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _print(*a):
    print(*a, flush=True)


def _np(t):
    return t.cpu().numpy()


def _small_bf16_inputs():
    base = W.get("small_bf16")
    w = W.scaled(base, "small_bf16_labels", n_layers=2, feat_layers=(0, 1), n_seq=2, seq_len=600,
                 anchors_per_seq=20, anchor_lo=100, anchor_hi=599, block=16)
    return W.Inputs(w, W.random_weights(w.shape, 91, scale=0.05, norm_gain="random"),
                    W.random_tokens(w.shape.vocab, (2, 600), 12, dist="zipf"),
                    *W.random_anchors(2, 600, 20, 100, 599, 13), None, None)


def _gpu_ranking(lp):
    """Top-8 ids of each row of the GPU's own log-probs: decreasing value, then id."""
    n, B, V = lp.shape
    flat = lp.reshape(-1, V)
    ids = np.zeros((flat.shape[0], 8), np.int64)
    for r in range(flat.shape[0]):
        ids[r] = np.lexsort((np.arange(V), -flat[r]))[:8]
    return ids.reshape(n, B, 8)


@pytest.mark.parametrize("name", ["tiny_fp32", "small_bf16"])
def test_rollout_topk_consistent_with_full_logprobs(name):
    """Same kernels, same logits: top-8 labels are exactly the GPU's own log-probs' top 8,
    with and without the full log-prob rows, and tokens/features do not change."""
    inp = W.make_inputs("tiny_fp32") if name == "tiny_fp32" else _small_bf16_inputs()
    w = inp.workload
    eng = make_engine(inp)
    prefill(eng, inp)
    tok, lp, ft = eng.rollout(inp.anchor_seq, inp.anchor_pos, w.block)
    t2, ids2, tl2, tt2, lp2, ft2 = eng.rollout_topk(inp.anchor_seq, inp.anchor_pos, w.block)
    t3, ids3, tl3, tt3, lp3, ft3 = eng.rollout_topk(inp.anchor_seq, inp.anchor_pos, w.block,
                                                    want_logprobs=True)
    torch.cuda.synchronize()
    assert lp2 is None
    for t in (t2, t3):
        assert torch.equal(t, tok)
    assert torch.equal(lp3, lp) and torch.equal(ft2, ft) and torch.equal(ft3, ft)
    assert torch.equal(ids2, ids3) and torch.equal(tl2, tl3) and torch.equal(tt2, tt3)
    lpn, ids, tl, tt = _np(lp), _np(ids2), _np(tl2), _np(tt2)
    np.testing.assert_array_equal(ids, _gpu_ranking(lpn))
    np.testing.assert_array_equal(ids[..., 0], _np(tok))
    np.testing.assert_array_equal(tl, np.take_along_axis(lpn, ids.astype(np.int64), axis=-1))
    mask = np.ones_like(lpn, dtype=bool)
    np.put_along_axis(mask, ids.astype(np.int64), False, axis=-1)
    tail_ref = np.where(mask, np.exp(lpn.astype(np.float64)), 0.0).sum(-1)
    np.testing.assert_allclose(tt, tail_ref, rtol=1e-4, atol=1e-7)
    _print(f"{name}: top-8 consistent over {tok.numel()} slots; max tail {tt.max():.3e}")
    eng.close()


def test_rollout_topk_matches_oracle_tiny():
    inp = W.make_inputs("tiny_fp32")
    w = inp.workload
    eng = make_engine(inp)
    prefill(eng, inp)
    tok, ids, tl, tt, _, _ = eng.rollout_topk(inp.anchor_seq, inp.anchor_pos, w.block)
    torch.cuda.synchronize()
    tok, ids, tl, tt = _np(tok).astype(np.int64), _np(ids), _np(tl), _np(tt)
    P = O.Params(inp.weights)
    o_tok, o_lp, _, margin = O.rollout_teacher_forced(P, w.shape, inp.tokens, inp.anchor_seq,
                                                      inp.anchor_pos, w.block, tok)
    conf = margin > 1e-4
    np.testing.assert_array_equal(tok[conf], o_tok[conf])
    o_ids, o_vals, o_tail = LB.topk_tail(o_lp)
    # the sorted top-8 log-probs are unique whatever the ties: compare values
    assert np.abs(tl - o_vals).max() <= 1e-4
    # every GPU id is a valid pick: its oracle log-prob equals the rank's value
    picked = np.take_along_axis(o_lp, ids.astype(np.int64), axis=-1)
    assert np.abs(picked - o_vals).max() <= 2e-4
    # ids agree exactly where the oracle's neighbouring ranks are separated
    srt = np.sort(o_lp, axis=-1)[..., ::-1][..., :9]
    gap_lo = np.concatenate([np.full(srt.shape[:-1] + (1,), np.inf),
                             srt[..., :-2] - srt[..., 1:-1]], axis=-1)
    gap_hi = srt[..., :-1] - srt[..., 1:]
    sep = (gap_lo > 1e-3) & (gap_hi > 1e-3)
    np.testing.assert_array_equal(ids[sep], o_ids[sep])
    assert np.abs(tt - o_tail).max() <= 1e-4
    _print(f"tiny top-8: value err {np.abs(tl - o_vals).max():.2e}, "
           f"tail err {np.abs(tt - o_tail).max():.2e}")
    eng.close()


def _corpus_case():
    base = W.get("tiny_fp32")
    w = W.scaled(base, "tiny_fp32_corpus", anchor_hi=127, block=6)
    inp = W.make_inputs("tiny_fp32")
    a_pos = np.array([0, 17, 60, 121, 122, 124, 125, 127, 37, 60], np.int32)
    a_seq = np.zeros(len(a_pos), np.int32)
    # positions 40 .. 49 hold given input rows instead of tokens
    d = w.shape.d_model
    rows = np.zeros((w.n_tokens, d), np.float32)
    mask = np.zeros(w.n_tokens, np.uint8)
    rng = np.random.default_rng(17)
    rows[40:50] = rng.standard_normal((10, d)).astype(np.float32)
    mask[40:50] = 1
    return W.Inputs(w, inp.weights, inp.tokens, a_seq, a_pos, rows, mask)


def test_corpus_labels_match_oracle_tiny():
    inp = _corpus_case()
    w = inp.workload
    B = w.block
    eng = make_engine(inp, max_anchors=len(inp.anchor_pos))
    prefill(eng, inp)
    r = eng.corpus_labels(inp.anchor_seq, inp.anchor_pos, B, want_topk=True, want_logprobs=True)
    torch.cuda.synchronize()
    g = {k: (None if v is None else _np(v)) for k, v in r.items()}
    P = O.Params(inp.weights)
    _, z = O.prefill_outputs(P, w.shape, inp.tokens[0], given_rows=inp.embeds,
                             given_mask=inp.embed_mask)
    lp_seq = O.log_softmax(z)
    is_tok = inp.embed_mask == 0
    valid, lab, am, clp, gs, gh = LB.corpus_labels(lp_seq, inp.tokens[0], inp.anchor_pos, B,
                                                   is_token=is_tok)
    np.testing.assert_array_equal(g["argmax"] >= 0, valid)
    srt = np.sort(lp_seq, axis=-1)
    marg = srt[:, -1] - srt[:, -2]
    pos = inp.anchor_pos[:, None] + np.arange(B)[None, :]
    conf = valid & (marg[np.minimum(pos, w.seq_len - 1)] > 1e-4)
    np.testing.assert_array_equal(g["argmax"][conf], am[conf])
    assert np.abs(g["logprobs"][valid] - lab[valid]).max() <= 1e-4
    assert np.isneginf(g["logprobs"][~valid]).all()
    np.testing.assert_array_equal(np.isnan(g["corpus_logp"]), np.isnan(clp))
    ok = ~np.isnan(clp)
    assert np.abs(g["corpus_logp"][ok] - clp[ok]).max() <= 1e-4
    assert np.abs(g["gate_soft"] - gs).max() <= 1e-4
    # hard gates: equal wherever every argmax they depend on is confident
    dep = np.cumprod(np.concatenate([np.ones((len(pos), 1), bool), conf[:, :-1] | ~valid[:, :-1]],
                                    axis=1), axis=1).astype(bool)
    np.testing.assert_array_equal(g["gate_hard"][dep], gh[dep])
    o_ids, o_vals, o_tail = LB.topk_tail(np.where(valid[..., None], lab, 0.0))
    assert np.abs(g["top_logp"][valid] - o_vals[valid]).max() <= 1e-4
    assert np.abs(g["tail"][valid] - o_tail[valid]).max() <= 1e-4
    assert (g["top_ids"][~valid] == -1).all() and (g["tail"][~valid] == 0).all()
    _print(f"corpus labels: {int(valid.sum())} valid slots of {valid.size}; gate err "
           f"{np.abs(g['gate_soft'] - gs).max():.2e}")
    eng.close()


def test_corpus_slot0_equals_rollout_slot0_bit_exact():
    """At slot 1 the KD labels and the ALR labels coincide: both come from the same GPU rows."""
    inp = _small_bf16_inputs()
    w = inp.workload
    eng = make_engine(inp)
    prefill(eng, inp)
    tok, ids, tl, tt, lp, _ = eng.rollout_topk(inp.anchor_seq, inp.anchor_pos, w.block,
                                               want_logprobs=True, want_feats=False)
    r = eng.corpus_labels(inp.anchor_seq, inp.anchor_pos, w.block, want_logprobs=True)
    torch.cuda.synchronize()
    assert torch.equal(r["logprobs"][:, 0], lp[:, 0])
    assert torch.equal(r["argmax"][:, 0], tok[:, 0])
    assert torch.equal(r["top_ids"][:, 0], ids[:, 0]) and torch.equal(r["tail"][:, 0], tt[:, 0])
    assert bool((r["gate_soft"][:, 0] == 1).all()) and bool((r["gate_hard"][:, 0] == 1).all())
    eng.close()


def test_ira_assemble_matches_oracle():
    inp = _small_bf16_inputs()
    w = inp.workload
    B = w.block
    eng = make_engine(inp)
    prefill(eng, inp)
    tok, ids, tl, tt, _, _ = eng.rollout_topk(inp.anchor_seq, inp.anchor_pos, B,
                                              want_feats=False)
    n = len(inp.anchor_seq)
    rng = np.random.default_rng(23)
    prim = rng.permutation(n)[: n // 2]
    offs = rng.integers(2, B - 1, size=len(prim))  # j ~ U{2 .. K-1}, K = B-1
    offs[:2] = [1, B - 1]  # the extreme offsets the ABI accepts
    t0, sids, slp, stail, sw = eng.ira_assemble(tok, ids, tl, tt, prim, offs, gamma=2.0)
    torch.cuda.synchronize()
    o_t0, o_ids, o_w, _ = LB.ira_secondary(_np(tok), _np(ids), prim, offs, gamma=2.0)
    _, o_lp, _, _ = LB.ira_secondary(_np(tok), _np(tl), prim, offs, gamma=2.0)
    _, o_tail, _, _ = LB.ira_secondary(_np(tok), _np(tt)[..., None], prim, offs, gamma=2.0)
    np.testing.assert_array_equal(_np(t0), o_t0)
    np.testing.assert_array_equal(_np(sids), o_ids)
    np.testing.assert_array_equal(_np(slp), o_lp)
    np.testing.assert_array_equal(_np(stail), np.where(np.isneginf(o_tail[..., 0]), 0.0,
                                                       o_tail[..., 0]))
    np.testing.assert_allclose(_np(sw), o_w, rtol=1e-6, atol=0)
    # out-of-range offsets are rejected on the host
    for bad in (0, B):
        with pytest.raises(binding.AlrError) as e:
            eng.ira_assemble(tok, ids, tl, tt, [0], [bad])
        assert e.value.status == 2
    eng.close()
