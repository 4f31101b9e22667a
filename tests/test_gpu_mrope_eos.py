"""GPU parity of multimodal RoPE positions and early-end masking through the C ABI."""
import numpy as np
import pytest

from oracle import labels as LB
from paper_2609_38795_amd import binding, workloads as W
from parity import compare
from gpu_util import make_engine

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _print(*a):
    print(*a, flush=True)


def _mrope_inputs(dtype, hd, H, G, sections, side, seed, d_model=256):
    base = W.get("tiny_fp32")
    L = 160
    w = W.scaled(base, f"mrope_{dtype}_{hd}_{d_model}", n_layers=2, d_model=d_model, n_heads=H,
                 n_kv_heads=G,
                 head_dim=hd, d_ffn=512, vocab=1024, feat_layers=(0, 1), dtype=dtype,
                 mrope_sections=sections, n_seq=2, seq_len=L, anchors_per_seq=6,
                 anchor_lo=side * side, anchor_hi=L - 1, block=6)
    a_seq, a_pos = W.random_anchors(2, L, 6, side * side, L - 1, seed)
    toks = W.random_tokens(1024, (2, L), seed + 1, dist="zipf")
    # the leading side x side positions are an image given as input rows
    d = w.shape.d_model
    rows = np.zeros((2 * L, d), np.float32)
    mask = np.zeros(2 * L, np.uint8)
    rng = np.random.default_rng(seed + 2)
    for q in range(2):
        rows[q * L:q * L + side * side] = rng.standard_normal((side * side, d)).astype(np.float32)
        mask[q * L:q * L + side * side] = 1
    if dtype == "bf16":
        rows = W.f32_to_bf16_bits(rows)
    inp = W.Inputs(w, W.random_weights(w.shape, seed + 3, scale=0.05, norm_gain="random"), toks,
                   a_seq, a_pos, rows, mask)
    pos = np.stack([W.grid_positions(L, side)] * 2)  # [n_seq, L, 3]
    return inp, pos


def _prefill(eng, inp, pos):
    w = inp.workload
    dev = eng.device
    toks = torch.from_numpy(inp.tokens.reshape(-1).astype(np.int32)).to(dev)
    e = inp.embeds
    emb = torch.from_numpy(e.view(np.int16) if e.dtype == np.uint16 else e).to(dev)
    mask = torch.from_numpy(inp.embed_mask).to(dev)
    eng.prefill(toks, [w.seq_len] * w.n_seq, emb, mask, positions=pos.reshape(-1, 3))


# the last case puts section boundaries (6 and 19) inside runs of four rotary dims and is wide
# enough (d_model 512) for the rollout's QKV product to be split over K, so the split-K reduce's
# four-column RoPE meets both a shared axis and the per-dim fallback
@pytest.mark.parametrize("dtype,hd,H,G,sections,d_model", [("f32", 32, 4, 2, (4, 6, 6), 256),
                                                           ("bf16", 128, 4, 2, (16, 24, 24), 256),
                                                           ("bf16", 64, 8, 2, (8, 12, 12), 256),
                                                           ("bf16", 64, 8, 2, (6, 13, 13), 512)])
def test_mrope_rollout_matches_oracle(dtype, hd, H, G, sections, d_model):
    inp, pos = _mrope_inputs(dtype, hd, H, G, sections, side=6, seed=hd + H, d_model=d_model)
    w = inp.workload
    eng = make_engine(inp)
    _prefill(eng, inp, pos)
    sel = np.arange(len(inp.anchor_seq))

    def gpu_run(forced):
        f = None if forced is None else torch.from_numpy(np.ascontiguousarray(forced, np.int32)).to(eng.device)
        tok, lp, ft = eng.rollout(inp.anchor_seq, inp.anchor_pos, w.block, forced=f)
        torch.cuda.synchronize()
        return tok.cpu().numpy().astype(np.int64), lp.cpu().numpy(), ft.cpu().numpy()

    rep = compare(inp, w.shape, sel, gpu_run, w.block, positions=pos)
    _print(f"mrope {dtype} hd {hd}: {rep}")
    assert rep.ok(), rep
    # the positions matter: a prefill with index positions gives other log-probs
    _prefill(eng, inp, np.repeat(np.arange(w.seq_len)[None, :, None], 3, axis=2).repeat(2, 0))
    _, lp_index, _ = gpu_run(None)
    _prefill(eng, inp, pos)
    _, lp_grid, _ = gpu_run(None)
    assert np.abs(lp_grid - lp_index).max() > 1e-3
    eng.close()


def test_positions_outside_max_pos_are_rejected():
    inp, pos = _mrope_inputs("f32", 32, 4, 2, (4, 6, 6), side=6, seed=1)
    w = inp.workload
    eng = make_engine(inp)
    for bad_val in (w.max_pos, -1):
        bad = pos.copy()
        bad[1, 5, 1] = bad_val
        with pytest.raises(binding.AlrError) as e:
            _prefill(eng, inp, bad)
        assert e.value.status == 2, e.value
    # a valid prefill still works afterwards
    _prefill(eng, inp, pos)
    tok, _, _ = eng.rollout(inp.anchor_seq, inp.anchor_pos, w.block)
    torch.cuda.synchronize()
    assert tok.shape == (len(inp.anchor_seq), w.block)
    eng.close()


def test_slot_weights_and_ira_stop_at_eos():
    base = W.get("small_bf16")
    w = W.scaled(base, "eos_case", n_layers=2, feat_layers=(0, 1), d_model=256, n_heads=4,
                 n_kv_heads=2, head_dim=64, d_ffn=512, vocab=64, n_seq=1, seq_len=300,
                 anchors_per_seq=24, anchor_lo=0, anchor_hi=299, block=12)
    inp = W.Inputs(w, W.random_weights(w.shape, 5, scale=0.3, norm_gain="random"),
                   W.random_tokens(64, (1, 300), 6), *W.random_anchors(1, 300, 24, 0, 299, 7),
                   None, None)
    eng = make_engine(inp)
    from gpu_util import prefill
    prefill(eng, inp)
    tok, ids, tl, tt, _, _ = eng.rollout_topk(inp.anchor_seq, inp.anchor_pos, w.block,
                                              want_feats=False)
    torch.cuda.synchronize()
    t = tok.cpu().numpy()
    # an EOS id that the rollouts actually produce, at different slots
    vals, counts = np.unique(t[:, 1:-1], return_counts=True)
    eos = int(vals[np.argmax(counts)])
    wg = eng.slot_weights(tok, eos_id=eos, gamma=2.0).cpu().numpy()
    wo = LB.slot_weights(t, eos, gamma=2.0)
    np.testing.assert_allclose(wg, wo, rtol=1e-6, atol=0)
    assert (wo == 0).any() and (wo > 0).sum() > len(t)
    np.testing.assert_allclose(eng.slot_weights(tok).cpu().numpy(), LB.slot_weights(t, None),
                               rtol=1e-6, atol=0)
    n = len(t)
    rng = np.random.default_rng(3)
    prim = rng.permutation(n)[: n // 2]
    offs = rng.integers(2, w.block - 1, size=len(prim))
    _, _, _, _, sw = eng.ira_assemble(tok, ids, tl, tt, prim, offs, gamma=2.0, eos_id=eos)
    _, _, o_w, _ = LB.ira_secondary(t, ids.cpu().numpy(), prim, offs, gamma=2.0, eos_id=eos)
    np.testing.assert_allclose(sw.cpu().numpy(), o_w, rtol=1e-6, atol=0)
    eng.close()
