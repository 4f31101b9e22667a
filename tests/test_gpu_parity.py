"""GPU parity: the HIP path through the C ABI against the CPU oracle on the same seeded inputs."""
import dataclasses

import numpy as np
import pytest

import oracle as O
from paper_2609_38795_amd import binding, workloads as W
from parity import compare
from gpu_util import make_engine, prefill, runner

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _print(*a):
    print(*a, flush=True)


# ------------------------------------------------------------------ GEMM kernels
@pytest.mark.parametrize("dtype,tile", [("bf16", 0), ("f32", 0), ("bf16", 1), ("bf16", 2),
                                        ("bf16", 3), ("bf16", 4), ("bf16", 5), ("bf16", 17),
                                        ("bf16", 18), ("bf16", 19), ("bf16", 20)])
@pytest.mark.parametrize("M,N,K", [(1, 64, 64), (300, 192, 256), (1024, 640, 1152),
                                   (257, 320, 1536)])
def test_gemm_kernel(dtype, tile, M, N, K):
    """Every GEMM kernel variant against a float64 product, ragged M and partial N tiles."""
    _print(f"gemm {dtype} tile {tile} {M}x{N}x{K}")
    rng = np.random.default_rng(M + N + K)
    a = rng.standard_normal((M, K)).astype(np.float32)
    w = rng.standard_normal((N, K)).astype(np.float32)
    if dtype == "bf16":
        a = O.bf16_round(a)
        w = O.bf16_round(w)
        ta = torch.from_numpy(a).to("cuda").to(torch.bfloat16)
        tw = torch.from_numpy(w).to("cuda").to(torch.bfloat16)
        code = binding.ALR_BF16
    else:
        ta, tw = torch.from_numpy(a).cuda(), torch.from_numpy(w).cuda()
        code = binding.ALR_F32
    c = torch.empty((M, N), dtype=torch.float32, device="cuda")
    binding.debug_gemm(code, ta, tw, c, tile=tile)
    torch.cuda.synchronize()
    ref = a.astype(np.float64) @ w.astype(np.float64).T
    err = np.abs(c.cpu().numpy() - ref).max()
    assert err <= 2e-5 * np.sqrt(K) * 4, err


# ------------------------------------------------------------------ fp32 workload
def _full_compare(inp, sel=None, block=None):
    w = inp.workload
    block = block or w.block
    sel = np.arange(w.n_anchors) if sel is None else np.asarray(sel)
    eng = make_engine(inp, max_anchors=len(sel), max_block=block)
    prefill(eng, inp)
    rep = compare(inp, w.shape, sel, runner(eng, inp.anchor_seq[sel], inp.anchor_pos[sel], block),
                  block)
    eng.close()
    _print(rep)
    return rep


def test_tiny_fp32_workload_matches_oracle():
    rep = _full_compare(W.make_inputs("tiny_fp32"))
    assert rep.ok()


def test_tiny_fp32_gqa_random_gains():
    base = W.get("tiny_fp32")
    w = W.scaled(base, "tiny_fp32_gqa", n_kv_heads=2, n_heads=4, head_dim=32)
    shape = w.shape
    inp = W.Inputs(w, W.random_weights(shape, 77, norm_gain="random", scale=0.05),
                   W.make_tokens(base), *W.make_anchors(base), None, None)
    rep = _full_compare(inp)
    assert rep.ok()


def test_zero_layer_bf16_iterated_map():
    base = W.get("tiny_fp32")
    w = W.scaled(base, "zero_layer_bf16", n_layers=0, feat_layers=(), dtype="bf16", vocab=1024,
                 d_model=256)
    inp = W.Inputs(w, W.random_weights(w.shape, 5, scale=0.5), W.random_tokens(1024, (1, 128), 3),
                   *W.make_anchors(base), None, None)
    rep = _full_compare(inp)
    assert rep.ok()


@pytest.mark.parametrize("hd,H,G", [(64, 8, 2), (128, 8, 2), (128, 7, 1), (32, 4, 4)])
def test_small_bf16_attention_paths(hd, H, G):
    """Both MFMA attention kernels (hd 64/128, rep 4 and 7) and the generic one (hd 32)."""
    base = W.get("small_bf16")
    w = W.scaled(base, f"small_bf16_{hd}_{H}_{G}", n_layers=2, d_model=256, n_heads=H,
                 n_kv_heads=G, head_dim=hd, d_ffn=512, vocab=2048, feat_layers=(0, 1),
                 n_seq=2, seq_len=300, anchors_per_seq=6, anchor_lo=0, anchor_hi=299, block=5)
    inp = W.Inputs(w, W.random_weights(w.shape, hd + H, scale=0.05, norm_gain="random"),
                   W.random_tokens(2048, (2, 300), 9, dist="zipf"),
                   *W.random_anchors(2, 300, 6, 0, 299, 4), None, None)
    rep = _full_compare(inp)
    assert rep.ok()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_wide_residual_rows(dtype):
    """d_model 8448: rows wider than the 8192 elements RMSNorm holds in registers, so every norm
    also runs its streaming tail; the GEMMs see K = 8448 and 33 column tiles of 256, and in bf16
    the rollout's down projection (K = 1024) is split over K with rows too wide for the reduce fused
    with the next norm, so the plain reduce and a separate norm run."""
    base = W.get("small_bf16")
    w = W.scaled(base, f"wide_{dtype}", n_layers=1, d_model=8448, n_heads=4, n_kv_heads=1,
                 head_dim=64, d_ffn=1024, vocab=512, feat_layers=(0,), dtype=dtype, n_seq=2,
                 seq_len=96, anchors_per_seq=3, anchor_lo=0, anchor_hi=95, block=4)
    inp = W.Inputs(w, W.random_weights(w.shape, 8448, scale=0.02, norm_gain="random"),
                   W.random_tokens(512, (2, 96), 29, dist="zipf"),
                   *W.random_anchors(2, 96, 3, 0, 95, 12), None, None)
    rep = _full_compare(inp)
    assert rep.ok()


def test_small_bf16_workload_subset():
    inp = W.make_inputs("small_bf16")
    sel = np.array([0, 1, 70, 130, 200, 255])
    rep = _full_compare(inp, sel=sel)
    assert rep.ok()


@pytest.mark.parametrize("dtype,hd,H,G", [("bf16", 128, 8, 2), ("bf16", 64, 8, 2), ("f32", 32, 4, 2)])
def test_ragged_sequences_and_edge_anchors(dtype, hd, H, G):
    """One prefill over sequences of ragged lengths (300, 129, 64 and 1 tokens: partial key tiles,
    a one-token prefix); anchors at each sequence's first and last position, one anchor twice, and
    rollout positions past the sequence end."""
    lens = [300, 129, 64, 1]
    base = W.get("small_bf16")
    w = W.scaled(base, f"ragged_{dtype}_{hd}", n_layers=2, d_model=256, n_heads=H, n_kv_heads=G,
                 head_dim=hd, d_ffn=512, vocab=2048, feat_layers=(0, 1), dtype=dtype,
                 n_seq=len(lens), seq_len=max(lens), block=5)
    tok_pad = W.random_tokens(2048, (len(lens), max(lens)), 17 + hd, dist="zipf")
    a_seq = np.array([0, 0, 0, 1, 1, 1, 2, 2, 3, 1], np.int32)
    a_pos = np.array([0, 299, 150, 0, 128, 128, 63, 31, 0, 64], np.int32)
    inp = W.Inputs(w, W.random_weights(w.shape, 31 + hd, scale=0.05, norm_gain="random"),
                   tok_pad, a_seq, a_pos, None, None)
    eng = make_engine(inp, max_anchors=len(a_seq), max_block=w.block)
    flat = np.concatenate([tok_pad[s, :n] for s, n in enumerate(lens)]).astype(np.int32)
    eng.prefill(torch.from_numpy(flat).to(eng.device), lens)
    rep = compare(inp, w.shape, np.arange(len(a_seq)), runner(eng, a_seq, a_pos, w.block), w.block)
    eng.close()
    _print(rep)
    assert rep.ok()


# ------------------------------------------------------------------ invariants (bit-exact)
def test_permutation_duplicates_and_slot0():
    inp = W.make_inputs("tiny_fp32")
    w = inp.workload
    eng = make_engine(inp, max_anchors=3 * w.n_anchors)
    fo = prefill(eng, inp, feats=True)
    a_s, a_p = inp.anchor_seq, inp.anchor_pos
    run = runner(eng, a_s, a_p, w.block)
    t0, l0, f0 = run(None)
    perm = np.random.default_rng(1).permutation(w.n_anchors)
    t1, l1, f1 = runner(eng, a_s[perm], a_p[perm], w.block)(None)
    np.testing.assert_array_equal(t1, t0[perm])
    np.testing.assert_array_equal(l1, l0[perm])
    np.testing.assert_array_equal(f1, f0[perm])
    dup = np.concatenate([np.arange(w.n_anchors), np.arange(w.n_anchors)[::-1]])
    t2, l2, f2 = runner(eng, a_s[dup], a_p[dup], w.block)(None)
    np.testing.assert_array_equal(t2, t0[dup])
    np.testing.assert_array_equal(l2, l0[dup])
    # slot-0 features equal the prefill's features at the anchor
    fpre = fo.cpu().numpy()
    np.testing.assert_array_equal(f0[:, 0], fpre[w.seq_len * a_s + a_p])
    eng.close()


def test_forced_corpus_continuation_matches_later_anchor_slot0():
    """Feeding the corpus continuation makes slot s of anchor a the prefill output at a+s."""
    inp = W.make_inputs("tiny_fp32")
    w = inp.workload
    a_p = np.array([10, 40, 77], np.int32)
    a_s = np.zeros(3, np.int32)
    B = 4
    eng = make_engine(inp, max_anchors=16, max_block=B)
    prefill(eng, inp)
    forced = np.stack([inp.tokens[0, a + 1:a + 1 + B] for a in a_p]).astype(np.int32)
    t, lp, ft = runner(eng, a_s, a_p, B)(forced)
    later_p = np.array([a + s for a in a_p for s in range(B)], np.int32)
    t0, lp0, ft0 = runner(eng, np.zeros(len(later_p), np.int32), later_p, 1)(None)
    np.testing.assert_allclose(lp.reshape(-1, w.shape.vocab), lp0[:, 0], atol=2e-5, rtol=0)
    np.testing.assert_allclose(ft.reshape(len(later_p), w.shape.n_feat, -1), ft0[:, 0], atol=2e-5,
                               rtol=0)
    eng.close()


@pytest.mark.parametrize("dtype,hd", [("bf16", 128), ("f32", 32)])
def test_second_prefill_replaces_the_first(dtype, hd):
    """A context reused for a second corpus (other lengths and tokens, after a rollout of the first)
    gives bit-identical rollouts to a fresh context: nothing of the first prefill, its cache layout
    or its rollout plan leaks into the second."""
    base = W.get("small_bf16")
    w = W.scaled(base, f"reuse_{dtype}_{hd}", n_layers=2, d_model=256, n_heads=8, n_kv_heads=2,
                 head_dim=hd, d_ffn=512, vocab=2048, feat_layers=(0, 1), dtype=dtype, n_seq=3,
                 seq_len=300, block=5)
    wts = W.random_weights(w.shape, 7 + hd, scale=0.05, norm_gain="random")
    lens_a, lens_b = [300, 200, 100], [129, 300]
    tok_a = W.random_tokens(2048, (3, 300), 1, dist="zipf")
    tok_b = W.random_tokens(2048, (2, 300), 2, dist="zipf")
    a_s_a, a_p_a = np.array([0, 1, 2, 0], np.int32), np.array([299, 150, 50, 10], np.int32)
    a_s_b, a_p_b = np.array([1, 0, 1, 0], np.int32), np.array([299, 128, 0, 64], np.int32)
    inp = W.Inputs(w, wts, tok_a, a_s_a, a_p_a, None, None)

    def pf(e, tok, lens):
        flat = np.concatenate([tok[q, :n] for q, n in enumerate(lens)]).astype(np.int32)
        e.prefill(torch.from_numpy(flat).to(e.device), lens)

    eng = make_engine(inp, max_anchors=8, max_block=w.block)
    pf(eng, tok_a, lens_a)
    runner(eng, a_s_a, a_p_a, w.block)(None)
    pf(eng, tok_b, lens_b)
    t1, l1, f1 = runner(eng, a_s_b, a_p_b, w.block)(None)
    eng.close()
    fresh = make_engine(inp, max_anchors=8, max_block=w.block)
    pf(fresh, tok_b, lens_b)
    t2, l2, f2 = runner(fresh, a_s_b, a_p_b, w.block)(None)
    fresh.close()
    np.testing.assert_array_equal(t1, t2)
    np.testing.assert_array_equal(l1, l2)
    np.testing.assert_array_equal(f1, f2)


def test_rollout_before_prefill_is_a_state_error():
    inp = W.make_inputs("tiny_fp32")
    eng = make_engine(inp)
    with pytest.raises(binding.AlrError) as e:
        eng.rollout(inp.anchor_seq, inp.anchor_pos, 4)
    assert e.value.status == 4
    eng.close()
