"""Rollout launch graphs (alr_set_rollout_graphs): every replay bit-exact against plain launches.

The graph of a rollout is recorded on the first call of a (anchor count, block, work-list size,
pointers) combination and replayed afterwards; anchors and plans are uploaded per call.  Each
replay here runs after eager work of the program itself (a new prefill, torch arithmetic, host
synchronisations) and is compared with the same call made with graphs off.
"""
import numpy as np
import pytest

from paper_2609_38795_amd import workloads as W
from gpu_util import make_engine, prefill

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _print(*a):
    print(*a, flush=True)


def _workload(dtype="bf16", hd=128):
    base = W.get("small_bf16")
    w = W.scaled(base, f"graphs_{dtype}_{hd}", n_layers=2, d_model=256, n_heads=8, n_kv_heads=2,
                 head_dim=hd, d_ffn=512, vocab=2048, feat_layers=(0, 1), dtype=dtype,
                 n_seq=2, seq_len=300, anchors_per_seq=6, anchor_lo=0, anchor_hi=299, block=5)
    return W.Inputs(w, W.random_weights(w.shape, 41 + hd, scale=0.05, norm_gain="random"),
                    W.random_tokens(2048, (2, 300), 23, dist="zipf"),
                    *W.random_anchors(2, 300, 6, 0, 299, 8), None, None)


def _host(ts):
    torch.cuda.synchronize()
    return [None if t is None else t.cpu().numpy().copy() for t in ts]


def _same(a, b, what):
    for x, y, name in zip(a, b, ("tokens", "log-probs", "features")):
        if x is None and y is None:
            continue
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), f"{what}: {name} differ"


@pytest.mark.parametrize("dtype,hd", [("bf16", 128), ("f32", 32)])
def test_rollout_graph_replays_match_eager(dtype, hd):
    inp = _workload(dtype, hd)
    w = inp.workload
    n = len(inp.anchor_seq)
    a_seq, a_pos = inp.anchor_seq, inp.anchor_pos
    # a second anchor set of the same size (same graph key when its work list has the same size)
    b_pos = np.clip(a_pos[::-1].copy() - 3, 0, w.seq_len - 1).astype(np.int32)
    b_seq = a_seq[::-1].copy()
    eng = make_engine(inp, max_anchors=n, max_block=w.block)
    prefill(eng, inp)
    _print(f"graphs {dtype} hd {hd}: {n} anchors, block {w.block}")

    eng.set_rollout_graphs(False)
    out = eng.alloc_outputs(n, w.block, True)
    ref_a = _host(eng.rollout(a_seq, a_pos, w.block, out=out))
    ref_b = _host(eng.rollout(b_seq, b_pos, w.block, out=out))
    forced = torch.from_numpy(np.ascontiguousarray(ref_a[0], np.int32)).to(eng.device)
    ref_f = _host(eng.rollout(b_seq, b_pos, w.block, forced=forced, out=out))

    eng.set_rollout_graphs(True)
    calls = [("A", a_seq, a_pos, None, ref_a), ("A", a_seq, a_pos, None, ref_a),
             ("B", b_seq, b_pos, None, ref_b), ("A", a_seq, a_pos, None, ref_a),
             ("B forced", b_seq, b_pos, forced, ref_f), ("B", b_seq, b_pos, None, ref_b),
             ("B forced", b_seq, b_pos, forced, ref_f)]
    for i, (name, s_, p_, f_, ref) in enumerate(calls):
        _print(f"  call {i}: anchors {name}")
        got = _host(eng.rollout(s_, p_, w.block, forced=f_, out=out))
        _same(got, ref, f"call {i} ({name})")
        # eager work of the program between replays: a fresh prefill of the same corpus,
        # torch arithmetic on the outputs, host synchronisation
        prefill(eng, inp)
        _ = (out[1] * 2.0).sum().item()
        torch.cuda.synchronize()
    # new output tensors: a new key, recorded and then replayed
    out2 = eng.alloc_outputs(n, w.block, True)
    for i in range(2):
        got = _host(eng.rollout(a_seq, a_pos, w.block, out=out2))
        _same(got, ref_a, f"new outputs, call {i}")
    eng.close()


def test_rollout_topk_graph_matches_eager_and_noalloc():
    inp = _workload()
    w = inp.workload
    n = len(inp.anchor_seq)
    eng = make_engine(inp, max_anchors=n, max_block=w.block)
    prefill(eng, inp)
    eng.set_rollout_graphs(False)
    ref = _host(eng.rollout_topk(inp.anchor_seq, inp.anchor_pos, w.block, want_logprobs=True))
    eng.set_rollout_graphs(True)
    outs = eng.rollout_topk(inp.anchor_seq, inp.anchor_pos, w.block, want_logprobs=True)
    for i in range(3):
        got = _host(eng.rollout_topk(inp.anchor_seq, inp.anchor_pos, w.block, out=outs))
        for x, y, name in zip(got, ref, ("tokens", "top ids", "top log-probs", "tail", "log-probs",
                                          "features")):
            assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), f"replay {i}: {name}"
        prefill(eng, inp)
        torch.cuda.synchronize()
    # the no-allocation entry point never records a graph; its results match as well
    tok, ti, tl, tt, ft = (torch.empty_like(t) for t in (outs[0], outs[1], outs[2], outs[3],
                                                          outs[5]))
    eng.rollout_topk_noalloc(inp.anchor_seq, inp.anchor_pos, w.block, (tok, ti, tl, tt, ft))
    got = _host((tok, ti, tl, tt, ft))
    for x, y in zip(got, (ref[0], ref[1], ref[2], ref[3], ref[5])):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8))
    eng.close()


def test_set_rollout_graphs_rejects_other_values():
    inp = _workload()
    w = inp.workload
    eng = make_engine(inp, max_anchors=len(inp.anchor_seq), max_block=w.block)
    st = eng.lib.alr_set_rollout_graphs(eng.ctx, 2)
    assert st != 0
    eng.close()


def test_rollout_graph_cache_eviction():
    """Five keys (five output tensor sets) cycled twice through the four-entry graph cache: every call
    after an eviction records again, and every result equals plain launches."""
    inp = _workload()
    w = inp.workload
    n = len(inp.anchor_seq)
    eng = make_engine(inp, max_anchors=n, max_block=w.block)
    prefill(eng, inp)
    eng.set_rollout_graphs(False)
    ref = _host(eng.rollout(inp.anchor_seq, inp.anchor_pos, w.block))
    eng.set_rollout_graphs(True)
    outs = [eng.alloc_outputs(n, w.block, True) for _ in range(5)]
    for rnd in range(2):
        for i, o in enumerate(outs):
            _print(f"  round {rnd}, output set {i}")
            got = _host(eng.rollout(inp.anchor_seq, inp.anchor_pos, w.block, out=o))
            _same(got, ref, f"round {rnd}, output set {i}")
    # switching graphs off drops the cache; plain launches still match
    eng.set_rollout_graphs(False)
    _same(_host(eng.rollout(inp.anchor_seq, inp.anchor_pos, w.block, out=outs[0])), ref, "graphs off")
    eng.close()
