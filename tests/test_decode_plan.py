"""Host-only checks of the decode attention's work plan (no GPU): the planner that alr_rollout runs,
reached through alr_debug_decode_plan.  Every (anchor group, kv head) must have its shared keys
0..a_max covered exactly once by chunk items, partial-output slots must be unique and dense, and
each XCD's items must run largest first."""
import numpy as np
import pytest

from paper_2609_38795_amd import binding, workloads as W

KT = 64


def _groups(shape, seq_len, a_s, a_p):
    """Sorted-anchor groups as the library forms them: up to 128/rep anchors of one sequence."""
    rep = shape.n_heads // shape.n_kv_heads
    ag = max(1, 128 // rep)
    order = sorted(range(len(a_s)), key=lambda i: (a_s[i], a_p[i], i))
    sq = [int(a_s[i]) for i in order]
    ps = [int(a_p[i]) for i in order]
    groups = []
    r0 = 0
    while r0 < len(sq):
        r1 = r0
        while r1 < len(sq) and sq[r1] == sq[r0]:
            r1 += 1
        for f in range(r0, r1, ag):
            cnt = min(ag, r1 - f)
            groups.append((f, cnt, ps[f + cnt - 1]))
        r0 = r1
    return groups


def _check_plan(shape, max_pos, n_cu, seq_len, a_s, a_p):
    ct, span, items = binding.decode_plan(shape, max_pos, n_cu, seq_len, a_s, a_p)
    G = shape.n_kv_heads
    groups = _groups(shape, seq_len, a_s, a_p)
    by_first = {f: (cnt, amax) for f, cnt, amax in groups}
    assert ct >= 1 and len(items) % 8 == 0
    covered = {}
    parts = []
    for b, (first, cnt, kvh, kb, ke, part) in enumerate(items):
        if cnt == 0:
            continue
        assert first in by_first and by_first[first][0] == cnt, (b, first, cnt)
        amax = by_first[first][1]
        assert 0 <= kvh < G
        assert kb % (ct * KT) == 0 and kb < ke <= min(amax + 1, kb + ct * KT), (b, kb, ke, amax)
        covered.setdefault((first, kvh), []).append((kb, ke))
        parts.append(part)
    # every (group, kv head) covers 0..a_max exactly once
    for f, cnt, amax in groups:
        for g in range(G):
            segs = sorted(covered[(f, g)])
            assert segs[0][0] == 0 and segs[-1][1] == amax + 1
            for (b0, e0), (b1, e1) in zip(segs, segs[1:]):
                assert e0 == b1
    # partial-output slots are unique and dense
    assert sorted(parts) == list(range(len(parts)))
    # each XCD runs its items largest first, padding last
    for x in range(8):
        tiles = [-(-(it[4] - it[3]) // KT) if it[1] else 0 for it in items[x::8]]
        assert all(a >= b for a, b in zip(tiles, tiles[1:])), (x, tiles)
    # the simulated makespan is at least the even share of the work
    work = sum(-(-(it[4] - it[3]) // KT) + 3 for it in items if it[1])
    assert span >= work / (2 * n_cu)
    return ct, span, items


@pytest.mark.parametrize("name,n_cu", [("llama8b_like", 256), ("long_ctx_8b", 256),
                                       ("vl_prefix_7b", 256), ("small_bf16", 256),
                                       ("llama8b_like", 80), ("small_bf16", 304)])
def test_plan_covers_every_group_once(name, n_cu):
    w = W.get(name)
    a_s, a_p = W.make_anchors(w)
    _check_plan(w.shape, w.max_pos, n_cu, [w.seq_len] * w.n_seq, a_s, a_p)


def test_plan_ragged_sequences_duplicates_and_edges():
    base = W.get("small_bf16")
    w = W.scaled(base, "plan_ragged", n_heads=8, n_kv_heads=2, head_dim=128, d_model=256,
                 n_seq=4, seq_len=300)
    lens = [300, 129, 64, 1]
    a_s = np.array([0, 0, 0, 1, 1, 1, 2, 2, 3, 1], np.int32)
    a_p = np.array([0, 299, 150, 0, 128, 128, 63, 31, 0, 64], np.int32)
    _check_plan(w.shape, w.max_pos, 256, lens, a_s, a_p)


def test_plan_of_the_headline_workload():
    """The split the measured runs used: 27-tile chunks, 584 items on 256 CUs (the largest chunk
    length with the smallest simulated makespan, 30 tiles)."""
    w = W.get("llama8b_like")
    a_s, a_p = W.make_anchors(w)
    ct, span, items = _check_plan(w.shape, w.max_pos, 256, [w.seq_len] * w.n_seq, a_s, a_p)
    assert ct == 27 and len(items) == 584 and span == 30


def test_plan_errors():
    w = W.get("small_bf16")
    a_s, a_p = W.make_anchors(w)
    sl = [w.seq_len] * w.n_seq
    with pytest.raises(binding.AlrError) as e:
        binding.decode_plan(W.get("tiny_fp32").shape, 256, 256, [128], [0], [0])
    assert e.value.status == 5  # fp32: no MFMA attention plan
    bad = a_p.copy()
    bad[0] = w.seq_len
    with pytest.raises(binding.AlrError) as e:
        binding.decode_plan(w.shape, w.max_pos, 256, sl, a_s, bad)
    assert e.value.status == 2
    with pytest.raises(binding.AlrError) as e:
        binding.decode_plan(w.shape, w.max_pos, 256, sl, a_s, a_p, max_items=8)
    assert e.value.status == 3
