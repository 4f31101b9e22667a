#!/usr/bin/env python3
"""Rollout throughput benchmark on one MI355X.

One step = one prefill over every corpus sequence of the workload (the shared
prefix key/value cache and features) plus the greedy rollout of every anchor
(block slots each: tokens, full-vocabulary log-probs, features).  Inputs are
resident in HBM before the timed region starts.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--gpus 1]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3    # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def site_work(site: str, w, anchor_seq=None, anchor_pos=None) -> dict:
    """Algorithmic FLOPs (or bytes) of one launch at a profiled site."""
    w_anchor_seq, w_anchor_pos = anchor_seq, anchor_pos
    s = w.shape
    d, F, V = s.d_model, s.d_ffn, s.vocab
    qd, kvd = s.n_heads * s.head_dim, s.n_kv_heads * s.head_dim
    T, NA = w.n_tokens, w.n_anchors
    gemm = {"prefill_qkv": (T, qd + 2 * kvd, d), "prefill_o": (T, d, qd),
            "prefill_gu": (T, 2 * F, d), "prefill_down": (T, d, F),
            "decode_qkv": (NA, qd + 2 * kvd, d), "decode_o": (NA, d, qd),
            "decode_gu": (NA, 2 * F, d), "decode_down": (NA, d, F), "lm_gemm": (NA, V, d)}
    if site in gemm:
        m, n, k = gemm[site]
        return {"bound": "mfma", "flops": 2.0 * m * n * k, "unit": "TFLOP/s"}
    if site == "lm_finalize":
        # the log-softmax rewrite of the logits: one fp32 read and one fp32 write per entry
        return {"bound": "hbm", "bytes": 8.0 * NA * V, "unit": "GB/s"}
    if site == "decode_attn":
        # unique bytes of one launch, averaged over the rollout steps s = 1 .. B-1: every
        # sequence's shared K and V up to its last anchor, each anchor's s private keys and
        # values, the queries read and the outputs written (bf16)
        hd, G, H = s.head_dim, s.n_kv_heads, s.n_heads
        a_max = [int(w_anchor_pos[w_anchor_seq == q].max()) for q in range(w.n_seq)
                 if (w_anchor_seq == q).any()]
        shared = sum(a + 1 for a in a_max) * G * hd * 2 * 2
        steps = max(w.block - 1, 1)
        private = NA * G * hd * 2 * 2 * (sum(range(1, w.block)) / steps)
        qo = 2 * NA * H * hd * 2
        # and the MFMA work: 4 hd FLOP per (query head, visible key), keys 0..a plus the
        # private ones (s of them at step s), averaged over the steps
        avg_priv = sum(range(1, w.block)) / steps
        flops = 4.0 * hd * H * float(sum(int(a) + 1 + avg_priv for a in w_anchor_pos))
        return {"bound": "hbm", "bytes": float(shared + private + qo), "unit": "GB/s",
                "flops": flops}
    if site == "prefill_attn":
        # causal: sum over positions of 4 * hd * (t+1) per head
        L = w.seq_len
        return {"bound": "mfma", "flops": 4.0 * s.head_dim * s.n_heads * w.n_seq * L * (L + 1) / 2,
                "unit": "TFLOP/s"}
    raise KeyError(site)


# rocprofv3 counter summaries: launch site -> (summary file, kernel sources it was taken on)
PROFILE_FILES = {
    "prefill_gu": ("profiles/gemm_gate_up_prefill_llama8b_like.md",
                   ("paper_2609_38795_amd/csrc/gemm_kernels.hpp",
                    "paper_2609_38795_amd/csrc/device_common.hpp")),
}


def measured_traffic(site: str):
    """HBM bytes per launch from the committed counter summary, or None when the kernel
    source has changed since the counters were taken (or none were taken)."""
    import hashlib
    import re

    if site not in PROFILE_FILES:
        return None
    path, srcs = PROFILE_FILES[site]
    try:
        text = open(os.path.join(ROOT, path)).read()
        h = hashlib.sha256()
        for f in srcs:
            h.update(open(os.path.join(ROOT, f), "rb").read())
    except OSError:
        return None
    m_t = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    m_h = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    if not m_t or not m_h or m_h.group(1) != h.hexdigest()[:16]:
        return None
    return float(m_t.group(1))


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform

    return platform.processor() or "unknown"


def cpu_baseline(inp, budget_layers=(2, 4)):
    """Time the oracle (teacher-forced, fp64, bf16-emulating) on the anchor with the median
    prefix of the workload, with the model cut to two depths, and extrapolate to the full
    depth: every decoder layer does the same work, so the time is affine in the depth (a
    fixed part for the embedding and the output head plus one equal share per layer)."""
    import numpy as np

    import oracle as O
    from paper_2609_38795_amd import workloads as W

    w = inp.workload
    order = np.argsort(inp.anchor_pos, kind="stable")
    sel = order[[len(order) // 2]]  # the median prefix
    a_seq, a_pos = inp.anchor_seq[sel], inp.anchor_pos[sel]
    feed = np.zeros((len(sel), w.block), np.int64)
    rows = mask = None
    if inp.embeds is not None:
        rows = inp.embeds.reshape(w.n_seq, w.seq_len, -1)
        mask = inp.embed_mask.reshape(w.n_seq, w.seq_len)
    times = {}
    for nl in sorted({min(x, w.shape.n_layers) for x in budget_layers}):
        shape = W.scaled(w, "trunc", n_layers=nl, feat_layers=tuple(range(min(nl, 1)))).shape
        wt = dict(inp.weights)
        wt["layers"] = inp.weights["layers"][:nl]
        P = O.Params(wt, cache=False)
        t0 = time.perf_counter()
        O.rollout_teacher_forced(P, shape, inp.tokens, a_seq, a_pos, w.block, feed,
                                 given_rows=rows, given_mask=mask,
                                 emulate_bf16=(w.shape.dtype == "bf16"))
        times[nl] = time.perf_counter() - t0
    l1, l2 = budget_layers
    l1, l2 = min(l1, w.shape.n_layers), min(l2, w.shape.n_layers)
    if l1 == l2:
        t_full = times[l1]
    else:
        per_layer = (times[l2] - times[l1]) / (l2 - l1)
        fixed = times[l1] - l1 * per_layer
        t_full = fixed + w.shape.n_layers * per_layer
    try:
        from threadpoolctl import threadpool_info

        cores = max(int(x.get("num_threads", 1)) for x in threadpool_info()) or 1
    except Exception:
        cores = os.cpu_count() or 1
    n = len(sel)
    extrap = (f"with the model cut to {l1} and {l2} decoder layers ({times[l1]:.1f} s, "
              f"{times[l2]:.1f} s) and extrapolated to {w.shape.n_layers} layers "
              f"({t_full:.1f} s; the time is affine in depth, and the median prefix makes the "
              f"anchor representative of the workload's prefix lengths)"
              if l1 != l2 else f"at full depth ({t_full:.1f} s)")
    return {"value": n * w.block / t_full, "unit": "rollout slots/s", "cores": cores,
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": (f"fp64 bf16-emulating teacher-forced oracle on the anchor with the median "
                       f"prefix (position {int(a_pos[0])} of positions "
                       f"{int(inp.anchor_pos.min())}..{int(inp.anchor_pos.max())}; {w.block} slots) "
                       + extrap)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="llama8b_like")
    ap.add_argument("--site", default="prefill_gu", help="kernel launch site for the roofline")
    ap.add_argument("--breakdown", action="store_true", help="time every launch site (extra steps)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the HBM-kernel timing steps (decode attention, output-head finalisation)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this path runs on one GPU; --gpus {args.gpus} is not supported "
              "(multi-GPU sharding by sequence is a design note, not built)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_38795_amd import binding, workloads as W

    w = W.get(args.workload)
    t0 = time.time()
    inp = W.make_inputs(w, progress=lambda m: log(f"[bench] {m} ({time.time() - t0:.0f}s)"))
    log(f"[bench] {w.name}: inputs drawn in {time.time() - t0:.1f}s")
    dev = torch.device("cuda:0")
    lim = binding.make_limits(w.n_tokens, w.n_seq, w.n_anchors, w.block)
    t0 = time.time()
    eng = binding.Engine(w.shape, inp.weights, w.max_pos, lim, device=dev)
    torch.cuda.synchronize()
    log(f"[bench] context created ({eng.ws_bytes / 2**30:.1f} GiB workspace) in {time.time() - t0:.1f}s")
    toks = torch.from_numpy(inp.tokens.reshape(-1).astype(np.int32)).to(dev)
    emb = mask = None
    if inp.embeds is not None:
        e = inp.embeds
        emb = torch.from_numpy(e.view(np.int16) if e.dtype == np.uint16 else e).to(dev)
        mask = torch.from_numpy(inp.embed_mask).to(dev)
    outs = eng.alloc_outputs(w.n_anchors, w.block, want_feats=True)
    seq_lens = [w.seq_len] * w.n_seq
    stream = eng.stream

    def step():
        eng.prefill(toks, seq_lens, emb, mask)
        eng.rollout(inp.anchor_seq, inp.anchor_pos, w.block, out=outs)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"[bench] warmup step {i + 1}/{args.warmup} done")

    # phase split (untimed): prefill vs rollout
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    e0.record(stream)
    eng.prefill(toks, seq_lens, emb, mask)
    e1.record(stream)
    eng.rollout(inp.anchor_seq, inp.anchor_pos, w.block, out=outs)
    e2.record(stream)
    torch.cuda.synchronize()
    prefill_ms, rollout_ms = e0.elapsed_time(e1), e1.elapsed_time(e2)
    log(f"[bench] phases: prefill {prefill_ms:.1f} ms, rollout {rollout_ms:.1f} ms")

    breakdown = {}
    if args.breakdown:
        for site in binding.PROF_SITES:
            binding.profile_start(eng, site, 8192)
            step()
            ms, n = binding.profile_stop(eng)
            breakdown[site] = {"ms_per_step": round(ms, 3), "launches": n}
            log(f"[bench] {site}: {ms:.2f} ms over {n} launches")

    # timed region: exactly K steps, synchronised on both sides
    binding.profile_start(eng, args.site, 8192)
    torch.cuda.synchronize()
    ev_a, ev_b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_start = time.perf_counter()
    ev_a.record(stream)
    for i in range(args.steps):
        step()
    ev_b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    site_ms, site_n = binding.profile_stop(eng)
    ms_per_step = max(wall * 1e3, ev_a.elapsed_time(ev_b)) / args.steps
    slots = w.n_anchors * w.block
    value = slots / (ms_per_step / 1e3)
    log(f"[bench] {args.steps} steps: {ms_per_step:.1f} ms/step, {value:.0f} slots/s")

    work = site_work(args.site, w, inp.anchor_seq, inp.anchor_pos)
    avg_s = site_ms / max(site_n, 1) / 1e3
    if work["bound"] == "mfma":
        achieved = work["flops"] / avg_s / 1e12
        peak = PEAK_BF16_TFLOPS if w.shape.dtype == "bf16" else PEAK_F32_TFLOPS
    else:
        achieved = work["bytes"] / avg_s / 1e9
        peak = PEAK_HBM_GBS
    roofline = {"bound": work["bound"], "achieved": round(achieved, 2), "peak": peak,
                "unit": work["unit"], "frac": round(achieved / peak, 4),
                "traffic": measured_traffic(args.site),
                "kernel": args.site, "avg_launch_ms": round(avg_s * 1e3, 4),
                "launches_timed": site_n}

    # HBM-side kernels the method also names (decode attention, output-head finalisation):
    # average launch time over one extra untimed step each, HIP events on the launch stream
    secondary = []
    for site2 in (() if args.no_secondary else ("decode_attn", "lm_finalize")):
        if site2 == args.site:
            continue
        binding.profile_start(eng, site2, 1024)
        step()
        ms2, n2 = binding.profile_stop(eng)
        wk2 = site_work(site2, w, inp.anchor_seq, inp.anchor_pos)
        gbs = wk2["bytes"] / (ms2 / max(n2, 1) / 1e3) / 1e9
        entry = {"kernel": site2, "bound": "hbm", "achieved": round(gbs, 1),
                 "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                 "avg_launch_ms": round(ms2 / max(n2, 1), 4), "launches_timed": n2,
                 "bytes_per_launch": wk2["bytes"]}
        if "flops" in wk2:  # the attention is at the MFMA/HBM ridge: report both sides
            tfs = wk2["flops"] / (ms2 / max(n2, 1) / 1e3) / 1e12
            entry["mfma_tflops"] = round(tfs, 1)
            entry["mfma_frac"] = round(tfs / PEAK_BF16_TFLOPS, 4)
        secondary.append(entry)
        log(f"[bench] {site2}: {gbs:.0f} GB/s of algorithmic bytes ({ms2 / max(n2, 1):.4f} ms/launch)")

    if args.copy_calibration:
        n = 1 << 28  # 2^28 fp32 = 1 GiB read + 1 GiB written per launch
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        log(f"[bench] copy calibration: 3 launches of {4 * n} bytes read + written")
        del src, dst

    cpu = None
    if not args.no_cpu_baseline:
        t0 = time.time()
        cpu = cpu_baseline(inp)
        log(f"[bench] cpu baseline: {cpu['value']:.4f} slots/s ({time.time() - t0:.1f}s)")

    line = {
        "metric": "rollout slots/sec (anchors x block) at 8B-like shapes; MFMA % and HBM GB/s",
        "value": round(value, 1), "unit": "slots/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w.shape.dtype == "bf16" else "f32",
        "data": "synthetic (seeded random weights and Zipf tokens)",
        "config": {"workload": w.name, "desc": w.description, "n_seq": w.n_seq,
                   "seq_len": w.seq_len, "anchors": w.n_anchors, "block": w.block,
                   "slots_per_step": slots},
        "phases_ms": {"prefill": round(prefill_ms, 2), "rollout": round(rollout_ms, 2),
                      "rollout_only_slots_per_s": round(slots / (rollout_ms / 1e3), 1)},
        "roofline": roofline,
        "roofline_hbm_kernels": secondary,
        "cpu_baseline": cpu,
    }
    if breakdown:
        line["breakdown_ms_per_step"] = breakdown
    print(json.dumps(line), flush=True)
    eng.close()


if __name__ == "__main__":
    main()
