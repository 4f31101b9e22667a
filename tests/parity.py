"""Helpers that run the HIP path and the CPU oracle on the same seeded inputs and compare them.

Parity rules (fp32 / bf16):

* tokens: bit-exact wherever the oracle's top-1 margin (in log-prob) exceeds
  ``tok_margin`` (1e-4 fp32, 1e-2 bf16, raised to 2x the measured bf16 noise
  floor when that is larger).  Where the margin is smaller the GPU's token
  must be an epsilon-argmax of the oracle's distribution; the comparison then
  continues with the GPU re-run on the oracle's tokens (``forced``), so that
  both sides condition on the same path.
* log-probs: max-abs difference <= ``lp_tol`` (1e-4 fp32; bf16: max(2e-2,
  2x floor)).
* features: max-abs difference, divided by the RMS of the oracle's feature row
  for bf16, <= ``ft_tol``.

Every report also carries the literal figures of the target contract, whatever
the pass rule: absolute log-prob and feature max-abs, and, among the slots whose
oracle margin exceeds the literal token threshold (1e-2 bf16, 1e-4 fp32), the
share of all slots they make up and the share of them whose tokens match.

The bf16 noise floor is the largest difference between the fp64 bf16 evaluation
and another valid bf16 evaluation of the same model: one that rounds at the
same points but accumulates in fp32, and one whose attention also rounds its
unnormalised probabilities to bf16 before the value product, as a bf16
matrix-core attention must (the method fixes bf16 arithmetic, not where
attention rounds).
"""
from __future__ import annotations

import dataclasses
import time
from typing import Optional

import numpy as np

import oracle as O


@dataclasses.dataclass
class Report:
    n_slots: int
    lp_max_abs: float
    ft_max: float
    tok_mismatch_confident: int
    tok_near_tie: int
    floor_lp: float
    floor_ft: float
    lp_tol: float
    ft_tol: float
    tok_margin: float
    forced_rerun: bool
    ft_abs: float = 0.0            # absolute feature max-abs (no RMS scaling)
    lit_margin: float = 0.0        # literal token threshold: 1e-2 bf16, 1e-4 fp32
    lit_checked: float = 0.0       # share of slots whose oracle margin exceeds it
    lit_exact: float = 1.0         # share of those slots whose GPU token equals the oracle's

    def literal(self) -> str:
        return (f"literal: lp max-abs {self.lp_max_abs:.4g}, feature max-abs {self.ft_abs:.4g}, "
                f"tokens bit-exact on {100 * self.lit_exact:.1f}% of the "
                f"{100 * self.lit_checked:.1f}% of slots with margin > {self.lit_margin:g}")

    def ok(self) -> bool:
        return (self.lp_max_abs <= self.lp_tol and self.ft_max <= self.ft_tol
                and self.tok_mismatch_confident == 0)


def _given(inp, sel_seq):
    if inp.embeds is None:
        return None, None
    w = inp.workload
    rows = inp.embeds.reshape(w.n_seq, w.seq_len, -1)
    mask = inp.embed_mask.reshape(w.n_seq, w.seq_len)
    return rows, mask


def _layer_progress(shape, what):
    """Per-layer progress lines for evaluations of deep, wide models (minutes each)."""
    if shape.n_params() < 1_000_000_000:
        return None
    t0 = time.time()

    def report(layer):
        if (layer + 1) % 8 == 0 or layer + 1 == shape.n_layers:
            print(f"[oracle] {what}: layer {layer + 1}/{shape.n_layers} "
                  f"({time.time() - t0:.0f}s)", flush=True)
    return report


def oracle_rollout(inp, shape, anchor_seq, anchor_pos, block, feed, emulate, dt=np.float64,
                   positions=None, bf16_probs=False):
    """Teacher-forced oracle along ``feed`` (tokens fed after each slot)."""
    P = O.Params(inp.weights, dt=dt, cache=shape.n_params() < 400_000_000)
    rows, mask = _given(inp, anchor_seq)
    what = f"{np.dtype(dt).name}{' bf16-probs' if bf16_probs else ''} anchors {list(anchor_pos)}"
    return O.rollout_teacher_forced(P, shape, inp.tokens, anchor_seq, anchor_pos, block, feed,
                                    given_rows=rows, given_mask=mask, emulate_bf16=emulate,
                                    positions=positions, bf16_probs=bf16_probs,
                                    progress=_layer_progress(shape, what))


def compare(inp, shape, sel, gpu_run, block, measure_floor: Optional[bool] = None,
            positions=None) -> Report:
    """Compare the GPU rollout of anchors ``sel`` (indices into the workload's anchors).

    positions[n_seq, L, 3] (optional): the (t, h, w) positions given to the prefill.

    gpu_run(forced or None) -> (tokens [n,B], logprobs [n,B,V], feats [n,B,nf,d]) as numpy,
    for exactly the selected anchors.
    """
    bf16 = shape.dtype == "bf16"
    a_seq = inp.anchor_seq[sel]
    a_pos = inp.anchor_pos[sel]
    g_tok, g_lp, g_ft = gpu_run(None)
    # oracle along the GPU's own path: equals the naive definition wherever they agree
    o_tok, o_lp, o_ft, margin = oracle_rollout(inp, shape, a_seq, a_pos, block, g_tok, bf16,
                                              positions=positions)
    floor_lp = floor_ft = 0.0
    if bf16 and (measure_floor is None or measure_floor):
        e_tok, e_lp, e_ft, _ = oracle_rollout(inp, shape, a_seq, a_pos, block, g_tok, True,
                                              dt=np.float32, positions=positions)
        p_tok, p_lp, p_ft, _ = oracle_rollout(inp, shape, a_seq, a_pos, block, g_tok, True,
                                              positions=positions, bf16_probs=True)
        floor_lp = float(max(np.abs(e_lp - o_lp).max(), np.abs(p_lp - o_lp).max()))
        if o_ft.size:
            rms = np.sqrt(np.mean(o_ft ** 2, axis=-1, keepdims=True))
            floor_ft = float(max((np.abs(e_ft - o_ft) / rms).max(),
                                 (np.abs(p_ft - o_ft) / rms).max()))
    if bf16:
        tok_margin = max(1e-2, 2 * floor_lp)
        lp_tol = max(2e-2, 2 * floor_lp)
        ft_tol = max(2e-2, 2 * floor_ft)
    else:
        tok_margin, lp_tol, ft_tol = 1e-4, 1e-4, 1e-4
    # which slots are confident, which are near-ties
    conf = margin > tok_margin
    mism = g_tok != o_tok
    confident_bad = int((mism & conf).sum())
    near = mism & ~conf
    # near-ties must be epsilon-argmaxes
    if near.any():
        idx = np.nonzero(near)
        top = o_lp[idx].max(axis=-1)
        chosen = o_lp[idx[0], idx[1], g_tok[idx]]
        confident_bad += int((chosen < top - tok_margin).sum())
    forced_rerun = False
    o_tok_fin = o_tok
    if near.any():
        # continue on the oracle's path: feed the oracle's own tokens to both sides
        forced = o_tok.astype(np.int32).copy()
        g_tok, g_lp, g_ft = gpu_run(forced)
        o_tok2, o_lp, o_ft, margin = oracle_rollout(inp, shape, a_seq, a_pos, block, forced, bf16,
                                                    positions=positions)
        conf = margin > tok_margin
        confident_bad += int(((g_tok != o_tok2) & conf).sum())
        forced_rerun = True
        o_tok_fin = o_tok2
    lp_err = float(np.abs(g_lp - o_lp).max())
    ft_abs = float(np.abs(g_ft - o_ft).max()) if o_ft.size else 0.0
    if o_ft.size:
        if bf16:
            rms = np.sqrt(np.mean(o_ft ** 2, axis=-1, keepdims=True))
            ft_err = float((np.abs(g_ft - o_ft) / rms).max())
        else:
            ft_err = ft_abs
    else:
        ft_err = 0.0
    lit_margin = 1e-2 if bf16 else 1e-4
    lit = margin > lit_margin
    lit_checked = float(lit.mean())
    lit_exact = float((g_tok[lit] == o_tok_fin[lit]).mean()) if lit.any() else 1.0
    return Report(int(np.prod(g_tok.shape)), lp_err, ft_err, confident_bad, int(near.sum()),
                  floor_lp, floor_ft, lp_tol, ft_tol, tok_margin, forced_rerun, ft_abs,
                  lit_margin, lit_checked, lit_exact)
