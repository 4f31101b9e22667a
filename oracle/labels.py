"""Plain fp64 reference of the label products built from the target's outputs
(test infrastructure only; never imported by the product path).

What is computed:

* :func:`topk_tail` -- the label format of the distillation loss (Sec. 3.1,
  Eq. 1, and the loss row of the training table in App. A): a slot's target
  distribution restricted to its 8 most probable tokens, the remaining
  probability mass grouped into one tail bucket.  Tokens are ranked by
  decreasing probability; equal probabilities rank the lower token id first,
  the same rule the paper applies to greedy ties (App. A, "Rollout
  implementation").
* :func:`slot_envelope` -- the decay envelope ``w_k = exp(-(k-1)/gamma)`` of
  Eq. 1.
* :func:`corpus_labels` -- the fixed-corpus distillation labels
  ``pi_{a,k} = p_T(. | x_{<a+k})`` of Sec. 3.1 and the survival gates of the
  erase objective (Eq. 2): the soft gate ``g_{a,k} = prod_{1<=j<k}
  p_T(x_{a+j} | x_{<a+j})`` and the hard gate, whose factors are the
  indicators ``1[x_{a+j} = argmax p_T(. | x_{<a+j})]``.
* :func:`slot_weights` -- the slot weights of ALR blocks: ``w_k`` on active
  slots, 0 on the slots that follow an early end of the rollout (Sec. 3.2: a
  slot is masked once an end-of-sequence token was fed before it).
* :func:`ira_secondary` -- the secondary blocks of in-rollout anchors (Sec. 3.2,
  Eq. 4): a block placed at offset ``j`` inside a primary rollout takes the
  target-generated token ``y*_j`` as its slot 0, inherits the primary label at
  position ``j+k`` for its slot ``k`` and gets the weight
  ``w_k 1[j+k <= K]``.

Slot convention shared with the rollout: index ``s = 0 .. B-1`` of a block is
the paper's slot ``k = s + 1`` and sits at position ``a + s``; ``K = B - 1``.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

TOPK = 8


def topk_tail(logp: np.ndarray, k: int = TOPK):
    """Top-k tokens of each log-distribution along the last axis, and the tail mass.

    Ranking: decreasing log-probability, equal values by increasing token id.
    Returns (ids int64 [..., k], their log-probs [..., k], tail [...]) where
    tail is the probability summed over every token outside the top k (0 when
    the vocabulary has at most k tokens; then the missing entries are id -1,
    log-prob -inf).
    """
    logp = np.asarray(logp, dtype=np.float64)
    lead, V = logp.shape[:-1], logp.shape[-1]
    flat = logp.reshape(-1, V)
    ids = np.full((flat.shape[0], k), -1, np.int64)
    vals = np.full((flat.shape[0], k), -np.inf)
    tail = np.zeros(flat.shape[0])
    for r in range(flat.shape[0]):
        # lexsort sorts by the last key first: -logp (descending value), then id
        order = np.lexsort((np.arange(V), -flat[r]))
        top = order[:k]
        ids[r, :len(top)] = top
        vals[r, :len(top)] = flat[r, top]
        rest = order[k:]
        tail[r] = float(np.sum(np.exp(flat[r, rest]))) if len(rest) else 0.0
    return ids.reshape(lead + (k,)), vals.reshape(lead + (k,)), tail.reshape(lead)


def slot_envelope(n_slots: int, gamma: float = 2.0) -> np.ndarray:
    """w_k = exp(-(k-1)/gamma) for k = 1 .. n_slots (Eq. 1), as an array indexed by k-1."""
    k = np.arange(1, n_slots + 1, dtype=np.float64)
    return np.exp(-(k - 1.0) / gamma)


def active_slots(tokens, eos_id: Optional[int]) -> np.ndarray:
    """active[i, s]: no end-of-sequence token among tokens[i, 0 .. s-1] (the tokens fed
    before index s; index s of a block is the paper's slot s+1).  eos_id None: all active."""
    tokens = np.asarray(tokens)
    act = np.ones(tokens.shape, bool)
    if eos_id is None or eos_id < 0:
        return act
    for i in range(tokens.shape[0]):
        for s in range(1, tokens.shape[1]):
            act[i, s] = act[i, s - 1] and int(tokens[i, s - 1]) != eos_id
    return act


def slot_weights(tokens, eos_id: Optional[int], gamma: float = 2.0) -> np.ndarray:
    """omega[i, s] = w_{s+1} on active slots, 0 after an early end (Eq. 1, Sec. 3.2)."""
    tokens = np.asarray(tokens)
    return slot_envelope(tokens.shape[1], gamma)[None, :] * active_slots(tokens, eos_id)


def corpus_labels(lp_seq: np.ndarray, tokens_seq: np.ndarray, anchor_pos, block: int,
                  is_token: Optional[np.ndarray] = None):
    """Fixed-corpus KD labels and erase gates for anchors of one corpus sequence.

    lp_seq[L, V]: the teacher-forced log-distribution at every position of the
    sequence (row p is log p_T(. | x_{<=p})); tokens_seq[L]: its tokens;
    is_token[L] (optional): False where the position holds a given input row
    instead of a token (such a position cannot be a corpus continuation).

    For anchor a and index s (paper slot k = s+1): the label is row a+s
    (``p_T(. | x_{<a+k})``), defined while a+s <= L-1.  The corpus log-prob of
    index s is ``log p_T(x_{a+s+1} | x_{<=a+s})``, defined while a+s+1 <= L-1
    and x_{a+s+1} is a token.  The gates of index s multiply the factors of
    indices 0 .. s-1 (so index 0 has gate 1); an undefined factor is 0.

    Returns (valid bool [n,B], labels [n,B,V] (-inf where invalid),
    argmax int64 [n,B] (-1 where invalid), corpus_logp [n,B] (nan where
    undefined), gate_soft [n,B], gate_hard [n,B]) with gates 0 where invalid.
    """
    lp_seq = np.asarray(lp_seq, dtype=np.float64)
    L, V = lp_seq.shape
    if is_token is None:
        is_token = np.ones(L, bool)
    n = len(anchor_pos)
    valid = np.zeros((n, block), bool)
    labels = np.full((n, block, V), -np.inf)
    amax = np.full((n, block), -1, np.int64)
    clp = np.full((n, block), np.nan)
    g_soft = np.zeros((n, block))
    g_hard = np.zeros((n, block))
    for i, a in enumerate(np.asarray(anchor_pos, dtype=np.int64)):
        soft, hard = 1.0, 1.0
        for s in range(block):
            p = a + s
            if p > L - 1:
                break
            valid[i, s] = True
            labels[i, s] = lp_seq[p]
            amax[i, s] = int(np.argmax(lp_seq[p]))  # first maximal index = lower id on ties
            g_soft[i, s], g_hard[i, s] = soft, hard
            nxt = p + 1
            if nxt <= L - 1 and is_token[nxt]:
                x = int(tokens_seq[nxt])
                clp[i, s] = lp_seq[p, x]
                soft *= float(np.exp(lp_seq[p, x]))
                hard *= 1.0 if amax[i, s] == x else 0.0
            else:
                soft, hard = 0.0, 0.0
    return valid, labels, amax, clp, g_soft, g_hard


def ira_secondary(tokens, labels, primary, offset, gamma: float = 2.0,
                  eos_id: Optional[int] = None):
    """Secondary blocks of in-rollout anchors (Eq. 4).

    tokens[n_prim, B]: the primary rollouts' greedy tokens (index s holds
    y*_{s+1}); labels[n_prim, B, ...]: any per-slot label arrays of the
    primaries (index s = paper slot s+1); primary[n_sec], offset[n_sec]: the
    primary block and offset j of each secondary (1 <= j <= B-1).

    Secondary index s' (paper slot k = s'+1) inherits the primary label at
    paper slot j+k, i.e. primary index j+s', where that exists (j+s' <= B-1;
    else the entry is left as fill).  Its weight is w_k 1[j+k <= K] with
    K = B-1, and 0 where the primary had ended before the inherited slot
    (an end-of-sequence token among tokens[p, 0 .. j+s'-1], with eos_id).
    Slot 0's token is y*_j = tokens[p, j-1]; the block's slot 0 sits
    at position a + j, so its context is the prefix up to a and the rollout
    positions a+1 .. a+j-1.

    Returns (token0 [n_sec], labels_sec (same trailing shape, fill = first
    label's fill: -1 for integer arrays, -inf for float arrays), weight
    [n_sec, B], pos_shift [n_sec] = j).
    """
    tokens = np.asarray(tokens)
    labels = np.asarray(labels)
    n_sec = len(primary)
    B = tokens.shape[1]
    K = B - 1
    w = slot_envelope(B, gamma)
    act = active_slots(tokens, eos_id)
    fill = -1 if np.issubdtype(labels.dtype, np.integer) else -np.inf
    out = np.full((n_sec,) + labels.shape[1:], fill, dtype=labels.dtype)
    weight = np.zeros((n_sec, B))
    token0 = np.zeros(n_sec, np.int64)
    for q in range(n_sec):
        p, j = int(primary[q]), int(offset[q])
        token0[q] = int(tokens[p, j - 1])
        for s2 in range(B):
            k = s2 + 1
            if j + s2 <= B - 1:
                out[q, s2] = labels[p, j + s2]
            alive = j + s2 <= B - 1 and bool(act[p, j + s2])
            weight[q, s2] = w[k - 1] if (j + k <= K and alive) else 0.0
    return token0, out, weight, np.asarray(offset, np.int64)
