"""Plain fp64 reference of anchor-branched greedy rollout (test infrastructure only).

What is computed (Eq. 3 of Sec. 3.2, and the "Rollout implementation"
paragraph of App. A):

* For an anchor position ``a`` of a corpus sequence ``x``, the frozen target
  continues ``x_{<=a}`` greedily: ``y_i = argmax_v p_T(v | x_{<=a}, y_{<i})``,
  ties going to the lower token id.
* Slot ``s`` (0-based, ``s = 0 .. B-1``) sits at position ``a + s``; its input
  token is ``x_a`` for ``s = 0`` and ``y_s`` afterwards.  It yields the
  next-token distribution ``log p_T(. | x_{<=a}, y_{1..s})`` (the paper's
  label for draft slot ``k = s + 1``), the greedy token ``y_{s+1}`` and the
  residual-stream outputs of the feature layers at that position (the stored
  layer outputs that in-rollout anchors reuse).
* Labels are read from the final normalised hidden state through the output
  head; rollout positions continue the anchor's position.

The target is a Llama-style decoder: per layer
``h += Wo . Attn(RoPE(Wq n1), RoPE(Wk n1), Wv n1)`` with ``n1 = RMSNorm(h)``,
then ``h += Wd . (SiLU(Wg n2) * (Wu n2))`` with ``n2 = RMSNorm(h)``; grouped-
query attention maps query head ``j`` to key/value head ``j // (H / G)``;
scores are scaled by ``1/sqrt(head_dim)``; RoPE rotates the pairs
``(i, i + head_dim/2)`` by ``pos * base^(-2i/head_dim)``.

``emulate_bf16=True`` rounds to bfloat16 (nearest, ties to even) at the points
where a bf16 implementation stores bf16 values: RMSNorm outputs, q and k after
RoPE, v, the attention output, the SwiGLU output and the final-norm output.
Everything else (residual stream, accumulations, scores, softmax, logits)
stays in the working precision ``dt`` (float64, or float32 to measure the
accumulation-order noise floor of bf16 evaluation).

Three rollout forms are provided:

* :func:`rollout_naive` -- the definition: one full causal forward over
  ``x_{<=a} . y_{1..s}`` for every slot, no key/value reuse;
* :func:`rollout_teacher_forced` -- one causal forward over
  ``x_{<=a} . y_{1..B-1}`` for given tokens ``y``, read at positions
  ``a .. a+B-1`` (equal to the naive form when ``y`` is its own greedy path,
  because a causal forward's output at position p depends only on inputs at
  positions <= p);
* :func:`rollout_kv_shared` -- all anchors batched per step, each query
  attending under one softmax to the corpus keys up to its anchor and to its
  own rollout keys (App. A, "Rollout implementation").  It exists only so the
  tests can show that this decomposition equals the definition.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np


# --------------------------------------------------------------------------
# bf16 rounding (round to nearest, ties to even) of float64 / float32 values
# --------------------------------------------------------------------------
def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round each value to the nearest bfloat16 (ties to even), keeping x's dtype.

    bfloat16 keeps the float32 sign and exponent and 7 explicit mantissa bits.
    A float64 keeps 52 mantissa bits, so rounding drops its low 45 bits; a
    float32 drops its low 16 bits.  Values are assumed finite and inside the
    normal float32 range.
    """
    x = np.ascontiguousarray(x)
    if x.dtype == np.float64:
        u = x.view(np.uint64)
        drop = np.uint64(45)
        half = np.uint64((1 << 44) - 1)
        r = (u + half + ((u >> drop) & np.uint64(1))) & ~np.uint64((1 << 45) - 1)
        return r.view(np.float64)
    if x.dtype == np.float32:
        u = x.view(np.uint32).astype(np.uint64)
        r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) & np.uint64(0xFFFF0000)
        return r.astype(np.uint32).view(np.float32)
    raise TypeError(f"bf16_round: unsupported dtype {x.dtype}")


def _ident(x):
    return x


# --------------------------------------------------------------------------
# Weights
# --------------------------------------------------------------------------
class Params:
    """Read-only view of the target's weights in the working precision.

    ``weights`` is the dict made by the input generator: matrices are float32
    arrays or uint16 bfloat16 bit patterns, [out, in] layout (y = W x).
    bfloat16 patterns widen exactly (bits << 16 reinterpreted as float32).
    """

    def __init__(self, weights: Dict, dt=np.float64, cache: bool = True):
        self.w = weights
        self.dt = dt
        self.cache = cache
        self._memo: Dict[Tuple[str, int], np.ndarray] = {}
        self.n_layers = len(weights["layers"])

    def _widen(self, a: np.ndarray) -> np.ndarray:
        if a.dtype == np.uint16:
            return (a.astype(np.uint32) << 16).view(np.float32).astype(self.dt)
        return np.asarray(a).astype(self.dt)

    def get(self, name: str, layer: int = -1) -> np.ndarray:
        key = (name, layer)
        if key in self._memo:
            return self._memo[key]
        src = self.w[name] if layer < 0 else self.w["layers"][layer][name]
        v = self._widen(src)
        if self.cache:
            self._memo[key] = v
        return v

    def embed_row(self, tok: int) -> np.ndarray:
        return self._widen(self.w["tok_embed"][tok])


# --------------------------------------------------------------------------
# Building blocks
# --------------------------------------------------------------------------
def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm: x * g / sqrt(mean(x^2) + eps) over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def rope_axis_of(half: int, sections) -> np.ndarray:
    """Position axis (0 = t, 1 = h, 2 = w) that drives frequency i < half under M-RoPE.

    Multimodal RoPE splits the frequency list into consecutive sections, one per
    position axis; sections (s_t, s_h, s_w) sum to head_dim / 2.  No sections
    (None or all zero) means one axis (plain RoPE).
    """
    if sections is None or sum(sections) == 0:
        return np.zeros(half, np.int64)
    assert sum(sections) == half, (sections, half)
    return np.repeat(np.arange(3), np.asarray(sections, dtype=np.int64))


def rope(x: np.ndarray, positions: np.ndarray, base: float, sections=None) -> np.ndarray:
    """Rotate-half RoPE on x[T, n_heads, head_dim]: pair (i, i+hd/2) rotates by pos*theta_i.

    positions[T] (one axis) or positions[T, 3] (t, h, w); with sections, frequency i
    takes the position of its axis (M-RoPE), else axis 0.
    """
    hd = x.shape[-1]
    half = hd // 2
    pos = np.asarray(positions, dtype=np.float64)
    if pos.ndim == 1:
        pos = pos[:, None]
    axis = rope_axis_of(half, sections)
    inv = np.power(float(base), -2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = pos[:, axis] * inv[None, :]  # [T, half]: frequency i at its axis' position
    cos = np.cos(ang).astype(x.dtype)[:, None, :]
    sin = np.sin(ang).astype(x.dtype)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def causal_gqa_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                         round_probs=None, q_pos=None) -> np.ndarray:
    """Causal softmax attention. q[Tq,H,hd], k/v[T,G,hd] -> out[Tq,H,hd].

    Query head j reads key/value head j // (H/G); scores are scaled by
    1/sqrt(hd); the query at position t sees keys 0..t.  q_pos[Tq] gives the
    position of each query row among the key rows (default: query row t is at
    position t, so Tq = T).  round_probs (optional): a rounding applied to the
    unnormalised probabilities exp(s - max) where they multiply the values, the
    normaliser staying in working precision (how a bf16 matrix-core attention
    evaluates the value product).
    """
    Tq, H, hd = q.shape
    T, G = k.shape[0], k.shape[1]
    rep = H // G
    qp = np.arange(Tq) if q_pos is None else np.asarray(q_pos, dtype=np.int64)
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(hd)
    mask = np.arange(T)[None, :] > qp[:, None]
    for j in range(H):
        g = j // rep
        s = (q[:, j, :] @ k[:, g, :].T) * scale
        s[mask] = -np.inf
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        if round_probs is None:
            p /= p.sum(axis=1, keepdims=True)
            out[:, j, :] = p @ v[:, g, :]
        else:
            out[:, j, :] = (round_probs(p) @ v[:, g, :]) / p.sum(axis=1, keepdims=True)
    return out


def log_softmax(z: np.ndarray) -> np.ndarray:
    m = z.max(axis=-1, keepdims=True)
    return z - (m + np.log(np.sum(np.exp(z - m), axis=-1, keepdims=True)))


def greedy_argmax(z: np.ndarray) -> np.ndarray:
    """Index of the largest value along the last axis; ties go to the lowest index."""
    return np.argmax(z, axis=-1)


# --------------------------------------------------------------------------
# Forward
# --------------------------------------------------------------------------
def embed_rows(P: Params, tokens: Sequence[int], given_rows: Optional[np.ndarray] = None,
               given_mask: Optional[np.ndarray] = None) -> np.ndarray:
    """Input rows of the decoder: token embeddings, or given rows where the mask is set."""
    E = P.w["tok_embed"]
    rows = P._widen(E[np.asarray(tokens, dtype=np.int64)])
    if given_rows is not None and given_mask is not None:
        m = np.asarray(given_mask, dtype=bool)
        if m.any():
            rows[m] = P._widen(given_rows[m])
    return rows


def decoder_forward(P: Params, shape, x0: np.ndarray, positions: np.ndarray,
                    emulate_bf16: bool = False, want_layers: bool = True,
                    bf16_probs: bool = False, progress=None):
    """Full causal forward.  Returns (outputs of every layer [L][T,d], final-normed [T,d]).

    bf16_probs: with emulate_bf16, attention also rounds its unnormalised
    probabilities to bf16 before the value product (a second valid bf16
    evaluation, used to size the bf16 noise floor).  progress(layer) (optional) is
    called after each layer (long evaluations report as they go)."""
    rnd = bf16_round if emulate_bf16 else _ident
    rp = bf16_round if (emulate_bf16 and bf16_probs) else None
    dt = P.dt
    H, G, hd = shape.n_heads, shape.n_kv_heads, shape.head_dim
    eps = shape.rms_eps
    T = x0.shape[0]
    h = x0.astype(dt).copy()
    outs: List[np.ndarray] = []
    for layer in range(shape.n_layers):
        n1 = rnd(rmsnorm(h, P.get("attn_norm", layer), eps))
        q = (n1 @ P.get("wq", layer).T).reshape(T, H, hd)
        k = (n1 @ P.get("wk", layer).T).reshape(T, G, hd)
        v = (n1 @ P.get("wv", layer).T).reshape(T, G, hd)
        q = rnd(rope(q, positions, shape.rope_base, _sections(shape)))
        k = rnd(rope(k, positions, shape.rope_base, _sections(shape)))
        v = rnd(v)
        o = rnd(causal_gqa_attention(q, k, v, rp).reshape(T, H * hd))
        h = h + o @ P.get("wo", layer).T
        n2 = rnd(rmsnorm(h, P.get("ffn_norm", layer), eps))
        act = rnd(silu(n2 @ P.get("w_gate", layer).T) * (n2 @ P.get("w_up", layer).T))
        h = h + act @ P.get("w_down", layer).T
        if want_layers:
            outs.append(h.copy())
        if progress is not None:
            progress(layer)
    hf = rnd(rmsnorm(h, P.get("final_norm"), eps))
    return outs, hf


def decoder_layer_at(P: Params, shape, layer: int, x: np.ndarray, positions: np.ndarray,
                     rows, emulate_bf16: bool = False, bf16_probs: bool = False) -> np.ndarray:
    """Output of decoder layer ``layer`` at the sequence positions ``rows`` only.

    x[T, d] is the layer's input at positions 0..T-1 (T > max(rows)) and
    positions[T] or [T, 3] their RoPE positions.  Causality makes a row's
    output depend on the keys and values of rows 0..row only, so keys and
    values are formed for every row and everything else only for ``rows``:
    the same arithmetic as one layer of :func:`decoder_forward`, restricted to
    the rows asked for.  Returns [len(rows), d].
    """
    rnd = bf16_round if emulate_bf16 else _ident
    rp = bf16_round if (emulate_bf16 and bf16_probs) else None
    dt = P.dt
    H, G, hd, eps = shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.rms_eps
    rows = np.asarray(rows, dtype=np.int64)
    T = int(rows.max()) + 1
    h_all = x[:T].astype(dt)
    pos = np.asarray(positions)[:T]
    n1 = rnd(rmsnorm(h_all, P.get("attn_norm", layer), eps))
    k = rnd(rope((n1 @ P.get("wk", layer).T).reshape(T, G, hd), pos, shape.rope_base,
                 _sections(shape)))
    v = rnd((n1 @ P.get("wv", layer).T).reshape(T, G, hd))
    q = rnd(rope((n1[rows] @ P.get("wq", layer).T).reshape(len(rows), H, hd), pos[rows],
                 shape.rope_base, _sections(shape)))
    o = rnd(causal_gqa_attention(q, k, v, rp, q_pos=rows).reshape(len(rows), H * hd))
    h = h_all[rows] + o @ P.get("wo", layer).T
    n2 = rnd(rmsnorm(h, P.get("ffn_norm", layer), eps))
    act = rnd(silu(n2 @ P.get("w_gate", layer).T) * (n2 @ P.get("w_up", layer).T))
    return h + act @ P.get("w_down", layer).T


def _sections(shape):
    return getattr(shape, "mrope_sections", None)


def slot_positions(pos_seq: Optional[np.ndarray], a: int, n_extra: int) -> np.ndarray:
    """Positions of the prefix 0..a and of n_extra rollout slots after it.

    pos_seq[L, 3] holds the corpus sequence's (t, h, w) positions (None: the
    index on every axis).  Rollout slot s continues the anchor's position with
    every axis advancing by s (App. A, "Rollout implementation").
    """
    if pos_seq is None:
        base = np.repeat(np.arange(a + 1, dtype=np.int64)[:, None], 3, axis=1)
    else:
        base = np.asarray(pos_seq, dtype=np.int64)[: a + 1]
    ext = base[a][None, :] + np.arange(1, n_extra + 1, dtype=np.int64)[:, None]
    return np.concatenate([base, ext], 0)


def head_logits(P: Params, hf: np.ndarray) -> np.ndarray:
    """Output-head logits of final-normed rows hf[n,d] -> [n,V]."""
    return hf @ P.get("lm_head").T


def _feats_at(outs: List[np.ndarray], feat_layers: Sequence[int], rows) -> np.ndarray:
    if not feat_layers:
        picked = outs[0][rows] if outs else None
        lead = () if picked is None else picked.shape[:-1]
        return np.zeros(lead + (0, 0))
    return np.stack([outs[layer][rows] for layer in feat_layers], axis=-2)


def prefill_outputs(P: Params, shape, tokens: np.ndarray, given_rows=None, given_mask=None,
                    emulate_bf16: bool = False, positions=None):
    """Teacher-forced forward of one whole corpus sequence.

    positions[T, 3] (optional): (t, h, w) positions; default the index.
    Returns (features [T, n_feat, d], logits [T, V]) at every position.
    """
    T = len(tokens)
    x0 = embed_rows(P, tokens, given_rows, given_mask)
    pos = np.arange(T) if positions is None else np.asarray(positions)
    outs, hf = decoder_forward(P, shape, x0, pos, emulate_bf16)
    return _feats_at(outs, shape.feat_layers, slice(None)), head_logits(P, hf)


# --------------------------------------------------------------------------
# Rollouts
# --------------------------------------------------------------------------
def _prefix_rows(P, tokens_seq, a, given_rows, given_mask):
    gr = None if given_rows is None else given_rows[: a + 1]
    gm = None if given_mask is None else given_mask[: a + 1]
    return embed_rows(P, tokens_seq[: a + 1], gr, gm)


def rollout_naive(P: Params, shape, tokens: np.ndarray, anchor_seq, anchor_pos, block: int,
                  forced: Optional[np.ndarray] = None, given_rows=None, given_mask=None,
                  emulate_bf16: bool = False, positions=None):
    """The definition: for every anchor and slot, a full causal forward with no reuse.

    tokens[n_seq, L]; given_rows/given_mask are per-sequence lists (or arrays
    [n_seq, L, d] / [n_seq, L]) of input rows that replace token embeddings.
    forced[n_anchor, block]: where >= 0, the token fed to the next slot
    instead of the greedy one.  positions[n_seq, L, 3] (optional): (t, h, w)
    positions of the corpus sequences (M-RoPE); default the index.
    Returns tokens_out int64 [n,B], logprobs [n,B,V], feats [n,B,n_feat,d].
    """
    n = len(anchor_seq)
    V, d, nf = shape.vocab, shape.d_model, len(shape.feat_layers)
    tok_out = np.zeros((n, block), np.int64)
    lp_out = np.zeros((n, block, V), P.dt)
    ft_out = np.zeros((n, block, nf, d), P.dt)
    for i in range(n):
        sq, a = int(anchor_seq[i]), int(anchor_pos[i])
        gr = None if given_rows is None else given_rows[sq]
        gm = None if given_mask is None else given_mask[sq]
        prefix = _prefix_rows(P, tokens[sq], a, gr, gm)
        fed: List[int] = []
        for s in range(block):
            rows = prefix if not fed else np.concatenate([prefix, embed_rows(P, fed)], 0)
            pos_seq = None if positions is None else positions[sq]
            outs, hf = decoder_forward(P, shape, rows, slot_positions(pos_seq, a, len(fed)),
                                       emulate_bf16)
            z = head_logits(P, hf[-1:])[0]
            lp_out[i, s] = log_softmax(z)
            tok_out[i, s] = int(greedy_argmax(z))
            if nf:
                ft_out[i, s] = _feats_at(outs, shape.feat_layers, -1)
            nxt = tok_out[i, s]
            if forced is not None and forced[i, s] >= 0:
                nxt = int(forced[i, s])
            fed.append(int(nxt))
    return tok_out, lp_out, ft_out


def rollout_teacher_forced(P: Params, shape, tokens: np.ndarray, anchor_seq, anchor_pos,
                           block: int, feed: np.ndarray, given_rows=None, given_mask=None,
                           emulate_bf16: bool = False, want_logprobs: bool = True,
                           positions=None, bf16_probs: bool = False, progress=None):
    """One causal forward per anchor over x_{<=a} . feed[i, :B-1], read at positions a..a+B-1.

    feed[n, B] holds the token fed *after* each slot (column B-1 is unused), i.e.
    the input of slot s+1 is feed[i, s].  Returns (argmax tokens [n,B],
    logprobs [n,B,V] or None, feats [n,B,n_feat,d], top-2 margins [n,B]).
    bf16_probs, progress: see :func:`decoder_forward`.
    """
    n = len(anchor_seq)
    V, d, nf = shape.vocab, shape.d_model, len(shape.feat_layers)
    tok_out = np.zeros((n, block), np.int64)
    lp_out = np.zeros((n, block, V), P.dt) if want_logprobs else None
    ft_out = np.zeros((n, block, nf, d), P.dt)
    margin = np.zeros((n, block), P.dt)
    for i in range(n):
        sq, a = int(anchor_seq[i]), int(anchor_pos[i])
        gr = None if given_rows is None else given_rows[sq]
        gm = None if given_mask is None else given_mask[sq]
        prefix = _prefix_rows(P, tokens[sq], a, gr, gm)
        fed = [int(t) for t in feed[i, : block - 1]]
        rows = np.concatenate([prefix, embed_rows(P, fed)], 0) if fed else prefix
        pos_seq = None if positions is None else positions[sq]
        outs, hf = decoder_forward(P, shape, rows, slot_positions(pos_seq, a, len(fed)),
                                   emulate_bf16, bf16_probs=bf16_probs, progress=progress)
        z = head_logits(P, hf[a:a + block])
        lp = log_softmax(z)
        if want_logprobs:
            lp_out[i] = lp
        tok_out[i] = greedy_argmax(z)
        srt = np.sort(lp, axis=-1)
        margin[i] = srt[:, -1] - srt[:, -2]
        if nf:
            ft_out[i] = _feats_at(outs, shape.feat_layers, slice(a, a + block))
    return tok_out, lp_out, ft_out, margin


def rollout_kv_shared(P: Params, shape, tokens: np.ndarray, anchor_seq, anchor_pos, block: int,
                      forced: Optional[np.ndarray] = None, given_rows=None, given_mask=None,
                      positions=None):
    """All anchors batched per step over a shared corpus key/value cache (fp64, no rounding).

    Step 0 reads the teacher-forced forward of each corpus sequence at the
    anchor.  Each later step runs every anchor's newest token through the
    decoder as one batch; the query of anchor i attends under one softmax to
    the cached corpus keys at positions 0..a_i and to its own rollout keys at
    positions a_i+1..a_i+s, kept apart from the corpus cache.
    """
    H, G, hd, eps = shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.rms_eps
    rep = H // G
    n = len(anchor_seq)
    V, d, nf, L = shape.vocab, shape.d_model, len(shape.feat_layers), shape.n_layers
    seqs = sorted(set(int(s) for s in anchor_seq))
    # corpus caches, one per sequence: K/V[layer][T,G,hd] after RoPE
    Kc: Dict[int, List[np.ndarray]] = {}
    Vc: Dict[int, List[np.ndarray]] = {}
    pref_feats: Dict[int, np.ndarray] = {}
    pref_hf: Dict[int, np.ndarray] = {}
    for sq in seqs:
        T = tokens.shape[1]
        gr = None if given_rows is None else given_rows[sq]
        gm = None if given_mask is None else given_mask[sq]
        h = embed_rows(P, tokens[sq], gr, gm)
        pos = np.arange(T) if positions is None else np.asarray(positions[sq])
        Ks, Vs, outs = [], [], []
        for layer in range(L):
            n1 = rmsnorm(h, P.get("attn_norm", layer), eps)
            q = rope((n1 @ P.get("wq", layer).T).reshape(T, H, hd), pos, shape.rope_base,
                     _sections(shape))
            k = rope((n1 @ P.get("wk", layer).T).reshape(T, G, hd), pos, shape.rope_base,
                     _sections(shape))
            v = (n1 @ P.get("wv", layer).T).reshape(T, G, hd)
            Ks.append(k)
            Vs.append(v)
            h = h + causal_gqa_attention(q, k, v).reshape(T, H * hd) @ P.get("wo", layer).T
            n2 = rmsnorm(h, P.get("ffn_norm", layer), eps)
            h = h + (silu(n2 @ P.get("w_gate", layer).T) * (n2 @ P.get("w_up", layer).T)) \
                @ P.get("w_down", layer).T
            outs.append(h.copy())
        Kc[sq], Vc[sq] = Ks, Vs
        pref_feats[sq] = _feats_at(outs, shape.feat_layers, slice(None))
        pref_hf[sq] = rmsnorm(h, P.get("final_norm"), eps)

    tok_out = np.zeros((n, block), np.int64)
    lp_out = np.zeros((n, block, V), P.dt)
    ft_out = np.zeros((n, block, nf, d), P.dt)
    a = np.asarray(anchor_pos, dtype=np.int64)
    # slot 0
    for i in range(n):
        sq = int(anchor_seq[i])
        z = head_logits(P, pref_hf[sq][a[i]:a[i] + 1])[0]
        lp_out[i, 0] = log_softmax(z)
        tok_out[i, 0] = int(greedy_argmax(z))
        ft_out[i, 0] = pref_feats[sq][a[i]]
    # private rollout keys/values: [layer][anchor] -> list of [G,hd]
    pk = [[[] for _ in range(n)] for _ in range(L)]
    pv = [[[] for _ in range(n)] for _ in range(L)]
    nxt = tok_out[:, 0].copy()
    if forced is not None:
        nxt = np.where(forced[:, 0] >= 0, forced[:, 0], nxt)
    for s in range(1, block):
        h = embed_rows(P, nxt)  # [n, d]
        if positions is None:
            pos = a + s
        else:  # every axis of the anchor's position advances by s
            pos = np.stack([np.asarray(positions[int(anchor_seq[i])])[a[i]] + s
                            for i in range(n)])
        outs = []
        for layer in range(L):
            n1 = rmsnorm(h, P.get("attn_norm", layer), eps)
            q = rope((n1 @ P.get("wq", layer).T).reshape(n, H, hd), pos, shape.rope_base,
                     _sections(shape))
            k = rope((n1 @ P.get("wk", layer).T).reshape(n, G, hd), pos, shape.rope_base,
                     _sections(shape))
            v = (n1 @ P.get("wv", layer).T).reshape(n, G, hd)
            o = np.zeros((n, H, hd), P.dt)
            for i in range(n):
                pk[layer][i].append(k[i])
                pv[layer][i].append(v[i])
                sq = int(anchor_seq[i])
                kk = np.concatenate([Kc[sq][layer][: a[i] + 1], np.stack(pk[layer][i])], 0)
                vv = np.concatenate([Vc[sq][layer][: a[i] + 1], np.stack(pv[layer][i])], 0)
                for j in range(H):
                    g = j // rep
                    sc = kk[:, g, :] @ q[i, j] / np.sqrt(hd)
                    p = np.exp(sc - sc.max())
                    o[i, j] = (p / p.sum()) @ vv[:, g, :]
            h = h + o.reshape(n, H * hd) @ P.get("wo", layer).T
            n2 = rmsnorm(h, P.get("ffn_norm", layer), eps)
            h = h + (silu(n2 @ P.get("w_gate", layer).T) * (n2 @ P.get("w_up", layer).T)) \
                @ P.get("w_down", layer).T
            outs.append(h.copy())
        z = head_logits(P, rmsnorm(h, P.get("final_norm"), eps))
        lp_out[:, s] = log_softmax(z)
        tok_out[:, s] = greedy_argmax(z)
        ft_out[:, s] = np.stack([outs[layer] for layer in shape.feat_layers], axis=1)
        nxt = tok_out[:, s].copy()
        if forced is not None:
            nxt = np.where(forced[:, s] >= 0, forced[:, s], nxt)
    return tok_out, lp_out, ft_out
