"""Seeded synthetic workloads for the anchor-branched greedy rollout.

This module only *draws inputs*: model shapes, random weights, corpus tokens,
anchor positions and image-embedding rows.  It holds none of the method's
arithmetic (no normalisation, attention, projection or softmax), so that both
the HIP path and the CPU oracle can be fed the very same arrays without sharing
any computation.

Shapes follow the paper's rollout workload: one corpus prefix per sequence,
128 anchors per sequence and a block of 16 slots (the drafter block of the
paper's training table, slot 0 being the anchor), with sequences of at most
4096 tokens (training table, maximum length).  The paper's corpora and target
weights are not available, so every workload is synthetic:

* weights: every matrix (token embedding, the attention and SwiGLU
  projections, the untied output head) is N(0, 0.02) drawn in float32, then
  rounded to bfloat16 (round-to-nearest-even) for bf16 workloads; RMSNorm gains
  are 1 unless ``norm_gain="random"`` is asked for;
* tokens: i.i.d. uniform, or Zipf(s) with P(id = r-1) proportional to r^-s
  over the vocabulary (rank r maps to id r-1), drawn by inverse CDF;
* anchors: distinct positions per sequence, drawn without replacement from an
  inclusive range and left unsorted;
* image rows (vision-language prefix): i.i.d. N(0, 1) vectors, bf16-rounded,
  given directly as input rows at the first positions of every sequence.
"""
from __future__ import annotations

import concurrent.futures as _fut
import dataclasses
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

SEED_BASE = 0x414C52  # ASCII "ALR"


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """Decoder-only (Llama-style) transformer shape."""

    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    rms_eps: float
    rope_base: float
    dtype: str  # "f32" or "bf16": storage type of weights and GEMM operands
    feat_layers: Tuple[int, ...]  # 0-based decoder layers whose outputs are features
    # multimodal RoPE: numbers of frequencies driven by the t, h and w position axes
    # (sum = head_dim / 2); all zero = one position axis (plain RoPE)
    mrope_sections: Tuple[int, int, int] = (0, 0, 0)

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def n_feat(self) -> int:
        return len(self.feat_layers)

    def n_params(self) -> int:
        d, f = self.d_model, self.d_ffn
        per_layer = d * (self.q_dim + 2 * self.kv_dim) + self.q_dim * d + 3 * d * f + 2 * d
        return self.n_layers * per_layer + 2 * self.vocab * d + d


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic rollout workload: corpus, anchors and block size."""

    name: str
    config_no: int
    shape: ModelShape
    n_seq: int
    seq_len: int
    token_dist: str  # "uniform" or "zipf"
    anchors_per_seq: int
    anchor_lo: int  # inclusive
    anchor_hi: int  # inclusive
    block: int
    zipf_s: float = 1.1
    image_rows: int = 0  # leading positions fed as given embedding rows
    weight_seed_config: Optional[int] = None  # reuse another workload's weights
    description: str = ""

    @property
    def n_anchors(self) -> int:
        return self.n_seq * self.anchors_per_seq

    @property
    def n_tokens(self) -> int:
        return self.n_seq * self.seq_len

    @property
    def max_pos(self) -> int:
        """Largest position any slot reaches, plus one."""
        return max(self.seq_len, self.anchor_hi + self.block)


def default_feat_layers(n_layers: int) -> Tuple[int, ...]:
    """Five layers spread from 1 to n_layers-3, the drafter's feature-layer spacing.

    The paper's drafter reads target layers 1, 9, 17, 25, 33 of a 36-layer
    target (training table); round(1 + i (n_layers - 4) / 4) reproduces that
    spacing for 36 layers and scales it to other depths.
    """
    if n_layers <= 5:
        return tuple(range(n_layers))
    return tuple(int(round(1 + i * (n_layers - 4) / 4.0)) for i in range(5))


_LLAMA8B = ModelShape(32, 4096, 32, 8, 128, 14336, 128256, 1e-5, 500000.0, "bf16",
                      (1, 8, 15, 22, 29))

WORKLOADS: Dict[str, Workload] = {
    "tiny_fp32": Workload(
        "tiny_fp32", 1,
        ModelShape(2, 128, 4, 4, 32, 512, 512, 1e-6, 10000.0, "f32", (0, 1)),
        n_seq=1, seq_len=128, token_dist="uniform", anchors_per_seq=8,
        anchor_lo=0, anchor_hi=123, block=4,
        description="2-layer fp32 decoder, d=128, 1 x 128 uniform tokens, 8 anchors, B=4"),
    "small_bf16": Workload(
        "small_bf16", 2,
        ModelShape(8, 1024, 16, 4, 64, 2816, 32000, 1e-6, 10000.0, "bf16", (1, 2, 3, 4, 5)),
        n_seq=4, seq_len=2048, token_dist="zipf", anchors_per_seq=64,
        anchor_lo=1024, anchor_hi=2047, block=16,
        description="8-layer bf16 decoder, d=1024, 4 x 2048 Zipf tokens, 256 anchors, B=16"),
    "llama8b_like": Workload(
        "llama8b_like", 3, _LLAMA8B,
        n_seq=8, seq_len=4096, token_dist="zipf", anchors_per_seq=128,
        anchor_lo=1024, anchor_hi=4080, block=16,
        description="Llama-3-8B shapes (32L, d=4096, GQA 32/8, V=128256), "
                    "8 x 4096 Zipf tokens, 1024 anchors, B=16"),
    "vl_prefix_7b": Workload(
        "vl_prefix_7b", 4,
        ModelShape(28, 3584, 28, 4, 128, 18944, 152064, 1e-6, 1000000.0, "bf16",
                   (1, 7, 13, 19, 25)),
        n_seq=8, seq_len=1600, token_dist="zipf", anchors_per_seq=96,
        anchor_lo=640, anchor_hi=1599, block=16, image_rows=576,
        description="Qwen2-7B shapes, 576 image rows + 64 prompt + 960 response tokens "
                    "per sequence, 8 sequences, 768 anchors in the response, B=16"),
    "long_ctx_8b": Workload(
        "long_ctx_8b", 5, _LLAMA8B,
        n_seq=4, seq_len=8192, token_dist="zipf", anchors_per_seq=512,
        anchor_lo=512, anchor_hi=8176, block=16, weight_seed_config=3,
        description="Llama-3-8B shapes, 4 x 8192 Zipf tokens, 2048 anchors, B=16"),
}

BY_NUMBER = {w.config_no: w for w in WORKLOADS.values()}


def get(name_or_no) -> Workload:
    if isinstance(name_or_no, int):
        return BY_NUMBER[name_or_no]
    return WORKLOADS[name_or_no]


def _streams(config_no: int) -> List[np.random.SeedSequence]:
    return np.random.SeedSequence(SEED_BASE + config_no).spawn(4)


def weight_names(shape: ModelShape) -> List[Tuple[str, int]]:
    """Fixed generation order of the weight tensors: (name, layer or -1)."""
    names: List[Tuple[str, int]] = [("tok_embed", -1)]
    for layer in range(shape.n_layers):
        for n in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down"):
            names.append((n, layer))
    names.append(("lm_head", -1))
    return names


def weight_shape(shape: ModelShape, name: str) -> Tuple[int, int]:
    d, f = shape.d_model, shape.d_ffn
    return {
        "tok_embed": (shape.vocab, d),
        "lm_head": (shape.vocab, d),
        "wq": (shape.q_dim, d),
        "wk": (shape.kv_dim, d),
        "wv": (shape.kv_dim, d),
        "wo": (d, shape.q_dim),
        "w_gate": (f, d),
        "w_up": (f, d),
        "w_down": (d, f),
    }[name]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    out = np.empty(x.shape, np.uint16)
    flat_u, flat_o = u.reshape(-1), out.reshape(-1)
    step = 1 << 22
    for i in range(0, flat_u.size, step):
        c = flat_u[i:i + step]
        t = c >> 16  # finite inputs only: the sum below cannot wrap
        t &= 1
        t += 0x7FFF
        t += c
        t >>= 16
        flat_o[i:i + step] = t
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _draw_matrix(ss: np.random.SeedSequence, shp: Tuple[int, int], scale: float,
                 dtype: str) -> np.ndarray:
    g = np.random.Generator(np.random.PCG64(ss))
    n = shp[0] * shp[1]
    out = np.empty(n, np.uint16 if dtype == "bf16" else np.float32)
    step = 1 << 24
    buf = np.empty(min(step, n), np.float32)
    for i in range(0, n, step):
        m = min(step, n - i)
        g.standard_normal(out=buf[:m], dtype=np.float32)
        buf[:m] *= np.float32(scale)
        if dtype == "bf16":
            out[i:i + m] = f32_to_bf16_bits(buf[:m])
        else:
            out[i:i + m] = buf[:m]
    return out.reshape(shp)


def _n_threads() -> int:
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:  # pragma: no cover
        return max(1, min(16, os.cpu_count() or 1))


def make_weights(shape: ModelShape, config_no: int, norm_gain: str = "ones",
                 threads: Optional[int] = None, progress=None) -> Dict:
    """Draw all weights of ``shape`` from the workload's weight stream.

    Returns ``{"tok_embed", "lm_head", "final_norm", "layers": [dict per layer]}``;
    matrices are uint16 bf16 bit patterns (bf16 shapes) or float32 arrays, in the
    [out, in] layout of a linear map y = W x.  Each tensor has its own child
    seed stream so that tensors can be drawn in parallel and in any order.
    """
    names = weight_names(shape)
    w_stream = _streams(config_no)[0]
    children = w_stream.spawn(len(names) + 1)
    jobs = {}
    with _fut.ThreadPoolExecutor(threads or _n_threads()) as ex:
        for (name, layer), ss in zip(names, children):
            jobs[(name, layer)] = ex.submit(_draw_matrix, ss, weight_shape(shape, name),
                                            0.02, shape.dtype)
        res = {}
        for i, (k, v) in enumerate(jobs.items()):
            res[k] = v.result()
            if progress is not None and (i + 1) % 32 == 0:
                progress(f"weights: {i + 1}/{len(jobs)} tensors drawn")

    def gain(i: int) -> np.ndarray:
        if norm_gain == "ones":
            g = np.ones(shape.d_model, np.float32)
        else:
            rng = np.random.Generator(np.random.PCG64(children[-1].spawn(2 * shape.n_layers + 1)[i]))
            g = (1.0 + 0.25 * rng.standard_normal(shape.d_model)).astype(np.float32)
        return f32_to_bf16_bits(g) if shape.dtype == "bf16" else g

    layers = []
    for layer in range(shape.n_layers):
        ld = {n: res[(n, layer)] for n in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")}
        ld["attn_norm"] = gain(2 * layer)
        ld["ffn_norm"] = gain(2 * layer + 1)
        layers.append(ld)
    return {"tok_embed": res[("tok_embed", -1)], "lm_head": res[("lm_head", -1)],
            "final_norm": gain(2 * shape.n_layers), "layers": layers, "dtype": shape.dtype}


def zipf_tokens(rng: np.random.Generator, n: int, vocab: int, s: float) -> np.ndarray:
    ranks = np.arange(1, vocab + 1, dtype=np.float64)
    cdf = np.cumsum(ranks ** (-s))
    cdf /= cdf[-1]
    u = rng.random(n)
    return np.minimum(np.searchsorted(cdf, u, side="right"), vocab - 1).astype(np.int32)


def make_tokens(w: Workload) -> np.ndarray:
    """Corpus tokens, int32 [n_seq, seq_len]."""
    rng = np.random.Generator(np.random.PCG64(_streams(w.config_no)[1]))
    n = w.n_seq * w.seq_len
    if w.token_dist == "uniform":
        t = rng.integers(0, w.shape.vocab, size=n, dtype=np.int64).astype(np.int32)
    else:
        t = zipf_tokens(rng, n, w.shape.vocab, w.zipf_s)
    return t.reshape(w.n_seq, w.seq_len)


def make_anchors(w: Workload) -> Tuple[np.ndarray, np.ndarray]:
    """Anchor (sequence, position) pairs, int32 [n_anchors] each, unsorted within a sequence."""
    rng = np.random.Generator(np.random.PCG64(_streams(w.config_no)[2]))
    seqs, poss = [], []
    span = w.anchor_hi - w.anchor_lo + 1
    for s in range(w.n_seq):
        p = w.anchor_lo + rng.choice(span, size=w.anchors_per_seq, replace=False)
        seqs.append(np.full(w.anchors_per_seq, s, np.int32))
        poss.append(p.astype(np.int32))
    return np.concatenate(seqs), np.concatenate(poss)


def make_image_rows(w: Workload) -> Tuple[Optional[np.ndarray], Optional[np.ndarray]]:
    """Given input rows for the image prefix: (rows [n_seq*seq_len, d], mask u8 [n_seq*seq_len]).

    Rows are stored in the weight dtype (bf16 bits or float32); rows outside the
    image prefix are zero and masked off.
    """
    if w.image_rows == 0:
        return None, None
    rng = np.random.Generator(np.random.PCG64(_streams(w.config_no)[3]))
    d = w.shape.d_model
    rows = np.zeros((w.n_seq, w.seq_len, d), np.float32)
    rows[:, :w.image_rows, :] = rng.standard_normal((w.n_seq, w.image_rows, d), dtype=np.float32)
    mask = np.zeros((w.n_seq, w.seq_len), np.uint8)
    mask[:, :w.image_rows] = 1
    rows = rows.reshape(w.n_seq * w.seq_len, d)
    if w.shape.dtype == "bf16":
        rows = f32_to_bf16_bits(rows)
    return rows, mask.reshape(-1)


def grid_positions(seq_len: int, image_side: int) -> np.ndarray:
    """(t, h, w) positions [seq_len, 3] of a sequence that starts with a square image of
    image_side x image_side rows, Qwen2-VL style: image row r, column c at (0, r, c); the
    text that follows starts one past the largest image position and advances all three
    axes together."""
    pos = np.zeros((seq_len, 3), np.int32)
    n_img = image_side * image_side
    r = np.arange(n_img)
    pos[:n_img, 1] = r // image_side
    pos[:n_img, 2] = r % image_side
    text = image_side + np.arange(seq_len - n_img, dtype=np.int32)
    pos[n_img:] = text[:, None]
    return pos


@dataclasses.dataclass
class Inputs:
    workload: Workload
    weights: Dict
    tokens: np.ndarray  # int32 [n_seq, seq_len]
    anchor_seq: np.ndarray  # int32 [n_anchors]
    anchor_pos: np.ndarray  # int32 [n_anchors]
    embeds: Optional[np.ndarray]  # [n_seq*seq_len, d] or None
    embed_mask: Optional[np.ndarray]  # uint8 [n_seq*seq_len] or None


def make_inputs(w, norm_gain: str = "ones", progress=None) -> Inputs:
    if not isinstance(w, Workload):
        w = get(w)
    wcfg = w.weight_seed_config or w.config_no
    weights = make_weights(w.shape, wcfg, norm_gain=norm_gain, progress=progress)
    a_seq, a_pos = make_anchors(w)
    emb, mask = make_image_rows(w)
    return Inputs(w, weights, make_tokens(w), a_seq, a_pos, emb, mask)


def scaled(w: Workload, name: str, **changes) -> Workload:
    """A variant of ``w`` with some fields (or shape fields) replaced."""
    shape_fields = {f.name for f in dataclasses.fields(ModelShape)}
    sc = {k: v for k, v in changes.items() if k in shape_fields}
    wc = {k: v for k, v in changes.items() if k not in shape_fields}
    shape = dataclasses.replace(w.shape, **sc) if sc else w.shape
    return dataclasses.replace(w, name=name, shape=shape, **wc)


def random_weights(shape: ModelShape, seed: int, norm_gain: str = "ones", scale: float = 0.02) -> Dict:
    """Weights for ad-hoc test shapes, from an explicit integer seed."""
    ss = np.random.SeedSequence([SEED_BASE, 0xA11, seed])
    names = weight_names(shape)
    children = ss.spawn(len(names) + 1)
    res = {k: _draw_matrix(c, weight_shape(shape, k[0]), scale, shape.dtype)
           for k, c in zip(names, children)}
    rng = np.random.Generator(np.random.PCG64(children[-1]))

    def gain() -> np.ndarray:
        g = np.ones(shape.d_model, np.float32)
        if norm_gain == "random":
            g = (1.0 + 0.25 * rng.standard_normal(shape.d_model)).astype(np.float32)
        return f32_to_bf16_bits(g) if shape.dtype == "bf16" else g

    layers = []
    for layer in range(shape.n_layers):
        ld = {n: res[(n, layer)] for n in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")}
        ld["attn_norm"] = gain()
        ld["ffn_norm"] = gain()
        layers.append(ld)
    return {"tok_embed": res[("tok_embed", -1)], "lm_head": res[("lm_head", -1)],
            "final_norm": gain(), "layers": layers, "dtype": shape.dtype}


def random_tokens(vocab: int, shape: Sequence[int], seed: int, dist: str = "uniform",
                  s: float = 1.1) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_BASE, 0x70C, seed])))
    n = int(np.prod(shape))
    if dist == "uniform":
        t = rng.integers(0, vocab, size=n).astype(np.int32)
    else:
        t = zipf_tokens(rng, n, vocab, s)
    return t.reshape(shape)


def random_anchors(n_seq: int, seq_len: int, per_seq: int, lo: int, hi: int,
                   seed: int) -> Tuple[np.ndarray, np.ndarray]:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_BASE, 0xA2C, seed])))
    seqs, poss = [], []
    for s in range(n_seq):
        p = lo + rng.choice(hi - lo + 1, size=per_seq, replace=False)
        seqs.append(np.full(per_seq, s, np.int32))
        poss.append(p.astype(np.int32))
    return np.concatenate(seqs), np.concatenate(poss)
