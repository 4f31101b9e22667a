"""Thin ctypes binding of libalr.so (argument marshalling only).

Every step of the rollout runs in the library's HIP kernels; this module only
turns Python/torch objects into the C ABI's plain pointers and sizes.  PyTorch
provides device memory and streams.  If the library is missing the binding
raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libalr.so")

ALR_F32, ALR_BF16 = 0, 1
ALR_MAX_FEAT = 8
STATUS = {0: "ALR_OK", 1: "ALR_E_INVALID_ARG", 2: "ALR_E_OUT_OF_RANGE", 3: "ALR_E_WORKSPACE",
          4: "ALR_E_STATE", 5: "ALR_E_UNSUPPORTED", 6: "ALR_E_HIP"}

# Every function the C headers declare (include/alr.h, include/alr_debug.h).
EXPORTS = ("alr_workspace_bytes", "alr_check_config", "alr_check_rollout", "alr_create",
           "alr_prefill", "alr_prefill_positions", "alr_rollout", "alr_rollout_topk",
           "alr_rollout_topk_noalloc",
           "alr_corpus_labels", "alr_ira_assemble", "alr_slot_weights", "alr_last_error", "alr_status_string", "alr_destroy",
           "alr_debug_gemm", "alr_debug_decode_plan", "alr_profile_start", "alr_profile_stop",
           "alr_set_rollout_graphs")
ALR_TOPK = 8


class AlrConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_base", ctypes.c_float), ("dtype", ctypes.c_int32),
                ("max_pos", ctypes.c_int32), ("n_feat", ctypes.c_int32),
                ("feat_layers", ctypes.c_int32 * ALR_MAX_FEAT),
                ("mrope_sections", ctypes.c_int32 * 3)]


class AlrLimits(ctypes.Structure):
    _fields_ = [("max_tokens", ctypes.c_int32), ("max_seqs", ctypes.c_int32),
                ("max_anchors", ctypes.c_int32), ("max_block", ctypes.c_int32)]


_PP = ctypes.POINTER(ctypes.c_void_p)


class AlrWeights(ctypes.Structure):
    _fields_ = [("tok_embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("lm_head", ctypes.c_void_p), ("attn_norm", _PP), ("wq", _PP), ("wk", _PP),
                ("wv", _PP), ("wo", _PP), ("ffn_norm", _PP), ("w_gate", _PP), ("w_up", _PP),
                ("w_down", _PP)]


class AlrError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


_lib: Optional[ctypes.CDLL] = None


def load_library() -> ctypes.CDLL:
    """Load libalr.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(the rollout has no non-HIP path)")
    lib = ctypes.CDLL(LIB_PATH)
    i32, vp, sz = ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t
    cfgp, limp = ctypes.POINTER(AlrConfig), ctypes.POINTER(AlrLimits)
    i32p = ctypes.POINTER(ctypes.c_int32)
    lib.alr_workspace_bytes.argtypes = [cfgp, limp]
    lib.alr_workspace_bytes.restype = sz
    lib.alr_check_config.argtypes = [cfgp, ctypes.c_char_p, sz]
    lib.alr_check_config.restype = ctypes.c_int
    lib.alr_check_rollout.argtypes = [cfgp, limp, i32, i32p, i32, i32p, i32p, i32,
                                      ctypes.c_char_p, sz]
    lib.alr_check_rollout.restype = ctypes.c_int
    lib.alr_create.argtypes = [cfgp, ctypes.POINTER(AlrWeights), limp, vp, sz, vp,
                               ctypes.POINTER(vp)]
    lib.alr_create.restype = ctypes.c_int
    lib.alr_prefill.argtypes = [vp, i32, i32p, vp, vp, vp, vp, vp]
    lib.alr_prefill.restype = ctypes.c_int
    lib.alr_prefill_positions.argtypes = [vp, i32, i32p, vp, i32p, vp, vp, vp, vp]
    lib.alr_prefill_positions.restype = ctypes.c_int
    lib.alr_slot_weights.argtypes = [vp, i32, i32, vp, i32, ctypes.c_float, vp, vp]
    lib.alr_slot_weights.restype = ctypes.c_int
    lib.alr_rollout.argtypes = [vp, i32, i32p, i32p, i32, vp, vp, vp, vp, vp]
    lib.alr_rollout.restype = ctypes.c_int
    lib.alr_rollout_topk.argtypes = [vp, i32, i32p, i32p, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.alr_rollout_topk.restype = ctypes.c_int
    lib.alr_rollout_topk_noalloc.argtypes = [vp, i32, i32p, i32p, i32, vp, vp, vp, vp, vp, vp, vp]
    lib.alr_rollout_topk_noalloc.restype = ctypes.c_int
    lib.alr_corpus_labels.argtypes = [vp, i32, i32p, i32p, i32, vp, vp, vp, vp, vp, vp, vp, vp,
                                      vp]
    lib.alr_corpus_labels.restype = ctypes.c_int
    lib.alr_ira_assemble.argtypes = [vp, i32, i32, vp, vp, vp, vp, i32, i32p, i32p,
                                     ctypes.c_float, i32, vp, vp, vp, vp, vp, vp]
    lib.alr_ira_assemble.restype = ctypes.c_int
    lib.alr_last_error.argtypes = [vp]
    lib.alr_last_error.restype = ctypes.c_char_p
    lib.alr_status_string.argtypes = [ctypes.c_int]
    lib.alr_status_string.restype = ctypes.c_char_p
    lib.alr_destroy.argtypes = [vp]
    lib.alr_destroy.restype = None
    lib.alr_debug_gemm.argtypes = [i32, vp, vp, vp, i32, i32, i32, i32, vp, sz, vp]
    lib.alr_debug_gemm.restype = ctypes.c_int
    lib.alr_debug_decode_plan.argtypes = [cfgp, i32, i32, i32p, i32, i32p, i32p, i32p, i32p, i32p,
                                          i32p, i32]
    lib.alr_debug_decode_plan.restype = ctypes.c_int
    lib.alr_profile_start.argtypes = [vp, i32, i32]
    lib.alr_profile_start.restype = ctypes.c_int
    lib.alr_profile_stop.argtypes = [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32)]
    lib.alr_profile_stop.restype = ctypes.c_int
    lib.alr_set_rollout_graphs.argtypes = [vp, i32]
    lib.alr_set_rollout_graphs.restype = ctypes.c_int
    _lib = lib
    return lib


def make_config(shape, max_pos: int) -> AlrConfig:
    c = AlrConfig()
    c.n_layers, c.d_model, c.n_heads = shape.n_layers, shape.d_model, shape.n_heads
    c.n_kv_heads, c.head_dim, c.d_ffn, c.vocab = (shape.n_kv_heads, shape.head_dim, shape.d_ffn,
                                                   shape.vocab)
    c.rms_eps, c.rope_base = shape.rms_eps, shape.rope_base
    c.dtype = ALR_BF16 if shape.dtype == "bf16" else ALR_F32
    c.max_pos = max_pos
    c.n_feat = len(shape.feat_layers)
    for i, f in enumerate(shape.feat_layers):
        c.feat_layers[i] = f
    for i, v in enumerate(getattr(shape, "mrope_sections", (0, 0, 0))):
        c.mrope_sections[i] = v
    return c


def make_limits(max_tokens: int, max_seqs: int, max_anchors: int, max_block: int) -> AlrLimits:
    lim = AlrLimits()
    lim.max_tokens, lim.max_seqs, lim.max_anchors, lim.max_block = (max_tokens, max_seqs,
                                                                    max_anchors, max_block)
    return lim


def _i32p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def check_rollout(shape, max_pos, limits: AlrLimits, seq_len: Sequence[int], anchor_seq,
                  anchor_pos, block: int):
    """Host-only validation of a rollout request (no GPU needed): (status, message)."""
    lib = load_library()
    cfg = make_config(shape, max_pos)
    sl = np.ascontiguousarray(seq_len, dtype=np.int32)
    a_s = np.ascontiguousarray(anchor_seq, dtype=np.int32)
    a_p = np.ascontiguousarray(anchor_pos, dtype=np.int32)
    buf = ctypes.create_string_buffer(256)
    st = lib.alr_check_rollout(ctypes.byref(cfg), ctypes.byref(limits), len(sl), _i32p(sl),
                               len(a_s), _i32p(a_s), _i32p(a_p), block, buf, 256)
    return st, buf.value.decode()


def decode_plan(shape, max_pos, n_cu: int, seq_len: Sequence[int], anchor_seq, anchor_pos,
                max_items: int = 1 << 16):
    """Host-only decode-attention work plan: (chunk tiles, makespan, items [n, 6] int32 with
    columns first sorted anchor, anchor count, kv head, first key, end key, partial index)."""
    lib = load_library()
    cfg = make_config(shape, max_pos)
    sl = np.ascontiguousarray(seq_len, dtype=np.int32)
    a_s = np.ascontiguousarray(anchor_seq, dtype=np.int32)
    a_p = np.ascontiguousarray(anchor_pos, dtype=np.int32)
    ct, span, n = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    items = np.zeros((max_items, 6), np.int32)
    st = lib.alr_debug_decode_plan(ctypes.byref(cfg), n_cu, len(sl), _i32p(sl), len(a_s),
                                   _i32p(a_s), _i32p(a_p), ctypes.byref(ct), ctypes.byref(span),
                                   ctypes.byref(n), _i32p(items), max_items)
    if st != 0:
        raise AlrError(st, "alr_debug_decode_plan")
    return ct.value, span.value, items[:n.value].copy()


class Engine:
    """One library context: weights repacked into a caller-owned workspace.

    ``weights`` is the generator's dict (numpy float32 or uint16 bf16 bits);
    they are uploaded, repacked by the library and released again.
    """

    def __init__(self, shape, weights: Dict, max_pos: int, limits: AlrLimits, device="cuda",
                 stream=None):
        import torch

        self.torch = torch
        self.lib = load_library()
        self.shape = shape
        self.device = torch.device(device)
        self.cfg = make_config(shape, max_pos)
        self.limits = limits
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        nbytes = self.lib.alr_workspace_bytes(ctypes.byref(self.cfg), ctypes.byref(limits))
        if nbytes == 0:
            buf = ctypes.create_string_buffer(256)
            st = self.lib.alr_check_config(ctypes.byref(self.cfg), buf, 256)
            raise AlrError(st or 1, buf.value.decode() or "invalid limits")
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self.ws_bytes = nbytes
        dev_w = self._upload_weights(weights)
        w = AlrWeights()
        keep = []

        def arr(name):
            a = (ctypes.c_void_p * max(1, shape.n_layers))(
                *[dev_w["layers"][l][name].data_ptr() for l in range(shape.n_layers)])
            keep.append(a)
            return ctypes.cast(a, _PP)

        w.tok_embed = dev_w["tok_embed"].data_ptr()
        w.final_norm = dev_w["final_norm"].data_ptr()
        w.lm_head = dev_w["lm_head"].data_ptr()
        for n in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down"):
            setattr(w, n, arr(n))
        ctx = ctypes.c_void_p()
        st = self.lib.alr_create(ctypes.byref(self.cfg), ctypes.byref(w), ctypes.byref(limits),
                                 self.workspace.data_ptr(), nbytes, self._sp(), ctypes.byref(ctx))
        if st != 0:
            raise AlrError(st, self.lib.alr_last_error(None).decode())
        self.ctx = ctx
        del dev_w, keep

    def _sp(self):
        return ctypes.c_void_p(self.stream.cuda_stream)

    def _to_dev(self, a: np.ndarray):
        torch = self.torch
        if a.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(self.device)
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(self.device)

    def _upload_weights(self, w: Dict) -> Dict:
        out = {k: self._to_dev(w[k]) for k in ("tok_embed", "final_norm", "lm_head")}
        out["layers"] = [{k: self._to_dev(v) for k, v in ld.items()} for ld in w["layers"]]
        return out

    def _err(self, st: int):
        raise AlrError(st, self.lib.alr_last_error(self.ctx).decode())

    def set_rollout_graphs(self, enable: bool):
        """alr_set_rollout_graphs: replay recorded launch graphs for repeated rollouts."""
        st = self.lib.alr_set_rollout_graphs(self.ctx, 1 if enable else 0)
        if st != 0:
            self._err(st)

    def close(self):
        if getattr(self, "ctx", None):
            self.lib.alr_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------------- calls
    def prefill(self, tokens, seq_len: Sequence[int], embeds=None, embed_mask=None,
                feats_out=None, positions=None):
        """tokens: device int32 tensor [sum seq_len]; embeds/embed_mask device tensors or None;
        positions: host int array [sum seq_len, 3] of (t, h, w) positions, or None."""
        sl = np.ascontiguousarray(seq_len, dtype=np.int32)
        self._seq_len = sl
        pos = None if positions is None else np.ascontiguousarray(positions, dtype=np.int32)
        st = self.lib.alr_prefill_positions(
            self.ctx, len(sl), _i32p(sl), tokens.data_ptr(), None if pos is None else _i32p(pos),
            None if embeds is None else embeds.data_ptr(),
            None if embed_mask is None else embed_mask.data_ptr(),
            None if feats_out is None else feats_out.data_ptr(), self._sp())
        if st != 0:
            self._err(st)

    def alloc_outputs(self, n_anchor: int, block: int, want_feats: bool = True):
        torch = self.torch
        tok = torch.empty((n_anchor, block), dtype=torch.int32, device=self.device)
        lp = torch.empty((n_anchor, block, self.shape.vocab), dtype=torch.float32,
                         device=self.device)
        ft = None
        if want_feats and self.shape.n_feat > 0:
            ft = torch.empty((n_anchor, block, self.shape.n_feat, self.shape.d_model),
                             dtype=torch.float32, device=self.device)
        return tok, lp, ft

    def rollout(self, anchor_seq, anchor_pos, block: int, forced=None, out=None,
                want_feats: bool = True):
        a_s = np.ascontiguousarray(anchor_seq, dtype=np.int32)
        a_p = np.ascontiguousarray(anchor_pos, dtype=np.int32)
        n = len(a_s)
        tok, lp, ft = out if out is not None else self.alloc_outputs(n, block, want_feats)
        st = self.lib.alr_rollout(self.ctx, n, _i32p(a_s), _i32p(a_p), block,
                                  None if forced is None else forced.data_ptr(), tok.data_ptr(),
                                  lp.data_ptr(), None if ft is None else ft.data_ptr(), self._sp())
        if st != 0:
            self._err(st)
        return tok, lp, ft


    def alloc_topk(self, n: int, block: int):
        torch = self.torch
        return (torch.empty((n, block, ALR_TOPK), dtype=torch.int32, device=self.device),
                torch.empty((n, block, ALR_TOPK), dtype=torch.float32, device=self.device),
                torch.empty((n, block), dtype=torch.float32, device=self.device))

    def rollout_topk(self, anchor_seq, anchor_pos, block: int, forced=None,
                     want_logprobs: bool = False, want_feats: bool = True, out=None):
        """-> (tokens, top_ids, top_logp, tail, logprobs or None, feats or None)."""
        torch = self.torch
        a_s = np.ascontiguousarray(anchor_seq, dtype=np.int32)
        a_p = np.ascontiguousarray(anchor_pos, dtype=np.int32)
        n = len(a_s)
        if out is None:
            tok = torch.empty((n, block), dtype=torch.int32, device=self.device)
            ti, tl, tt = self.alloc_topk(n, block)
            lp = (torch.empty((n, block, self.shape.vocab), dtype=torch.float32,
                              device=self.device) if want_logprobs else None)
            ft = None
            if want_feats and self.shape.n_feat > 0:
                ft = torch.empty((n, block, self.shape.n_feat, self.shape.d_model),
                                 dtype=torch.float32, device=self.device)
        else:
            tok, ti, tl, tt, lp, ft = out
        st = self.lib.alr_rollout_topk(
            self.ctx, n, _i32p(a_s), _i32p(a_p), block,
            None if forced is None else forced.data_ptr(), tok.data_ptr(), ti.data_ptr(),
            tl.data_ptr(), tt.data_ptr(), None if lp is None else lp.data_ptr(),
            None if ft is None else ft.data_ptr(), self._sp())
        if st != 0:
            self._err(st)
        return tok, ti, tl, tt, lp, ft

    def rollout_topk_noalloc(self, anchor_seq, anchor_pos, block: int, out, forced=None):
        """alr_rollout_topk_noalloc into caller tensors out = (tokens, top_ids, top_logp, tail,
        feats or None); the library's fixed scratch holds the per-step logits."""
        a_s = np.ascontiguousarray(anchor_seq, dtype=np.int32)
        a_p = np.ascontiguousarray(anchor_pos, dtype=np.int32)
        tok, ti, tl, tt, ft = out
        st = self.lib.alr_rollout_topk_noalloc(
            self.ctx, len(a_s), _i32p(a_s), _i32p(a_p), block,
            None if forced is None else forced.data_ptr(), tok.data_ptr(), ti.data_ptr(),
            tl.data_ptr(), tt.data_ptr(), None if ft is None else ft.data_ptr(), self._sp())
        if st != 0:
            self._err(st)
        return tok, ti, tl, tt, ft

    def corpus_labels(self, anchor_seq, anchor_pos, block: int, want_topk: bool = True,
                      want_logprobs: bool = False):
        """-> dict of argmax, top_ids, top_logp, tail, logprobs, corpus_logp, gate_soft,
        gate_hard (device tensors; absent forms are None)."""
        torch = self.torch
        a_s = np.ascontiguousarray(anchor_seq, dtype=np.int32)
        a_p = np.ascontiguousarray(anchor_pos, dtype=np.int32)
        n = len(a_s)
        f32 = dict(dtype=torch.float32, device=self.device)
        r = {"argmax": torch.empty((n, block), dtype=torch.int32, device=self.device),
             "top_ids": None, "top_logp": None, "tail": None, "logprobs": None,
             "corpus_logp": torch.empty((n, block), **f32),
             "gate_soft": torch.empty((n, block), **f32),
             "gate_hard": torch.empty((n, block), **f32)}
        if want_topk:
            r["top_ids"], r["top_logp"], r["tail"] = self.alloc_topk(n, block)
        if want_logprobs:
            r["logprobs"] = torch.empty((n, block, self.shape.vocab), **f32)
        ptr = (lambda t: None if t is None else t.data_ptr())
        st = self.lib.alr_corpus_labels(
            self.ctx, n, _i32p(a_s), _i32p(a_p), block, ptr(r["argmax"]), ptr(r["top_ids"]),
            ptr(r["top_logp"]), ptr(r["tail"]), ptr(r["logprobs"]), ptr(r["corpus_logp"]),
            ptr(r["gate_soft"]), ptr(r["gate_hard"]), self._sp())
        if st != 0:
            self._err(st)
        return r

    def ira_assemble(self, tokens, top_ids, top_logp, tail, sec_primary, sec_offset,
                     gamma: float = 2.0, eos_id: int = -1):
        """Secondary blocks from primary rollout labels -> (token0, top_ids, top_logp, tail,
        weight) device tensors."""
        torch = self.torch
        n_prim, block = tokens.shape
        sp = np.ascontiguousarray(sec_primary, dtype=np.int32)
        so = np.ascontiguousarray(sec_offset, dtype=np.int32)
        q = len(sp)
        t0 = torch.empty(q, dtype=torch.int32, device=self.device)
        ti, tl, tt = self.alloc_topk(q, block)
        w = torch.empty((q, block), dtype=torch.float32, device=self.device)
        st = self.lib.alr_ira_assemble(self.ctx, n_prim, block, tokens.data_ptr(),
                                       top_ids.data_ptr(), top_logp.data_ptr(), tail.data_ptr(),
                                       q, _i32p(sp), _i32p(so), gamma, eos_id, t0.data_ptr(),
                                       ti.data_ptr(), tl.data_ptr(), tt.data_ptr(), w.data_ptr(),
                                       self._sp())
        if st != 0:
            self._err(st)
        return t0, ti, tl, tt, w

    def slot_weights(self, tokens, eos_id: int = -1, gamma: float = 2.0):
        """ALR slot weights [n, block] from rollout tokens (device int32 [n, block])."""
        torch = self.torch
        n, block = tokens.shape
        w = torch.empty((n, block), dtype=torch.float32, device=self.device)
        st = self.lib.alr_slot_weights(self.ctx, n, block, tokens.data_ptr(), eos_id, gamma,
                                       w.data_ptr(), self._sp())
        if st != 0:
            self._err(st)
        return w


PROF_SITES = {"prefill_qkv": 1, "prefill_attn": 2, "prefill_o": 3, "prefill_gu": 4,
              "prefill_down": 5, "decode_qkv": 6, "decode_attn": 7, "decode_o": 8, "decode_gu": 9,
              "decode_down": 10, "lm_gemm": 11, "lm_finalize": 12, "decode_combine": 13}


def profile_start(eng: "Engine", site: str, capacity: int = 4096):
    st = eng.lib.alr_profile_start(eng.ctx, PROF_SITES[site], capacity)
    if st != 0:
        eng._err(st)


def profile_stop(eng: "Engine"):
    """-> (total device ms, number of timed launches)"""
    ms = ctypes.c_double()
    n = ctypes.c_int32()
    st = eng.lib.alr_profile_stop(eng.ctx, ctypes.byref(ms), ctypes.byref(n))
    if st != 0:
        eng._err(st)
    return ms.value, n.value


def debug_gemm(dtype: int, A, W, C, stream=None, tile: int = 0):
    """C = A W^T on the library's GEMM kernel (device tensors, fp32 C)."""
    import torch

    lib = load_library()
    s = stream if stream is not None else torch.cuda.current_stream()
    M, K = A.shape
    N = W.shape[0]
    scratch = None
    nbytes = 0
    if dtype == ALR_BF16 and tile in (18, 20):
        nbytes = 4 * M * N * 4
        scratch = torch.empty(nbytes, dtype=torch.uint8, device=A.device)
    st = lib.alr_debug_gemm(dtype, A.data_ptr(), W.data_ptr(), C.data_ptr(), M, N, K, tile,
                            None if scratch is None else scratch.data_ptr(), nbytes,
                            ctypes.c_void_p(s.cuda_stream))
    if st != 0:
        raise AlrError(st, "alr_debug_gemm")
