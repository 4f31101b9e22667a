"""Host-side checks of the C ABI: the library loads, exports every declared symbol,
and rejects bad arguments before touching the GPU (no compute calls here)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2609_38795_amd import binding, workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in ("alr.h", "alr_debug.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        names |= set(re.findall(r"\b(alr_[a-z_]+)\s*\(", src))
    return names


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.LIB_PATH):
        from paper_2609_38795_amd import build
        build.build()
    return binding.load_library()


def test_every_declared_symbol_is_exported(lib):
    declared = _declared()
    assert declared == set(binding.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code, name in binding.STATUS.items():
        assert lib.alr_status_string(code).decode() == name


def _cfg(name="small_bf16"):
    w = W.get(name)
    return w, binding.make_config(w.shape, w.max_pos)


def test_config_checks(lib):
    w, cfg = _cfg()
    buf = ctypes.create_string_buffer(256)
    assert lib.alr_check_config(ctypes.byref(cfg), buf, 256) == 0
    bad = binding.make_config(W.scaled(w, "x", n_kv_heads=3).shape, w.max_pos)
    assert lib.alr_check_config(ctypes.byref(bad), buf, 256) == 1
    assert b"n_kv_heads" in buf.value
    bad = binding.make_config(W.scaled(w, "x", d_model=1000).shape, w.max_pos)
    assert lib.alr_check_config(ctypes.byref(bad), buf, 256) == 5
    bad = binding.make_config(W.scaled(w, "x", feat_layers=(1, 9)).shape, w.max_pos)
    assert lib.alr_check_config(ctypes.byref(bad), buf, 256) == 2
    bad = binding.make_config(W.scaled(w, "x", feat_layers=(1, 1)).shape, w.max_pos)
    assert lib.alr_check_config(ctypes.byref(bad), buf, 256) == 1
    bad = binding.make_config(w.shape, w.max_pos)
    bad.dtype = 7
    assert lib.alr_check_config(ctypes.byref(bad), buf, 256) == 1
    # multimodal RoPE sections: all zero, or non-negative with sum head_dim/2 (= 32 here)
    ok = binding.make_config(W.scaled(w, "x", mrope_sections=(8, 12, 12)).shape, w.max_pos)
    assert lib.alr_check_config(ctypes.byref(ok), buf, 256) == 0
    for secs in ((8, 12, 11), (-2, 17, 17), (0, 0, 33)):
        bad = binding.make_config(W.scaled(w, "x", mrope_sections=secs).shape, w.max_pos)
        assert lib.alr_check_config(ctypes.byref(bad), buf, 256) == 1
        assert b"mrope_sections" in buf.value


def test_workspace_bytes_monotone_and_zero_on_invalid(lib):
    w, cfg = _cfg()
    l1 = binding.make_limits(4096, 2, 64, 16)
    l2 = binding.make_limits(8192, 4, 256, 16)
    b1 = lib.alr_workspace_bytes(ctypes.byref(cfg), ctypes.byref(l1))
    b2 = lib.alr_workspace_bytes(ctypes.byref(cfg), ctypes.byref(l2))
    assert 0 < b1 < b2 and b1 % 256 == 0
    assert b1 > 2 * w.shape.n_params()  # bf16 weights are repacked into the workspace
    assert lib.alr_workspace_bytes(ctypes.byref(cfg), ctypes.byref(binding.make_limits(0, 1, 1, 1))) == 0


def test_workspace_fits_long_context_workload_on_one_gpu(lib):
    w = W.get("long_ctx_8b")
    cfg = binding.make_config(w.shape, w.max_pos)
    lim = binding.make_limits(w.n_tokens, w.n_seq, w.n_anchors, w.block)
    b = lib.alr_workspace_bytes(ctypes.byref(cfg), ctypes.byref(lim))
    assert 0 < b < 200 * 2 ** 30


def test_rollout_checks(lib):
    w = W.get("small_bf16")
    lim = binding.make_limits(w.n_tokens, w.n_seq, w.n_anchors, w.block)
    seq_len = [w.seq_len] * w.n_seq
    a_s, a_p = W.make_anchors(w)
    st, msg = binding.check_rollout(w.shape, w.max_pos, lim, seq_len, a_s, a_p, w.block)
    assert st == 0, msg
    bad_p = a_p.copy()
    bad_p[3] = w.seq_len
    st, msg = binding.check_rollout(w.shape, w.max_pos, lim, seq_len, a_s, bad_p, w.block)
    assert st == 2 and "anchor 3" in msg
    bad_s = a_s.copy()
    bad_s[0] = w.n_seq
    assert binding.check_rollout(w.shape, w.max_pos, lim, seq_len, bad_s, a_p, w.block)[0] == 2
    bad_s[0] = -1
    assert binding.check_rollout(w.shape, w.max_pos, lim, seq_len, bad_s, a_p, w.block)[0] == 2
    assert binding.check_rollout(w.shape, w.max_pos, lim, seq_len, a_s, a_p, 0)[0] == 1
    assert binding.check_rollout(w.shape, w.max_pos, lim, seq_len, a_s, a_p, w.block + 1)[0] == 1
    # the last slot must stay below max_pos
    st, msg = binding.check_rollout(w.shape, w.seq_len, lim, seq_len, a_s, a_p, w.block)
    assert st == 2 and "max_pos" in msg
    # too many anchors for the context's limits
    lim_small = binding.make_limits(w.n_tokens, w.n_seq, 8, w.block)
    assert binding.check_rollout(w.shape, w.max_pos, lim_small, seq_len, a_s, a_p, w.block)[0] == 1
    # an empty request is an argument error, not a silent no-op
    st, msg = binding.check_rollout(w.shape, w.max_pos, lim, seq_len, a_s[:0], a_p[:0], w.block)
    assert st == 1 and "n_anchor 0" in msg


def test_create_rejects_bad_arguments_without_gpu(lib):
    w, cfg = _cfg("tiny_fp32")
    lim = binding.make_limits(128, 1, 8, 4)
    ctx = ctypes.c_void_p()
    wts = binding.AlrWeights()
    st = lib.alr_create(ctypes.byref(cfg), ctypes.byref(wts), ctypes.byref(lim), None, 0, None,
                        ctypes.byref(ctx))
    assert st == 1 and not ctx.value
    assert b"tok_embed" in lib.alr_last_error(None)
    st = lib.alr_create(ctypes.byref(cfg), None, ctypes.byref(lim), None, 0, None, ctypes.byref(ctx))
    assert st == 1


def test_rollout_and_prefill_reject_null_context(lib):
    z = np.zeros(1, np.int32)
    assert lib.alr_rollout(None, 1, binding._i32p(z), binding._i32p(z), 1, None, None, None,
                           None, None) == 1
    assert lib.alr_prefill(None, 1, binding._i32p(z), None, None, None, None, None) == 1


def test_graph_switch_rejects_null_context(lib):
    assert lib.alr_set_rollout_graphs(None, 1) == 1  # ALR_E_INVALID_ARG
    assert lib.alr_set_rollout_graphs(None, 0) == 1


def test_operands_of_4gib_are_rejected(lib):
    """The bf16 GEMM kernels address operand chunks by 32-bit byte offsets: a context whose
    activation operand (max(max_tokens, max_anchors) rows of max(d, F, H hd) bf16) or any weight
    matrix reaches 4 GiB is refused before anything is allocated or launched."""
    w, cfg = _cfg("llama8b_like")
    F = w.shape.d_ffn
    r_ok = (2 ** 32 - 1) // (2 * F)  # largest row count whose F-wide bf16 operand is < 4 GiB
    ok = binding.make_limits(r_ok, 8, 1024, 16)
    assert lib.alr_workspace_bytes(ctypes.byref(cfg), ctypes.byref(ok)) > 0
    for lim in (binding.make_limits(r_ok + 1, 8, 1024, 16),
                binding.make_limits(4096, 8, r_ok + 1, 16)):
        assert lib.alr_workspace_bytes(ctypes.byref(cfg), ctypes.byref(lim)) == 0
        ctx = ctypes.c_void_p()
        st = lib.alr_create(ctypes.byref(cfg), ctypes.byref(binding.AlrWeights()), ctypes.byref(lim),
                            None, 0, None, ctypes.byref(ctx))
        assert st == 5 and not ctx.value
        assert b"4 GiB" in lib.alr_last_error(None)
    # a weight matrix of 4 GiB: vocab x d_model bf16
    big = binding.make_config(W.scaled(w, "x", vocab=2 ** 31 // w.shape.d_model).shape, w.max_pos)
    assert lib.alr_workspace_bytes(ctypes.byref(big), ctypes.byref(ok)) == 0
    # fp32 contexts use the FMA kernel with 64-bit offsets: no such limit
    wf, cf = _cfg("tiny_fp32")
    assert lib.alr_workspace_bytes(ctypes.byref(cf), ctypes.byref(binding.make_limits(200000, 1, 8, 4))) > 0
