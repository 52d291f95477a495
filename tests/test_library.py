"""The C-ABI library builds for gfx950, loads without a GPU and exports every declared symbol."""
import ctypes
import os
import re

import pytest

import paper_2604_09603_amd as pkg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    with open(os.path.join(ROOT, "include", "echo.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:int32_t|size_t|const char\*)\s+(echo_\w+)\(", text, re.M)))


def test_header_and_binding_agree():
    assert _declared() == sorted(pkg.EXPORTS)


def test_library_exports_every_symbol():
    if not os.path.exists(pkg.LIB_PATH):
        pytest.skip("libecho.so not built (run __graft_entry__.build())")
    lib = ctypes.CDLL(pkg.LIB_PATH)
    for name in _declared():
        assert hasattr(lib, name), name
    lib = pkg.load()
    assert "gfx950" in pkg.version()
    assert pkg.status_string(pkg.ERR_WORKSPACE).startswith("workspace")


def test_host_side_errors_need_no_gpu():
    """Argument checks run on the host and return before touching the device."""
    if not os.path.exists(pkg.LIB_PATH):
        pytest.skip("libecho.so not built")
    lib = pkg.load()
    P = ctypes.c_void_p
    # R = 0, negative budget, head_dim != 128, Hq % Hkv != 0, max_depth > 16
    assert lib.echo_gate(None, None, None, 0, 0, 0, None, None, None, None, 0, None, None) == pkg.ERR_INVALID_ARG
    assert lib.echo_gate(P(8), P(8), P(8), 1, 1, -1, None, P(8), P(8), P(256), 1 << 20, None, None) == pkg.ERR_INVALID_ARG
    assert lib.echo_gate(P(256), P(256), P(256), 1, 1, 4, None, P(256), P(256), P(256), 0, None, None) == pkg.ERR_WORKSPACE
    # sparse gating: checkpoint depth outside 1..16, NaN ln tau, too many checkpoints
    I = lambda *v: ctypes.cast((ctypes.c_int32 * len(v))(*v), P)
    F = lambda *v: ctypes.cast((ctypes.c_float * len(v))(*v), P)
    ws = lib.echo_gate_sparse_workspace_size(1, 1, 4)
    assert ws == lib.echo_gate_workspace_size(1, 1, 4)
    sparse = lambda d, t, n: lib.echo_gate_sparse(P(256), P(256), P(256), 1, 1, 4, d, t, n, None,
                                                  P(256), P(256), None, P(256), ws, None, None)
    assert sparse(I(0), F(-1.0), 1) == pkg.ERR_INVALID_ARG
    assert sparse(I(17), F(-1.0), 1) == pkg.ERR_INVALID_ARG
    assert sparse(I(2), F(float("nan")), 1) == pkg.ERR_INVALID_ARG
    assert sparse(I(*range(1, 18)), F(*([-1.0] * 17)), 17) == pkg.ERR_INVALID_ARG
    assert sparse(None, None, 1) == pkg.ERR_INVALID_ARG
    assert lib.echo_gate_sparse(P(256), P(256), P(256), 1, 1, 4, I(2), F(-1.0), 1, None, P(256),
                                P(256), None, P(256), ws - 1, None, None) == pkg.ERR_WORKSPACE
    # elastic scheduler: w_topk < 1, w_max < 0, bad checkpoint, workspace too small
    wse = lib.echo_gate_elastic_workspace_size(1, 1, 4)
    assert wse > ws
    elastic = lambda d, t, n, wt, wm, sz: lib.echo_gate_elastic(
        P(256), P(256), P(256), 1, 1, 4, d, t, n, wt, wm, None, P(256), P(256), None, P(256), sz,
        None, None)
    assert elastic(I(2), F(-1.0), 1, 0, 4, wse) == pkg.ERR_INVALID_ARG
    assert elastic(I(2), F(-1.0), 1, 2, -1, wse) == pkg.ERR_INVALID_ARG
    assert elastic(I(0), F(-1.0), 1, 2, 4, wse) == pkg.ERR_INVALID_ARG
    assert elastic(I(2), F(float("nan")), 1, 2, 4, wse) == pkg.ERR_INVALID_ARG
    assert elastic(I(2), F(-1.0), 1, 2, 4, wse - 1) == pkg.ERR_WORKSPACE
    # paged attention: page size not a power of two >= 32, missing block table
    wsa = lib.echo_tree_verify_attn_workspace_size(1, 4, 8, 8, 128)
    paged = lambda page, bt: lib.echo_tree_verify_attn_paged(
        P(256), P(256), P(256), P(256), P(256), 8, page, bt, 4, P(256), P(256), P(256), 1, 1, 4,
        8, 8, 128, 1.0, P(256), None, P(256), wsa, None, None)
    assert paged(48, P(256)) == pkg.ERR_UNSUPPORTED
    assert paged(16, P(256)) == pkg.ERR_UNSUPPORTED
    assert paged(64, None) == pkg.ERR_INVALID_ARG
    # acceptance from logits: vocab < 1, missing target output
    al = lambda vocab, tgt: lib.echo_accept_logits(P(256), P(256), P(256), P(256), vocab, 1, 4, 4,
                                                   tgt, P(256), P(256), P(256), None, None)
    assert al(0, P(256)) == pkg.ERR_INVALID_ARG
    assert al(100, None) == pkg.ERR_INVALID_ARG
    # commit: misaligned K/V, max_depth out of range
    cm = lambda kn, depth: lib.echo_commit_kv(P(256), P(256), P(256), depth, kn, P(256), 1, 4, 1,
                                              P(256), P(256), 8, 16, P(256), 4, P(256), None, None)
    assert cm(P(258), 4) == pkg.ERR_INVALID_ARG
    assert cm(P(256), 17) == pkg.ERR_UNSUPPORTED
    assert lib.echo_tree_verify_attn_workspace_size(4, 20, 8, 8, 64) == 0
    assert lib.echo_tree_verify_attn(P(16), P(16), P(16), P(16), P(16), P(16), 10, P(16), P(16), 1,
                                     1, 4, 6, 4, 128, 1.0, P(16), None, P(256), 1 << 30, None,
                                     None) == pkg.ERR_INVALID_ARG
    assert lib.echo_tree_verify_attn(P(16), P(16), P(16), P(16), P(16), P(16), 10, P(16), P(16), 1,
                                     1, 4, 8, 8, 64, 1.0, P(16), None, P(256), 1 << 30, None,
                                     None) == pkg.ERR_UNSUPPORTED
    assert lib.echo_accept(P(8), P(8), P(8), P(8), 1, 4, 17, P(8), P(8), P(8), None, None) == pkg.ERR_UNSUPPORTED
    assert lib.echo_build_tree_mask(P(8), P(8), P(8), P(8), P(8), P(8), 1, 1, 64, P(8), P(8), P(8),
                                    P(8), P(8), P(8), 1, None, 0, None, None) == pkg.ERR_INVALID_ARG


def test_attention_scale_and_timing_events_checked_on_host():
    """sm_scale must be finite and positive (the softmax takes the largest raw logit
    of a row as its reference before scaling); the timed entry points need both
    events; the read probe checks its mode and head count.  All host-side."""
    if not os.path.exists(pkg.LIB_PATH):
        pytest.skip("libecho.so not built")
    lib = pkg.load()
    P = ctypes.c_void_p
    ws = lib.echo_tree_verify_attn_workspace_size(1, 4, 8, 8, 128)
    attn = lambda scale: lib.echo_tree_verify_attn(
        P(256), P(256), P(256), P(256), P(256), P(256), 10, P(256), P(256), 1, 1, 4, 8, 8, 128,
        scale, P(256), None, P(256), ws, None, None)
    paged = lambda scale: lib.echo_tree_verify_attn_paged(
        P(256), P(256), P(256), P(256), P(256), 8, 64, P(256), 4, P(256), P(256), P(256), 1, 1, 4,
        8, 8, 128, scale, P(256), None, P(256), ws, None, None)
    for bad in (0.0, -0.125, float("nan"), float("inf"), -float("inf")):
        assert attn(bad) == pkg.ERR_INVALID_ARG, bad
        assert paged(bad) == pkg.ERR_INVALID_ARG, bad
    timed = lambda a, b: lib.echo_tree_verify_attn_timed(
        P(256), P(256), P(256), P(256), P(256), P(256), 10, P(256), P(256), 1, 1, 4, 8, 8, 128,
        0.088, P(256), None, P(256), ws, None, a, b, None)
    assert timed(None, None) == pkg.ERR_INVALID_ARG
    assert timed(P(256), None) == pkg.ERR_INVALID_ARG
    assert timed(None, P(256)) == pkg.ERR_INVALID_ARG
    ptimed = lambda a, b: lib.echo_tree_verify_attn_paged_timed(
        P(256), P(256), P(256), P(256), P(256), 8, 64, P(256), 4, P(256), P(256), P(256), 1, 1, 4,
        8, 8, 128, 0.088, P(256), None, P(256), ws, None, a, b, None)
    assert ptimed(None, P(256)) == pkg.ERR_INVALID_ARG
    # the timed calls check their other arguments exactly as the untimed ones
    timed_bad_scale = lib.echo_tree_verify_attn_timed(
        P(256), P(256), P(256), P(256), P(256), P(256), 10, P(256), P(256), 1, 1, 4, 8, 8, 128,
        -1.0, P(256), None, P(256), ws, None, P(256), P(256), None)
    assert timed_bad_scale == pkg.ERR_INVALID_ARG
    probe = lambda heads, mode, k=P(256): lib.echo_probe_stream_read(k, P(256), 64, heads, mode,
                                                                     P(256), None)
    assert probe(4, 3) == pkg.ERR_INVALID_ARG
    assert lib.echo_probe_stream_read(P(256), P(256), 7, 1, 2, P(256), None) == pkg.ERR_UNSUPPORTED
    assert probe(6, 1) == pkg.ERR_UNSUPPORTED
    assert probe(4, 0, P(264)) == pkg.ERR_INVALID_ARG
    assert probe(0, 0) == pkg.ERR_INVALID_ARG


def test_verify_step_checked_on_host():
    """echo_verify_step runs every check of the four calls before it launches
    anything: each failing check gives that call's code (no GPU needed)."""
    if not os.path.exists(pkg.LIB_PATH):
        pytest.skip("libecho.so not built")
    lib = pkg.load()
    P = ctypes.c_void_p
    R, N, B, W, cap = 1, 4, 4, 1, 5
    gws = lib.echo_gate_workspace_size(R, N, B)
    aws = lib.echo_tree_verify_attn_workspace_size(R, cap, 8, 8, 128)
    base = dict(cand_offsets=P(256), parent=P(256), logq=P(256), token=P(256), R=R, N=N,
                budget=B, path_score=None, selected=P(256), num_selected=P(256),
                gate_ws=P(256), gate_ws_bytes=gws, root_token=P(256), prefix_len=P(256),
                q_offsets=P(256), slot_cand=P(256), slot_parent=P(256), slot_token=P(256),
                position_ids=P(256), tree_mask=P(256), mask_words=W, q=P(256), k_new=P(256),
                v_new=P(256), k_cache=P(256), v_cache=P(256), kv_offsets=P(256), kv_rows=10,
                max_rows=cap, hq=8, hkv=8, head_dim=128, scale=0.088, out=P(256), lse=None,
                attn_ws=P(256), attn_ws_bytes=aws, target=P(256), max_depth=4,
                accept_len=P(256), accept_slots=P(256), bonus=P(256), status=None, stream=None)

    def step(**kw):
        a = dict(base, **kw)
        return lib.echo_verify_step(*a.values())

    assert step(R=0) == pkg.ERR_INVALID_ARG
    assert step(budget=16385) == pkg.ERR_UNSUPPORTED                 # ECHO_MAX_BUDGET + 1
    assert step(token=None) == pkg.ERR_INVALID_ARG                  # the mask's tokens
    assert step(gate_ws=P(257)) == pkg.ERR_WORKSPACE
    assert step(gate_ws_bytes=gws - 1) == pkg.ERR_WORKSPACE
    assert step(mask_words=0) == pkg.ERR_INVALID_ARG
    assert step(tree_mask=None) == pkg.ERR_INVALID_ARG
    assert step(head_dim=64) == pkg.ERR_UNSUPPORTED
    assert step(hq=6, hkv=4) == pkg.ERR_INVALID_ARG
    assert step(scale=-1.0) == pkg.ERR_INVALID_ARG
    assert step(q=P(264)) == pkg.ERR_INVALID_ARG                     # not 16-byte aligned
    assert step(attn_ws_bytes=aws - 1) == pkg.ERR_WORKSPACE
    assert step(max_depth=0) == pkg.ERR_INVALID_ARG
    assert step(max_depth=pkg.MAX_DEPTH + 1) == pkg.ERR_UNSUPPORTED
    assert step(bonus=None) == pkg.ERR_INVALID_ARG
    assert step(target=None) == pkg.ERR_INVALID_ARG
    assert len(base) == 44
