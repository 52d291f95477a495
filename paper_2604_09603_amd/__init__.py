"""MI355X (gfx950) batch super-tree verification: Python binding of libecho.

The four calls of one verification step live in ``libecho.so`` (HIP kernels
behind a C ABI, declared in ``include/echo.h``).  This module only marshals
arguments: torch device tensors are passed as raw pointers together with the
current HIP stream.  There is no CPU fallback: if the library is missing or
cannot be loaded every call raises.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libecho.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_UNSUPPORTED = -2
ERR_WORKSPACE = -3
ERR_HIP = -4

DATA_NAN_LOGQ = 1 << 0
DATA_POS_LOGQ = 1 << 1
DATA_BAD_PARENT = 1 << 2
DATA_TOO_DEEP = 1 << 3
DATA_NOT_CLOSED = 1 << 4
DATA_OVER_CAPACITY = 1 << 5
DATA_BAD_SLOT_PARENT = 1 << 6
DATA_BAD_OFFSETS = 1 << 7

MAX_DEPTH = 16
MAX_CHECKPOINTS = 16
HEAD_DIM = 128

EXPORTS = [
    "echo_gate", "echo_gate_workspace_size", "echo_gate_sparse", "echo_gate_sparse_workspace_size",
    "echo_gate_elastic", "echo_gate_elastic_workspace_size",
    "echo_build_tree_mask", "echo_build_tree_mask_workspace_size",
    "echo_tree_verify_attn", "echo_tree_verify_attn_workspace_size",
    "echo_tree_verify_attn_paged", "echo_accept_logits", "echo_commit_kv",
    "echo_accept", "echo_tree_verify_attn_timed", "echo_tree_verify_attn_paged_timed",
    "echo_probe_stream_read", "echo_gate_noalloc", "echo_verify_step", "echo_status_string",
    "echo_version",
]
GATE_SCRATCH_BYTES = 8 << 20

_lib = None

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_F32 = ctypes.c_float

_SIGS = {
    "echo_gate": (_I32, [_P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _P, _SZ, _P, _P]),
    "echo_gate_workspace_size": (_SZ, [_I32, _I32, _I32]),
    "echo_gate_noalloc": (_I32, [_P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _P, _P]),
    "echo_gate_sparse": (_I32, [_P, _P, _P, _I32, _I32, _I32, _P, _P, _I32, _P, _P, _P, _P, _P,
                                _SZ, _P, _P]),
    "echo_gate_sparse_workspace_size": (_SZ, [_I32, _I32, _I32]),
    "echo_gate_elastic": (_I32, [_P, _P, _P, _I32, _I32, _I32, _P, _P, _I32, _I32, _I32, _P, _P,
                                 _P, _P, _P, _SZ, _P, _P]),
    "echo_gate_elastic_workspace_size": (_SZ, [_I32, _I32, _I32]),
    "echo_build_tree_mask": (_I32, [_P, _P, _P, _P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P,
                                    _I32, _P, _SZ, _P, _P]),
    "echo_build_tree_mask_workspace_size": (_SZ, [_I32, _I32, _I32]),
    "echo_tree_verify_attn": (_I32, [_P, _P, _P, _P, _P, _P, _I64, _P, _P, _I32, _I32, _I32, _I32,
                                     _I32, _I32, _F32, _P, _P, _P, _SZ, _P, _P]),
    "echo_tree_verify_attn_workspace_size": (_SZ, [_I32, _I32, _I32, _I32, _I32]),
    "echo_accept": (_I32, [_P, _P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _P, _P]),
    "echo_tree_verify_attn_paged": (_I32, [_P, _P, _P, _P, _P, _I64, _I32, _P, _I32, _P, _P, _P,
                                           _I32, _I32, _I32, _I32, _I32, _I32, _F32, _P, _P, _P,
                                           _SZ, _P, _P]),
    "echo_accept_logits": (_I32, [_P, _P, _P, _P, _I64, _I32, _I32, _I32, _P, _P, _P, _P, _P,
                                  _P]),
    "echo_commit_kv": (_I32, [_P, _P, _P, _I32, _P, _P, _I32, _I32, _I32, _P, _P, _I64, _I32, _P,
                              _I32, _P, _P, _P]),
    "echo_tree_verify_attn_timed": (_I32, [_P, _P, _P, _P, _P, _P, _I64, _P, _P, _I32, _I32, _I32,
                                           _I32, _I32, _I32, _F32, _P, _P, _P, _SZ, _P, _P, _P,
                                           _P]),
    "echo_tree_verify_attn_paged_timed": (_I32, [_P, _P, _P, _P, _P, _I64, _I32, _P, _I32, _P, _P,
                                                 _P, _I32, _I32, _I32, _I32, _I32, _I32, _F32, _P,
                                                 _P, _P, _SZ, _P, _P, _P, _P]),
    "echo_probe_stream_read": (_I32, [_P, _P, _I64, _I32, _I32, _P, _P]),
    "echo_verify_step": (_I32, [_P, _P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _P, _SZ,
                                _P, _P, _P, _P, _P, _P, _P, _P, _I32,
                                _P, _P, _P, _P, _P, _P, _I64, _I32, _I32, _I32, _I32, _F32, _P,
                                _P, _P, _SZ,
                                _P, _I32, _P, _P, _P, _P, _P]),
    "echo_status_string": (ctypes.c_char_p, [_I32]),
    "echo_version": (ctypes.c_char_p, []),
}


class EchoError(RuntimeError):
    pass


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libecho (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise EchoError(f"{path} is missing: build it with "
                        "`python -m paper_2604_09603_amd.build` (there is no CPU fallback)")
    # torch ships its own HIP runtime under the same soname; load it first so that the
    # library and torch's streams and allocations share one runtime instance
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check(code: int, what: str):
    if code != OK:
        raise EchoError(f"{what}: {load().echo_status_string(code).decode()} ({code})")


def _event(e):
    return ctypes.c_void_p(e.cuda_event)


def echo_probe_stream_read(k, v, rows, heads, mode, sink, stream=None, check=True):
    """Measurement helper: read two [rows, heads, 128] bf16 tensors once (mode 0: plain
    vector loads; mode 1: the attention's tile copies into LDS)."""
    code = load().echo_probe_stream_read(_ptr(k), _ptr(v), int(rows), int(heads), int(mode),
                                         _ptr(sink), _stream(stream))
    if check:
        _check(code, "echo_probe_stream_read")
    return code


def version() -> str:
    return load().echo_version().decode()


def status_string(code: int) -> str:
    return load().echo_status_string(code).decode()


def gate_workspace_size(R, N, budget) -> int:
    return int(load().echo_gate_workspace_size(R, N, budget))


def build_tree_mask_workspace_size(R, N, budget) -> int:
    return int(load().echo_build_tree_mask_workspace_size(R, N, budget))


def tree_verify_attn_workspace_size(R, max_rows, hq, hkv, head_dim=HEAD_DIM) -> int:
    return int(load().echo_tree_verify_attn_workspace_size(R, max_rows, hq, hkv, head_dim))


def echo_gate(cand_offsets, parent, logq, R, N, budget, path_score, selected, num_selected,
              workspace, status=None, stream=None, check=True):
    """Path scores and global top-B selection (eq. 5, eq. 4).  Device tensors."""
    code = load().echo_gate(_ptr(cand_offsets), _ptr(parent), _ptr(logq), R, N, budget,
                            _ptr(path_score), _ptr(selected), _ptr(num_selected), _ptr(workspace),
                            workspace.numel() * workspace.element_size(), _ptr(status),
                            _stream(stream))
    if check:
        _check(code, "echo_gate")
    return code


def echo_gate_noalloc(cand_offsets, parent, logq, R, N, budget, path_score, selected,
                      num_selected, status=None, stream=None, check=True):
    """echo_gate with the library's fixed per-device workspace (no allocation;
    overlapping calls on one device race)."""
    code = load().echo_gate_noalloc(_ptr(cand_offsets), _ptr(parent), _ptr(logq), R, N, budget,
                                    _ptr(path_score), _ptr(selected), _ptr(num_selected),
                                    _ptr(status), _stream(stream))
    if check:
        _check(code, "echo_gate_noalloc")
    return code


def echo_gate_sparse(cand_offsets, parent, logq, R, N, budget, sig_depth, log_tau, path_score,
                     selected, num_selected, workspace, trunc_depth=None, status=None,
                     stream=None, check=True):
    """Sparse checkpoint gating (eq. 6-7) then the global top-B.  ``sig_depth`` and
    ``log_tau`` are host sequences (checkpoint depths and ln tau); the rest are
    device tensors."""
    n = len(sig_depth)
    if len(log_tau) != n:
        raise ValueError("sig_depth and log_tau differ in length")
    depths = (ctypes.c_int32 * max(n, 1))(*[int(x) for x in sig_depth])
    taus = (ctypes.c_float * max(n, 1))(*[float(x) for x in log_tau])
    code = load().echo_gate_sparse(_ptr(cand_offsets), _ptr(parent), _ptr(logq), R, N, budget,
                                   ctypes.cast(depths, _P), ctypes.cast(taus, _P), n,
                                   _ptr(path_score), _ptr(selected), _ptr(num_selected),
                                   _ptr(trunc_depth), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _ptr(status),
                                   _stream(stream))
    if check:
        _check(code, "echo_gate_sparse")
    return code


def gate_elastic_workspace_size(R, N, budget) -> int:
    return int(load().echo_gate_elastic_workspace_size(R, N, budget))


def echo_gate_elastic(cand_offsets, parent, logq, R, N, budget, sig_depth, log_tau, w_topk, w_max,
                      path_score, selected, num_selected, workspace, trunc_depth=None,
                      status=None, stream=None, check=True):
    """Alg. 1's elastic budget scheduler as a selection.  ``sig_depth`` and
    ``log_tau`` are host sequences; the rest are device tensors."""
    n = len(sig_depth)
    if len(log_tau) != n:
        raise ValueError("sig_depth and log_tau differ in length")
    depths = (ctypes.c_int32 * max(n, 1))(*[int(x) for x in sig_depth])
    taus = (ctypes.c_float * max(n, 1))(*[float(x) for x in log_tau])
    code = load().echo_gate_elastic(_ptr(cand_offsets), _ptr(parent), _ptr(logq), R, N, budget,
                                    ctypes.cast(depths, _P), ctypes.cast(taus, _P), n, w_topk,
                                    w_max, _ptr(path_score), _ptr(selected), _ptr(num_selected),
                                    _ptr(trunc_depth), _ptr(workspace),
                                    workspace.numel() * workspace.element_size(), _ptr(status),
                                    _stream(stream))
    if check:
        _check(code, "echo_gate_elastic")
    return code


def echo_build_tree_mask(cand_offsets, parent, token, selected, root_token, prefix_len, R, N,
                         budget, q_offsets, slot_cand, slot_parent, slot_token, position_ids,
                         tree_mask, mask_words, workspace=None, status=None, stream=None,
                         check=True):
    """Flatten & pack the selection into verify slots.  Device tensors."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    code = load().echo_build_tree_mask(
        _ptr(cand_offsets), _ptr(parent), _ptr(token), _ptr(selected), _ptr(root_token),
        _ptr(prefix_len), R, N, budget, _ptr(q_offsets), _ptr(slot_cand), _ptr(slot_parent),
        _ptr(slot_token), _ptr(position_ids), _ptr(tree_mask), mask_words, _ptr(workspace),
        ws_bytes, _ptr(status), _stream(stream))
    if check:
        _check(code, "echo_build_tree_mask")
    return code


def echo_tree_verify_attn(q, k_new, v_new, k_cache, v_cache, kv_offsets, kv_rows, q_offsets,
                          tree_mask, mask_words, R, max_rows, hq, hkv, head_dim, sm_scale, out,
                          lse, workspace, status=None, stream=None, check=True):
    """Tree-masked GQA verification attention.  bf16 inputs as int16/uint16/bfloat16 tensors."""
    code = load().echo_tree_verify_attn(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(kv_offsets),
        int(kv_rows), _ptr(q_offsets), _ptr(tree_mask), mask_words, R, max_rows, hq, hkv, head_dim,
        float(sm_scale), _ptr(out), _ptr(lse), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(status), _stream(stream))
    if check:
        _check(code, "echo_tree_verify_attn")
    return code


def echo_tree_verify_attn_timed(q, k_new, v_new, k_cache, v_cache, kv_offsets, kv_rows, q_offsets,
                                tree_mask, mask_words, R, max_rows, hq, hkv, head_dim, sm_scale,
                                out, lse, workspace, ev_start, ev_stop, status=None, stream=None,
                                check=True):
    """echo_tree_verify_attn with two torch.cuda.Event objects recorded around its
    main kernel on its stream (measurement only)."""
    code = load().echo_tree_verify_attn_timed(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(kv_offsets),
        int(kv_rows), _ptr(q_offsets), _ptr(tree_mask), mask_words, R, max_rows, hq, hkv, head_dim,
        float(sm_scale), _ptr(out), _ptr(lse), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(status), _event(ev_start),
        _event(ev_stop), _stream(stream))
    if check:
        _check(code, "echo_tree_verify_attn_timed")
    return code


def echo_accept(q_offsets, slot_parent, slot_token, target_token, R, max_rows, max_depth,
                accept_len, accept_slots, bonus_token, status=None, stream=None, check=True):
    """Greedy acceptance of the longest matching path per request."""
    code = load().echo_accept(_ptr(q_offsets), _ptr(slot_parent), _ptr(slot_token),
                              _ptr(target_token), R, max_rows, max_depth, _ptr(accept_len),
                              _ptr(accept_slots), _ptr(bonus_token), _ptr(status),
                              _stream(stream))
    if check:
        _check(code, "echo_accept")
    return code


def echo_verify_step(cand_offsets, parent, logq, token, R, N, budget, path_score, selected,
                     num_selected, gate_workspace, root_token, prefix_len, q_offsets, slot_cand,
                     slot_parent, slot_token, position_ids, tree_mask, mask_words, q, k_new, v_new,
                     k_cache, v_cache, kv_offsets, kv_rows, max_rows, hq, hkv, head_dim, sm_scale,
                     out, lse, attn_workspace, target_token, max_depth, accept_len, accept_slots,
                     bonus_token, status=None, stream=None, check=True):
    """The four stages of a step in one call (gate, flatten & pack, attention over a
    contiguous cache, acceptance); the arguments of the four calls in order."""
    code = load().echo_verify_step(
        _ptr(cand_offsets), _ptr(parent), _ptr(logq), _ptr(token), R, N, budget, _ptr(path_score),
        _ptr(selected), _ptr(num_selected), _ptr(gate_workspace),
        gate_workspace.numel() * gate_workspace.element_size(), _ptr(root_token),
        _ptr(prefix_len), _ptr(q_offsets), _ptr(slot_cand), _ptr(slot_parent), _ptr(slot_token),
        _ptr(position_ids), _ptr(tree_mask), mask_words, _ptr(q), _ptr(k_new), _ptr(v_new),
        _ptr(k_cache), _ptr(v_cache), _ptr(kv_offsets), int(kv_rows), max_rows, hq, hkv, head_dim,
        float(sm_scale), _ptr(out), _ptr(lse), _ptr(attn_workspace),
        attn_workspace.numel() * attn_workspace.element_size(), _ptr(target_token), max_depth,
        _ptr(accept_len), _ptr(accept_slots), _ptr(bonus_token), _ptr(status), _stream(stream))
    if check:
        _check(code, "echo_verify_step")
    return code


def echo_tree_verify_attn_paged(q, k_new, v_new, k_pages, v_pages, page_size, block_table,
                                prefix_len, q_offsets, tree_mask, mask_words, R, max_rows, hq,
                                hkv, head_dim, sm_scale, out, lse, workspace, status=None,
                                stream=None, check=True):
    """Verification attention over a paged KV cache.  Device tensors; k_pages is
    [num_pages, page_size, Hkv, 128] bf16 bits, block_table [R, max_pages]."""
    code = load().echo_tree_verify_attn_paged(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_pages), _ptr(v_pages), k_pages.shape[0],
        page_size, _ptr(block_table), block_table.shape[1], _ptr(prefix_len), _ptr(q_offsets),
        _ptr(tree_mask), mask_words, R, max_rows, hq, hkv, head_dim, sm_scale, _ptr(out),
        _ptr(lse), _ptr(workspace), workspace.numel() * workspace.element_size(), _ptr(status),
        _stream(stream))
    if check:
        _check(code, "echo_tree_verify_attn_paged")
    return code


def echo_tree_verify_attn_paged_timed(q, k_new, v_new, k_pages, v_pages, page_size, block_table,
                                      prefix_len, q_offsets, tree_mask, mask_words, R, max_rows,
                                      hq, hkv, head_dim, sm_scale, out, lse, workspace, ev_start,
                                      ev_stop, status=None, stream=None, check=True):
    """echo_tree_verify_attn_paged with events around its main kernel (measurement only)."""
    code = load().echo_tree_verify_attn_paged_timed(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_pages), _ptr(v_pages), k_pages.shape[0],
        page_size, _ptr(block_table), block_table.shape[1], _ptr(prefix_len), _ptr(q_offsets),
        _ptr(tree_mask), mask_words, R, max_rows, hq, hkv, head_dim, sm_scale, _ptr(out),
        _ptr(lse), _ptr(workspace), workspace.numel() * workspace.element_size(), _ptr(status),
        _event(ev_start), _event(ev_stop), _stream(stream))
    if check:
        _check(code, "echo_tree_verify_attn_paged_timed")
    return code


def echo_accept_logits(q_offsets, slot_parent, slot_token, logits, R, max_rows, max_depth,
                       target_token, accept_len, accept_slots, bonus_token, status=None,
                       stream=None, check=True):
    """Target argmax of bf16 logits [max_rows, V] followed by greedy acceptance."""
    code = load().echo_accept_logits(_ptr(q_offsets), _ptr(slot_parent), _ptr(slot_token),
                                     _ptr(logits), logits.shape[1], R, max_rows, max_depth,
                                     _ptr(target_token), _ptr(accept_len), _ptr(accept_slots),
                                     _ptr(bonus_token), _ptr(status), _stream(stream))
    if check:
        _check(code, "echo_accept_logits")
    return code


def echo_commit_kv(q_offsets, accept_len, accept_slots, max_depth, k_new, v_new, R, max_rows,
                   hkv, k_pages, v_pages, page_size, block_table, prefix_len, status=None,
                   stream=None, check=True):
    """Append each request's root and accepted slots to its paged KV cache."""
    code = load().echo_commit_kv(_ptr(q_offsets), _ptr(accept_len), _ptr(accept_slots),
                                 max_depth, _ptr(k_new), _ptr(v_new), R, max_rows, hkv,
                                 _ptr(k_pages), _ptr(v_pages), k_pages.shape[0], page_size,
                                 _ptr(block_table), block_table.shape[1], _ptr(prefix_len),
                                 _ptr(status), _stream(stream))
    if check:
        _check(code, "echo_commit_kv")
    return code
