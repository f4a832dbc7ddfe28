"""Thin ctypes binding of libsegpa.so (same entry-point names as include/segpa.h).

Argument marshalling only: torch tensors supply device memory and the HIP
stream; every step of selection and attention runs in the library's kernels.
There is no fallback: if the library is missing or a call fails, this raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsegpa.so")

SPA_OK = 0
SPA_ERR_WORKSPACE = -3
SPA_NOALLOC_SCRATCH_BYTES = 32 << 20
SPA_SEL_ALL, SPA_SEL_HEAD_CLASS, SPA_SEL_RANDOM_HASH, SPA_SEL_TOPK_MEANKEY = 0, 1, 2, 3


class SegpaError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} failed: {msg} (status {status})")
        self.status = status


class spa_dims_t(ctypes.Structure):
    _fields_ = [("num_requests", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("pages_per_segment", ctypes.c_int32),
                ("max_segments", ctypes.c_int32), ("max_q_len", ctypes.c_int32),
                ("total_q", ctypes.c_int32), ("reserved0", ctypes.c_int32),
                ("num_virtual_pages", ctypes.c_int64), ("num_phys_pages", ctypes.c_int64),
                ("softmax_scale", ctypes.c_float)]


class spa_select_params_t(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("n_sink_tokens", ctypes.c_int32),
                ("window_tokens", ctypes.c_int32), ("forced_head_pages", ctypes.c_int32),
                ("forced_tail_pages", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("seed", ctypes.c_uint64), ("head_policy", ctypes.c_void_p),
                ("budget_pages", ctypes.c_void_p)]


_lib: Optional[ctypes.CDLL] = None
_P = ctypes.c_void_p


def lib() -> ctypes.CDLL:
    """Load libsegpa.so (built in-tree); raise if it is not there."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_06256_amd.build_lib`")
    L = ctypes.CDLL(LIB_PATH)
    L.seg_paged_attn_workspace_size.restype = ctypes.c_size_t
    L.seg_paged_attn_workspace_size.argtypes = [ctypes.POINTER(spa_dims_t), ctypes.c_int32]
    L.seg_paged_attn_select.restype = ctypes.c_int
    L.seg_paged_attn_select.argtypes = [ctypes.POINTER(spa_dims_t), ctypes.POINTER(spa_select_params_t),
                                        _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_int64, _P,
                                        ctypes.c_size_t, _P]
    L.seg_paged_attn_fwd.restype = ctypes.c_int
    L.seg_paged_attn_fwd.argtypes = [ctypes.POINTER(spa_dims_t), _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                     ctypes.c_int64, _P, _P, _P, ctypes.c_size_t, _P]
    L.seg_paged_attn_fwd_noalloc.restype = ctypes.c_int
    L.seg_paged_attn_fwd_noalloc.argtypes = [ctypes.POINTER(spa_dims_t), _P, _P, _P, _P, _P, _P, _P,
                                             _P, _P, ctypes.c_int64, _P, _P, _P]
    L.seg_paged_attn_page_summary.restype = ctypes.c_int
    L.seg_paged_attn_page_summary.argtypes = [ctypes.POINTER(spa_dims_t), _P, _P, _P, _P]
    L.seg_paged_attn_append.restype = ctypes.c_int
    L.seg_paged_attn_append.argtypes = [ctypes.POINTER(spa_dims_t), _P, _P, _P, _P, ctypes.c_int64,
                                         _P, _P, _P, _P, _P, _P]
    L.seg_paged_attn_rope_align.restype = ctypes.c_int
    L.seg_paged_attn_rope_align.argtypes = [ctypes.POINTER(spa_dims_t), _P, _P, _P, ctypes.c_int64,
                                             ctypes.c_double, _P]
    L.seg_paged_attn_token_mass.restype = ctypes.c_int
    L.seg_paged_attn_token_mass.argtypes = [ctypes.POINTER(spa_dims_t), _P, _P, _P, _P, _P, _P, _P,
                                            _P, ctypes.c_int64, _P, _P, _P]
    L.seg_paged_attn_select_tokens.restype = ctypes.c_int
    L.seg_paged_attn_select_tokens.argtypes = [ctypes.POINTER(spa_dims_t), _P, _P, ctypes.c_int32,
                                               ctypes.c_double, ctypes.c_int32, _P, _P, _P, _P, _P]
    L.seg_paged_attn_validate.restype = ctypes.c_int
    L.seg_paged_attn_validate.argtypes = [ctypes.POINTER(spa_dims_t), _P, _P, _P, _P, _P, _P,
                                          ctypes.c_int64, ctypes.POINTER(ctypes.c_int32),
                                          ctypes.POINTER(ctypes.c_int64), _P, ctypes.c_size_t, _P]
    L.seg_paged_attn_status_string.restype = ctypes.c_char_p
    L.seg_paged_attn_status_string.argtypes = [ctypes.c_int]
    L.seg_paged_attn_profile_begin.restype = ctypes.c_int
    L.seg_paged_attn_profile_begin.argtypes = []
    L.seg_paged_attn_profile_end.restype = ctypes.c_int32
    L.seg_paged_attn_profile_end.argtypes = [ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_int32),
                                             ctypes.POINTER(ctypes.c_double), ctypes.c_int32]
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().seg_paged_attn_status_string(status).decode()


def _check(fn: str, st: int):
    if st != SPA_OK:
        raise SegpaError(fn, st, status_string(st))


def _ptr(t: Optional[torch.Tensor], dtype=None, name: str = "") -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name}: expected a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name}: expected {dtype}, got {t.dtype}")
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def make_dims(*, num_requests, num_q_heads, num_kv_heads, head_dim, page_size, pages_per_segment,
              max_segments, max_q_len, total_q, num_virtual_pages, num_phys_pages,
              softmax_scale=0.0) -> spa_dims_t:
    return spa_dims_t(num_requests, num_q_heads, num_kv_heads, head_dim, page_size,
                      pages_per_segment, max_segments, max_q_len, total_q, 0, num_virtual_pages,
                      num_phys_pages, softmax_scale)


def make_select_params(mode: int, *, n_sink_tokens=4, window_tokens=256, forced_head_pages=0,
                       forced_tail_pages=0, seed=0, head_policy: Optional[torch.Tensor] = None,
                       budget_pages: Optional[torch.Tensor] = None) -> spa_select_params_t:
    return spa_select_params_t(mode, n_sink_tokens, window_tokens, forced_head_pages,
                               forced_tail_pages, 0, seed & ((1 << 64) - 1),
                               _ptr(head_policy, torch.int8, "head_policy"),
                               _ptr(budget_pages, torch.int32, "budget_pages"))


def seg_paged_attn_workspace_size(dims: spa_dims_t, sel_mode: int) -> int:
    return int(lib().seg_paged_attn_workspace_size(ctypes.byref(dims), sel_mode))


def seg_paged_attn_select(dims: spa_dims_t, params: spa_select_params_t, ctx_lens, q, q_indptr,
                          page_ksum, seg_table, page_table, sel_indptr, sel_pages, workspace,
                          stream=None):
    st = lib().seg_paged_attn_select(
        ctypes.byref(dims), ctypes.byref(params), _ptr(ctx_lens, torch.int32, "ctx_lens"),
        _ptr(q, torch.bfloat16, "q"), _ptr(q_indptr, torch.int32, "q_indptr"),
        _ptr(page_ksum, torch.float32, "page_ksum"), _ptr(seg_table, torch.int32, "seg_table"),
        _ptr(page_table, torch.int32, "page_table"), _ptr(sel_indptr, torch.int32, "sel_indptr"),
        _ptr(sel_pages, torch.int32, "sel_pages"), sel_pages.numel(),
        _ptr(workspace, torch.uint8, "workspace"), 0 if workspace is None else workspace.numel(),
        _stream(stream))
    _check("seg_paged_attn_select", st)


def seg_paged_attn_fwd(dims: spa_dims_t, q, q_indptr, ctx_lens, k_pool, v_pool, seg_table,
                       page_table, sel_indptr, sel_pages, out, lse, workspace, stream=None):
    st = lib().seg_paged_attn_fwd(
        ctypes.byref(dims), _ptr(q, torch.bfloat16, "q"), _ptr(q_indptr, torch.int32, "q_indptr"),
        _ptr(ctx_lens, torch.int32, "ctx_lens"), _ptr(k_pool, torch.bfloat16, "k_pool"),
        _ptr(v_pool, torch.bfloat16, "v_pool"), _ptr(seg_table, torch.int32, "seg_table"),
        _ptr(page_table, torch.int32, "page_table"), _ptr(sel_indptr, torch.int32, "sel_indptr"),
        _ptr(sel_pages, torch.int32, "sel_pages"), sel_pages.numel(),
        _ptr(out, torch.bfloat16, "out"), _ptr(lse, torch.float32, "lse"),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream))
    _check("seg_paged_attn_fwd", st)


def seg_paged_attn_fwd_noalloc(dims: spa_dims_t, q, q_indptr, ctx_lens, k_pool, v_pool, seg_table,
                               page_table, sel_indptr, sel_pages, out, lse, stream=None):
    """seg_paged_attn_fwd over the library's own per-GPU scratch (no workspace)."""
    st = lib().seg_paged_attn_fwd_noalloc(
        ctypes.byref(dims), _ptr(q, torch.bfloat16, "q"), _ptr(q_indptr, torch.int32, "q_indptr"),
        _ptr(ctx_lens, torch.int32, "ctx_lens"), _ptr(k_pool, torch.bfloat16, "k_pool"),
        _ptr(v_pool, torch.bfloat16, "v_pool"), _ptr(seg_table, torch.int32, "seg_table"),
        _ptr(page_table, torch.int32, "page_table"), _ptr(sel_indptr, torch.int32, "sel_indptr"),
        _ptr(sel_pages, torch.int32, "sel_pages"), sel_pages.numel(),
        _ptr(out, torch.bfloat16, "out"), _ptr(lse, torch.float32, "lse"), _stream(stream))
    _check("seg_paged_attn_fwd_noalloc", st)


def seg_paged_attn_page_summary(dims: spa_dims_t, k_pool, page_valid_tokens, page_ksum, stream=None):
    st = lib().seg_paged_attn_page_summary(
        ctypes.byref(dims), _ptr(k_pool, torch.bfloat16, "k_pool"),
        _ptr(page_valid_tokens, torch.int32, "page_valid_tokens"),
        _ptr(page_ksum, torch.float32, "page_ksum"), _stream(stream))
    _check("seg_paged_attn_page_summary", st)


def seg_paged_attn_append(dims: spa_dims_t, ctx_lens, new_indptr, k_new, v_new, seg_table, page_table,
                          k_pool, v_pool, page_ksum=None, stream=None):
    """Writes the new tokens' keys and values into their pages (and refreshes
    the key sums of the pages written when page_ksum is given)."""
    n_new = k_new.shape[0]
    if v_new.shape != k_new.shape:
        raise ValueError("k_new and v_new differ in shape")
    st = lib().seg_paged_attn_append(
        ctypes.byref(dims), _ptr(ctx_lens, torch.int32, "ctx_lens"),
        _ptr(new_indptr, torch.int32, "new_indptr"), _ptr(k_new, torch.bfloat16, "k_new"),
        _ptr(v_new, torch.bfloat16, "v_new"), n_new, _ptr(seg_table, torch.int32, "seg_table"),
        _ptr(page_table, torch.int32, "page_table"), _ptr(k_pool, torch.bfloat16, "k_pool"),
        _ptr(v_pool, torch.bfloat16, "v_pool"), _ptr(page_ksum, torch.float32, "page_ksum"),
        _stream(stream))
    _check("seg_paged_attn_append", st)


def seg_paged_attn_rope_align(dims: spa_dims_t, k_pool, pages, deltas, rope_base: float = 10000.0,
                              stream=None):
    """Rotates the listed physical pages of k_pool in place by their deltas."""
    if pages.numel() != deltas.numel():
        raise ValueError("pages and deltas differ in length")
    st = lib().seg_paged_attn_rope_align(
        ctypes.byref(dims), _ptr(k_pool, torch.bfloat16, "k_pool"), _ptr(pages, torch.int32, "pages"),
        _ptr(deltas, torch.int32, "deltas"), pages.numel(), float(rope_base), _stream(stream))
    _check("seg_paged_attn_rope_align", st)


def seg_paged_attn_token_mass(dims: spa_dims_t, q, q_indptr, ctx_lens, k_pool, seg_table, page_table,
                              sel_indptr, sel_pages, lse, mass, stream=None):
    """mass [total_q, Hkv]: softmax mass each chunk token receives per KV head."""
    st = lib().seg_paged_attn_token_mass(
        ctypes.byref(dims), _ptr(q, torch.bfloat16, "q"), _ptr(q_indptr, torch.int32, "q_indptr"),
        _ptr(ctx_lens, torch.int32, "ctx_lens"), _ptr(k_pool, torch.bfloat16, "k_pool"),
        _ptr(seg_table, torch.int32, "seg_table"), _ptr(page_table, torch.int32, "page_table"),
        _ptr(sel_indptr, torch.int32, "sel_indptr"), _ptr(sel_pages, torch.int32, "sel_pages"),
        sel_pages.numel(), _ptr(lse, torch.float32, "lse"), _ptr(mass, torch.float32, "mass"),
        _stream(stream))
    _check("seg_paged_attn_token_mass", st)


def seg_paged_attn_select_tokens(dims: spa_dims_t, q_indptr, mass, tau: float, recent: int, keep,
                                 keep_count, kept=None, token_mass=None, stream=None):
    """Per request: tokens of the smallest mass-ranked set reaching tau of the
    total, plus the last `recent` tokens (keep mask, kept rows, counts)."""
    cols = 1 if mass.dim() == 1 else mass.shape[1]
    st = lib().seg_paged_attn_select_tokens(
        ctypes.byref(dims), _ptr(q_indptr, torch.int32, "q_indptr"), _ptr(mass, torch.float32, "mass"),
        cols, float(tau), int(recent), _ptr(keep, torch.uint8, "keep"), _ptr(kept, torch.int32, "kept"),
        _ptr(keep_count, torch.int32, "keep_count"), _ptr(token_mass, torch.float32, "token_mass"),
        _stream(stream))
    _check("seg_paged_attn_select_tokens", st)


def seg_paged_attn_validate(dims: spa_dims_t, ctx_lens, q_indptr, seg_table, page_table,
                            sel_indptr, sel_pages, workspace, stream=None):
    """Returns (status, bad_code, bad_index); does not raise on SPA_ERR_BAD_DATA."""
    code = ctypes.c_int32(0)
    idx = ctypes.c_int64(-1)
    st = lib().seg_paged_attn_validate(
        ctypes.byref(dims), _ptr(ctx_lens, torch.int32, "ctx_lens"),
        _ptr(q_indptr, torch.int32, "q_indptr"), _ptr(seg_table, torch.int32, "seg_table"),
        _ptr(page_table, torch.int32, "page_table"), _ptr(sel_indptr, torch.int32, "sel_indptr"),
        _ptr(sel_pages, torch.int32, "sel_pages"), sel_pages.numel(), ctypes.byref(code),
        ctypes.byref(idx), _ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
        _stream(stream))
    return st, code.value, idx.value


def profile_begin():
    _check("seg_paged_attn_profile_begin", lib().seg_paged_attn_profile_begin())


def profile_end(cap: int = 16) -> dict:
    names = (ctypes.c_char_p * cap)()
    launches = (ctypes.c_int32 * cap)()
    ms = (ctypes.c_double * cap)()
    n = lib().seg_paged_attn_profile_end(names, launches, ms, cap)
    if n < 0:
        raise SegpaError("seg_paged_attn_profile_end", n, "event timing failed")
    return {names[i].decode(): (int(launches[i]), float(ms[i])) for i in range(min(n, cap))}
