"""C-ABI surface (CPU): the library loads, exports every declared entry point,
and rejects bad host arguments with the documented status codes before it
launches anything."""
import ctypes
import os
import re

import pytest

from paper_2606_06256_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "segpa.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(seg_paged_attn_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared_functions()
    for n in ("seg_paged_attn_select", "seg_paged_attn_fwd", "seg_paged_attn_workspace_size",
              "seg_paged_attn_page_summary", "seg_paged_attn_validate",
              "seg_paged_attn_status_string"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(B.LIB_PATH)
    missing = [n for n in _declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings():
    for code, text in [(0, "ok"), (-1, "invalid argument"), (-3, "workspace"), (-4, "sel_capacity"),
                       (-6, "invalid table")]:
        assert text in B.status_string(code)
    assert B.status_string(-99) == "unknown status"


def _dims(**kw):
    base = dict(num_requests=2, num_q_heads=8, num_kv_heads=2, head_dim=128, page_size=16,
                pages_per_segment=4, max_segments=4, max_q_len=1, total_q=2,
                num_virtual_pages=64, num_phys_pages=64)
    base.update(kw)
    return B.make_dims(**base)


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every case fails its host checks first


def _select(dims, params, cap=1 << 20, ws=None, ctx=FAKE, indptr=FAKE, pages=FAKE):
    return B.lib().seg_paged_attn_select(ctypes.byref(dims), ctypes.byref(params) if params else None,
                                         ctx, FAKE, FAKE, FAKE, FAKE, FAKE, indptr, pages, cap, ws,
                                         0 if ws is None else 1 << 20, None)


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=96), -2), (dict(page_size=24), -2), (dict(page_size=8), -2),
    (dict(num_q_heads=6, num_kv_heads=4), -1), (dict(num_requests=0), -1),
    (dict(max_q_len=0), -1), (dict(num_phys_pages=0), -1), (dict(num_requests=2000, num_kv_heads=8), -2),
    (dict(num_phys_pages=1 << 28), -2), (dict(num_phys_pages=1 << 24, page_size=256), -2),
])
def test_bad_dims_rejected(kw, code):
    params = B.spa_select_params_t(0, 4, 256, 0, 0, 0, 0, None, None)
    assert _select(_dims(**kw), params) == code


def test_bad_select_args_rejected():
    d = _dims()
    ok_params = B.spa_select_params_t(0, 4, 256, 0, 0, 0, 0, None, None)
    assert _select(d, None) == -1
    assert _select(d, ok_params, ctx=None) == -1
    assert _select(d, ok_params, cap=2 * 2 * 16 - 1) == -4            # below units * max_pages
    assert _select(d, B.spa_select_params_t(7, 4, 256, 0, 0, 0, 0, None, None)) == -1
    # HEAD_CLASS needs the head policy; RANDOM_HASH needs budgets
    assert _select(d, B.spa_select_params_t(1, 4, 256, 0, 0, 0, 0, None, None)) == -1
    assert _select(d, B.spa_select_params_t(2, 4, 256, 0, 0, 0, 0, None, None)) == -1
    assert _select(d, B.spa_select_params_t(1, -1, 256, 0, 0, 0, 0, 0x1000, None)) == -1
    # TOPK needs a workspace for the page scores
    L = B.lib()
    st = L.seg_paged_attn_select(ctypes.byref(d), ctypes.byref(B.spa_select_params_t(3, 4, 256, 0, 0, 0, 0, None, 0x1000)),
                                 FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, None, 0, None)
    assert st == -3


def test_bad_fwd_args_rejected():
    d = _dims()
    L = B.lib()
    args = [FAKE] * 9
    # null output
    st = L.seg_paged_attn_fwd(ctypes.byref(d), *args, 1 << 20, None, None, FAKE, 1 << 20, None)
    assert st == -1
    # misaligned pool
    bad = [FAKE] * 9
    bad[3] = ctypes.c_void_p(0x1002)
    st = L.seg_paged_attn_fwd(ctypes.byref(d), *bad, 1 << 20, FAKE, None, FAKE, 1 << 20, None)
    assert st == -1
    # unsupported head dim
    st = L.seg_paged_attn_fwd(ctypes.byref(_dims(head_dim=80)), *args, 1 << 20, FAKE, None, FAKE,
                              1 << 20, None)
    assert st == -2
    assert L.seg_paged_attn_workspace_size(ctypes.byref(_dims(head_dim=80)), 0) == 0


def test_validate_needs_workspace():
    d = _dims()
    L = B.lib()
    st = L.seg_paged_attn_validate(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 100,
                                   None, None, None, 0, None)
    assert st == -3


def test_bad_rope_align_args_rejected():
    d = _dims()
    L = B.lib()
    assert L.seg_paged_attn_rope_align(ctypes.byref(d), FAKE, FAKE, FAKE, -1, 1e4, None) == -1
    assert L.seg_paged_attn_rope_align(ctypes.byref(d), FAKE, FAKE, FAKE, 1 << 31, 1e4, None) == -1
    assert L.seg_paged_attn_rope_align(ctypes.byref(d), FAKE, FAKE, FAKE, 4, 1.0, None) == -1
    assert L.seg_paged_attn_rope_align(ctypes.byref(d), FAKE, FAKE, FAKE, 4, float("nan"), None) == -1
    assert L.seg_paged_attn_rope_align(ctypes.byref(d), FAKE, None, FAKE, 4, 1e4, None) == -1
    assert L.seg_paged_attn_rope_align(ctypes.byref(d), ctypes.c_void_p(0x1002), FAKE, FAKE, 4, 1e4,
                                       None) == -1
    # nothing to do: no launch, no pointer needed
    assert L.seg_paged_attn_rope_align(ctypes.byref(d), None, None, None, 0, 1e4, None) == 0


def test_bad_append_args_rejected():
    d = _dims()
    L = B.lib()
    f = lambda **kw: L.seg_paged_attn_append(
        ctypes.byref(d), kw.get("ctx", FAKE), kw.get("ind", FAKE), kw.get("kn", FAKE), kw.get("vn", FAKE),
        kw.get("n", 4), FAKE, FAKE, kw.get("kp", FAKE), FAKE, kw.get("ks", None), None)
    assert f(n=-1) == -1
    assert f(ctx=None) == -1
    assert f(kn=None) == -1
    assert f(kp=ctypes.c_void_p(0x1008)) == -1
    assert f(ks=ctypes.c_void_p(0x1004)) == -1
    # nothing to append: no launch, no pointer needed
    assert L.seg_paged_attn_append(ctypes.byref(d), None, None, None, None, 0, None, None, None, None,
                                   None, None) == 0


def test_bad_token_mass_args_rejected():
    d = _dims()
    L = B.lib()
    f = lambda **kw: L.seg_paged_attn_token_mass(
        ctypes.byref(kw.get("d", d)), kw.get("q", FAKE), FAKE, FAKE, kw.get("kp", FAKE), FAKE, FAKE,
        FAKE, FAKE, kw.get("cap", 1 << 10), kw.get("lse", FAKE), kw.get("mass", FAKE), None)
    assert f(q=None) == -1
    assert f(lse=None) == -1
    assert f(mass=None) == -1
    assert f(cap=-1) == -1
    assert f(q=ctypes.c_void_p(0x1008)) == -1
    assert f(kp=ctypes.c_void_p(0x1008)) == -1
    assert f(mass=ctypes.c_void_p(0x1002)) == -1
    assert f(d=_dims(head_dim=96)) == -2
    # no rows: nothing launched
    assert f(d=_dims(total_q=0)) == 0


def test_bad_select_tokens_args_rejected():
    d = _dims()
    L = B.lib()
    f = lambda **kw: L.seg_paged_attn_select_tokens(
        ctypes.byref(kw.get("d", d)), kw.get("ind", FAKE), kw.get("mass", FAKE), kw.get("cols", 2),
        kw.get("tau", 0.5), kw.get("recent", 0), kw.get("keep", FAKE), None, kw.get("cnt", FAKE),
        kw.get("tm", None), None)
    assert f(ind=None) == -1
    assert f(mass=None) == -1
    assert f(keep=None) == -1
    assert f(cnt=None) == -1
    for tau in (0.0, -0.5, 1.5, float("nan"), float("inf")):
        assert f(tau=tau) == -1
    assert f(recent=-1) == -1
    assert f(cols=0) == -1
    assert f(cols=4097) == -1
    assert f(tm=ctypes.c_void_p(0x1002)) == -1
    assert f(d=_dims(max_q_len=16385)) == -2
