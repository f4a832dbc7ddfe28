"""Pins of the KV append / key-sum refresh oracle (Sections 4.3, 4.4) against
the independently pinned pool reader and key-sum definition."""
import numpy as np
import pytest
import torch

from oracle import build_oracle as BO
from oracle import segpa_oracle as S
from paper_2606_06256_amd import inputs as I


def _state(P=16, D=64, ctx=(40, 17), seg_tokens=32, Hkv=2, extra=6, seed=5):
    sp = I.Spec(name="append", B=len(ctx), Hq=2 * Hkv, Hkv=Hkv, D=D, P=P, seg_tokens=seg_tokens,
                ctx_lens=list(ctx), q_lens=[1] * len(ctx), seed=seed, extra_phys_pages=extra)
    wl = I.build(sp)
    k, v = wl.build_pool("cpu")
    bits = lambda t: t.view(torch.int16).numpy().view(np.uint16).copy()
    return wl, bits(k), bits(v)


def _new_tokens(n, Hkv, D, seed):
    rng = np.random.default_rng(seed)
    f = lambda: torch.from_numpy(rng.standard_normal((n, Hkv, D)).astype(np.float32)).to(
        torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    return f(), f()


def _f64(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def test_append_reads_back_as_old_then_new():
    n_new = [5, 20]               # crosses page and segment boundaries
    L0s = [40, 17]
    # tables and pages are allocated for the final lengths; the append starts
    # from the shorter ones
    wl, kp, vp = _state(ctx=tuple(a + b for a, b in zip(L0s, n_new)))
    indptr = np.concatenate([[0], np.cumsum(n_new)])
    kn, vn = _new_tokens(indptr[-1], wl.Hkv, wl.D, 1)
    L1 = [int(x) for x in wl.ctx_lens]
    k2, v2, touched = BO.append(kp, vp, wl.seg_table, wl.page_table, L0s, indptr, kn, vn,
                                wl.Hkv, wl.P, wl.pps)
    seg = wl.seg_table.reshape(wl.B * wl.Hkv, -1)
    for r in range(wl.B):
        L0 = L0s[r]
        for g in range(wl.Hkv):
            row = seg[r * wl.Hkv + g]
            K0, V0 = S.unit_kv_from_pool(_f64(kp), _f64(vp), row, wl.page_table, wl.pps, L0, wl.P, wl.D)
            K1, V1 = S.unit_kv_from_pool(_f64(k2), _f64(v2), row, wl.page_table, wl.pps, L1[r], wl.P, wl.D)
            np.testing.assert_array_equal(K1[:L0], K0)
            np.testing.assert_array_equal(V1[:L0], V0)
            np.testing.assert_array_equal(K1[L0:], _f64(kn[indptr[r]:indptr[r + 1], g]))
            np.testing.assert_array_equal(V1[L0:], _f64(vn[indptr[r]:indptr[r + 1], g]))
    # pages that received nothing are unchanged
    other = np.setdiff1d(np.arange(kp.shape[0]), list(touched))
    np.testing.assert_array_equal(k2[other], kp[other])
    np.testing.assert_array_equal(v2[other], vp[other])


def test_two_appends_equal_one():
    wl, kp, vp = _state(ctx=(47, 22), seed=6)
    L0s = np.array([40, 17])
    kn, vn = _new_tokens(12, wl.Hkv, wl.D, 2)
    one = BO.append(kp, vp, wl.seg_table, wl.page_table, L0s, [0, 7, 12], kn, vn, wl.Hkv, wl.P, wl.pps)
    a = BO.append(kp, vp, wl.seg_table, wl.page_table, L0s, [0, 3, 5], kn[[0, 1, 2, 7, 8]],
                  vn[[0, 1, 2, 7, 8]], wl.Hkv, wl.P, wl.pps)
    ctx = L0s + [3, 2]
    b = BO.append(a[0], a[1], wl.seg_table, wl.page_table, ctx, [0, 4, 7], kn[[3, 4, 5, 6, 9, 10, 11]],
                  vn[[3, 4, 5, 6, 9, 10, 11]], wl.Hkv, wl.P, wl.pps)
    np.testing.assert_array_equal(b[0], one[0])
    np.testing.assert_array_equal(b[1], one[1])


def test_unmapped_segment_drops_its_tokens():
    wl, kp, vp = _state(ctx=(40, 30), seed=7)
    seg = wl.seg_table.copy()
    seg.reshape(wl.B * wl.Hkv, -1)[0, 1] = -1      # unit 0, segment 1 (positions 32..63)
    kn, vn = _new_tokens(10, wl.Hkv, wl.D, 3)
    k2, v2, touched = BO.append(kp, vp, seg, wl.page_table, [30, 30], [0, 10, 10], kn, vn,
                                wl.Hkv, wl.P, wl.pps)
    seg_row = seg.reshape(wl.B * wl.Hkv, -1)
    # unit 0: positions 30, 31 land in segment 0; 32..39 are dropped
    K, _ = S.unit_kv_from_pool(_f64(k2), _f64(v2), seg_row[0], wl.page_table, wl.pps, 32, wl.P, wl.D)
    np.testing.assert_array_equal(K[30:32], _f64(kn[0:2, 0]))
    # unit 1 (KV head 1 of request 0) has its segment 1 mapped: all 10 written
    K1, _ = S.unit_kv_from_pool(_f64(k2), _f64(v2), seg_row[1], wl.page_table, wl.pps, 40, wl.P, wl.D)
    np.testing.assert_array_equal(K1[30:40], _f64(kn[:, 1]))


def test_refreshed_key_sums_equal_a_full_recompute():
    wl, kp, vp = _state(P=32, D=128, ctx=(64, 80), seg_tokens=64, seed=8)
    kn, vn = _new_tokens(30, wl.Hkv, wl.D, 4)
    k2, v2, touched = BO.append(kp, vp, wl.seg_table, wl.page_table, [50, 64], [0, 14, 30], kn, vn,
                                wl.Hkv, wl.P, wl.pps)
    assert any(v < wl.P for v in touched.values())   # a partial page is among them
    # slots past a page's valid tokens hold anything (here 1.0): never summed
    for ph, valid in touched.items():
        kt = k2[ph].reshape(wl.P // 16, wl.D // 8, 16, 8)
        for slot in range(valid, wl.P):
            kt[slot // 16, :, slot % 16, :] = 0x3F80
    ksum0 = np.full((kp.shape[0], wl.D), np.float32(7.0))
    ks = BO.refresh_key_sums(ksum0, k2, touched, wl.P, wl.D)
    seg = wl.seg_table.reshape(wl.B * wl.Hkv, -1)
    L1 = [50 + 14, 64 + 16]
    for r in range(wl.B):
        for g in range(wl.Hkv):
            row = seg[r * wl.Hkv + g]
            K, _ = S.unit_kv_from_pool(_f64(k2), _f64(v2), row, wl.page_table, wl.pps, L1[r], wl.P, wl.D)
            sums, valid = S.unit_key_sums(K, wl.P)
            for j in range(len(valid)):
                ph = S.translate(row, wl.page_table, wl.pps, j)
                if ph in touched:
                    np.testing.assert_array_equal(ks[ph], sums[j])
                    assert touched[ph] == valid[j]
    untouched = np.setdiff1d(np.arange(kp.shape[0]), list(touched))
    assert (ks[untouched] == 7.0).all()
