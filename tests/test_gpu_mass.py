"""GPU parity of attention-mass token selection through the C-ABI.

seg_paged_attn_token_mass (after select + fwd on the GPU) against the fp64
oracle's masses, which the oracle derives itself (its own selection, its own
softmax normalisation); seg_paged_attn_select_tokens bit-exact against the
oracle on seeded synthetic masses; the two chained, checked where the result
is unique; and the head-class prefill workload at full size on sampled tokens
and by properties of the selection that hold at any size.

Tolerance for the masses: every weight is exp(scale q.k - lse) with the
score an exact product of bf16 values accumulated in fp32 (relative error
~1e-6 of |score|, below 1e-5 here) and lse the forward's fp32 log-sum-exp
(its own error is of the same order: the scores are the same products); a
token's mass is an fp32 sum over at most 4 * 512 rows, whose rounding is
bounded by n * 2^-24 < 1.3e-4 relative. Hence |got - want| <= 3e-4 * want +
1e-6; a dropped or doubled row, which moves the mass of the chunk's last
tokens by a quarter or more, fails it.
"""
import math

import numpy as np
import pytest
import torch

from oracle import mass_oracle as M
from paper_2606_06256_amd import binding as B
from paper_2606_06256_amd import inputs as I
from paper_2606_06256_amd.device import DeviceWorkload

import parity_util as PU

pytestmark = pytest.mark.gpu

MASS_RTOL = 3e-4
MASS_ATOL = 1e-6


def _require_gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"


def _spec(**kw):
    base = dict(name="mass", B=2, Hq=8, Hkv=2, D=128, P=16, seg_tokens=256, ctx_lens=[700, 333],
                q_lens=[40, 33], seed=5151)
    base.update(kw)
    return I.Spec(**base)


def _gpu_masses(wl, label):
    print(f"[mass] {label}: B={wl.B} Hq={wl.Hq} Hkv={wl.Hkv} D={wl.D} P={wl.P} "
          f"q_lens={np.diff(wl.q_indptr).tolist()[:4]} mode={wl.spec.sel_mode}", flush=True)
    dw = DeviceWorkload(wl)
    if wl.spec.sel_mode == I.SEL_TOPK_MEANKEY:
        dw.summary()
    dw.select()
    dw.fwd()
    dw.token_mass()
    torch.cuda.synchronize()
    return dw


def _check_unit_masses(wl, dw, q64, sel, units):
    mass = dw.mass.cpu().numpy()
    scale = 1.0 / math.sqrt(wl.D)
    G = wl.G
    worst = 0.0
    for u in units:
        r, g = divmod(u, wl.Hkv)
        q0, q1 = int(wl.q_indptr[r]), int(wl.q_indptr[r + 1])
        if q1 == q0:
            continue
        K, _ = PU.kv64(wl, r, g)
        want = M.unit_chunk_mass(q64[q0:q1, g * G:(g + 1) * G], K, sel[u], wl.P, scale)
        got = mass[q0:q1, g].astype(np.float64)
        err = np.abs(got - want) - (MASS_RTOL * want + MASS_ATOL)
        bad = np.nonzero(err > 0)[0]
        assert bad.size == 0, (f"unit {u}: token {bad[0]} got {got[bad[0]]:.9g} want {want[bad[0]]:.9g}")
        # unselected chunk tokens have exactly zero mass
        assert np.all(got[want == 0] == 0)
        nz = want > 1e-3
        if np.any(nz):
            worst = max(worst, float(np.max(np.abs(got[nz] - want[nz]) / want[nz])))
    return worst


MASS_CASES = {
    "two_key_groups_ragged": dict(q_lens=[300, 77], ctx_lens=[900, 77]),
    # chunks longer than one block's 512 keys: several key groups per unit
    "key_groups_2_and_3": dict(Hq=4, Hkv=2, q_lens=[700, 1100], ctx_lens=[1500, 1100],
                               seg_tokens=512),
    "key_groups_d64_g8": dict(D=64, Hq=16, Hkv=2, q_lens=[530, 513], ctx_lens=[600, 800]),
    "chunk_is_whole_stream": dict(q_lens=[64, 16], ctx_lens=[64, 16]),
    "decode_rows": dict(q_lens=[1, 1], ctx_lens=[700, 5]),
    "short_chunks": dict(q_lens=[3, 7], ctx_lens=[300, 129]),
    "d64_p32_g8": dict(D=64, P=32, Hq=16, Hkv=2, q_lens=[70, 40], ctx_lens=[400, 300]),
    "mha": dict(Hq=2, Hkv=2, q_lens=[130, 33], ctx_lens=[400, 200]),
    "g3": dict(Hq=6, Hkv=2, q_lens=[50, 20], ctx_lens=[500, 90]),
    "g16": dict(Hq=32, Hkv=2, q_lens=[33, 17], ctx_lens=[600, 256]),
    "page64": dict(P=64, seg_tokens=512, q_lens=[100, 70], ctx_lens=[700, 400]),
    "page256_key_groups": dict(P=256, seg_tokens=512, D=64, q_lens=[600, 90],
                               ctx_lens=[1300, 300]),
    "page128_random_gaps": dict(P=128, seg_tokens=256, sel_mode=I.SEL_RANDOM_HASH, budgets=[4, 2],
                                q_lens=[300, 60], ctx_lens=[1500, 400], sel_seed=41),
    # a small page budget without the forced tail leaves chunk pages unselected
    "random_chunk_gaps": dict(sel_mode=I.SEL_RANDOM_HASH, budgets=[10, 6], q_lens=[64, 40],
                              ctx_lens=[600, 300], sel_seed=31),
    "random_empty_unit": dict(sel_mode=I.SEL_RANDOM_HASH, budgets=[0, 4], q_lens=[20, 40],
                              ctx_lens=[500, 300], sel_seed=32),
    "head_class": dict(sel_mode=I.SEL_HEAD_CLASS, Hkv=4, Hq=16, head_policy=[1, 0, 1, 0], n_sink=4,
                       window=40, q_lens=[90, 30], ctx_lens=[1000, 300]),
    "topk": dict(sel_mode=I.SEL_TOPK_MEANKEY, budgets=[12, 8], forced_tail=2, q_lens=[30, 20],
                 ctx_lens=[800, 400]),
}


@pytest.mark.parametrize("name", sorted(MASS_CASES))
def test_token_mass_matches_oracle(name):
    _require_gpu()
    wl = I.build(_spec(name=name, **MASS_CASES[name]))
    dw = _gpu_masses(wl, name)
    q64 = wl.q("cpu").double().numpy()
    sel = PU.oracle_selection(wl, q64)
    ties = PU.compare_selection(wl, dw, q64, sel)
    units = [u for u in range(wl.num_units) if u not in ties]
    worst = _check_unit_masses(wl, dw, q64, sel, units)
    print(f"[mass] {name}: worst relative error {worst:.3e}", flush=True)


@pytest.mark.parametrize("i,div,batch", [(9, 32, 2), (4, 64, 2)])
def test_token_mass_scaled_prefill_workloads(i, div, batch):
    """The two chunked-prefill workloads at reduced context (512-token chunks)."""
    _require_gpu()
    sp = I.scaled_spec(i, div, batch)
    wl = I.build(sp)
    dw = _gpu_masses(wl, sp.name)
    q64 = wl.q("cpu").double().numpy()
    units = PU.sample_units(wl.num_units, 3)
    sel = PU.oracle_selection(wl, q64, units=units)
    PU.compare_selection(wl, dw, q64, sel)
    worst = _check_unit_masses(wl, dw, q64, sel, units)
    print(f"[mass] {sp.name}: worst relative error {worst:.3e}", flush=True)


def test_token_mass_is_reproducible():
    _require_gpu()
    wl = I.build(_spec(name="repro", q_lens=[300, 77], ctx_lens=[900, 400]))
    dw = _gpu_masses(wl, "repro")
    first = dw.mass.clone()
    dw.token_mass()
    torch.cuda.synchronize()
    assert torch.equal(first, dw.mass)


# --------------------------------------------------------------------------
# token selection on synthetic masses: bit-exact
# --------------------------------------------------------------------------
def _sel_dims(lens, cols):
    total = int(sum(lens))
    return B.make_dims(num_requests=len(lens), num_q_heads=cols, num_kv_heads=cols, head_dim=64,
                       page_size=16, pages_per_segment=1, max_segments=1,
                       max_q_len=max(1, max(lens)), total_q=total, num_virtual_pages=1,
                       num_phys_pages=1)


def _run_select(lens, cols_np, tau, recent, label):
    print(f"[select_tokens] {label}: n={list(lens)[:6]} cols={cols_np.shape[1]} tau={tau} "
          f"recent={recent}", flush=True)
    dev = torch.device("cuda")
    indptr = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    total = int(indptr[-1])
    dims = _sel_dims(lens, cols_np.shape[1])
    mass = torch.from_numpy(cols_np).to(dev)
    keep = torch.full((max(1, total),), 7, dtype=torch.uint8, device=dev)
    kept = torch.full((max(1, total),), -5, dtype=torch.int32, device=dev)
    cnt = torch.full((len(lens),), -1, dtype=torch.int32, device=dev)
    tm = torch.zeros(max(1, total), dtype=torch.float32, device=dev)
    B.seg_paged_attn_select_tokens(dims, torch.from_numpy(indptr).to(dev), mass, tau, recent, keep,
                                   cnt, kept, tm)
    torch.cuda.synchronize()
    return indptr, keep.cpu().numpy(), kept.cpu().numpy(), cnt.cpu().numpy(), tm.cpu().numpy()


def _compare_select(lens, cols_np, tau, recent, label):
    indptr, keep, kept, cnt, tm = _run_select(lens, cols_np, tau, recent, label)
    want_tm = M.columns_to_token_mass(cols_np)
    np.testing.assert_array_equal(tm[:indptr[-1]].view(np.uint32), want_tm.view(np.uint32))
    for r in range(len(lens)):
        q0, q1 = int(indptr[r]), int(indptr[r + 1])
        want = M.select_tokens(want_tm[q0:q1].astype(np.float64), tau, recent)
        mask = np.zeros(q1 - q0, dtype=np.uint8)
        mask[want] = 1
        np.testing.assert_array_equal(keep[q0:q1], mask, err_msg=f"{label} request {r}")
        assert cnt[r] == want.size, (label, r, cnt[r], want.size)
        np.testing.assert_array_equal(kept[q0:q0 + want.size], q0 + want)
    return cnt


def test_select_tokens_full_size_shape():
    """64 chunks of 512 tokens with 8 KV-head columns (the head-class prefill
    shape), at the thresholds of the paper's sparse-FFN settings."""
    _require_gpu()
    lens = [512] * 64
    cols = I.synthetic_masses(11, sum(lens), 8, "lognormal")
    for tau, recent in [(0.2, 128), (0.05, 128), (0.7, 256), (0.6, 0), (1.0, 0), (0.99, 0)]:
        cnt = _compare_select(lens, cols, tau, recent, f"lognormal tau={tau}")
        assert cnt.min() >= min(recent, 512)


@pytest.mark.parametrize("kind", ["dyadic", "sparse", "lognormal"])
def test_select_tokens_ragged_and_long(kind):
    """Every LDS size class (up to 16384 tokens), empty and one-token chunks."""
    _require_gpu()
    lens = [0, 1, 2, 3, 31, 1000, 1024, 1025, 4096, 4097, 16384, 0, 777]
    cols = I.synthetic_masses(12, sum(lens), 3, kind)
    for tau, recent in [(0.5, 0), (0.9, 5), (1.0, 2000)]:
        _compare_select(lens, cols, tau, recent, f"{kind} tau={tau}")
    small = [5, 1024, 17]
    _compare_select(small, I.synthetic_masses(13, sum(small), 1, kind), 0.3, 1, f"{kind} small")
    mid = [4096, 3000]
    _compare_select(mid, I.synthetic_masses(14, sum(mid), 2, kind), 0.8, 64, f"{kind} mid")


def test_select_tokens_special_values():
    """Ties, all-zero chunks, negative and NaN entries, an infinite mass."""
    _require_gpu()
    lens = [8, 6, 5, 4]
    cols = np.zeros((sum(lens), 2), dtype=np.float32)
    cols[0:8] = [[1, 1], [2, 0], [1, 1], [0.5, 0], [2, 0], [0, 0], [1, 1], [0.25, 0.25]]  # ties
    cols[8:14] = 0.0                                                                    # all zero
    cols[14:19] = [[1, -3], [np.nan, 1], [2, 0], [-0.0, -0.0], [1, 0]]
    cols[19:23] = [[1, 0], [np.inf, 0], [5, 0], [np.inf, 1]]
    for tau, recent in [(0.5, 0), (0.5, 1), (1.0, 0), (1e-9, 0)]:
        _compare_select(lens, cols, tau, recent, f"special tau={tau}")


# --------------------------------------------------------------------------
# the chain: GPU masses -> GPU selection, checked where the answer is unique
# --------------------------------------------------------------------------
def test_mass_then_select_end_to_end():
    _require_gpu()
    wl = I.build(_spec(name="chain", Hq=8, Hkv=2, q_lens=[300, 90], ctx_lens=[1200, 400]))
    dw = _gpu_masses(wl, "chain")
    tau, recent = 0.5, 16
    dw.select_tokens(tau, recent)
    torch.cuda.synchronize()
    q64 = wl.q("cpu").double().numpy()
    sel = PU.oracle_selection(wl, q64)
    scale = 1.0 / math.sqrt(wl.D)
    keep = dw.keep.cpu().numpy()
    tm = dw.tok_mass.cpu().numpy().astype(np.float64)
    for r in range(wl.B):
        q0, q1 = int(wl.q_indptr[r]), int(wl.q_indptr[r + 1])
        want_m = sum(M.unit_chunk_mass(q64[q0:q1, g * wl.G:(g + 1) * wl.G], PU.kv64(wl, r, g)[0],
                                       sel[r * wl.Hkv + g], wl.P, scale) for g in range(wl.Hkv))
        assert np.all(np.abs(tm[q0:q1] - want_m) <= MASS_RTOL * want_m + wl.Hkv * MASS_ATOL)
        # The GPU ranks and sums its own masses, each within the bound above of
        # the oracle's. A token is decided when every masses within the bounds
        # give the same answer: kept if even the most mass that can rank
        # before it stays below tau of the least possible total, dropped if
        # the least mass that must rank before it reaches tau of the most.
        n = q1 - q0
        lo = np.maximum(0.0, want_m * (1 - MASS_RTOL) - wl.Hkv * MASS_ATOL)
        hi = want_m * (1 + MASS_RTOL) + wl.Hkv * MASS_ATOL
        got = keep[q0:q1].astype(bool)
        assert got[n - recent:].all()
        decided = 0
        for k in range(n - recent):
            others = np.arange(n) != k
            may = others & (hi >= lo[k])
            must = others & (lo > hi[k])
            if hi[may].sum() < tau * lo.sum():
                assert got[k], (r, k)
                decided += 1
            elif lo[must].sum() >= tau * hi.sum():
                assert not got[k], (r, k)
                decided += 1
        want = M.select_tokens(want_m, tau, recent)
        print(f"[mass] chain request {r}: {decided}/{n - recent} decided, oracle keeps {want.size}, "
              f"GPU keeps {int(got.sum())}", flush=True)
        assert decided >= 0.9 * (n - recent)
        assert abs(int(got.sum()) - want.size) <= (n - recent) - decided


# --------------------------------------------------------------------------
# full size: 64 layers of Qwen3-32B-shaped heads, 512-token chunk at 32K
# --------------------------------------------------------------------------
def _selection_properties(tm, keep, kept, cnt, q0, n, tau, recent):
    """A valid SelectImportantTokens result for masses tm (checked in float64):
    outside the recent window the kept tokens are the top of the ranking (mass
    descending, position ascending), they reach tau of the total, and the top
    one fewer would not."""
    got = keep[q0:q0 + n].astype(bool)
    assert cnt == int(got.sum())
    np.testing.assert_array_equal(kept[q0:q0 + cnt], q0 + np.nonzero(got)[0])
    assert got[max(0, n - recent):].all()
    m = tm[q0:q0 + n].astype(np.float64)
    order = sorted(range(n), key=lambda k: (-m[k], k))
    run, last_old, gap = 0, 0, False
    for j, k in enumerate(order):
        if not got[k]:
            gap = True
        elif gap:
            assert k >= n - recent, f"token {k} kept below an unkept one"
        else:
            run = j + 1
            if k < n - recent:
                last_old = j + 1
    total = m.sum()
    if total > 0:
        s = np.cumsum(m[order])
        assert s[run - 1] >= tau * total * (1 - 1e-12)
        if last_old >= 2:
            assert s[last_old - 2] < tau * total * (1 + 1e-12)


def test_full_size_headclass_prefill_sampled():
    _require_gpu()
    wl = I.config(9)
    dw = _gpu_masses(wl, wl.spec.name + "/full")
    tau, recent = 0.2, 128
    dw.select_tokens(tau, recent)
    torch.cuda.synchronize()
    mass = dw.mass.cpu().numpy()
    keep = dw.keep.cpu().numpy()
    kept = dw.kept.cpu().numpy()
    cnt = dw.keep_count.cpu().numpy()
    tm = dw.tok_mass.cpu().numpy()
    # token mass = column sum of the per-head masses (float32, head order)
    ref = np.zeros(mass.shape[0], dtype=np.float32)
    for g in range(wl.Hkv):
        ref = (ref + mass[:, g]).astype(np.float32)
    np.testing.assert_array_equal(tm[:wl.total_q].view(np.uint32), ref[:wl.total_q].view(np.uint32))
    for r in [0, 17, wl.B - 1]:
        q0, n = int(wl.q_indptr[r]), int(wl.q_indptr[r + 1] - wl.q_indptr[r])
        _selection_properties(tm, keep, kept, int(cnt[r]), q0, n, tau, recent)
    # sampled tokens of sampled units against the oracle's own masses
    q64 = wl.q("cpu").double().numpy()
    units = [0, 1, 5 * wl.Hkv + 6, wl.num_units - 1]       # global and local heads
    sel = PU.oracle_selection(wl, q64, units=units)
    PU.compare_selection(wl, dw, q64, sel)
    scale = 1.0 / math.sqrt(wl.D)
    G = wl.G
    for u in units:
        r, g = divmod(u, wl.Hkv)
        q0, q1 = int(wl.q_indptr[r]), int(wl.q_indptr[r + 1])
        n = q1 - q0
        K, _ = PU.kv64(wl, r, g)
        qq = q64[q0:q1, g * G:(g + 1) * G]
        for k in (n - 1, n - 2, n - 33, n - 100):
            want = M.chunk_token_mass(qq, K, sel[u], wl.P, scale, k)
            got = float(mass[q0 + k, g])
            assert abs(got - want) <= MASS_RTOL * want + MASS_ATOL, (u, k, got, want)
