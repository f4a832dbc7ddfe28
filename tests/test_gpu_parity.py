"""GPU parity: the HIP path through the C-ABI against the fp64 oracle.

Sizes the oracle finishes in seconds that still span many tiles, several
waves per unit and ragged tails; then every named workload at full size in
the benchmark's launch configuration, on sampled units. Each case prints
its name before it touches the GPU.
"""
import os

import numpy as np
import pytest
import torch

from paper_2606_06256_amd import inputs as I
from paper_2606_06256_amd.device import DeviceWorkload

import parity_util as PU

pytestmark = pytest.mark.gpu


def _require_gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"


def _spec(**kw):
    base = dict(name="edge", B=2, Hq=8, Hkv=2, D=128, P=16, seg_tokens=256, ctx_lens=[700, 333],
                q_lens=[1, 1], seed=4242)
    base.update(kw)
    return I.Spec(**base)


# --------------------------------------------------------------------------
# the named workloads, scaled down (all units compared)
# --------------------------------------------------------------------------
def test_tiny_config_full():
    _require_gpu()
    PU.run_parity(I.config(1), label="tiny")


@pytest.mark.parametrize("i,div,batch", [(2, 16, 4), (3, 32, 6), (5, 32, 3), (10, 16, 3)])
def test_scaled_decode_configs(i, div, batch):
    _require_gpu()
    PU.run_parity(I.build(I.scaled_spec(i, div, batch)))


@pytest.mark.parametrize("i,div,batch", [(6, 1, 4), (7, 8, 3), (8, 32, 2), (9, 16, 3)])
def test_scaled_headclass_configs(i, div, batch):
    """The head-class micro-benchmark shape (global and local KV heads, one
    batched call over layers), decode and chunked prefill, at reduced sizes."""
    _require_gpu()
    PU.run_parity(I.build(I.scaled_spec(i, div, batch)))


def test_scaled_prefill_config():
    _require_gpu()
    sp = I.scaled_spec(4, 32, 2)
    sp.q_lens = [48, 31]
    sp.ctx_lens = [2048 + 48, 1500 + 31]
    sp.budgets = [40, 30]
    sp.forced_tail = 3
    PU.run_parity(I.build(sp), label="chunked_prefill/small")


# --------------------------------------------------------------------------
# shapes and edge cases
# --------------------------------------------------------------------------
EDGE = {
    "mha_d64": dict(Hq=4, Hkv=4, D=64),
    "gqa2": dict(Hq=4, Hkv=2),
    "gqa8": dict(Hq=16, Hkv=2),
    "gqa16": dict(Hq=32, Hkv=2),
    "page32": dict(P=32, seg_tokens=256),
    "page64_d64": dict(P=64, seg_tokens=512, D=64),
    "ctx_below_page": dict(ctx_lens=[5, 1]),
    "single_page": dict(ctx_lens=[16, 16]),
    "multi_query_causal": dict(q_lens=[3, 4], ctx_lens=[300, 129]),
    "chunk_g8": dict(Hq=16, Hkv=2, q_lens=[2, 2]),
    "rows_cross_blocks": dict(Hq=24, Hkv=2, q_lens=[5, 3], ctx_lens=[400, 64]),
    "random_forced": dict(sel_mode=I.SEL_RANDOM_HASH, budgets=[9, 4], forced_head=2, forced_tail=3,
                          sel_seed=77),
    "random_zero_budget": dict(sel_mode=I.SEL_RANDOM_HASH, budgets=[0, 2], sel_seed=5),
    "topk_p32": dict(sel_mode=I.SEL_TOPK_MEANKEY, P=32, budgets=[5, 3], shift_pages=2,
                     shift_mag=3.0),
    "topk_partial": dict(sel_mode=I.SEL_TOPK_MEANKEY, budgets=[7, 30], forced_tail=1,
                         ctx_lens=[701, 333]),
    "head_class": dict(sel_mode=I.SEL_HEAD_CLASS, Hkv=4, Hq=8, head_policy=[1, 0, 0, 1],
                       n_sink=4, window=100, ctx_lens=[1001, 300]),
    "head_class_chunk": dict(sel_mode=I.SEL_HEAD_CLASS, Hkv=2, Hq=4, head_policy=[0, 1],
                             n_sink=20, window=40, q_lens=[6, 2], ctx_lens=[900, 70]),
    "aliased_prefix": dict(B=3, ctx_lens=[600, 512, 300], q_lens=[1, 1, 1],
                           shared_prefix_segments=1),
    "spare_phys_pages": dict(extra_phys_pages=37),
    "scaled_keys": dict(k_page_scale_sigma=0.5, sel_mode=I.SEL_RANDOM_HASH, budgets=[20, 10]),
    # chunks of >= 128 query rows per unit run the matrix-core prefill kernel
    "prefill_g4": dict(q_lens=[40, 33], ctx_lens=[700, 333]),
    "prefill_d64_p32": dict(D=64, P=32, seg_tokens=256, q_lens=[64, 70], ctx_lens=[400, 300]),
    "prefill_mha": dict(Hq=2, Hkv=2, q_lens=[130, 200], ctx_lens=[400, 200]),
    "prefill_random_empty": dict(sel_mode=I.SEL_RANDOM_HASH, budgets=[0, 3], q_lens=[50, 40],
                                 ctx_lens=[500, 300], sel_seed=21),
    "prefill_forced_tail": dict(sel_mode=I.SEL_RANDOM_HASH, budgets=[12, 9], forced_tail=3,
                                q_lens=[45, 38], ctx_lens=[1500, 800], sel_seed=22),
    "prefill_head_class": dict(sel_mode=I.SEL_HEAD_CLASS, head_policy=[0, 1], n_sink=8, window=64,
                               q_lens=[40, 40], ctx_lens=[900, 300]),
    "prefill_rows_g16": dict(Hq=32, Hkv=2, q_lens=[33, 17], ctx_lens=[600, 256]),
    # either side of the switch between the two kernels (max_q_len * G = 128)
    "decode_rows_124": dict(q_lens=[31, 20], ctx_lens=[700, 333]),
    "prefill_rows_128": dict(q_lens=[32, 5], ctx_lens=[700, 333]),
    "decode_rows_112_g16": dict(Hq=32, Hkv=2, q_lens=[7, 3], ctx_lens=[500, 90]),
    "prefill_rows_128_g16": dict(Hq=32, Hkv=2, q_lens=[8, 8], ctx_lens=[500, 90]),
    "prefill_many_entries": dict(ctx_lens=[20000, 3000], q_lens=[40, 8], seg_tokens=4096),
    # per-page key scales (LogNormal): scores far apart within a row, so the
    # prefill's running reference max moves several times mid-stream
    "prefill_scaled_keys": dict(k_page_scale_sigma=1.0, q_lens=[60, 40], ctx_lens=[1500, 700]),
    "prefill_scaled_keys_d64": dict(D=64, k_page_scale_sigma=1.5, q_lens=[70, 35],
                                    ctx_lens=[1200, 400], sel_mode=I.SEL_RANDOM_HASH,
                                    budgets=[40, 20], forced_tail=5, sel_seed=13),
    # the largest page sizes: several 16-token tiles per page, partial last pages
    "page128": dict(P=128, seg_tokens=512, ctx_lens=[1000, 130]),
    "page256_d64": dict(P=256, seg_tokens=1024, D=64, ctx_lens=[2000, 257], q_lens=[3, 1]),
    "page128_prefill": dict(P=128, seg_tokens=512, ctx_lens=[900, 400], q_lens=[70, 40]),
    "page256_random": dict(P=256, seg_tokens=1024, sel_mode=I.SEL_RANDOM_HASH, budgets=[3, 2],
                           forced_tail=1, ctx_lens=[3000, 1500], q_lens=[1, 1], sel_seed=9),
    "page128_topk": dict(P=128, seg_tokens=512, sel_mode=I.SEL_TOPK_MEANKEY, budgets=[4, 2],
                         ctx_lens=[1800, 700]),
    # between 4096 and 8192 candidate pages: key high halves held in LDS
    "topk_4300_pages": dict(sel_mode=I.SEL_TOPK_MEANKEY, D=64, seg_tokens=4096, budgets=[300, 40],
                            ctx_lens=[4300 * 16 + 5, 900], shift_pages=40, shift_mag=3.0,
                            forced_tail=2),
    "random_4500_pages": dict(sel_mode=I.SEL_RANDOM_HASH, D=64, seg_tokens=4096, budgets=[350, 20],
                              ctx_lens=[4500 * 16 - 3, 700], forced_head=3, forced_tail=2,
                              sel_seed=31),
    # more candidate pages than the selection kernel keeps in LDS (8192): the
    # keys are recomputed in every radix pass
    "topk_uncached": dict(sel_mode=I.SEL_TOPK_MEANKEY, D=64, seg_tokens=4096, budgets=[500, 40],
                          ctx_lens=[8300 * 16 + 5, 900], shift_pages=60, shift_mag=3.0,
                          forced_tail=2),
    "random_uncached": dict(sel_mode=I.SEL_RANDOM_HASH, D=64, seg_tokens=4096, budgets=[700, 20],
                            ctx_lens=[8500 * 16 - 3, 700], forced_head=3, forced_tail=2,
                            sel_seed=31),
}


def test_topk_equal_scores_take_the_lowest_pages():
    """TOPK where every page of a unit scores the same (its key sums zeroed
    after the summary build): all 64 key bits tie, the radix passes run down
    to the low half of the keys and the threshold is decided by the page
    index; the selection must be the oracle's, i.e. the lowest pages. Units
    with whole keys in LDS (3,000 pages), with their high halves (6,000) and
    with none (9,000)."""
    _require_gpu()
    from oracle import segpa_oracle as O
    wl = I.build(_spec(name="topk_ties", B=3, sel_mode=I.SEL_TOPK_MEANKEY, D=64, seg_tokens=4096,
                       ctx_lens=[9000 * 16 - 5, 3000 * 16 + 3, 6000 * 16], q_lens=[1, 1, 1],
                       budgets=[600, 50, 400], forced_head=2, forced_tail=3))
    dw = DeviceWorkload(wl)
    dw.summary()
    dw.page_ksum.zero_()
    dw.select()
    torch.cuda.synchronize()
    ind, pages = dw.selection()
    q64 = wl.q("cpu").double().numpy()
    for u in range(wl.num_units):
        r, g = divmod(u, wl.Hkv)
        L, n = int(wl.ctx_lens[r]), int(wl.n_pages[r])
        valid = np.minimum(wl.P, L - np.arange(n) * wl.P)
        last = int(wl.q_indptr[r + 1]) - 1
        want, _ = O.pages_topk_meankey(q64[last, g * wl.G:(g + 1) * wl.G], np.zeros((n, wl.D)), valid,
                                       int(wl.budgets[r]), wl.spec.forced_head, wl.spec.forced_tail)
        got = pages[ind[u]:ind[u + 1]].tolist()
        assert got == list(want), f"unit {u}: {got[:8]} ... vs {list(want)[:8]} ..."



@pytest.mark.parametrize("name", sorted(EDGE))
def test_edge_cases(name):
    _require_gpu()
    PU.run_parity(I.build(_spec(name=name, **EDGE[name])), label=name)


def _random_spec(k: int):
    """A seeded random small workload: shapes, page sizes, chunk lengths,
    selection rules and their parameters all drawn from the supported ranges."""
    rng = np.random.default_rng(900 + k)
    Hkv = int(rng.choice([1, 2, 4]))
    G = int(rng.choice([1, 2, 3, 4, 8, 16]))
    D = int(rng.choice([64, 128]))
    P = int(rng.choice([16, 32, 64, 128, 256]))
    seg = P * int(rng.choice([1, 2, 4, 8]))
    B = int(rng.integers(1, 4))
    ctx = rng.integers(1, 1500, size=B)
    ql = [int(min(c, rng.choice([1, 1, 2, 5, 17, 40, 64]))) for c in ctx]
    mode = int(rng.choice([I.SEL_ALL, I.SEL_HEAD_CLASS, I.SEL_RANDOM_HASH, I.SEL_TOPK_MEANKEY]))
    npg = [-(-int(c) // P) for c in ctx]
    kw = dict(name=f"random{k}", B=B, Hq=Hkv * G, Hkv=Hkv, D=D, P=P, seg_tokens=seg,
              ctx_lens=ctx.tolist(), q_lens=ql, seed=5000 + k, sel_mode=mode)
    if mode in (I.SEL_RANDOM_HASH, I.SEL_TOPK_MEANKEY):
        kw["budgets"] = [int(rng.integers(0, n + 2)) for n in npg]
        kw["forced_head"] = int(rng.integers(0, 3))
        kw["forced_tail"] = int(rng.integers(0, 3))
        kw["sel_seed"] = int(rng.integers(0, 1 << 62))
    if mode == I.SEL_HEAD_CLASS:
        kw["head_policy"] = rng.integers(0, 2, size=Hkv).tolist()
        kw["n_sink"] = int(rng.integers(0, 40))
        kw["window"] = int(rng.integers(0, 600))
    return I.Spec(**kw)


@pytest.mark.parametrize("k", range(16))
def test_random_small_workloads(k):
    _require_gpu()
    sp = _random_spec(k)
    PU.run_parity(I.build(sp), label=f"{sp.name} B={sp.B} G={sp.Hq // sp.Hkv} D={sp.D} P={sp.P} "
                  f"q={list(sp.q_lens)} mode={sp.sel_mode}")


def test_many_units_short_lists():
    _require_gpu()
    B = 40
    rng = np.random.default_rng(8)
    ctx = rng.integers(1, 200, size=B).tolist()
    sp = _spec(name="many_units", B=B, Hq=8, Hkv=4, ctx_lens=ctx, q_lens=[1] * B,
               sel_mode=I.SEL_RANDOM_HASH, budgets=rng.integers(0, 6, size=B).tolist(), sel_seed=3)
    PU.run_parity(I.build(sp), label="many_units")


def test_max_units_per_call():
    """The largest unit count one call takes (B * Hkv = 8192): every unit's
    page list compared bit for bit, the outputs on a sample of units."""
    _require_gpu()
    B = 1024
    rng = np.random.default_rng(11)
    ctx = rng.integers(1, 160, size=B).tolist()
    sp = _spec(name="max_units", B=B, Hq=32, Hkv=8, ctx_lens=ctx, q_lens=[1] * B,
               sel_mode=I.SEL_RANDOM_HASH, budgets=rng.integers(0, 8, size=B).tolist(), sel_seed=5)
    wl = I.build(sp)
    assert wl.num_units == 8192
    PU.run_parity(wl, units=PU.sample_units(wl.num_units, 64), label="max_units")


def test_explicit_lists_with_empty_units():
    _require_gpu()
    wl = I.build(_spec(name="explicit", B=3, ctx_lens=[900, 40, 300], q_lens=[2, 1, 1]))
    dw = DeviceWorkload(wl)
    rng = np.random.default_rng(1)
    lists = []
    for u in range(wl.num_units):
        r = u // wl.Hkv
        n = int(wl.n_pages[r])
        k = 0 if u % 3 == 1 else int(rng.integers(1, n + 1))
        lists.append(sorted(rng.choice(n, size=k, replace=False).tolist()))
    dw.set_selection(lists)
    dw.fwd()
    torch.cuda.synchronize()
    q64 = wl.q("cpu").double().numpy()
    stats = PU.compare_outputs(wl, dw, q64, dict(enumerate(lists)), range(wl.num_units))
    print("[parity] explicit lists:", stats, flush=True)
    stats.check("explicit")
    lse = dw.lse.cpu().numpy()
    assert np.all(np.isneginf(lse[:2, 4:8]))           # request 0, KV head 1: empty list
    assert np.all(dw.out.float().cpu().numpy()[:2, 4:8] == 0)


# --------------------------------------------------------------------------
# invariances of the GPU path
# --------------------------------------------------------------------------
def test_split_count_invariance_and_determinism(monkeypatch):
    _require_gpu()
    wl = I.build(I.scaled_spec(2, 8, 4))
    outs = []
    for blocks in ("1", "3", "8"):
        monkeypatch.setenv("SEGPA_DECODE_BLOCKS_PER_CU", blocks)
        print(f"[split] blocks per CU {blocks}", flush=True)
        dw = DeviceWorkload(wl)
        dw.step()
        dw.fwd()
        torch.cuda.synchronize()
        first = dw.out.clone()
        dw.fwd()
        torch.cuda.synchronize()
        assert torch.equal(first, dw.out), "run-to-run results differ"
        outs.append(first.float())
        del dw
    for o in outs[1:]:
        assert float((o - outs[0]).abs().max()) <= 1e-2


@pytest.mark.parametrize("cfg", ["decode", "topk", "prefill"])
def test_step_replays_from_a_hip_graph(cfg):
    """select + fwd captured once in a HIP graph (torch.cuda.graph records the
    library's launches on its capture stream) replay to the eager result, bit
    for bit, on several replays with eager work and synchronisations between
    them (the library records no memset or host sync in these calls)."""
    _require_gpu()
    spec = {"decode": I.scaled_spec(2, 8, 4), "topk": I.scaled_spec(5, 32, 2),
            "prefill": I.scaled_spec(4, 64, 2)}[cfg]
    wl = I.build(spec)
    print(f"[graph] {wl.spec.name}", flush=True)
    dw = DeviceWorkload(wl)
    if wl.spec.sel_mode == I.SEL_TOPK_MEANKEY:
        dw.summary()
    dw.step()
    torch.cuda.synchronize()
    ref_o, ref_l = dw.out.clone(), dw.lse.clone()
    ref_ind, ref_pages = dw.selection()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        dw.step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        dw.step()
    torch.cuda.synchronize()
    for it in range(3):
        dw.out.zero_()
        dw.lse.zero_()
        dw.sel_pages.zero_()
        dw.sel_indptr.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(dw.out, ref_o), f"replay {it}: output differs from eager"
        assert torch.equal(dw.lse, ref_l), f"replay {it}: lse differs from eager"
        ind, pages = dw.selection()
        assert np.array_equal(ind, ref_ind) and np.array_equal(pages, ref_pages), f"replay {it}: selection"
        float((dw.out.float() * 2.0).sum())   # eager work between replays


def test_two_streams_run_independently():
    """Two workloads with their own workspaces, stepped on two streams at the
    same time (several rounds), give the results each gives alone."""
    _require_gpu()
    wa = I.build(I.scaled_spec(2, 8, 4))
    wb = I.build(I.scaled_spec(4, 64, 2))      # a chunked prefill next to a decode
    da, db = DeviceWorkload(wa), DeviceWorkload(wb)
    da.step()
    db.step()
    torch.cuda.synchronize()
    ref = [(da.out.clone(), da.lse.clone()), (db.out.clone(), db.lse.clone())]
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    for it in range(3):
        for dw in (da, db):
            dw.out.zero_()
            dw.lse.zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(sa):
            da.step()
        with torch.cuda.stream(sb):
            db.step()
        torch.cuda.synchronize()
        for dw, (ro, rl) in zip((da, db), ref):
            assert torch.equal(dw.out, ro) and torch.equal(dw.lse, rl), f"{dw.wl.spec.name} round {it}"


@pytest.mark.parametrize("cfg", ["decode", "prefill"])
def test_fwd_without_lse(cfg):
    """lse may be NULL: the output is the same as with it (decode with split
    partials, and the chunked prefill)."""
    _require_gpu()
    from paper_2606_06256_amd import binding as B
    spec = {"decode": I.scaled_spec(2, 8, 4), "prefill": I.scaled_spec(4, 64, 2)}[cfg]
    dw = DeviceWorkload(I.build(spec))
    dw.step()
    torch.cuda.synchronize()
    ref = dw.out.clone()
    dw.out.zero_()
    B.seg_paged_attn_fwd(dw.dims, dw.q, dw.q_indptr, dw.ctx_lens, dw.k_pool, dw.v_pool, dw.seg_table,
                         dw.page_table, dw.sel_indptr, dw.sel_pages, dw.out, None, dw.workspace)
    torch.cuda.synchronize()
    assert torch.equal(dw.out, ref)


def test_physical_placement_invariance():
    _require_gpu()
    wl = I.build(_spec(name="placement", P=32, ctx_lens=[1200, 555], q_lens=[2, 1],
                       sel_mode=I.SEL_RANDOM_HASH, budgets=[20, 9], sel_seed=11))
    a = DeviceWorkload(wl)
    a.step()
    perm = torch.from_numpy(np.random.default_rng(2).permutation(wl.num_phys)).cuda()
    b = DeviceWorkload(wl)
    b.k_pool = torch.empty_like(a.k_pool)
    b.v_pool = torch.empty_like(a.v_pool)
    b.k_pool[perm] = a.k_pool
    b.v_pool[perm] = a.v_pool
    b.page_table = perm.to(torch.int32)[a.page_table.long()].contiguous()
    b.step()
    torch.cuda.synchronize()
    assert torch.equal(a.sel_indptr, b.sel_indptr) and torch.equal(a.sel_pages, b.sel_pages)
    assert torch.equal(a.out, b.out) and torch.equal(a.lse, b.lse)


@pytest.mark.parametrize("q_lens", [[1, 1], [40, 33]])
def test_stale_slots_never_reach_the_result(q_lens):
    """Slots past the context in a page and unused pages may hold anything (here
    NaN): they never enter the softmax, so results are bitwise unchanged."""
    _require_gpu()
    wl = I.build(_spec(name="stale", P=32, ctx_lens=[701, 333], q_lens=q_lens, extra_phys_pages=9))
    clean = DeviceWorkload(wl)
    clean.step()
    dirty = DeviceWorkload(wl)
    nan = torch.tensor(float("nan"), dtype=torch.bfloat16, device="cuda")
    used = torch.zeros(wl.num_phys, dtype=torch.bool)
    for r in range(wl.B):
        L = int(wl.ctx_lens[r])
        for g in range(wl.Hkv):
            ph = wl.unit_phys_pages(r, g)
            used[torch.from_numpy(ph.astype(np.int64))] = True
            last = int(ph[-1])
            valid = L - (len(ph) - 1) * wl.P
            kt = dirty.k_pool[last].view(wl.P // 16, wl.D // 8, 16, 8)
            vt = dirty.v_pool[last].view(wl.P // 16, wl.D, 16)
            for t in range(valid, wl.P):
                kt[t // 16, :, t % 16, :] = nan
                vt[t // 16, :, t % 16] = nan
    dirty.k_pool[~used.cuda()] = nan
    dirty.v_pool[~used.cuda()] = nan
    dirty.step()
    torch.cuda.synchronize()
    assert torch.equal(clean.out, dirty.out) and torch.equal(clean.lse, dirty.lse)
    assert torch.isfinite(dirty.out.float()).all()


def test_page_summary_bit_exact():
    _require_gpu()
    from oracle import segpa_oracle as O
    wl = I.build(_spec(name="ksum", P=32, ctx_lens=[1000, 77], sel_mode=I.SEL_TOPK_MEANKEY,
                       budgets=[3, 2], shift_pages=3, shift_mag=3.0))
    dw = DeviceWorkload(wl)
    dw.summary()
    torch.cuda.synchronize()
    ks = dw.page_ksum.cpu().numpy()
    for r in range(wl.B):
        for g in range(wl.Hkv):
            K, _ = PU.kv64(wl, r, g)
            want, _ = O.unit_key_sums(K, wl.P)
            got = ks[wl.unit_phys_pages(r, g)]
            assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_generated_pool_matches_cpu_generation():
    _require_gpu()
    wl = I.build(I.scaled_spec(3, 16, 3))
    dw = DeviceWorkload(wl)
    kp, vp = dw.k_pool.cpu(), dw.v_pool.cpu()
    for r in range(wl.B):
        for g in (0, wl.Hkv - 1):
            K, V = wl.unit_kv(r, g, "cpu")
            kt, vt = wl.tile_unit(K, V, int(wl.n_pages[r]))
            ph = torch.from_numpy(wl.unit_phys_pages(r, g).astype(np.int64))
            assert torch.equal(kp[ph], kt) and torch.equal(vp[ph], vt)


def test_validate_reports_bad_lists():
    _require_gpu()
    wl = I.build(_spec(name="validate", sel_mode=I.SEL_RANDOM_HASH, budgets=[10, 5], sel_seed=9))
    dw = DeviceWorkload(wl)
    dw.select()
    st, code, idx = dw.validate()
    assert (st, code) == (0, 0)
    good = dw.sel_pages.clone()
    n0 = int(wl.n_pages[0])
    dw.sel_pages[3] = n0 + 5                    # page id past the context
    st, code, idx = dw.validate()
    assert st == -6 and code == 4 and idx == 3
    dw.fwd()                                    # never faults: the bad page is skipped
    torch.cuda.synchronize()
    dw.sel_pages.copy_(good)
    dw.sel_pages[2], dw.sel_pages[3] = good[3], good[2]   # not ascending
    st, code, idx = dw.validate()
    assert st == -6 and code == 4 and idx in (2, 3)
    dw.sel_pages.copy_(good)
    ind = dw.sel_indptr.clone()
    dw.sel_indptr[1] = ind[2] + 1
    st, code, idx = dw.validate()
    assert st == -6 and code == 3


def test_validate_switch_stops_fwd_on_bad_lists(monkeypatch):
    """With SEGPA_VALIDATE set, fwd runs the list check first and refuses bad
    data (SPA_ERR_BAD_DATA, nothing launched); good data gives the ordinary
    result; unset, the bad page is skipped as usual."""
    _require_gpu()
    from paper_2606_06256_amd import binding as B
    wl = I.build(_spec(name="validate_switch", sel_mode=I.SEL_RANDOM_HASH, budgets=[10, 5],
                       sel_seed=9))
    dw = DeviceWorkload(wl)
    dw.select()
    dw.fwd()
    torch.cuda.synchronize()
    want = dw.out.clone()
    monkeypatch.setenv("SEGPA_VALIDATE", "1")
    dw.out.zero_()
    dw.fwd()                                    # good lists: checked, then the same result
    torch.cuda.synchronize()
    assert torch.equal(dw.out, want)
    good = dw.sel_pages.clone()
    dw.sel_pages[3] = int(wl.n_pages[0]) + 5    # page id past the context
    dw.out.fill_(3.0)
    with pytest.raises(B.SegpaError) as e:
        dw.fwd()
    assert e.value.status == -6
    torch.cuda.synchronize()
    assert bool((dw.out == 3.0).all())          # nothing was launched
    monkeypatch.setenv("SEGPA_VALIDATE", "0")
    dw.fwd()                                    # switch off: the bad page is skipped
    torch.cuda.synchronize()
    dw.sel_pages.copy_(good)


# --------------------------------------------------------------------------
# full-size workloads in the benchmark's launch configuration
# --------------------------------------------------------------------------
@pytest.mark.parametrize("i", [2, 3, 4, 5, 6, 7, 8, 9, 10])
def test_full_size_config(i):
    _require_gpu()
    wl = I.config(i)
    U = wl.num_units
    units = PU.sample_units(U, 3)
    # selections: every unit for the seeded rules, sampled units for TOPK
    sel_units = units if wl.spec.sel_mode == I.SEL_TOPK_MEANKEY else None
    PU.run_parity(wl, units=units, sel_units=sel_units, label=wl.spec.name + "/full")
