"""Pins of the fp64 oracle against facts other than itself.

Each test checks the oracle against something it does not compute itself:
a value the paper prints, a library routine on a special case, pure-Python
brute force on tiny inputs, a closed form, or an invariant. The tests are
chosen so that a plausible slip in the oracle fails at least one of them.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import segpa_oracle as O
from paper_2606_06256_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _rng(seed):
    return np.random.default_rng(seed)


# --------------------------------------------------------------------------
# worked example and closed forms for the head-class policy
# --------------------------------------------------------------------------
def test_window_worked_example():
    g = _golden("window_example.json")
    W = O.visible_window(g["i"], g["w"], sink=[])
    assert min(W) == g["window_first"] and max(W) == g["window_last"]
    assert W == set(range(g["window_first"], g["window_last"] + 1))
    Ws = O.visible_window(g["i"], g["w"], sink=range(4))
    assert Ws == set(range(4)) | set(range(744, 1001))


def test_window_clamps_at_zero():
    assert O.visible_window(10, 256, sink=[]) == set(range(0, 11))


def test_head_class_decode_example_pages():
    # decode query at i = 1000 (L = 1001), w = 256, page 16, 4 sink tokens:
    # sink page 0 plus the pages covering 744..1000 = pages 46..62
    pages = O.pages_head_class(O.LOCAL, L=1001, n_q=1, P=16, n_sink=4, w=256)
    assert pages == [0] + list(range(46, 63))


def _local_pages_closed_form(L, n_q, P, n_sink, w):
    # union over the chunk's queries of [max(0, i - w), i] is one interval
    lo, hi = max(0, L - n_q - w), L - 1
    out = []
    for p in range((L + P - 1) // P):
        a, b = p * P, min(L, (p + 1) * P) - 1
        if (n_sink > 0 and a <= min(n_sink, L) - 1) or (a <= hi and b >= lo):
            out.append(p)
    return out


@pytest.mark.parametrize("seed", range(40))
def test_head_class_local_matches_interval_overlap(seed):
    r = _rng(seed)
    P = int(r.choice([16, 32]))
    L = int(r.integers(1, 700))
    n_q = int(r.integers(1, min(L, 40) + 1))
    n_sink = int(r.integers(0, 40))
    w = int(r.integers(0, 300))
    got = O.pages_head_class(O.LOCAL, L, n_q, P, n_sink, w)
    assert got == _local_pages_closed_form(L, n_q, P, n_sink, w)


def test_head_class_global_is_all():
    for L in (1, 15, 16, 17, 1000):
        assert O.pages_head_class(O.GLOBAL, L, 1, 16, 4, 256) == list(range(-(-L // 16)))


# --------------------------------------------------------------------------
# SplitMix64 and the seeded sampler
# --------------------------------------------------------------------------
def test_splitmix64_published_outputs():
    g = _golden("splitmix64_seed0.json")
    state = g["state0"]
    for want in g["outputs_hex"]:
        assert O.splitmix64(state) == int(want, 16)
        state = (state + 0x9E3779B97F4A7C15) & O.MASK64


def test_splitmix64_mix_is_bijective_on_sample():
    # the mixer is a composition of invertible steps: no collisions on a sample
    xs = list(range(0, 1 << 16)) + [(1 << 63) + i for i in range(1 << 12)]
    assert len({O.splitmix64_mix(x) for x in xs}) == len(xs)


@pytest.mark.parametrize("n,budget,fh,ft", [(10, 3, 0, 0), (10, 3, 2, 2), (10, 0, 1, 1),
                                            (5, 9, 0, 0), (8, 4, 6, 6), (1, 1, 0, 0),
                                            (0, 3, 1, 1), (2048, 512, 128, 128)])
def test_selection_count_closed_form(n, budget, fh, ft):
    forced = len(set(range(min(n, fh))) | set(range(max(0, n - ft), n)))
    assert forced == min(n, min(n, fh) + min(n, ft))
    want = min(n, max(budget, forced))
    assert O.selection_count(n, budget, fh, ft) == want
    pages = O.pages_random_hash(7, 1, 2, n, budget, fh, ft)
    assert len(pages) == want
    assert pages == sorted(set(pages))
    assert set(range(min(n, fh))) <= set(pages)
    assert set(range(max(0, n - ft), n)) <= set(pages)


def test_random_hash_is_smallest_keys():
    seed, r, g, n, k = 99, 3, 5, 300, 40
    keys = [(O.page_hash(seed, r, g, p), p) for p in range(n)]
    want = sorted(p for _, p in sorted(keys)[:k])
    assert O.pages_random_hash(seed, r, g, n, k, 0, 0) == want


def test_random_hash_uniform_inclusion():
    # every non-forced page is included with probability k'/n'; chi-square over seeds
    n, k, fh, ft, trials = 24, 8, 2, 2, 1500
    counts = np.zeros(n)
    for s in range(trials):
        for p in O.pages_random_hash(s, 0, 0, n, k, fh, ft):
            counts[p] += 1
    assert np.all(counts[:2] == trials) and np.all(counts[-2:] == trials)
    mid = counts[2:-2]
    expect = trials * (k - 4) / (n - 4)
    chi2 = float(np.sum((mid - expect) ** 2 / expect))
    # 19 degrees of freedom (inclusion counts are mildly negatively correlated,
    # which only lowers chi2); 45 is beyond the 0.999 quantile (43.8)
    assert chi2 < 45.0, chi2


def test_random_hash_depends_on_unit_and_seed():
    a = O.pages_random_hash(1, 0, 0, 500, 50, 0, 0)
    assert a != O.pages_random_hash(2, 0, 0, 500, 50, 0, 0)
    assert a != O.pages_random_hash(1, 1, 0, 500, 50, 0, 0)
    assert a != O.pages_random_hash(1, 0, 1, 500, 50, 0, 0)
    assert a == O.pages_random_hash(1, 0, 0, 500, 50, 0, 0)


# --------------------------------------------------------------------------
# page key sums and mean-key top-k
# --------------------------------------------------------------------------
def _f32_round_exact(fr: Fraction) -> float:
    """Independent round-to-nearest-even of an exact rational to float32 (normal range)."""
    if fr == 0:
        return 0.0
    sign = -1 if fr < 0 else 1
    a = abs(fr)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    quantum = Fraction(2) ** (e - 23)
    q = a / quantum
    n = math.floor(q)
    rem = q - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return sign * float(n * quantum)


def test_page_key_sum_rounding_cases():
    cases = [
        [1.0, 2.0 ** -24],                 # tie: 1 + 2^-24 -> 1 (even)
        [1.0, 3 * 2.0 ** -24],             # 1 + 3*2^-24 -> 1 + 2^-22
        [3.0, -3.0, 2.0 ** -30],           # cancellation
        [1.0, 2.0 ** -24, 2.0 ** -40],     # just above the tie -> rounds up
        [0.0, 0.0],
    ]
    for vals in cases:
        got = O.page_key_sum(np.array(vals)[:, None])[0]
        exact = sum(Fraction(v) for v in vals)
        assert float(got) == _f32_round_exact(exact), vals
    assert float(O.page_key_sum(np.array([1.0, 2.0 ** -24, 2.0 ** -40])[:, None])[0]) == 1.0 + 2.0 ** -23


def test_page_key_sum_matches_exact_on_bf16_data():
    r = _rng(5)
    x = torch.from_numpy(r.standard_normal((32, 16)) * 3).to(torch.bfloat16).double().numpy()
    got = O.page_key_sum(x)
    for d in range(16):
        assert float(got[d]) == _f32_round_exact(sum(Fraction(v) for v in x[:, d].tolist()))


def test_meankey_scores_exact_against_fractions():
    r = _rng(11)
    G, D, n = 4, 16, 9
    q = torch.from_numpy(r.standard_normal((G, D))).to(torch.bfloat16).double().numpy()
    K = torch.from_numpy(r.standard_normal((n * 16 - 5, D))).to(torch.bfloat16).double().numpy()
    ksum, valid = O.unit_key_sums(K, 16)
    assert list(valid) == [16] * 8 + [11]
    got = O.meankey_scores(q, ksum, valid)
    qbar = [sum(Fraction(v) for v in q[:, d].tolist()) for d in range(D)]
    for p in range(n):
        want = sum(qbar[d] * Fraction(float(ksum[p, d])) for d in range(D)) / int(valid[p])
        assert got[p] == want
        approx = float(np.dot(q.sum(0), ksum[p].astype(np.float64)) / valid[p])
        assert abs(float(got[p]) - approx) <= 1e-12 * max(1.0, abs(approx))


def test_topk_ties_go_to_lower_index():
    # identical pages -> identical scores: the budget takes the lowest indices
    P, n = 16, 12
    K = np.ones((n * P, 8))
    q = np.ones((2, 8))
    ksum, valid = O.unit_key_sums(K, P)
    got, _ = O.pages_topk_meankey(q, ksum, valid, budget=5, forced_head=0, forced_tail=2)
    assert got == [0, 1, 2, 10, 11]
    K[7 * P:8 * P] = 2.0          # one strictly better page enters first
    ksum, valid = O.unit_key_sums(K, P)
    got, _ = O.pages_topk_meankey(q, ksum, valid, budget=3)
    assert got == [0, 1, 7]


@pytest.mark.parametrize("seed", range(24))
def test_topk_matches_subset_bruteforce(seed):
    r = _rng(100 + seed)
    n = int(r.integers(3, 11))
    P, G = 16, 2
    D = 2 if seed % 2 else 4
    L = n * P - int(r.integers(0, P))
    # small integers create exact ties between page scores
    lim = 1 if seed % 2 else 2
    K = r.integers(-lim, lim + 1, size=(L, D)).astype(np.float64)
    if seed % 3 == 0:
        K[: (L // P) * P] = np.repeat(K[:P][None], L // P, axis=0).reshape(-1, D)
    q = r.integers(-2, 3, size=(G, D)).astype(np.float64)
    budget = int(r.integers(0, n + 1))
    fh, ft = int(r.integers(0, 2)), int(r.integers(0, 2))
    ksum, valid = O.unit_key_sums(K, P)
    got, scores = O.pages_topk_meankey(q, ksum, valid, budget, fh, ft)
    # brute force: among subsets that contain the forced pages and have the
    # right size, maximise the exact score sum; ties -> lexicographically smallest
    forced = set(range(min(n, fh))) | set(range(max(0, n - ft), n))
    size = min(n, max(budget, len(forced)))
    exact = []
    for p in range(n):
        s = sum(Fraction(float(q[:, d].sum())) * Fraction(float(ksum[p, d])) for d in range(D))
        exact.append(s / int(valid[p]))
    best = None
    for sub in itertools.combinations(range(n), size):
        if not forced <= set(sub):
            continue
        key = (-sum(exact[p] for p in sub), sub)
        if best is None or key < best:
            best = key
    assert got == list(best[1])


# --------------------------------------------------------------------------
# attention: library routine, brute force, invariants
# --------------------------------------------------------------------------
def _bf16(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float32)).to(torch.bfloat16).double().numpy()


def _random_unit(seed, L, D, G, n_q):
    r = _rng(seed)
    q = _bf16(r.standard_normal((n_q, G, D)))
    K = _bf16(r.standard_normal((L, D)))
    V = _bf16(r.standard_normal((L, D)))
    return q, K, V


def _sdpa_on_tokens(q, K, V, T, L, scale):
    """torch SDPA (float64, CPU) over the gathered tokens T with a bottom-right causal mask."""
    n_q, G, D = q.shape
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]                     # [1, G, n_q, D]
    kt = torch.from_numpy(K[T])[None, None].expand(1, G, len(T), D)
    vt = torch.from_numpy(V[T])[None, None].expand(1, G, len(T), D)
    pos = torch.arange(n_q)[:, None] + (L - n_q)
    mask = torch.from_numpy(T)[None, :] <= pos                          # [n_q, |T|]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)
    return o[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("L,D,G,n_q,P", [(1024, 64, 1, 1, 16), (333, 128, 4, 1, 16),
                                         (200, 64, 8, 5, 32), (64, 128, 2, 64, 16)])
def test_full_selection_equals_sdpa(L, D, G, n_q, P):
    q, K, V = _random_unit(L + D, L, D, G, n_q)
    scale = 1 / math.sqrt(D)
    Oo, _ = O.attend_unit(q, K, V, O.pages_all(L, P), P, scale)
    ref = _sdpa_on_tokens(q, K, V, np.arange(L), L, scale)
    np.testing.assert_allclose(Oo, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_sparse_equals_sdpa_on_gathered_tokens(seed):
    r = _rng(seed)
    P = 16
    L = int(r.integers(40, 400))
    n = -(-L // P)
    n_q = int(r.integers(1, 6))
    pages = sorted(r.choice(n, size=int(r.integers(1, n + 1)), replace=False).tolist())
    q, K, V = _random_unit(seed, L, 64, 4, n_q)
    Oo, _ = O.attend_unit(q, K, V, pages, P, 0.125)
    T = np.array([t for p in pages for t in range(p * P, min(L, p * P + P))])
    # queries with no visible token are excluded from the library check
    ok = np.array([np.any(T <= L - n_q + i) for i in range(n_q)])
    ref = _sdpa_on_tokens(q, K, V, T, L, 0.125)
    np.testing.assert_allclose(Oo[ok], ref[ok], rtol=0, atol=1e-12)


def test_bruteforce_loops_tiny():
    P = 16
    for seed, (B, L, n_q) in enumerate([(1, 37, 1), (2, 64, 3)]):
        r = _rng(200 + seed)
        D, G = 8, 2
        for b in range(B):
            q, K, V = _random_unit(300 + 10 * seed + b, L, D, G, n_q)
            pages = sorted(r.choice(-(-L // P), size=2, replace=False).tolist())
            Oo, LSE = O.attend_unit(q, K, V, pages, P, 0.3)
            for i in range(n_q):
                for h in range(G):
                    toks = [t for p in pages for t in range(p * P, p * P + P)
                            if t < L and t <= L - n_q + i]
                    if not toks:
                        assert LSE[i, h] == -math.inf and np.all(Oo[i, h] == 0)
                        continue
                    s = []
                    for t in toks:
                        acc = 0.0
                        for d in range(D):
                            acc += q[i, h, d] * K[t, d]
                        s.append(0.3 * acc)
                    m = max(s)
                    z = sum(math.exp(x - m) for x in s)
                    for d in range(D):
                        o = sum(math.exp(x - m) * V[t, d] for x, t in zip(s, toks)) / z
                        assert abs(o - Oo[i, h, d]) < 1e-12
                    assert abs(m + math.log(z) - LSE[i, h]) < 1e-12


def test_weights_sum_to_one_and_output_in_hull():
    q, K, V = _random_unit(7, 500, 64, 4, 1)
    pages = [0, 3, 7, 30, 31]
    T = O.selected_tokens(pages, 500, 16)
    Oo, _ = O.attend_unit(q, K, V, pages, 16, 0.125)
    for h in range(4):
        w = O.attention_weights(q[0, h], K, T, 0.125)
        assert abs(w.sum() - 1.0) < 1e-13 and np.all(w >= 0)
        np.testing.assert_allclose(w @ V[T], Oo[0, h], atol=1e-13)
        assert np.all(Oo[0, h] <= V[T].max(0) + 1e-12) and np.all(Oo[0, h] >= V[T].min(0) - 1e-12)


def test_empty_selection():
    q, K, V = _random_unit(8, 100, 64, 2, 3)
    Oo, LSE = O.attend_unit(q, K, V, [], 16, 0.125)
    assert np.all(Oo == 0) and np.all(LSE == -np.inf)


def test_lse_merge_exact_split():
    """Section 4.4: attention over A U B equals the LSE merge of A and B."""
    q, K, V = _random_unit(9, 900, 128, 4, 2)
    pages = list(range(0, 57, 2))
    A, Bp = pages[::3], [p for p in pages if p not in pages[::3]]
    whole = O.attend_unit(q, K, V, pages, 16, 1 / math.sqrt(128))
    a = O.attend_unit(q, K, V, A, 16, 1 / math.sqrt(128))
    b = O.attend_unit(q, K, V, Bp, 16, 1 / math.sqrt(128))
    m = O.lse_merge([a, b])
    np.testing.assert_allclose(m[0], whole[0], atol=1e-13)
    np.testing.assert_allclose(m[1], whole[1], atol=1e-12)
    # an empty part changes nothing
    e = O.attend_unit(q, K, V, [], 16, 1 / math.sqrt(128))
    m2 = O.lse_merge([whole, e])
    np.testing.assert_allclose(m2[0], whole[0], atol=1e-15)
    np.testing.assert_allclose(m2[1], whole[1], atol=1e-15)


def test_true_eviction_differs_from_zero_fill():
    """Section 5.4: an evicted page contributes no mass; a zero-filled one does."""
    L, D, P = 256, 64, 16
    q, K, V = _random_unit(10, L, D, 1, 1)
    keep = [0, 1, 2, 5, 15]
    evicted = O.attend_unit(q, K, V, keep, P, 0.125)
    Kz = K.copy()
    Kz[9 * P:10 * P] = 0.0
    zero = O.attend_unit(q, Kz, V, keep + [9], P, 0.125)
    # zero keys score 0: the merge adds 16 * exp(0) mass of page 9's values
    Z = math.exp(evicted[1][0, 0])
    extra = P * 1.0
    want = (Z * evicted[0][0, 0] + V[9 * P:10 * P].sum(0)) / (Z + extra)
    np.testing.assert_allclose(zero[0][0, 0], want, atol=1e-12)
    assert np.max(np.abs(zero[0] - evicted[0])) > 1e-3
    # pages outside the selection never matter
    Kx = K.copy()
    Kx[9 * P:10 * P] = 1e6
    again = O.attend_unit(q, Kx, V, keep, P, 0.125)
    np.testing.assert_array_equal(again[0], evicted[0])


# --------------------------------------------------------------------------
# paging: pool layout and placement invariance
# --------------------------------------------------------------------------
def _small_workload(**kw):
    base = dict(name="t", B=2, Hq=8, Hkv=2, D=64, P=16, seg_tokens=64, ctx_lens=[150, 64],
                q_lens=[1, 2], seed=77)
    base.update(kw)
    return I.build(I.Spec(**base))


def test_pool_roundtrip_through_tables():
    w = _small_workload()
    kp, vp = w.build_pool("cpu")
    for r in range(w.B):
        for g in range(w.Hkv):
            K, V = w.unit_kv(r, g)
            Kp, Vp = O.unit_kv_from_pool(kp.double().numpy(), vp.double().numpy(),
                                         w.seg_table[r, g], w.page_table, w.pps,
                                         int(w.ctx_lens[r]), w.P, w.D)
            np.testing.assert_array_equal(Kp, K.double().numpy())
            np.testing.assert_array_equal(Vp, V.double().numpy())


def test_placement_invariance():
    w = _small_workload(P=32, seg_tokens=64, ctx_lens=[300, 97])
    kp, vp = w.build_pool("cpu")
    r = _rng(3)
    perm = r.permutation(w.num_phys)          # physical page x moves to perm[x]
    kp2 = torch.zeros_like(kp)
    vp2 = torch.zeros_like(vp)
    kp2[torch.from_numpy(perm)] = kp
    vp2[torch.from_numpy(perm)] = vp
    pt2 = perm[w.page_table]
    q = w.q().double().numpy()
    for u in range(w.num_units):
        rr, g = divmod(u, w.Hkv)
        L = int(w.ctx_lens[rr])
        a = O.unit_kv_from_pool(kp.double().numpy(), vp.double().numpy(), w.seg_table[rr, g],
                                w.page_table, w.pps, L, w.P, w.D)
        b = O.unit_kv_from_pool(kp2.double().numpy(), vp2.double().numpy(), w.seg_table[rr, g],
                                pt2, w.pps, L, w.P, w.D)
        pages = list(range(0, -(-L // w.P), 2))
        oa = O.forward_unit(q, w.q_indptr, w.ctx_lens, w.Hq, w.Hkv, w.P, u, pages, *a)
        ob = O.forward_unit(q, w.q_indptr, w.ctx_lens, w.Hq, w.Hkv, w.P, u, pages, *b)
        np.testing.assert_array_equal(oa[0], ob[0])
        np.testing.assert_array_equal(oa[1], ob[1])


def test_aliased_segments_read_the_same_pages():
    w = _small_workload(B=3, ctx_lens=[256, 200, 130], q_lens=[1, 1, 1], shared_prefix_segments=2)
    assert np.array_equal(w.seg_table[1, :, :2], w.seg_table[0, :, :2])
    kp, vp = w.build_pool("cpu")
    for r in (1, 2):
        for g in range(w.Hkv):
            K, _ = w.unit_kv(r, g)
            Kp, _ = O.unit_kv_from_pool(kp.double().numpy(), vp.double().numpy(), w.seg_table[r, g],
                                        w.page_table, w.pps, int(w.ctx_lens[r]), w.P, w.D)
            np.testing.assert_array_equal(Kp, K.double().numpy())
            K0, _ = w.unit_kv(0, g)
            np.testing.assert_array_equal(K.double().numpy()[:128], K0.double().numpy()[:128])


def test_translate_rejects_unmapped_segment():
    with pytest.raises(ValueError):
        O.translate([3, -1], [0, 1, 2, 3, 4, 5, 6, 7], 2, 2)


def test_forward_unit_bruteforce_gqa_rows_and_default_scale():
    """forward_unit against pure-Python loops over the whole call's layout.

    Two requests with ragged query chunks (so request 1's rows start at a
    nonzero offset of q_indptr), Hq = 8 query heads over Hkv = 2 KV heads
    (G = 4). Query head h must read KV head h // G (contiguous groups), its
    rows must be q_indptr[r] .. q_indptr[r+1]-1, and the default scale must
    be 1/sqrt(D). Each KV head has its own keys, so a wrong head map, a wrong
    row offset or another scale changes the result.
    """
    P, D, Hq, Hkv = 16, 8, 8, 2
    G = Hq // Hkv
    ctx = [45, 70]
    q_lens = [3, 5]
    q_indptr = np.array([0, 3, 8])
    r0 = _rng(4242)
    q_all = _bf16(r0.standard_normal((8, Hq, D)))
    KV = {(r, g): (_bf16(r0.standard_normal((ctx[r], D))), _bf16(r0.standard_normal((ctx[r], D))))
          for r in range(2) for g in range(Hkv)}
    pages = {(0, 0): [0, 2], (0, 1): [1, 2], (1, 0): [0, 3, 4], (1, 1): [2, 4]}
    scale = 1.0 / math.sqrt(D)
    for r in range(2):
        L, n_q = ctx[r], q_lens[r]
        for h in range(Hq):
            kv = h // G                                # the head map under test
            K, V = KV[(r, kv)]
            Oo, LSE = O.forward_unit(q_all, q_indptr, np.array(ctx), Hq, Hkv, P, r * Hkv + kv,
                                     pages[(r, kv)], K, V)
            assert Oo.shape == (n_q, G, D) and LSE.shape == (n_q, G)
            for i in range(n_q):
                row = int(q_indptr[r]) + i
                pos = L - n_q + i
                toks = [t for p in pages[(r, kv)] for t in range(p * P, p * P + P)
                        if t < L and t <= pos]
                if not toks:
                    assert LSE[i, h % G] == -math.inf
                    continue
                s = []
                for t in toks:
                    acc = 0.0
                    for d in range(D):
                        acc += q_all[row, h, d] * K[t, d]
                    s.append(scale * acc)
                m = max(s)
                z = sum(math.exp(x - m) for x in s)
                for d in range(D):
                    o = sum(math.exp(x - m) * V[t, d] for x, t in zip(s, toks)) / z
                    assert abs(o - Oo[i, h % G, d]) < 1e-12
                assert abs(m + math.log(z) - LSE[i, h % G]) < 1e-12
