"""Property pins of the fp64 oracle over tiny random shapes (hypothesis).

Each property is checked against something the oracle does not compute
itself: a pure-Python softmax over lists of floats, the Section 4.4 merge
identity for any partition of a page set, and the definition of a seeded
sample (the count in closed form, the forced pages, key order).
"""
import math

import numpy as np
from hypothesis import given, settings, strategies as st

from oracle import segpa_oracle as O

SETTINGS = settings(max_examples=60, deadline=None)


@st.composite
def units(draw):
    """One unit: q [n_q, G, D], K, V [L, D], page size P, selected pages."""
    P = draw(st.sampled_from([2, 4, 8]))
    L = draw(st.integers(1, 70))
    D = draw(st.sampled_from([4, 8]))
    G = draw(st.sampled_from([1, 2, 4]))
    n_q = draw(st.integers(1, min(4, L)))
    seed = draw(st.integers(0, 2**31 - 1))
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((n_q, G, D))
    K = rng.standard_normal((L, D)) * draw(st.sampled_from([0.5, 1.0, 3.0]))
    V = rng.standard_normal((L, D))
    n = (L + P - 1) // P
    pages = sorted(draw(st.sets(st.integers(0, n - 1), max_size=n)))
    return q, K, V, P, pages


def _brute(q, K, V, P, pages, scale):
    """Per query row and head: softmax over the visible selected tokens, with
    Python floats and math.exp only."""
    n_q, G, D = q.shape
    L = K.shape[0]
    O_ = [[[0.0] * D for _ in range(G)] for _ in range(n_q)]
    LSE = [[-math.inf] * G for _ in range(n_q)]
    for i in range(n_q):
        pos = L - n_q + i
        toks = [t for p in pages for t in range(p * P, (p + 1) * P) if t < L and t <= pos]
        for h in range(G):
            if not toks:
                continue
            s = [scale * sum(float(q[i, h, d]) * float(K[t, d]) for d in range(D)) for t in toks]
            m = max(s)
            e = [math.exp(x - m) for x in s]
            z = sum(e)
            for d in range(D):
                O_[i][h][d] = sum(e[k] * float(V[t, d]) for k, t in enumerate(toks)) / z
            LSE[i][h] = m + math.log(z)
    return np.array(O_), np.array(LSE)


@SETTINGS
@given(units())
def test_attend_unit_equals_pure_python_softmax(u):
    q, K, V, P, pages = u
    scale = 1.0 / math.sqrt(q.shape[-1])
    Oo, LSE = O.attend_unit(q, K, V, pages, P, scale)
    Ob, Lb = _brute(q, K, V, P, pages, scale)
    np.testing.assert_allclose(Oo, Ob, atol=1e-12, rtol=0)
    assert np.array_equal(np.isneginf(LSE), np.isneginf(Lb))
    fin = np.isfinite(Lb)
    np.testing.assert_allclose(LSE[fin], Lb[fin], atol=1e-12, rtol=0)


@SETTINGS
@given(units(), st.data())
def test_lse_merge_of_any_partition_equals_the_union(u, data):
    """Section 4.4: attention over the union of disjoint page sets is the LSE
    merge of the attention over each (empty parts included)."""
    q, K, V, P, pages = u
    n_parts = data.draw(st.integers(1, 4))
    owner = data.draw(st.lists(st.integers(0, n_parts - 1), min_size=len(pages),
                               max_size=len(pages)))
    parts = [[p for p, o in zip(pages, owner) if o == k] for k in range(n_parts)]
    scale = 0.7
    whole = O.attend_unit(q, K, V, pages, P, scale)
    merged = O.lse_merge([O.attend_unit(q, K, V, ps, P, scale) for ps in parts])
    np.testing.assert_allclose(merged[0], whole[0], atol=1e-12, rtol=0)
    assert np.array_equal(np.isneginf(merged[1]), np.isneginf(whole[1]))
    fin = np.isfinite(whole[1])
    np.testing.assert_allclose(merged[1][fin], whole[1][fin], atol=1e-12, rtol=0)


@SETTINGS
@given(st.integers(1, 60), st.integers(0, 70), st.integers(0, 8), st.integers(0, 8),
       st.integers(0, 2**64 - 1), st.integers(0, 31), st.integers(0, 15))
def test_random_hash_is_the_budget_of_smallest_keys(n, budget, fh, ft, seed, r, g):
    sel = O.pages_random_hash(seed, r, g, n, budget, fh, ft)
    forced = set(range(min(n, fh))) | set(range(max(0, n - ft), n))
    assert len(sel) == min(n, max(budget, len(forced)))
    assert sel == sorted(set(sel)) and all(0 <= p < n for p in sel)
    assert forced <= set(sel)
    # no unselected free page beats a selected one under (key, page) order
    key = {p: (O.page_hash(seed, r, g, p), p) for p in range(n)}
    chosen = [key[p] for p in sel if p not in forced]
    left = [key[p] for p in range(n) if p not in forced and p not in sel]
    if chosen and left:
        assert max(chosen) < min(left)


@SETTINGS
@given(units())
def test_all_pages_equal_dense_causal_attention(u):
    """A global head (every page) is dense causal attention, computed here with
    torch-free numpy over the whole prefix."""
    q, K, V, P, _ = u
    L = K.shape[0]
    n = (L + P - 1) // P
    scale = 0.5
    Oo, LSE = O.attend_unit(q, K, V, list(range(n)), P, scale)
    n_q = q.shape[0]
    for i in range(n_q):
        vis = L - n_q + i + 1
        s = scale * np.einsum("hd,td->ht", q[i], K[:vis])
        w = np.exp(s - s.max(axis=1, keepdims=True))
        w /= w.sum(axis=1, keepdims=True)
        np.testing.assert_allclose(Oo[i], w @ V[:vis], atol=1e-12, rtol=0)
