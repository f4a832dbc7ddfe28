"""Pins of the attention-mass token selection oracle: dense softmax column
sums from torch, brute force over subsets, tie order, and the recent window."""
import itertools

import numpy as np
import pytest
import torch

from oracle import mass_oracle as M


def test_mass_equals_dense_softmax_column_sums():
    rng = np.random.default_rng(0)
    L, n_q, G, D, P = 40, 12, 3, 16, 8
    K = rng.standard_normal((L, D))
    q = rng.standard_normal((n_q, G, D))
    scale = D ** -0.5
    pages = list(range((L + P - 1) // P))           # every page: plain causal attention
    got = M.unit_chunk_mass(q, K, pages, P, scale)
    # dense causal softmax with torch (float64), rows (i, h), columns = positions
    s = torch.einsum("igd,td->igt", torch.from_numpy(q), torch.from_numpy(K)) * scale
    pos = torch.arange(L)
    mask = pos[None, None, :] <= (L - n_q + torch.arange(n_q))[:, None, None]
    w = torch.softmax(s.masked_fill(~mask, float("-inf")), dim=-1)
    want = w.sum(dim=(0, 1))[L - n_q:].numpy()
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)
    # each row puts mass 1 on its keys; the chunk's share is below n_q * G
    assert got.sum() < n_q * G


def test_unselected_pages_get_no_mass_and_rows_renormalise():
    rng = np.random.default_rng(1)
    L, n_q, G, D, P = 64, 16, 2, 8, 16
    K = rng.standard_normal((L, D))
    q = rng.standard_normal((n_q, G, D))
    m_all = M.unit_chunk_mass(q, K, [0, 1, 2, 3], P, 0.3)
    m_sub = M.unit_chunk_mass(q, K, [3], P, 0.3)      # only the chunk's own page
    # with only chunk keys visible every row's mass lands on the chunk
    assert abs(m_sub.sum() - n_q * G) < 1e-9
    assert (m_sub >= m_all - 1e-15).all()              # fewer keys: no token loses mass


def test_selection_is_a_smallest_set_brute_force():
    rng = np.random.default_rng(2)
    for trial in range(60):
        n = int(rng.integers(1, 9))
        mass = rng.choice([0.0, 0.5, 1.0, 1.5, 2.0, 3.0], size=n) if trial % 2 else rng.random(n)
        tau = float(rng.choice([0.2, 0.5, 0.9, 0.99, 1.0]))
        got = M.select_tokens(mass, tau, 0)
        total = mass.sum()
        assert mass[got].sum() >= tau * total - 1e-12
        best = min((len(c) for r in range(n + 1) for c in itertools.combinations(range(n), r)
                    if mass[list(c)].sum() >= tau * total - 1e-12), default=0)
        assert got.size == best, (mass, tau, got)


def test_ties_go_to_the_earlier_token_and_recent_tokens_are_kept():
    mass = np.array([1.0, 2.0, 2.0, 0.5, 2.0, 0.1])
    # 2.0 x3 = 6 of 7.6: tau 0.5 -> 3.8 needs two of the three 2.0 tokens: the earlier ones
    np.testing.assert_array_equal(M.select_tokens(mass, 0.5, 0), [1, 2])
    np.testing.assert_array_equal(M.select_tokens(mass, 0.5, 2), [1, 2, 4, 5])
    np.testing.assert_array_equal(M.select_tokens(np.zeros(4), 0.5, 1), [3])
    assert M.mass_cover_fraction(np.array([8.0, 1.0, 0.5, 0.5])) == 1.0
    assert M.mass_cover_fraction(np.array([99.0, 1.0, 0.0, 0.0]), 0.99) == 0.25


def test_single_token_mass_equals_dense_column_sum():
    rng = np.random.default_rng(3)
    L, n_q, G, D, P = 50, 20, 2, 8, 8
    K = rng.standard_normal((L, D))
    q = rng.standard_normal((n_q, G, D))
    pages = [0, 2, 4, 6]                               # chunk tokens 30..49: page 5 (40..47) missing
    s = torch.einsum("igd,td->igt", torch.from_numpy(q), torch.from_numpy(K)) * 0.4
    pos = torch.arange(L)
    sel = torch.zeros(L, dtype=torch.bool)
    for p in pages:
        sel[p * P:(p + 1) * P] = True
    mask = (pos[None, None, :] <= (L - n_q + torch.arange(n_q))[:, None, None]) & sel[None, None, :]
    w = torch.softmax(s.masked_fill(~mask, float("-inf")), dim=-1)
    want = w.sum(dim=(0, 1))[L - n_q:].numpy()
    for k in range(n_q):
        assert abs(M.chunk_token_mass(q, K, pages, P, 0.4, k) - want[k]) < 1e-12, k
    np.testing.assert_allclose(M.unit_chunk_mass(q, K, pages, P, 0.4), want, rtol=1e-12, atol=1e-14)
    assert all(want[k] == 0 for k in range(n_q) if not sel[L - n_q + k])


def test_columns_to_token_mass_float32_order_and_sanitising():
    cols = np.array([[1.0, 2.0, 3.0], [2.0 ** 24, 1.0, 1.0], [-5.0, 1.0, 1.0], [np.nan, 1.0, 0.0],
                     [-0.0, -0.0, -0.0]], dtype=np.float32)
    m = M.columns_to_token_mass(cols)
    assert m.dtype == np.float32
    # 2^24 + 1 rounds back to 2^24 in float32 at each step (column order), not 2^24 + 2
    np.testing.assert_array_equal(m, np.array([6.0, 2.0 ** 24, 0.0, 0.0, 0.0], dtype=np.float32))
    assert not np.signbit(m[4])
