"""fp64 CPU oracle for attention-mass token selection (SelectImportantTokens).

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
baseline leg may import or call this module; the product path never does.
It shares no code with the HIP library and imports nothing from it.

What it follows (RedKnot, arXiv 2606.06256): Algorithm 1 applies the FFN only
to the tokens SelectImportantTokens picks from a layer's attention; Section
4.4 describes the pick as the smallest set of tokens whose cumulative
attention mass exceeds a threshold tau, and the experiments (Section 5) also
always keep the most recent N tokens; the denoising study reports the minimum
fraction of tokens that covers 99% of the attention mass.

Readings where the paper is silent (listed in the design notes):
  * the candidates are the tokens of the current query chunk (the tokens the
    FFN runs on); the mass of chunk token t is the sum, over every query row
    (query i, head h) of the request that sees t, of the softmax weight of t in
    that row, the softmax taken over the row's attended keys exactly as the
    attention forward defines them (selected pages, causal);
  * "exceeds tau" is read as: the chosen tokens carry at least tau of the total
    mass of the candidates;
  * the smallest such set is the longest-mass-first prefix: tokens in
    descending mass, equal masses in ascending position, taken until the
    cumulative mass reaches tau * total; the most recent N candidates are kept
    in any case;
  * tau is in (0, 1]; with tau * total reached by no prefix (total mass 0) the
    mass part is empty.
"""
from __future__ import annotations

from typing import Sequence

import numpy as np

from . import segpa_oracle as S


def unit_chunk_mass(q: np.ndarray, K: np.ndarray, pages: Sequence[int], P: int, scale: float) -> np.ndarray:
    """Mass received by each of a unit's chunk tokens from that unit's rows.

    q: [n_q, G, D] (the G query heads of one KV head), K: [L, D] logical keys;
    query i sits at position L - n_q + i. Returns [n_q] (chunk token k is
    position L - n_q + k)."""
    n_q, G, _ = q.shape
    L = K.shape[0]
    tok = S.selected_tokens(pages, L, P)
    m = np.zeros(n_q)
    for i in range(n_q):
        T = tok[tok <= L - n_q + i]
        if T.size == 0:
            continue
        for h in range(G):
            w = S.attention_weights(q[i, h], K, T, scale)
            in_chunk = T >= L - n_q
            np.add.at(m, T[in_chunk] - (L - n_q), w[in_chunk])
    return m


def chunk_token_mass(q: np.ndarray, K: np.ndarray, pages: Sequence[int], P: int, scale: float,
                     k: int) -> float:
    """Mass of chunk token k alone (same definition as unit_chunk_mass), for
    sampling long chunks: only the rows i >= k are visited."""
    n_q, G, _ = q.shape
    L = K.shape[0]
    tok = S.selected_tokens(pages, L, P)
    pos = L - n_q + k
    if pos < 0 or pos not in set(tok.tolist()):
        return 0.0
    KT = K[tok]
    at = int(np.searchsorted(tok, pos))
    total = 0.0
    for i in range(k, n_q):
        n_i = int(np.searchsorted(tok, L - n_q + i, side="right"))   # keys at or before query i
        s = scale * (KT[:n_i] @ q[i].T)                # [n_i, G]
        e = np.exp(s - s.max(axis=0))
        total += float(np.sum(e[at] / e.sum(axis=0)))
    return total


def columns_to_token_mass(cols: np.ndarray) -> np.ndarray:
    """Token masses from per-column masses [n, c]: the float32 sum of a row's
    columns in column order; a sum that is negative or NaN counts as 0."""
    cols = np.asarray(cols, dtype=np.float32)
    m = np.zeros(cols.shape[0], dtype=np.float32)
    for c in range(cols.shape[1]):
        m = (m + cols[:, c]).astype(np.float32)
    return np.where(m >= 0, m, np.float32(0)).astype(np.float32)


def select_tokens(mass: np.ndarray, tau: float, recent: int) -> np.ndarray:
    """Kept positions (ascending) of one request's chunk given its token masses."""
    n = mass.size
    order = sorted(range(n), key=lambda k: (-float(mass[k]), k))
    total = float(np.sum(mass))
    keep = set(range(max(0, n - recent), n))
    if total > 0:
        acc = 0.0
        for k in order:
            if acc >= tau * total:
                break
            keep.add(k)
            acc += float(mass[k])
    return np.array(sorted(keep), dtype=np.int64)


def mass_cover_fraction(mass: np.ndarray, frac: float = 0.99) -> float:
    """Smallest fraction of the candidates whose mass covers `frac` of the total
    (the paper's 99%-mass sparsity measurement)."""
    if mass.size == 0:
        return 0.0
    return select_tokens(mass, frac, 0).size / mass.size
