"""fp64 CPU oracle for SegPagedAttention with per-head page selection.

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
baseline leg may import or call this module; the product path never does.
It shares no code with the HIP library and imports nothing from it.

What it follows (RedKnot, arXiv 2606.06256):
  * Algorithm 2 (SegPagedAttention): a KV head stream is split into head
    segments; the segment table maps a segment to consecutive virtual pages and
    the page table maps a virtual page to a physical page (Section 4.3). A head
    attends only to its selected pages U_h; a global head keeps the full range
    (U_h = V_h), a local head keeps sink pages and recent-window pages.
  * Section 4.2 (head-aware attention recovery): the local visible set
    W(i) = S_sink U [max(0, i - w), i], both ends inclusive.
  * Section 4.3: a local head accesses "only the pages that overlap with its
    visible region", i.e. whole pages.
  * Section 4.4 (DeepSeek-V4 adapter): splitting the key set in two parts and
    merging the two attention results with log-sum-exp gives the same result
    as softmax attention over the union.
  * Section 5.4 (prefix compression): true eviction means an evicted key never
    enters the softmax; zero-filling it would still add exp(0)-type mass.
  * Section 5.3: the fused kernel is mask-free over each head's own page list.

Readings where the paper is silent (each listed in the design notes):
  softmax scale 1/sqrt(D); q head h uses KV head h // (Hq/Hkv); a chunk of n_q
  queries sits at the end of the context (query i at position L - n_q + i) and
  is causal; the sink set is the first n_sink token positions; an empty key set
  gives O = 0 and LSE = -inf; budgets are whole pages per request; RANDOM_HASH
  and TOPK_MEANKEY are content/seeded rules defined here, not in the paper (its
  only KV page rule is the head-class policy, HEAD_CLASS here).

All floating point is float64; bf16 inputs convert exactly.
"""
from __future__ import annotations

import math
from fractions import Fraction
from typing import Callable, Iterable, Sequence

import numpy as np

GLOBAL, LOCAL = 1, 0
MASK64 = (1 << 64) - 1


# --------------------------------------------------------------------------
# Paging (Algorithm 2: segment table, page table, Translate)
# --------------------------------------------------------------------------
def n_pages(L: int, P: int) -> int:
    """Number of logical pages of a head stream of L tokens (the last may be partial)."""
    return (L + P - 1) // P


def translate(seg_row: Sequence[int], page_table: Sequence[int], pps: int, j: int) -> int:
    """Logical page j of one head stream -> physical page (Algorithm 2, Translate).

    Page j lies in head segment s = j // pps at offset o = j % pps; the segment
    table gives the segment's first virtual page; the page table maps the
    virtual page to its physical page.
    """
    s, o = divmod(j, pps)
    first_virtual = int(seg_row[s])
    if first_virtual < 0:
        raise ValueError(f"segment {s} is not mapped")
    return int(page_table[first_virtual + o])


def unit_kv_from_pool(k_pool: np.ndarray, v_pool: np.ndarray, seg_row, page_table,
                      pps: int, L: int, P: int, D: int):
    """Logical K, V [L, D] (float64) of one head stream, read through the tables.

    Physical page layout: P/16 tiles of 16 tokens; a K tile is [D/8][16][8]
    (head-dimension chunks of 8, chunk-major), a V tile is [D][16].
    """
    n = n_pages(L, P)
    K = np.zeros((n * P, D))
    V = np.zeros((n * P, D))
    nt = P // 16
    for j in range(n):
        ph = translate(seg_row, page_table, pps, j)
        kt = np.asarray(k_pool[ph], dtype=np.float64).reshape(nt, D // 8, 16, 8)
        vt = np.asarray(v_pool[ph], dtype=np.float64).reshape(nt, D, 16)
        for t in range(nt):
            for u in range(16):
                row = j * P + t * 16 + u
                K[row] = kt[t, :, u, :].reshape(D)
                V[row] = vt[t, :, u]
    return K[:L], V[:L]


# --------------------------------------------------------------------------
# Selection rules (Algorithm 2 policy step, plus the two ranked rules)
# --------------------------------------------------------------------------
def pages_all(L: int, P: int) -> list[int]:
    """Global head: U_h = V_h, every page of the stream."""
    return list(range(n_pages(L, P)))


def visible_window(i: int, w: int, sink: Iterable[int]) -> set[int]:
    """W(i) = S_sink U [max(0, i - w), i] (Section 4.2), inclusive."""
    return set(sink) | set(range(max(0, i - w), i + 1))


def pages_head_class(policy: int, L: int, n_q: int, P: int, n_sink: int, w: int) -> list[int]:
    """Head-class policy of Algorithm 2.

    GLOBAL keeps every page. LOCAL keeps the pages that overlap the visible
    region of any query of the chunk: the sink positions and each query's
    window W(i), for query positions i = L - n_q .. L - 1.
    """
    if policy == GLOBAL:
        return pages_all(L, P)
    sink = range(min(n_sink, L))
    tokens: set[int] = set()
    for i in range(L - n_q, L):
        tokens |= visible_window(i, w, sink)
    tokens = {t for t in tokens if 0 <= t < L}
    return sorted({t // P for t in tokens})


def splitmix64_mix(z: int) -> int:
    """Output function of SplitMix64 (Steele, Lea, Flood, OOPSLA 2014)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def splitmix64(state: int) -> int:
    """One SplitMix64 output from `state`: advance by the golden gamma, then mix."""
    return splitmix64_mix((state + 0x9E3779B97F4A7C15) & MASK64)


def page_hash(seed: int, r: int, g: int, p: int) -> int:
    """RANDOM_HASH key of logical page p of unit (request r, KV head g)."""
    assert 0 <= r < (1 << 24) and 0 <= g < (1 << 8) and 0 <= p < (1 << 32)
    return splitmix64(splitmix64(seed & MASK64) ^ ((r << 40) | (g << 32) | p))


def forced_pages(n: int, forced_head: int, forced_tail: int) -> set[int]:
    return set(range(min(n, forced_head))) | set(range(max(0, n - forced_tail), n))


def selection_count(n: int, budget: int, forced_head: int, forced_tail: int) -> int:
    """Pages a ranked rule returns: the budget, never fewer than the forced pages, at most n."""
    return min(n, max(budget, len(forced_pages(n, forced_head, forced_tail))))


def select_ranked(n: int, budget: int, forced_head: int, forced_tail: int,
                  rank: Callable[[int], object]) -> list[int]:
    """Forced pages plus the best-ranked other pages, ascending.

    `rank(p)` orders pages, smaller first; equal ranks go to the lower index.
    """
    forced = forced_pages(n, forced_head, forced_tail)
    count = selection_count(n, budget, forced_head, forced_tail)
    rest = sorted((p for p in range(n) if p not in forced), key=lambda p: (rank(p), p))
    return sorted(forced | set(rest[:count - len(forced)]))


def pages_random_hash(seed: int, r: int, g: int, n: int, budget: int,
                      forced_head: int, forced_tail: int) -> list[int]:
    """Seeded uniform sample without replacement: the non-forced pages with the
    smallest SplitMix64 keys (the prefix of a uniformly random order)."""
    return select_ranked(n, budget, forced_head, forced_tail,
                         lambda p: page_hash(seed, r, g, p))


def page_key_sum(k_page: np.ndarray) -> np.ndarray:
    """Per-dimension sum of a page's valid keys, rounded to float32.

    The sum is taken with math.fsum (exact, then rounded once to float64) and
    then rounded to float32; for bf16 keys whose magnitudes span less than
    2^40 the float64 value is the exact sum, so this is the float32 rounding of
    the exact sum.
    """
    k = np.asarray(k_page, dtype=np.float64)
    return np.array([math.fsum(k[:, d].tolist()) for d in range(k.shape[1])], dtype=np.float64
                    ).astype(np.float32)


def unit_key_sums(K: np.ndarray, P: int) -> tuple[np.ndarray, np.ndarray]:
    """Key sums [n_pages, D] (float32) and valid-token counts of one head stream."""
    L, D = K.shape
    n = n_pages(L, P)
    sums = np.zeros((n, D), dtype=np.float32)
    valid = np.zeros(n, dtype=np.int64)
    for p in range(n):
        blk = K[p * P:min(L, (p + 1) * P)]
        sums[p] = page_key_sum(blk)
        valid[p] = blk.shape[0]
    return sums, valid


def _dyadic_ints(x: np.ndarray, shift: int) -> list[int]:
    """Exact integers x * 2^shift for float64 values that are multiples of 2^-shift."""
    out = []
    for v in np.asarray(x, dtype=np.float64).ravel().tolist():
        s = math.ldexp(v, shift)
        if s != math.floor(s):
            raise ValueError("value is not a multiple of the quantum")
        out.append(int(s))
    return out


def meankey_scores(q_group: np.ndarray, ksum: np.ndarray, valid: np.ndarray) -> list[Fraction]:
    """Exact page scores (q_bar . ksum_p) / n_valid(p) as rationals.

    q_bar is the sum of the group's query heads (last query token); ksum_p is
    the float32 key sum of page p. bf16 values are multiples of 2^-133 and
    float32 values multiples of 2^-149, so the dot product is an integer
    multiple of 2^-282 and is computed exactly in integers.
    """
    qbar = [math.fsum(col) for col in np.asarray(q_group, dtype=np.float64).T.tolist()]
    qi = _dyadic_ints(np.array(qbar), 133)
    n, D = ksum.shape
    ki = _dyadic_ints(np.asarray(ksum, dtype=np.float64), 149)
    scores = []
    denom_q = 1 << 282
    for p in range(n):
        row = ki[p * D:(p + 1) * D]
        dot = sum(a * b for a, b in zip(qi, row))
        if valid[p] <= 0:
            raise ValueError("a logical page holds at least one valid token")
        scores.append(Fraction(dot, denom_q * int(valid[p])))
    return scores


def pages_topk_meankey(q_group: np.ndarray, ksum: np.ndarray, valid: np.ndarray, budget: int,
                       forced_head: int = 0, forced_tail: int = 0):
    """Top-budget pages by exact mean-key score, higher first, ties to the lower index.

    Returns (pages ascending, exact scores)."""
    scores = meankey_scores(q_group, ksum, valid)
    n = len(scores)
    pages = select_ranked(n, budget, forced_head, forced_tail, lambda p: -scores[p])
    return pages, scores


# --------------------------------------------------------------------------
# Attention over the selected pages (Algorithm 2, FusedVarlenAttention)
# --------------------------------------------------------------------------
def selected_tokens(pages: Sequence[int], L: int, P: int) -> np.ndarray:
    """Token positions of the selected pages that lie inside the context."""
    toks = [t for p in sorted(pages) for t in range(p * P, min(L, (p + 1) * P))]
    return np.asarray(toks, dtype=np.int64)


def attention_weights(q: np.ndarray, K: np.ndarray, T: np.ndarray, scale: float) -> np.ndarray:
    """Softmax weights of one query row q [D] over keys K[T] (float64)."""
    s = scale * (K[T] @ q)
    e = np.exp(s - s.max())
    return e / e.sum()


def attend_unit(q: np.ndarray, K: np.ndarray, V: np.ndarray, pages: Sequence[int], P: int,
                scale: float):
    """Softmax attention of one unit's queries over its selected pages.

    q: [n_q, G, D] (the G query heads of one KV head); K, V: [L, D] logical.
    Query i sits at position L - n_q + i and sees selected tokens t <= that
    position. Returns O [n_q, G, D] and natural-log LSE [n_q, G]; a query with
    no visible key gets O = 0 and LSE = -inf.
    """
    n_q, G, D = q.shape
    L = K.shape[0]
    tok = selected_tokens(pages, L, P)
    O = np.zeros((n_q, G, D))
    LSE = np.full((n_q, G), -np.inf)
    for i in range(n_q):
        T = tok[tok <= L - n_q + i]
        if T.size == 0:
            continue
        s = scale * (q[i] @ K[T].T)          # [G, |T|]
        M = s.max(axis=1, keepdims=True)
        e = np.exp(s - M)
        Z = e.sum(axis=1, keepdims=True)
        O[i] = (e @ V[T]) / Z
        LSE[i] = (M + np.log(Z))[:, 0]
    return O, LSE


def lse_merge(parts: Sequence[tuple[np.ndarray, np.ndarray]]):
    """Merge attention results over disjoint key sets with log-sum-exp (Section 4.4)."""
    lses = np.stack([p[1] for p in parts])                # [S, ...]
    Os = np.stack([p[0] for p in parts])                  # [S, ..., D]
    M = lses.max(axis=0)
    Mf = np.where(np.isfinite(M), M, 0.0)
    w = np.exp(lses - Mf)                                 # 0 for empty parts
    Z = w.sum(axis=0)
    with np.errstate(invalid="ignore", divide="ignore"):
        O = np.where(Z[..., None] > 0, (w[..., None] * Os).sum(axis=0) / np.where(Z > 0, Z, 1)[..., None], 0.0)
        lse = np.where(Z > 0, Mf + np.log(np.where(Z > 0, Z, 1)), -np.inf)
    return O, lse


# --------------------------------------------------------------------------
# Whole-call references
# --------------------------------------------------------------------------
def select(mode: int, ctx_lens, q_indptr, Hq: int, Hkv: int, P: int, *, budgets=None,
           forced_head: int = 0, forced_tail: int = 0, seed: int = 0, head_policy=None,
           n_sink: int = 4, window: int = 256, q=None, kv_of_unit=None, units=None):
    """Selected logical pages for every unit u = r * Hkv + g (or for `units`).

    mode 0 ALL, 1 HEAD_CLASS, 2 RANDOM_HASH, 3 TOPK_MEANKEY. TOPK needs q
    [total_q, Hq, D] and kv_of_unit(r, g) -> (K, V) logical float64 arrays; the
    oracle derives the key sums from the logical keys itself.
    Returns {u: pages}.
    """
    G = Hq // Hkv
    B = len(ctx_lens)
    out = {}
    todo = range(B * Hkv) if units is None else units
    for u in todo:
        r, g = divmod(u, Hkv)
        L = int(ctx_lens[r])
        n = n_pages(L, P)
        nq = int(q_indptr[r + 1]) - int(q_indptr[r])
        if mode == 0:
            pages = pages_all(L, P)
        elif mode == 1:
            pages = pages_head_class(int(head_policy[g]), L, nq, P, n_sink, window)
        elif mode == 2:
            pages = pages_random_hash(seed, r, g, n, int(budgets[r]), forced_head, forced_tail)
        elif mode == 3:
            K, _ = kv_of_unit(r, g)
            ksum, valid = unit_key_sums(K, P)
            last = int(q_indptr[r + 1]) - 1
            qg = np.asarray(q[last, g * G:(g + 1) * G], dtype=np.float64)
            pages, _ = pages_topk_meankey(qg, ksum, valid, int(budgets[r]), forced_head, forced_tail)
        else:
            raise ValueError(mode)
        out[u] = pages
    return out


def forward_unit(q_all: np.ndarray, q_indptr, ctx_lens, Hq: int, Hkv: int, P: int, u: int,
                 pages: Sequence[int], K: np.ndarray, V: np.ndarray, scale: float | None = None):
    """O [n_q, G, D] and LSE [n_q, G] of unit u from logical K, V."""
    G = Hq // Hkv
    r, g = divmod(u, Hkv)
    D = q_all.shape[-1]
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    q0, q1 = int(q_indptr[r]), int(q_indptr[r + 1])
    q = np.asarray(q_all[q0:q1, g * G:(g + 1) * G], dtype=np.float64)
    return attend_unit(q, np.asarray(K, dtype=np.float64), np.asarray(V, dtype=np.float64),
                       pages, P, scale)
