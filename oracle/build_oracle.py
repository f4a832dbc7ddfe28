"""CPU oracle for building head-segmented KV state: appending new tokens'
keys and values to their pages and refreshing the pages' key sums.

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
baseline leg may import or call this module; the product path never does.
It shares no code with the HIP library and imports nothing from it.

What it follows (RedKnot, arXiv 2606.06256):
  * Section 4.4: BuildState constructs the reusable state of cached chunks;
    for explicit KV pages that is the keys and values written into their
    pages (and here the page key sums the mean-key rule reads).
  * Section 4.3 and Algorithm 2 (Translate): token position t of the head
    stream of (request r, KV head g) lies in logical page t // P at slot
    t % P; the segment table gives the segment's first virtual page, the page
    table the physical page.

Readings where the paper is silent (listed in the design notes):
  * the new tokens of request r take positions ctx_lens[r], ctx_lens[r] + 1, ...
    in order, for every KV head;
  * a token whose segment is unmapped, or whose position lies past the
    segment table, is dropped (nothing is written for it);
  * a page's key sum is the float32 rounding of the exact sum of its valid
    keys (as for the mean-key rule), valid = min(P, new length - page start);
    it is refreshed for every page that received a token.
Pools are handled as raw bf16 bits (uint16), so writes are exact.
"""
from __future__ import annotations

import numpy as np

from . import segpa_oracle as S

TILE = 16


def token_page_slot(seg_row, page_table, pps: int, P: int, pos: int):
    """(physical page, slot) of position pos, or None when unmapped."""
    j, slot = divmod(pos, P)
    if j // pps >= len(seg_row) or int(seg_row[j // pps]) < 0:
        return None
    return S.translate(seg_row, page_table, pps, j), slot


def write_token(k_page: np.ndarray, v_page: np.ndarray, slot: int, k_tok: np.ndarray,
                v_tok: np.ndarray, P: int, D: int) -> None:
    """Store one token's key and value (bf16 bits, [D]) at `slot` of a page in
    the tile layout: K tile [D/8][16][8], V tile [D][16]."""
    t, u = divmod(slot, TILE)
    kt = k_page.reshape(P // TILE, D // 8, TILE, 8)
    vt = v_page.reshape(P // TILE, D, TILE)
    kt[t, :, u, :] = np.asarray(k_tok, dtype=np.uint16).reshape(D // 8, 8)
    vt[t, :, u] = np.asarray(v_tok, dtype=np.uint16)


def append(k_pool: np.ndarray, v_pool: np.ndarray, seg_table: np.ndarray, page_table: np.ndarray,
           ctx_lens, new_indptr, k_new: np.ndarray, v_new: np.ndarray, Hkv: int, P: int, pps: int):
    """Pools after appending; k_new, v_new are bf16 bits [n_new, Hkv, D].
    Returns (k_pool, v_pool, touched) with touched = {physical page: valid
    tokens after the append}."""
    D = k_new.shape[-1]
    kp = np.array(k_pool, dtype=np.uint16, copy=True)
    vp = np.array(v_pool, dtype=np.uint16, copy=True)
    seg = np.asarray(seg_table).reshape(len(ctx_lens) * Hkv, -1)
    touched: dict[int, int] = {}
    for r in range(len(ctx_lens)):
        L0 = int(ctx_lens[r])
        i0, i1 = int(new_indptr[r]), int(new_indptr[r + 1])
        L1 = L0 + (i1 - i0)
        for g in range(Hkv):
            row = seg[r * Hkv + g]
            for i in range(i0, i1):
                pos = L0 + (i - i0)
                loc = token_page_slot(row, page_table, pps, P, pos)
                if loc is None:
                    continue
                ph, slot = loc
                write_token(kp[ph], vp[ph], slot, k_new[i, g], v_new[i, g], P, D)
                touched[ph] = min(P, L1 - (pos // P) * P)
    return kp, vp, touched


def refresh_key_sums(page_ksum: np.ndarray, k_pool: np.ndarray, touched: dict, P: int, D: int) -> np.ndarray:
    """Key sums (float32 [n_phys, D]) with every touched page recomputed from
    its first `valid` keys."""
    out = np.array(page_ksum, dtype=np.float32, copy=True)
    for ph, valid in touched.items():
        kt = k_pool[ph].reshape(P // TILE, D // 8, TILE, 8).transpose(0, 2, 1, 3).reshape(P, D)
        keys = (kt[:valid].astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        out[ph] = S.page_key_sum(keys)
    return out
