"""fp64 CPU oracle for RoPE positional alignment of cached key pages.

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
baseline leg may import or call this module; the product path never does.
It shares no code with the HIP library and imports nothing from it.

What it follows (RedKnot, arXiv 2606.06256), Section 4.2, "RoPE-based
positional alignment": a key cached at offline position p_off and reused at
online position p_on is replaced by R(p_on) R(p_off)^-1 K(p_off), R(p) being
the RoPE rotation at position p. Rotations of one 2-D plane commute, so this
is the rotation by the relative shift delta = p_on - p_off.

Readings where the paper is silent (listed in the design notes):
  * pairing: dimension i is rotated together with dimension i + D/2
    (i < D/2), the "rotate half" layout of Llama/Qwen checkpoints;
  * angle of pair i at position p: p * theta_i, theta_i = base^(-2 i / D);
    the base is a parameter (10000 unless stated);
  * the aligned key is computed in float64 from the bf16 key and rounded
    once to bf16, to nearest with ties to even;
  * every token slot of a listed page is rotated (slots past the context
    hold values nobody reads).
"""
from __future__ import annotations

import numpy as np

TILE = 16


def inv_freq(D: int, base: float) -> np.ndarray:
    """theta_i = base^(-2 i / D) for the D/2 rotation planes."""
    i = np.arange(D // 2, dtype=np.float64)
    return np.power(float(base), -(2.0 * i) / D)


def rotate(x: np.ndarray, p, base: float) -> np.ndarray:
    """RoPE rotation of x[..., D] by position p (a number, or an array that
    broadcasts against x[..., 0]): pair (i, i + D/2) turns by p * theta_i."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    h = D // 2
    ang = np.asarray(p, dtype=np.float64)[..., None] * inv_freq(D, base)
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def align(k: np.ndarray, p_off, p_on, base: float) -> np.ndarray:
    """R(p_on) R(p_off)^-1 k = rotation by p_on - p_off (fp64, no rounding)."""
    return rotate(k, np.asarray(p_on, dtype=np.int64) - np.asarray(p_off, dtype=np.int64), base)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """float64 -> bf16 bits, rounded to nearest with ties to even, directly
    (not through float32, which would round twice)."""
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    out = np.zeros(x.shape, dtype=np.uint16)
    fin = np.isfinite(x) & (a > 0)
    m, e = np.frexp(np.where(fin, a, 1.0))      # a = m 2^e, m in [0.5, 1)
    q = np.maximum(e - 8, -133)                  # exponent of the bf16 quantum at a
    r = np.round(np.ldexp(np.where(fin, a, 0.0), -q))   # half to even; exact scaling
    val = np.ldexp(r, q)                         # representable in bf16 (or 2^128)
    with np.errstate(over="ignore"):
        f32 = val.astype(np.float32)             # exact, or inf past the range
    mag = (f32.view(np.uint32) >> 16).astype(np.uint16)
    out = np.where(fin, mag, out)
    out = np.where(np.isinf(x), np.uint16(0x7F80), out)
    out = np.where(np.isnan(x), np.uint16(0x7FC0), out)
    sign = np.signbit(x) & ~np.isnan(x)
    return np.where(sign, out | np.uint16(0x8000), out).astype(np.uint16)


def page_tokens(page_bits: np.ndarray, P: int, D: int) -> np.ndarray:
    """One pool page (bf16 bits, P*D in tile layout: per 16-token tile,
    [D/8][16][8]) -> [P, D] bits."""
    t = np.asarray(page_bits, dtype=np.uint16).reshape(P // TILE, D // 8, TILE, 8)
    return t.transpose(0, 2, 1, 3).reshape(P, D)


def tokens_page(tok_bits: np.ndarray, P: int, D: int) -> np.ndarray:
    """Inverse of page_tokens."""
    t = np.asarray(tok_bits, dtype=np.uint16).reshape(P // TILE, TILE, D // 8, 8)
    return t.transpose(0, 2, 1, 3).reshape(P * D)


def align_pages(k_pool_bits: np.ndarray, pages, deltas, P: int, D: int, base: float) -> np.ndarray:
    """Aligned copy of a K pool (bf16 bits, [n_phys, P*D]): each listed page
    rotated by its delta = p_on - p_off; other pages unchanged."""
    out = np.array(k_pool_bits, dtype=np.uint16, copy=True)
    for ph, dl in zip(pages, deltas):
        tok = bf16_bits_to_f64(page_tokens(out[int(ph)], P, D))
        out[int(ph)] = tokens_page(round_bf16(rotate(tok, int(dl), base)), P, D)
    return out
