"""Pins of the RoPE alignment oracle (Section 4.2) against things other than
itself: an explicit rotation matrix inverted with numpy, complex
multiplication, torch's float32 -> bf16 rounding, and hand-made ties."""
import numpy as np
import pytest
import torch

from oracle import rope_oracle as R


def rope_matrix(p: int, D: int, base: float) -> np.ndarray:
    """RoPE at position p as a D x D matrix, built entry by entry."""
    M = np.zeros((D, D))
    h = D // 2
    for i in range(h):
        a = p * base ** (-2.0 * i / D)
        M[i, i] = np.cos(a)
        M[i, i + h] = -np.sin(a)
        M[i + h, i] = np.sin(a)
        M[i + h, i + h] = np.cos(a)
    return M


@pytest.mark.parametrize("D,base", [(64, 10000.0), (128, 10000.0), (128, 1.0e6)])
def test_align_equals_rotation_matrices(D, base):
    rng = np.random.default_rng(D)
    x = rng.standard_normal((5, D))
    for p_off, p_on in [(0, 7), (100, 33), (4096, 131071), (5, 5)]:
        want = (rope_matrix(p_on, D, base) @ np.linalg.inv(rope_matrix(p_off, D, base)) @ x.T).T
        got = R.align(x, p_off, p_on, base)
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-9)


def test_rotation_is_complex_multiplication():
    rng = np.random.default_rng(1)
    D, base, p = 16, 10000.0, 37
    x = rng.standard_normal(D)
    z = x[:D // 2] + 1j * x[D // 2:]
    w = z * np.exp(1j * p * base ** (-2.0 * np.arange(D // 2) / D))
    got = R.rotate(x, p, base)
    np.testing.assert_allclose(got, np.concatenate([w.real, w.imag]), atol=1e-13)


def test_identity_inverse_and_norm():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 128))
    np.testing.assert_array_equal(R.align(x, 9, 9, 1e4), x)
    back = R.align(R.align(x, 0, 12345, 1e4), 12345, 0, 1e4)
    np.testing.assert_allclose(back, x, atol=1e-12)
    y = R.rotate(x, 777, 1e4)
    np.testing.assert_allclose(np.hypot(y[:, :64], y[:, 64:]), np.hypot(x[:, :64], x[:, 64:]), atol=1e-12)


def test_round_bf16_matches_torch_on_float32_values():
    rng = np.random.default_rng(3)
    v = np.concatenate([(rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000)).astype(np.float32),
                        np.array([0.0, -0.0, 1e-40, -3e-39, 3.3e38, -3.3e38], dtype=np.float32)])
    assert v.dtype == np.float32          # torch then rounds float32 -> bf16 once
    want = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(R.round_bf16(v.astype(np.float64)), want)


def test_round_bf16_ties_and_double_rounding():
    q = 2.0 ** -8                         # half a bf16 quantum at 1.0
    one = 0x3F80
    cases = {1.0 + q: one,                # tie -> even (1.0)
             1.0 + 3 * q: one + 2,        # tie -> even (1 + 2 quanta)
             1.0 + q + 2.0 ** -30: one + 1,   # just above the tie: float32 first would give 1.0
             -(1.0 + q + 2.0 ** -30): 0x8000 | (one + 1),
             float("inf"): 0x7F80, float("-inf"): 0xFF80}
    for x, bits in cases.items():
        assert int(R.round_bf16(np.array([x]))[0]) == bits, x
    assert int(R.round_bf16(np.array([np.nan]))[0]) & 0x7FFF > 0x7F80


def test_page_layout_roundtrip_and_align_pages():
    rng = np.random.default_rng(4)
    P, D = 32, 64
    pool = rng.integers(0, 1 << 16, size=(5, P * D), dtype=np.uint16)
    pool &= 0x3FFF                        # finite values only
    for ph in range(5):
        np.testing.assert_array_equal(R.tokens_page(R.page_tokens(pool[ph], P, D), P, D), pool[ph])
    out = R.align_pages(pool, [3, 1], [0, 100], P, D, 1e4)
    np.testing.assert_array_equal(out[[0, 2, 3, 4]], pool[[0, 2, 3, 4]])   # delta 0 and unlisted: unchanged
    tok = R.bf16_bits_to_f64(R.page_tokens(pool[1], P, D))
    want = R.round_bf16(rope_matrix(100, D, 1e4) @ tok.T).T
    np.testing.assert_array_equal(R.page_tokens(out[1], P, D), want)
