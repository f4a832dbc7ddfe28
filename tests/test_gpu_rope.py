"""GPU parity of RoPE alignment of cached key pages (Section 4.2) against the
fp64 oracle: every bit of the pool must match, listed pages rotated, all
other pages untouched."""
import numpy as np
import pytest
import torch

from oracle import rope_oracle as R
from paper_2606_06256_amd import binding as B
from paper_2606_06256_amd import inputs as I

pytestmark = pytest.mark.gpu


def _require_gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"


def _pool(D, P, n_phys, seed):
    sp = I.Spec(name="rope", B=1, Hq=2, Hkv=1, D=D, P=P, seg_tokens=P, ctx_lens=[P * n_phys],
                q_lens=[1], seed=seed)
    wl = I.build(sp)
    k, _ = wl.build_pool("cpu")
    dims = B.make_dims(num_requests=1, num_q_heads=2, num_kv_heads=1, head_dim=D, page_size=P,
                       pages_per_segment=1, max_segments=n_phys, max_q_len=1, total_q=1,
                       num_virtual_pages=n_phys, num_phys_pages=k.shape[0])
    return k, dims


@pytest.mark.parametrize("D,P,base", [(128, 16, 1e4), (64, 32, 1e4), (128, 64, 1e6), (128, 256, 5e5)])
def test_rope_align_matches_oracle_bitwise(D, P, base):
    _require_gpu()
    n_phys = 96 if P <= 64 else 24
    k, dims = _pool(D, P, n_phys, seed=D + P)
    n_phys = k.shape[0]
    rng = np.random.default_rng(P)
    pages = rng.permutation(n_phys)[: n_phys // 2].astype(np.int32)
    deltas = rng.integers(-131072, 131072, size=pages.size).astype(np.int32)
    deltas[:3] = [0, 1, -1]
    # ids outside the pool are skipped
    pages_dev = np.concatenate([pages, np.array([-1, n_phys, 1 << 30], dtype=np.int32)])
    deltas_dev = np.concatenate([deltas, np.array([5, 5, 5], dtype=np.int32)])
    kd = k.cuda()
    B.seg_paged_attn_rope_align(dims, kd, torch.from_numpy(pages_dev).cuda(),
                                torch.from_numpy(deltas_dev).cuda(), base)
    torch.cuda.synchronize()
    got = kd.cpu().view(torch.int16).numpy().view(np.uint16)
    want = R.align_pages(k.view(torch.int16).numpy().view(np.uint16), pages, deltas, P, D, base)
    diff = np.nonzero(got != want)
    print(f"[rope] D={D} P={P} base={base:g}: pages {pages.size}, differing elements {diff[0].size}")
    assert diff[0].size == 0


def test_rope_align_twice_matches_oracle_twice():
    """Two alignments in a row (d, then -d, as when a chunk moves back) give
    the oracle's two-step result bit for bit, and come back to the original
    keys up to the two roundings."""
    _require_gpu()
    D, P = 128, 16
    k, dims = _pool(D, P, 64, seed=7)
    kd = k.cuda()
    pages = np.arange(64, dtype=np.int32)
    d = np.full(64, 4099, dtype=np.int32)
    for dl in (d, -d):
        B.seg_paged_attn_rope_align(dims, kd, torch.from_numpy(pages).cuda(), torch.from_numpy(dl).cuda())
    torch.cuda.synchronize()
    bits0 = k.view(torch.int16).numpy().view(np.uint16)
    want = R.align_pages(R.align_pages(bits0, pages, d, P, D, 1e4), pages, -d, P, D, 1e4)
    got = kd.cpu().view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(got, want)
    x0 = R.bf16_bits_to_f64(bits0)
    x2 = R.bf16_bits_to_f64(got)
    assert np.abs(x2 - x0).max() <= 2.0 ** -6 * np.abs(x0).max()


def test_rope_align_empty_list_is_a_no_op():
    _require_gpu()
    k, dims = _pool(128, 16, 8, seed=9)
    kd = k.cuda()
    B.seg_paged_attn_rope_align(dims, kd, torch.zeros(0, dtype=torch.int32, device="cuda"),
                                torch.zeros(0, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    assert torch.equal(kd.cpu().view(torch.int16), k.view(torch.int16))
