"""GPU parity of appending tokens to head-segmented pages and refreshing page
key sums (Sections 4.3, 4.4) against the CPU oracle, bit for bit."""
import numpy as np
import pytest
import torch

from oracle import build_oracle as BO
from paper_2606_06256_amd import binding as B
from paper_2606_06256_amd import inputs as I
from paper_2606_06256_amd.device import DeviceWorkload

pytestmark = pytest.mark.gpu


def _require_gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"


def _bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16).copy()


CASES = {
    # final lengths allocate the tables and pages; appends start from L0
    "decode_one_token": dict(D=128, P=16, seg=256, L1=[700, 333, 1024], n=[1, 1, 1]),
    "chunks_cross_pages": dict(D=64, P=32, seg=64, L1=[300, 129, 64], n=[70, 1, 64]),
    "some_requests_idle": dict(D=128, P=64, seg=128, L1=[500, 260, 90], n=[0, 130, 0]),
    "past_the_table": dict(D=128, P=16, seg=64, L1=[100, 40], n=[20, 5], extra=[9, 0]),
    "unmapped_segment": dict(D=128, P=16, seg=32, L1=[200, 150], n=[60, 10], unmap=(0, 1, 5)),
    "page128": dict(D=128, P=128, seg=256, L1=[250, 129, 600], n=[10, 129, 300]),
    "page256_d64": dict(D=64, P=256, seg=512, L1=[600, 200], n=[300, 56]),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_append_matches_oracle(name):
    _require_gpu()
    c = CASES[name]
    Hkv = 2
    sp = I.Spec(name=name, B=len(c["L1"]), Hq=4, Hkv=Hkv, D=c["D"], P=c["P"], seg_tokens=c["seg"],
                ctx_lens=c["L1"], q_lens=[1] * len(c["L1"]), seed=31, extra_phys_pages=3)
    wl = I.build(sp)
    dw = DeviceWorkload(wl)
    n = list(c["n"])
    L0 = [L - k for L, k in zip(c["L1"], n)]
    extra = c.get("extra", [0] * len(n))       # tokens that run past the table
    n_app = [k + e for k, e in zip(n, extra)]
    indptr = np.concatenate([[0], np.cumsum(n_app)]).astype(np.int32)
    seg = wl.seg_table.reshape(-1).astype(np.int32).copy()
    if "unmap" in c:
        r, g, s = c["unmap"]
        seg.reshape(wl.B, Hkv, -1)[r, g, s] = -1
    rng = np.random.default_rng(len(name))
    mk = lambda: torch.from_numpy(rng.standard_normal((int(indptr[-1]), Hkv, wl.D)).astype(np.float32)).to(
        torch.bfloat16)
    kn, vn = mk(), mk()
    k0, v0 = _bits(dw.k_pool), _bits(dw.v_pool)
    ks = torch.full((wl.num_phys, wl.D), 7.0, dtype=torch.float32, device="cuda")
    B.seg_paged_attn_append(dw.dims, torch.tensor(L0, dtype=torch.int32, device="cuda"),
                            torch.from_numpy(indptr).cuda(), kn.cuda(), vn.cuda(),
                            torch.from_numpy(seg).cuda(), dw.page_table, dw.k_pool, dw.v_pool, ks)
    torch.cuda.synchronize()
    kw, vw, touched = BO.append(k0, v0, seg, wl.page_table, L0, indptr, _bits(kn), _bits(vn), Hkv, wl.P, wl.pps)
    want_ks = BO.refresh_key_sums(np.full((wl.num_phys, wl.D), 7.0, np.float32), kw, touched, wl.P, wl.D)
    print(f"[append] {name}: tokens {int(indptr[-1])}, pages touched {len(touched)}")
    np.testing.assert_array_equal(_bits(dw.k_pool), kw)
    np.testing.assert_array_equal(_bits(dw.v_pool), vw)
    np.testing.assert_array_equal(ks.cpu().numpy(), want_ks)


def test_append_without_key_sums_and_empty():
    _require_gpu()
    sp = I.Spec(name="nosum", B=1, Hq=2, Hkv=1, D=128, P=16, seg_tokens=64, ctx_lens=[64], q_lens=[1], seed=3)
    wl = I.build(sp)
    dw = DeviceWorkload(wl)
    k0 = _bits(dw.k_pool)
    e = torch.zeros(0, 1, 128, dtype=torch.bfloat16, device="cuda")
    B.seg_paged_attn_append(dw.dims, torch.tensor([0], dtype=torch.int32, device="cuda"),
                            torch.zeros(2, dtype=torch.int32, device="cuda"), e, e, dw.seg_table,
                            dw.page_table, dw.k_pool, dw.v_pool)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_bits(dw.k_pool), k0)
    kn = torch.ones(3, 1, 128, dtype=torch.bfloat16, device="cuda")
    B.seg_paged_attn_append(dw.dims, torch.tensor([10], dtype=torch.int32, device="cuda"),
                            torch.tensor([0, 3], dtype=torch.int32, device="cuda"), kn, kn, dw.seg_table,
                            dw.page_table, dw.k_pool, dw.v_pool)
    torch.cuda.synchronize()
    kw, _, _ = BO.append(k0, _bits(dw.v_pool), wl.seg_table.reshape(-1), wl.page_table, [10], [0, 3],
                         _bits(kn), _bits(kn), 1, 16, wl.pps)
    np.testing.assert_array_equal(_bits(dw.k_pool), kw)
