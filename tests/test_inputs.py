"""Seeded input generator: determinism, distribution, tables (CPU)."""
import math

import numpy as np
import torch

from paper_2606_06256_amd import inputs as I


def test_normals_deterministic_and_standard():
    key = I.stream_key(123, I.KIND_K, 4, 5)
    a = I.normals_f64(key, 0, 200000, "cpu")
    b = I.normals_f64(key, 0, 200000, "cpu")
    assert torch.equal(a, b)
    # counters are independent of the chunking
    c = torch.cat([I.normals_f64(key, 0, 70000, "cpu"), I.normals_f64(key, 70000, 130000, "cpu")])
    assert torch.equal(a, c)
    x = a.numpy()
    assert abs(x.mean()) < 0.01 and abs(x.std() - 1) < 0.01
    # Kolmogorov-Smirnov distance to N(0,1)
    xs = np.sort(x)
    cdf = 0.5 * (1 + np.array([math.erf(v / math.sqrt(2)) for v in xs[::50]]))
    emp = (np.arange(0, len(xs), 50) + 0.5) / len(xs)
    assert np.max(np.abs(cdf - emp)) < 0.01
    other = I.normals_f64(I.stream_key(123, I.KIND_K, 4, 6), 0, 1000, "cpu")
    assert not torch.equal(a[:1000], other)


def test_bf16_rounding_is_two_step_rne():
    x = torch.tensor([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -2.5e-3], dtype=torch.float64)
    y = I.to_bf16(x)
    assert y.dtype == torch.bfloat16
    assert y[0].item() == 1.0 and y[1].item() == 1.0 + 2.0 ** -6


def test_workloads_shapes():
    w = I.config(2)
    assert w.B == 16 and w.G == 4 and w.P == 16 and w.pps == 128
    assert int(w.budgets[0]) == 512 and w.spec.forced_head == 128 and w.spec.forced_tail == 128
    assert w.num_phys == 16 * 8 * 2048
    assert sorted(w.page_table.tolist()) == list(range(w.num_phys))
    w5 = I.config(5)
    assert w5.G == 8 and w5.P == 32 and int(w5.budgets[0]) == 410 and w5.spec.shift_pages == 82
    w4 = I.config(4)
    assert int(w4.ctx_lens[0]) == 66048 and int(w4.budgets[0]) == 852 and w4.spec.forced_tail == 32
    w3 = I.config(3)
    L = w3.ctx_lens.astype(np.int64)
    assert L.min() >= 4096 and L.max() <= 131072
    frac = w3.budgets / w3.n_pages
    assert frac.min() >= 0.05 - 1e-9 and frac.max() <= 0.5 + 1.0 / w3.n_pages.min()


def test_page_valid_counts():
    sp = I.Spec(name="t", B=2, Hq=2, Hkv=1, D=64, P=16, seg_tokens=32, ctx_lens=[40, 16],
                q_lens=[1, 1], seed=1, extra_phys_pages=3)
    w = I.build(sp)
    assert w.num_phys == 4 + 2 + 3   # whole segments are allocated: 2x2 + 1x2 virtual, + 3 spare
    v = w.page_valid
    # request 0: pages of 16, 16, 8 tokens; request 1: one page of 16
    assert sorted(v[v > 0].tolist()) == [8, 16, 16, 16]
    assert int(np.sum(v == 0)) == w.num_phys - 4


def test_shifted_pages_and_scale():
    sp = I.config_spec(5)
    sp.B, sp.ctx_lens, sp.q_lens, sp.budgets = 1, [32 * 200], [1], [20]
    sp.seg_tokens = 32 * 50
    sp.shift_pages = 4
    w = I.build(sp)
    pages = w.shifted_pages(0, 3)
    assert len(pages) == 4 and len(set(pages.tolist())) == 4
    sv = w.shift_vector()
    assert abs(np.linalg.norm(sv) - 3.0) < 1e-12
    K, _ = w.unit_kv(0, 3)
    Kf = K.double().numpy().reshape(200, 32, -1)
    means = Kf.mean(axis=1) @ (sv / 3.0)
    top = set(np.argsort(-means)[:4].tolist())
    assert top == set(pages.tolist())
