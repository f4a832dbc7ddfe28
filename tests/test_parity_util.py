"""Host checks of the GPU-parity helpers (no GPU needed)."""
import gc

import numpy as np

import parity_util as PU
from paper_2606_06256_amd import inputs as I


def _spec(name, D, P, ctx, Hkv=2, Hq=4, seed=1):
    return I.Spec(name=name, B=1, Hq=Hq, Hkv=Hkv, D=D, P=P, seg_tokens=4 * P, ctx_lens=[ctx],
                  q_lens=[1], seed=seed)


def test_kv64_never_returns_another_workloads_keys():
    # Workloads of different shapes built and dropped in turn: CPython reuses
    # object ids after collection, so a cache keyed by id() would hand a new
    # workload an old workload's arrays. Each call must return the keys of
    # the workload it was given.
    shapes = [(64, 32, 400), (128, 16, 64), (64, 16, 150), (128, 32, 333)] * 3
    for n, (D, P, L) in enumerate(shapes):
        wl = I.build(_spec(f"w{n}", D, P, L, seed=10 + n))
        for g in range(wl.Hkv):
            K, V = PU.kv64(wl, 0, g)
            Kr, Vr = wl.unit_kv(0, g)
            assert K.shape == (L, D) and V.shape == (L, D)
            np.testing.assert_array_equal(K, Kr.double().numpy())
            np.testing.assert_array_equal(V, Vr.double().numpy())
        del wl
        gc.collect()


def test_kv64_cache_is_bounded_per_workload():
    wl = I.build(I.Spec(name="many", B=2, Hq=8, Hkv=8, D=64, P=16, seg_tokens=64,
                        ctx_lens=[40, 50], q_lens=[1, 1], seed=3))
    for r in range(2):
        for g in range(8):
            PU.kv64(wl, r, g)
    assert len(wl.__dict__["_kv64_cache"]) <= PU.KV_CACHE_UNITS
