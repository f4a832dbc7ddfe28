"""The LDS-poison debug build against the oracle.

libsegpa_poison.so is the library built with SEGPA_LDS_POISON: the kernels
that stage key and value tiles through LDS (chunked prefill, token masses)
write NaN into each slot before the copy that fills it. A read that is not
ordered after its copy's wait and barrier, or a read of a slot that no copy
fills, then puts NaN into the outputs, which fails the same parity checks as
the ordinary build (chunked prefill over many key steps and ragged tails,
partial tiles, empty units; token masses over several key groups and
unselected chunk pages).
"""
import os

import pytest
import torch

from paper_2606_06256_amd import binding as B
from paper_2606_06256_amd import build_lib
from paper_2606_06256_amd import inputs as I

import parity_util as PU
import test_gpu_mass as TM
import test_gpu_parity as TP

pytestmark = pytest.mark.gpu


@pytest.fixture
def poison_library():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    assert os.path.exists(build_lib.POISON_LIB), "build the library first (build_lib.build())"
    old_lib, old_path = B._lib, B.LIB_PATH
    B._lib, B.LIB_PATH = None, build_lib.POISON_LIB
    try:
        yield B.lib()
    finally:
        B._lib, B.LIB_PATH = old_lib, old_path


@pytest.mark.parametrize("name", ["prefill_g4", "prefill_random_empty", "prefill_scaled_keys",
                                  "page128_prefill", "prefill_d64_p32", "prefill_many_entries"])
def test_poisoned_prefill_matches_oracle(poison_library, name):
    PU.run_parity(I.build(TP._spec(name=name, **TP.EDGE[name])), label="poison/" + name)


def test_poisoned_headclass_prefill_matches_oracle(poison_library):
    PU.run_parity(I.build(I.scaled_spec(9, 16, 3)), label="poison/headclass-prefill")


@pytest.mark.parametrize("name", ["key_groups_2_and_3", "random_chunk_gaps", "random_empty_unit",
                                  "page256_key_groups"])
def test_poisoned_token_mass_matches_oracle(poison_library, name):
    wl = I.build(TM._spec(name=name, **TM.MASS_CASES[name]))
    dw = TM._gpu_masses(wl, "poison/" + name)
    q64 = wl.q("cpu").double().numpy()
    sel = PU.oracle_selection(wl, q64)
    TM._check_unit_masses(wl, dw, q64, sel, list(range(wl.num_units)))
