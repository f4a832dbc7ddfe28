"""The README's usage example runs as written and attends over the pages it
selected (fp64 oracle over the same tokens)."""
import math
import os
import re

import numpy as np
import pytest
import torch

from oracle import segpa_oracle as O

README = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "README.md")


def _example_code():
    text = open(README).read()
    sec = text[text.index("## Using the library"):]
    return re.search(r"```python\n(.*?)```", sec, re.S).group(1)


@pytest.mark.gpu
def test_readme_example_runs_and_matches_the_oracle():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    torch.manual_seed(0)
    ns = {}
    exec(compile(_example_code(), "README.md example", "exec"), ns)
    Hq, Hkv, D, P, L = ns["Hq"], ns["Hkv"], ns["D"], ns["P"], ns["L"]
    G = Hq // Hkv
    ind = ns["sel_indptr"].cpu().numpy()
    pages = ns["sel_pages"].cpu().numpy()
    q = ns["q"].float().cpu().double().numpy()            # [1, Hq, D]
    K = ns["k_new"].float().cpu().double().numpy()        # [L, Hkv, D] logical order
    V = ns["v_new"].float().cpu().double().numpy()
    out = ns["out"].float().cpu().numpy()
    lse = ns["lse"].cpu().numpy()
    n = (L + P - 1) // P
    for g in range(Hkv):
        sel = [int(p) for p in pages[ind[g]:ind[g + 1]]]
        assert len(sel) == 16 and sel == sorted(set(sel)) and all(0 <= p < n for p in sel)
        assert set(range(4)) <= set(sel) and set(range(n - 4, n)) <= set(sel)
        Oo, LSE = O.attend_unit(q[:, g * G:(g + 1) * G], K[:, g], V[:, g], sel, P, 1 / math.sqrt(D))
        np.testing.assert_allclose(out[:, g * G:(g + 1) * G], Oo, atol=2e-2, rtol=0)
        np.testing.assert_allclose(lse[:, g * G:(g + 1) * G], LSE, atol=1e-3, rtol=0)
