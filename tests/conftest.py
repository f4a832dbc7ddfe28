import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Run order of the test modules. The hot-path parity suite (selection,
# translation, split-KV attention, LSE combine, chunked prefill) runs first, so
# that with -x a failure in a later state-building or token-selection module
# can never hide it. Modules not listed keep their collection order after
# these; test_zz_* modules always run last.
FIRST = ("test_gpu_parity.py",)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: oracle runs at full workload size (seconds to minutes)")


def _rank(item):
    name = os.path.basename(str(item.fspath))
    if name in FIRST:
        return FIRST.index(name)
    if name.startswith("test_zz_"):
        return len(FIRST) + 2
    return len(FIRST) + 1


def pytest_collection_modifyitems(config, items):
    # stable sort: the order inside a module is unchanged. Nothing is skipped
    # silently: GPU tests fail loudly when no GPU or no library is present.
    items.sort(key=_rank)
