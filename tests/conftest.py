import functools
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size parity runs (seconds to minutes of oracle time)")


@functools.lru_cache(maxsize=None)
def blob_for(name, init=None):
    import workloads
    return workloads.make_blob(workloads.get_config(name), init=init)


@functools.lru_cache(maxsize=None)
def oracle_model(name):
    import oracle
    return oracle.load_blob(blob_for(name))
