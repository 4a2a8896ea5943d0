"""Helpers for the GPU tests: device upload and cached library handles."""
import functools

import numpy as np
import pytest

torch = pytest.importorskip("torch")


def gpu_available():
    return torch.cuda.is_available()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


@functools.lru_cache(maxsize=None)
def model(name, prec, max_rows=8, init=None):
    from conftest import blob_for
    from paper_2511_22009_amd import Model, Precision
    return Model(blob_for(name, init), Precision[prec.upper()], max_rows)
