"""The allocation-free conditioning entry point (sf_modulation_noalloc) against
sf_modulation: the same table bit for bit, on two calls in a row (the second with
fewer samples and other timesteps), from a model whose max_rows is smaller than the
batch; and sizes beyond the fixed scratch array are refused without writing."""
import numpy as np
import pytest

import oracle
import workloads as W
from conftest import blob_for, oracle_model
from helpers import TOL_BF16, TOL_FP32, rel_l2

pytestmark = pytest.mark.gpu

from gpu_util import host, torch  # noqa: E402

TOL = {"fp32": TOL_FP32, "bf16": TOL_BF16}


@pytest.mark.parametrize("prec", ["bf16", "fp32"])
@pytest.mark.parametrize("name", ["tiny_tsens", "ragged"])
def test_modulation_noalloc_equals_modulation(name, prec):
    from paper_2511_22009_amd import Model, Precision
    cfg = W.get_config(name)
    m = Model(blob_for(name), Precision[prec.upper()], 2)
    mw = m.info["mod_width"]
    rng = np.random.default_rng(90)
    om = oracle_model(name)
    for B in (9, 3):                        # the second call is smaller than the first
        t = rng.uniform(0.0, 1.0, B).astype(np.float32)
        got = torch.full((B, mw), np.nan, device="cuda")
        m.modulation_noalloc(t, got)
        ref = torch.empty((B, mw), device="cuda")
        for k0 in range(0, B, 2):           # the workspace entry point takes max_rows samples at a time
            m.modulation(t[k0:k0 + 2], out=ref[k0:k0 + 2])
        np.testing.assert_array_equal(host(got), host(ref))
        for k in range(B):
            assert rel_l2(host(got)[k], oracle.modulation_table(om, t[k])) <= TOL[prec]
    m.close()


def test_modulation_noalloc_rejects_more_than_the_array_holds():
    from paper_2511_22009_amd import Model, Precision, SFError
    m = Model(blob_for("tiny"), Precision.BF16, 4)
    out = torch.full((65, m.info["mod_width"]), 7.0, device="cuda")
    with pytest.raises(SFError) as e:
        m.modulation_noalloc(np.full(65, 0.5, np.float32), out)
    assert e.value.code == -1
    assert bool((host(out) == 7.0).all())
    m.modulation_noalloc(np.full(64, 0.5, np.float32), out)
    assert np.isfinite(host(out)[:64]).all() and bool((host(out)[64] == 7.0).all())
    m.close()
