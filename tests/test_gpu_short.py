"""GPU parity for attention over at most 32 keys: the bf16 attention kernels split each
64-key step into two halves of 32 keys, so with 32 or fewer keys (a 4x8x8 latent, or a
short cross-attention context) the second half holds no key at all. Its wavefronts must
contribute nothing, not NaN. Velocity against the oracle, relative L2 per sample."""
import numpy as np
import pytest

import oracle
import workloads as W
from conftest import oracle_model
from helpers import TOL_BF16, TOL_FP32, rel_l2

pytestmark = pytest.mark.gpu

from gpu_util import dev, host, model  # noqa: E402

TOL = {"fp32": TOL_FP32, "bf16": TOL_BF16}
PRECS = ["fp32", "bf16"]


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("name", ["short16", "short16_dh72", "short32_dh64"])
def test_short_sequence_velocity_parity(name, prec):
    cfg = W.get_config(name)
    t, _ = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    got = host(model(name, prec).velocity(dev(x), t))
    assert np.isfinite(got).all()
    ref = oracle.velocity(oracle_model(name), x, t)
    errs = [rel_l2(got[k], ref[k]) for k in range(cfg.K)]
    assert max(errs) <= TOL[prec], errs


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("name", ["tiny_cfg_ctx20", "tiny_cfg_ctx32"])
def test_short_context_guided_velocity_parity(name, prec):
    from paper_2511_22009_amd import Cond
    cfg = W.get_config(name)
    t, _ = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    ctx, nctx = W.context(cfg, cfg.K), W.null_context(cfg)
    got = host(model(name, prec).velocity(dev(x), t, Cond(dev(ctx), dev(nctx), cfg.guidance)))
    assert np.isfinite(got).all()
    ref = oracle.velocity(oracle_model(name), x, t, ctx, nctx, cfg.guidance)
    errs = [rel_l2(got[k], ref[k]) for k in range(cfg.K)]
    assert max(errs) <= TOL[prec], errs
