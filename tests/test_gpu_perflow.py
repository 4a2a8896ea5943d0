"""PeRFlow time windows on the GPU (sf_set_scheduler): the per-slot window update
against the oracle (Sec. 2 windows, Sec. 3.3, Alg. 1), composed with the queue shift
and with the network; bookkeeping bit-exact."""
import numpy as np
import pytest

import workloads as W
from conftest import blob_for, oracle_model
from helpers import TOL_BF16, TOL_FP32, rel_l2
from oracle import perflow as pf

pytestmark = pytest.mark.gpu

from gpu_util import dev, host, torch  # noqa: E402

TOL = {"fp32": TOL_FP32, "bf16": TOL_BF16}
ABAR = pf.alphas_cumprod()


def _fresh(name, prec="fp32"):
    from paper_2511_22009_amd import Model, Precision
    return Model(blob_for(name), Precision[prec.upper()], 8)


CASES = {
    # uniform 4 steps on 4 windows: every step ends on its window's end
    "uniform": (np.array([1.0, 0.75, 0.5, 0.25], np.float32), np.full(4, -0.25, np.float32)),
    # irregular times inside windows, steps that stay inside or cross a window end
    "irregular": (np.array([0.97, 0.8, 0.51, 0.3], np.float32), np.array([-0.17, -0.29, -0.21, -0.3], np.float32)),
    # times a hair above and below window boundaries
    "edges": (np.array([0.7500019, 0.7499981, 0.2500019, 0.0100001], np.float32),
              np.array([-0.01, -0.2, -0.05, -0.01], np.float32)),
}


@pytest.mark.parametrize("steady", [True, False], ids=["steady", "fill"])
@pytest.mark.parametrize("case", sorted(CASES))
@pytest.mark.parametrize("B", [1, 3, 4])
def test_window_update_and_shift_match_oracle(case, B, steady):
    cfg = W.get_config("tiny")
    t, dt = CASES[case]
    t, dt = t[:B], dt[:B]
    rng = np.random.default_rng(B * 10 + len(case))
    x = rng.standard_normal((B + 1,) + cfg.latent_shape).astype(np.float32)
    e = rng.standard_normal((B,) + cfg.latent_shape).astype(np.float32)
    z = rng.standard_normal(cfg.latent_shape).astype(np.float32)
    m = _fresh("tiny")
    m.set_scheduler(windows=4)
    xd = dev(x)
    done = torch.full(cfg.latent_shape, np.nan, device="cuda") if steady else None
    m.scheduler_shift(xd, dev(e), t, dt, B, dev(z), done)
    got = host(xd)
    ref, _ = pf.batched_velocity_step(e, x[:B], t, dt, 4, ABAR)
    np.testing.assert_array_equal(got[0], z)
    new = np.concatenate([got[1:B], host(done)[None]]) if steady else got[1:B + 1]
    np.testing.assert_allclose(new, ref, rtol=2e-6, atol=2e-6)
    if steady:
        np.testing.assert_array_equal(got[B], x[B])      # the slot past the queue is untouched
    m.close()


def test_uniform_steps_land_on_the_window_prediction():
    """dt = t^e - t: the update lands on X_pred = lambda_t x + eta_t eps."""
    cfg = W.get_config("tiny")
    t, dt = CASES["uniform"]
    rng = np.random.default_rng(5)
    x = rng.standard_normal((5,) + cfg.latent_shape).astype(np.float32)
    e = rng.standard_normal((4,) + cfg.latent_shape).astype(np.float32)
    m = _fresh("tiny")
    m.set_scheduler(windows=4)
    xd, done = dev(x), torch.empty(cfg.latent_shape, device="cuda")
    m.scheduler_shift(xd, dev(e), t, dt, 4, dev(x[4]), done)
    new = np.concatenate([host(xd)[1:4], host(done)[None]])
    p = pf.batch_params(t, 4, ABAR)
    pred = p["lam_t"][:, None, None, None] * x[:4].astype(np.float64) + p["eta_t"][:, None, None, None] * e
    np.testing.assert_allclose(new, pred, rtol=2e-6, atol=2e-6)
    m.close()


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
@pytest.mark.parametrize("name", ["tiny_tsens", "ragged"])
def test_window_stream_step_parity(name, prec):
    """sf_stream_step with the scheduler set: the network output read as eps, every
    slot's update x' - x against the oracle's (same tolerances as the Euler step)."""
    cfg = W.get_config(name)
    t, dt = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    z = W.z_new_for_image(cfg, 9)
    xn_ref, done_ref, _ = pf.stream_step(oracle_model(name), x, t, dt, z, cfg.K, ABAR)
    m = _fresh(name, prec)
    m.set_scheduler(windows=cfg.K)
    xd, done = dev(x), torch.empty(cfg.latent_shape, device="cuda")
    m.stream_step(xd, t, dt, cfg.K, dev(z), done)
    got = host(xd)
    np.testing.assert_array_equal(got[0], z)
    new = np.concatenate([got[1:], host(done)[None]])
    ref = np.concatenate([xn_ref[1:], done_ref[None]])
    for k in range(cfg.K):
        assert rel_l2(new[k] - x[k], ref[k] - x[k]) <= TOL[prec], k
    m.close()


def test_clearing_the_scheduler_restores_euler_and_graphs_follow():
    cfg = W.get_config("tiny_tsens")
    t, dt = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    z = dev(W.z_new_for_image(cfg, 1))
    m = _fresh("tiny_tsens")
    s = torch.cuda.Stream()
    m.graph_enable(True)

    def run():
        xd, done = dev(x), torch.empty(cfg.latent_shape, device="cuda")
        torch.cuda.synchronize()
        m.stream_step(xd, t, dt, cfg.K, z, done, stream=s)
        s.synchronize()
        return host(xd), host(done)

    euler = run()
    m.set_scheduler(windows=4)
    win = [run(), run()]                                  # capture, then replay
    m.clear_scheduler()
    back = run()
    np.testing.assert_array_equal(back[0], euler[0])
    np.testing.assert_array_equal(back[1], euler[1])
    np.testing.assert_array_equal(win[0][0], win[1][0])
    assert rel_l2(win[0][1], euler[1]) > 1e-3             # the window update is a different map
    m.close()


def test_scheduler_rejects_bad_parameters():
    from paper_2511_22009_amd import SFError
    m = _fresh("tiny")
    for kw in [dict(windows=0), dict(train_steps=1), dict(beta_start=0.0), dict(beta_end=0.0001),
               dict(beta_end=1.5), dict(eps=0.5), dict(eps=-1.0)]:
        with pytest.raises(SFError):
            m.set_scheduler(**kw)
    m.close()
