"""Error paths of the C ABI on a GPU: a rejected call returns its code and leaves every
output untouched, a failed device allocation comes back as SF_E_OOM without a handle,
and a scheduler whose allocation fails is cleared (Euler on the velocity), never left
half set."""
import ctypes
import os

import numpy as np
import pytest

import oracle
import workloads as W
from conftest import blob_for

pytestmark = pytest.mark.gpu

from gpu_util import dev, host, model, torch  # noqa: E402

SF_E_INVAL, SF_E_OOM = -1, -4


def _sentinel(shape, value=7.0):
    return torch.full(shape, value, device="cuda")


@pytest.mark.parametrize("bad", [np.nan, np.inf, -np.inf])
def test_non_finite_times_are_rejected_and_write_nothing(bad):
    from paper_2511_22009_amd import SFError
    cfg = W.get_config("tiny")
    m = model("tiny", "bf16")
    t, dt = W.slot_times(cfg)
    x0 = W.latents(cfg, cfg.K)
    z = dev(W.z_new_for_image(cfg, 1))
    for which in ("t", "dt"):
        tt, dd = t.copy(), dt.copy()
        (tt if which == "t" else dd)[2] = bad
        xd, done = dev(x0), _sentinel(cfg.latent_shape)
        with pytest.raises(SFError) as e:
            m.stream_step(xd, tt, dd, cfg.K, z, done)
        assert e.value.code == SF_E_INVAL
        np.testing.assert_array_equal(host(xd), x0)
        assert bool((host(done) == 7.0).all())
    out = _sentinel((cfg.K,) + cfg.latent_shape)
    tt = t.copy()
    tt[0] = bad
    with pytest.raises(SFError) as e:
        m.velocity(dev(x0), tt, out=out)
    assert e.value.code == SF_E_INVAL and bool((host(out) == 7.0).all())
    with pytest.raises(SFError) as e:
        m.euler_shift(dev(x0), dev(x0), np.where(np.arange(cfg.K) == 1, bad, dt).astype(np.float32), cfg.K, z,
                      _sentinel(cfg.latent_shape))
    assert e.value.code == SF_E_INVAL


@pytest.mark.parametrize("bad", [np.nan, np.inf])
def test_non_finite_guidance_is_rejected(bad):
    from paper_2511_22009_amd import Cond, SFError
    cfg = W.get_config("tiny_cfg")
    m = model("tiny_cfg", "bf16")
    t, dt = W.slot_times(cfg)
    x0 = W.latents(cfg, cfg.K)
    cond = Cond(dev(W.context(cfg, cfg.K)), dev(W.null_context(cfg)), bad)
    out = _sentinel((cfg.K,) + cfg.latent_shape)
    with pytest.raises(SFError) as e:
        m.velocity(dev(x0), t, cond, out=out)
    assert e.value.code == SF_E_INVAL and bool((host(out) == 7.0).all())
    xd, done = dev(x0), _sentinel(cfg.latent_shape)
    with pytest.raises(SFError) as e:
        m.stream_step(xd, t, dt, cfg.K, dev(W.z_new_for_image(cfg, 1)), done, cond)
    assert e.value.code == SF_E_INVAL
    np.testing.assert_array_equal(host(xd), x0)
    assert bool((host(done) == 7.0).all())


@pytest.fixture
def fail_alloc(monkeypatch):
    def set_n(n):
        monkeypatch.setenv("SF_FAIL_ALLOC_AFTER", str(n))
    yield set_n
    monkeypatch.delenv("SF_FAIL_ALLOC_AFTER", raising=False)


@pytest.mark.parametrize("n", [0, 1])
def test_forced_allocation_failure_returns_oom_without_handle(fail_alloc, n):
    """SF_FAIL_ALLOC_AFTER=n fails the (n+1)-th device allocation of a load (weights,
    then workspace): SF_E_OOM and no handle; the next load without it succeeds."""
    from paper_2511_22009_amd import load_library
    blob = bytes(blob_for("tiny"))
    L = load_library()
    fail_alloc(n)
    h = ctypes.c_void_p()
    assert L.sf_load_weights(blob, len(blob), 0, 4, ctypes.byref(h)) == SF_E_OOM
    assert not h.value
    os.environ.pop("SF_FAIL_ALLOC_AFTER")
    assert L.sf_load_weights(blob, len(blob), 0, 4, ctypes.byref(h)) == 0 and h.value
    L.sf_free(h)


def test_failed_scheduler_set_leaves_euler(fail_alloc):
    """A scheduler set whose schedule allocation fails returns SF_E_OOM and leaves the
    model on plain Euler: the next stream step's update equals x + dt v bit for bit."""
    from paper_2511_22009_amd import Model, Precision, SFError
    cfg = W.get_config("tiny")
    m = Model(blob_for("tiny"), Precision.FP32, 4)
    m.set_scheduler(windows=4, train_steps=1000)
    fail_alloc(0)
    with pytest.raises(SFError) as e:
        m.set_scheduler(windows=4, train_steps=500)          # a new length needs a new buffer
    assert e.value.code == SF_E_OOM
    os.environ.pop("SF_FAIL_ALLOC_AFTER")
    rng = np.random.default_rng(5)
    x = rng.standard_normal((cfg.K,) + cfg.latent_shape).astype(np.float32)
    v = rng.standard_normal((cfg.K,) + cfg.latent_shape).astype(np.float32)
    t, dt = W.slot_times(cfg)
    xd, done = dev(x), torch.empty(cfg.latent_shape, device="cuda")
    m.scheduler_shift(xd, dev(v), t, dt, cfg.K, dev(W.z_new_for_image(cfg, 2)), done)
    got = np.concatenate([host(xd)[1:], host(done)[None]])
    np.testing.assert_array_equal(got, oracle.euler(x, v, dt))
    m.set_scheduler(windows=4, train_steps=500)                # recovers once memory is there
    m.close()
