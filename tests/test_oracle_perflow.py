"""Pins for the oracle's PeRFlow time-window conversion (Sec. 2 time windows, Sec. 3.3,
Alg. 1), each against something other than the oracle's own formula: brute force,
closed forms and identities the equations imply."""
import math

import numpy as np
import pytest

import oracle
from oracle import perflow as pf


def test_alphas_cumprod_brute_force():
    """The scaled-linear schedule, recomputed with a pure-Python loop (beta from the
    square of a linear interpolation of sqrt(beta), running product)."""
    T, b0, b1 = 1000, 0.00085, 0.012
    prod, ref = 1.0, []
    for i in range(T):
        s = math.sqrt(b0) + (math.sqrt(b1) - math.sqrt(b0)) * i / (T - 1)
        prod *= 1.0 - s * s
        ref.append(prod)
    np.testing.assert_allclose(pf.alphas_cumprod(T, b0, b1), ref, rtol=1e-13)
    a = pf.alphas_cumprod()
    assert a[0] == pytest.approx(1 - b0) and np.all(np.diff(a) < 0) and 0.004 < a[-1] < 0.005


@pytest.mark.parametrize("K_w", [1, 2, 4, 8])
def test_window_lookup_matches_argmax_definition(K_w):
    """k = argmax_k {t > t_k^e + eps}: the largest window whose end lies below t."""
    rng = np.random.default_rng(7)
    t = np.concatenate([rng.uniform(0.0, 1.0, 200), np.arange(K_w + 1) / K_w,
                        np.arange(1, K_w + 1) / K_w + 2e-6, np.arange(1, K_w + 1) / K_w - 2e-6])
    t = t[(t > 2e-6) & (t <= 1.0)]
    got = pf.window_lookup(t, K_w)
    for ti, ki in zip(t, got):
        best = max(k for k in range(1, K_w + 1) if ti > (k - 1) / K_w + 1e-6)
        assert ki == best, (ti, ki, best)
        # t lies in its window: t^e < t <= t^s (up to the tolerance)
        assert (ki - 1) / K_w < ti <= ki / K_w + 1e-6


def test_window_boundaries_belong_to_the_window_they_start():
    """A time exactly on a boundary starts the lower window (the tolerance pushes it
    down), so a uniform K-step schedule on K windows takes one window per step."""
    k = pf.window_lookup(np.array([1.0, 0.75, 0.5, 0.25]), 4)
    np.testing.assert_array_equal(k, [4, 3, 2, 1])


def test_lambda_eta_identity_and_limits():
    a = pf.alphas_cumprod()
    t = np.array([1.0, 0.9, 0.75, 0.6, 0.5, 0.31, 0.25, 0.1])
    p = pf.batch_params(t, 4, a)
    # lambda_s^2 - eta_s^2 = (1 - (1 - gamma^2)) / gamma^2 = 1
    np.testing.assert_allclose(p["lam_s"] ** 2 - p["eta_s"] ** 2, 1.0, rtol=1e-12)
    assert np.all(p["gamma"] < 1) and np.all(p["lam_s"] > 1) and np.all(p["eta_s"] < 0)
    # at the window start the time-dependent parameters equal the window's own
    at_start = np.isclose(t, p["ts"])
    assert at_start.sum() == 4
    np.testing.assert_allclose(p["lam_t"][at_start], p["lam_s"][at_start], rtol=1e-14)
    np.testing.assert_allclose(p["eta_t"][at_start], p["eta_s"][at_start], rtol=1e-14)
    # approaching the window end, lambda_t -> 1 and eta_t -> 0 (X_pred -> X)
    near_end = pf.batch_params(p["te"][:4] + 1e-5, 4, a)
    np.testing.assert_allclose(near_end["lam_t"], 1.0, atol=1e-4)
    np.testing.assert_allclose(near_end["eta_t"], 0.0, atol=1e-4)


def test_gamma_from_schedule_values():
    a = pf.alphas_cumprod()
    p = pf.batch_params(np.array([1.0]), 4, a)
    np.testing.assert_allclose(p["gamma"], [math.sqrt(a[999] / a[round(0.75 * 999)])], rtol=1e-14)


def test_step_ending_on_window_end_lands_on_the_prediction():
    """dt = t^e - t: X_next = X + (t^e - t) (X_pred - X) / (t^e - t) = X_pred."""
    a = pf.alphas_cumprod()
    rng = np.random.default_rng(3)
    t = np.array([1.0, 0.8, 0.55, 0.3], np.float32)
    p = pf.batch_params(t, 4, a)
    dt = (p["te"] - t.astype(np.float64)).astype(np.float32)
    X = rng.standard_normal((4, 2, 3, 5)).astype(np.float32)
    E = rng.standard_normal((4, 2, 3, 5)).astype(np.float32)
    xn, _ = pf.batched_velocity_step(E, X, t, dt, 4, a)
    sh = (-1, 1, 1, 1)
    x_pred = p["lam_t"].reshape(sh) * X.astype(np.float64) + p["eta_t"].reshape(sh) * E.astype(np.float64)
    # dt was rounded to fp32, so the landing is exact up to that rounding
    np.testing.assert_allclose(xn, x_pred, rtol=2e-6, atol=2e-6)


def test_update_is_the_stated_affine_map_and_per_sample():
    """X_next = (1 + c (lambda_t - 1)) X + c eta_t eps with c = dt / (t^e - t), slot by
    slot; a batch equals each slot alone."""
    a = pf.alphas_cumprod()
    rng = np.random.default_rng(11)
    t = np.array([0.97, 0.71, 0.44, 0.12], np.float32)
    dt = np.array([-0.1, -0.05, -0.2, -0.12], np.float32)
    X = rng.standard_normal((4, 4, 8, 8)).astype(np.float32)
    E = rng.standard_normal((4, 4, 8, 8)).astype(np.float32)
    xn, v = pf.batched_velocity_step(E, X, t, dt, 4, a)
    for k in range(4):
        p = pf.batch_params(t[k:k + 1], 4, a)
        c = float(dt[k]) / (p["te"][0] - float(t[k]))
        ref = (1 + c * (p["lam_t"][0] - 1)) * X[k].astype(np.float64) + c * p["eta_t"][0] * E[k].astype(np.float64)
        np.testing.assert_allclose(xn[k], ref, rtol=1e-6, atol=1e-6)
        alone, _ = pf.batched_velocity_step(E[k:k + 1], X[k:k + 1], t[k:k + 1], dt[k:k + 1], 4, a)
        np.testing.assert_array_equal(alone[0], xn[k])


def test_perflow_stream_step_shift_and_fill():
    """The window update composes with Alg. 2's shift exactly like the Euler update."""
    import workloads as W
    cfg = W.get_config("tiny")
    m = oracle.load_blob(W.make_blob(cfg))
    t, dt = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    z = W.z_new_for_image(cfg, 4)
    a = pf.alphas_cumprod()
    xn, done, e = pf.stream_step(m, x, t, dt, z, 4, a)
    ref, _ = pf.batched_velocity_step(e, x, t, dt, 4, a)
    np.testing.assert_array_equal(xn[0], z)
    np.testing.assert_array_equal(xn[1:], ref[:-1])
    np.testing.assert_array_equal(done, ref[-1])
    xf, none, _ = pf.stream_step(m, x[:2], t[:2], dt[:2], z, 4, a, steady=False)
    assert none is None and xf.shape[0] == 3
