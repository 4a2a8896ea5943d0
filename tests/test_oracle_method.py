"""The method's own invariants, checked on the oracle (CPU only).

(a) a heterogeneous-t batch equals each sample run alone at its own t (Eq. 5);
(b) Euler integration reproduces closed forms for a constant field and a
    straight-line field (Sec. 3.1.1);
and the Alg. 2 queue: stream output equals independent per-image samplers, the
network-call count of Eq. 7, and exact bookkeeping of the shift.
"""
import os

import numpy as np
import pytest

import oracle
import workloads as W
from conftest import oracle_model
from helpers import TOL_BF16, rel_l2

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("name", ["tiny", "tiny_tsens", "ragged"])
def test_heterogeneous_batch_equals_each_sample_alone(name):
    cfg = W.get_config(name)
    m = oracle_model(name)
    t, _ = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    v = oracle.velocity(m, x, t)
    for k in range(cfg.K):
        np.testing.assert_array_equal(v[k], oracle.velocity(m, x[k:k + 1], t[k:k + 1])[0])


def test_sample_independence():
    cfg = W.get_config("tiny_tsens")
    m = oracle_model("tiny_tsens")
    t, _ = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    v = oracle.velocity(m, x, t)
    x2, t2 = x.copy(), t.copy()
    x2[2] += 0.5
    t2[2] = 0.1
    v2 = oracle.velocity(m, x2, t2)
    for k in (0, 1, 3):
        np.testing.assert_array_equal(v[k], v2[k])
    assert rel_l2(v2[2], v[2]) > 1e-2


def test_tsens_negative_control():
    """Same latent at the K schedule times: every pair of outputs must differ by at
    least 10x the bf16 tolerance, so broadcasting one sample's t to all would fail."""
    cfg = W.get_config("tiny_tsens")
    m = oracle_model("tiny_tsens")
    t, _ = W.slot_times(cfg)
    x = np.repeat(W.latents(cfg, 1), cfg.K, axis=0)
    v = oracle.velocity(m, x, t)
    worst = min(rel_l2(v[i], v[j]) for i in range(cfg.K) for j in range(cfg.K) if i != j)
    assert worst >= 10 * TOL_BF16


def _constant_field_model(cfg, c):
    tens = W.make_weights(cfg, init="zero")
    tens["b_f"] = c
    return oracle.load_blob(W.write_blob(cfg, tens))


def test_constant_field_stream_is_exact():
    """v == c everywhere: after the S-step schedule each image is z + (sum dt) c,
    bit-exact with dyadic data (x in 2^-8 Z, c in 2^-4 Z, dt = -1/4)."""
    cfg = W.get_config("tiny")
    rng = np.random.default_rng(12)
    c = (rng.integers(-32, 33, cfg.patch_dim) / 16.0).astype(np.float32)
    m = _constant_field_model(cfg, c)
    grid = W.schedule(cfg)
    noise = lambda j: (np.round(W.z_new_for_image(cfg, j) * 256) / 256).astype(np.float32)
    imgs = oracle.run_stream(m, grid, 5, noise)
    cf = oracle.unpatchify(np.tile(c, (cfg.N, 1)), cfg.C, cfg.H, cfg.W, cfg.p)
    total = np.float32(grid[-1] - grid[0])
    for i, img in enumerate(imgs):
        np.testing.assert_array_equal(img, noise(i + 1) + total * cf)


def test_straight_line_field_lands_on_data():
    """x_t = t z + (1 - t) x_data has velocity (x_t - x_data) / t; Euler is exact on
    a straight line, so from noise at t = 1 the last step lands on x_data."""
    for name in ("tiny", "s512_cfg"):    # uniform and irregular schedules
        cfg = W.get_config(name)
        grid = W.schedule(cfg)
        z = W.latents(cfg, 1, seed=21)[0].astype(np.float64)
        xd = W.latents(cfg, 1, seed=22)[0].astype(np.float64)
        x = z[None]
        for i in range(len(grid) - 1):
            v = (x - xd) / np.float64(grid[i])
            x = oracle.euler(x, v, [np.float64(grid[i + 1]) - np.float64(grid[i])])
        assert rel_l2(x[0], xd) < 1e-12


@pytest.mark.parametrize("name", ["tiny", "tiny_cfg"])
def test_stream_equals_sequential(name):
    cfg = W.get_config(name)
    m = oracle_model(name)
    grid = W.schedule(cfg)
    M = 6
    noise = lambda j: W.z_new_for_image(cfg, j)
    kw = {}
    if cfg.cfg:
        ctxs = W.context(cfg, M + cfg.K)
        kw = dict(ctx_of=lambda j: ctxs[j - 1], null_ctx=W.null_context(cfg), guidance=cfg.guidance)
    imgs = oracle.run_stream(m, grid, M, noise, **kw)
    assert len(imgs) == M
    for i in range(M):
        skw = {} if not cfg.cfg else dict(ctx=ctxs[i], null_ctx=kw["null_ctx"], guidance=cfg.guidance)
        np.testing.assert_array_equal(imgs[i], oracle.sequential_sample(m, noise(i + 1), grid, **skw))


def _golden_rows():
    rows = []
    with open(os.path.join(GOLDEN, "eq7_network_calls.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                rows.append(tuple(int(v) for v in line.split()))
    return rows


@pytest.mark.parametrize("M,S,pipelined,sequential", _golden_rows())
def test_eq7_network_call_count(monkeypatch, M, S, pipelined, sequential):
    from dataclasses import replace
    cfg = replace(W.get_config("tiny"), L=0, schedule=f"uniform{S}", K=S)
    m = oracle.load_blob(W.make_blob(cfg))
    calls = []
    real = oracle.stream.velocity
    monkeypatch.setattr(oracle.stream, "velocity", lambda *a, **k: calls.append(a[1].shape[0]) or real(*a, **k))
    oracle.run_stream(m, W.schedule(cfg), M, lambda j: W.z_new_for_image(cfg, j))
    assert len(calls) == pipelined
    assert max(calls) == min(S, M + S - 1)
    assert M * S == sequential


def test_dt_zero_step_is_pure_rotation():
    cfg = W.get_config("tiny")
    m = oracle_model("tiny")
    t, _ = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    z = W.z_new_for_image(cfg, 1)
    xn, done, _ = oracle.stream_step(m, x, t, np.zeros(cfg.K, np.float32), z)
    np.testing.assert_array_equal(xn[0], z)
    np.testing.assert_array_equal(xn[1:], x[:-1])
    np.testing.assert_array_equal(done, x[-1])


def test_fill_phase_grows_queue():
    cfg = W.get_config("tiny")
    m = oracle_model("tiny")
    t, dt = W.slot_times(cfg)
    x = W.latents(cfg, 2)
    z = W.z_new_for_image(cfg, 3)
    xn, done, v = oracle.stream_step(m, x, t[:2], dt[:2], z, steady=False)
    assert done is None and xn.shape[0] == 3
    np.testing.assert_array_equal(xn[0], z)
    np.testing.assert_array_equal(xn[1:], oracle.euler(x, v, dt[:2]))


# ------------------------------------------------- image-to-image and one-step runs

def test_noise_latent_endpoints_and_line():
    """x = (1 - t0) x_ref + t0 z: t0 = 1 gives z, t0 = 0 gives x_ref, and at dyadic t0 on
    dyadic data the point is exact."""
    rng = np.random.default_rng(21)
    ref = (rng.integers(-64, 65, (4, 8, 8)) / 16.0).astype(np.float32)
    z = (rng.integers(-64, 65, (4, 8, 8)) / 16.0).astype(np.float32)
    np.testing.assert_array_equal(oracle.noise_latent(ref, z, 1.0), z)
    np.testing.assert_array_equal(oracle.noise_latent(ref, z, 0.0), ref)
    np.testing.assert_array_equal(oracle.noise_latent(ref, z, 0.25), 0.75 * ref + 0.25 * z)
    mid = oracle.noise_latent(ref, z, 0.5)
    np.testing.assert_array_equal(mid - ref, 0.5 * (z - ref))


def test_img2img_stream_equals_sequential_from_the_noised_reference():
    """A schedule starting at t0 < 1 with noised references admitted: every image equals
    the one-image sampler started from its own noised reference."""
    cfg = W.get_config("tiny_tsens")
    m = oracle.load_blob(W.make_blob(cfg))
    grid = np.array([0.5, 0.25, 0.0], np.float32)
    refs = {j: W.latents(cfg, 1, seed=500 + j)[0] for j in range(1, 8)}
    noisy = lambda j: oracle.noise_latent(refs[j], W.z_new_for_image(cfg, j), grid[0])  # noqa: E731
    imgs = oracle.run_stream(m, grid, 4, noisy)
    for i, img in enumerate(imgs):
        np.testing.assert_array_equal(img, oracle.sequential_sample(m, noisy(i + 1), grid))


def test_one_step_queue():
    """K = 1: every call finishes one image in a single Euler step from t = 1 to 0."""
    cfg = W.get_config("tiny_tsens")
    m = oracle.load_blob(W.make_blob(cfg))
    grid = np.array([1.0, 0.0], np.float32)
    imgs = oracle.run_stream(m, grid, 3, lambda j: W.z_new_for_image(cfg, j))
    for i, img in enumerate(imgs):
        z = W.z_new_for_image(cfg, i + 1)
        v = oracle.velocity(m, z[None], grid[:1])[0]
        np.testing.assert_array_equal(img, z + np.float32(-1.0) * v)
