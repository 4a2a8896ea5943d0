"""GPU parity: the HIP path through the C ABI against the oracle, on the same seeded
inputs. Tolerances: relative L2 per sample <= 1e-4 (fp32 mode) and <= 2e-2 (bf16
mode) on v and on the Euler update x' - x; bookkeeping bit-exact."""
import numpy as np
import pytest

import oracle
import workloads as W
from conftest import oracle_model
from helpers import TOL_BF16, TOL_FP32, rel_l2

pytestmark = pytest.mark.gpu

from gpu_util import dev, host, model, torch  # noqa: E402

TOL = {"fp32": TOL_FP32, "bf16": TOL_BF16}
PRECS = ["fp32", "bf16"]
SMALL = ["tiny", "tiny_tsens", "ragged", "dh72", "dh64"]


def _inputs(name):
    cfg = W.get_config(name)
    t, dt = W.slot_times(cfg)
    return cfg, W.latents(cfg, cfg.K), t, dt


# ------------------------------------------------------------------ K6 bookkeeping

@pytest.mark.parametrize("steady", [True, False], ids=["steady", "fill"])
@pytest.mark.parametrize("B", [1, 3, 4])
def test_euler_shift_bit_exact(steady, B):
    cfg = W.get_config("tiny")
    rng = np.random.default_rng(30 + B)
    x = rng.standard_normal((B + 1,) + cfg.latent_shape).astype(np.float32)
    v = rng.standard_normal((B,) + cfg.latent_shape).astype(np.float32)
    dt = -rng.uniform(0.01, 0.5, B).astype(np.float32)
    z = rng.standard_normal(cfg.latent_shape).astype(np.float32)
    xd = dev(x)
    done = torch.full(cfg.latent_shape, np.nan, device="cuda") if steady else None
    model("tiny", "fp32").euler_shift(xd, dev(v), dt, B, dev(z), done)
    got = host(xd)
    xp = oracle.euler(x[:B], v, dt)
    np.testing.assert_array_equal(got[0], z)
    if steady:
        np.testing.assert_array_equal(got[1:B], xp[:B - 1])
        np.testing.assert_array_equal(host(done), xp[B - 1])
        np.testing.assert_array_equal(got[B], x[B])          # slot past the queue untouched
    else:
        np.testing.assert_array_equal(got[1:B + 1], xp)


def test_euler_shift_dt_zero_is_rotation():
    cfg = W.get_config("tiny")
    x = W.latents(cfg, 4)
    v = W.latents(cfg, 4, seed=9)
    z = W.z_new_for_image(cfg, 1)
    xd, done = dev(x), torch.empty(cfg.latent_shape, device="cuda")
    model("tiny", "fp32").euler_shift(xd, dev(v), np.zeros(4, np.float32), 4, dev(z), done)
    got = host(xd)
    np.testing.assert_array_equal(got[0], z)
    np.testing.assert_array_equal(got[1:], x[:3])
    np.testing.assert_array_equal(host(done), x[3])


# ------------------------------------------------------------------ K1 conditioning

@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("name", ["tiny_tsens", "ragged"])
def test_modulation_table_parity(name, prec):
    cfg, _, t, _ = _inputs(name)
    om = oracle_model(name)
    got = host(model(name, prec).modulation(t))
    for k in range(cfg.K):
        ref = oracle.modulation_table(om, t[k])
        assert rel_l2(got[k], ref) <= TOL[prec], (k, rel_l2(got[k], ref))


@pytest.mark.parametrize("prec", PRECS)
def test_modulation_table_rows_are_per_sample(prec):
    """Each sample's table row depends only on its own t: the batched table equals
    each t run alone, bit for bit."""
    cfg, _, t, _ = _inputs("tiny_tsens")
    m = model("tiny_tsens", prec)
    full = host(m.modulation(t))
    for k in range(cfg.K):
        np.testing.assert_array_equal(full[k], host(m.modulation(t[k:k + 1]))[0])


# ------------------------------------------------------------- residual per block

@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("name", ["tiny_tsens", "ragged", "dh72", "dh64"])
def test_residual_stream_per_block(name, prec):
    cfg, x, t, _ = _inputs(name)
    om = oracle_model(name)
    m = model(name, prec)
    for blocks in range(cfg.L + 1):
        got = host(m.residual(dev(x), t, blocks))
        for k in range(cfg.K):
            ref, _ = oracle.residual_one(om, x[k], t[k], None, blocks)
            err = rel_l2(got[k], ref)
            assert err <= TOL[prec], (blocks, k, err)


# ------------------------------------------------------------------ velocity

@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("name", SMALL)
def test_velocity_parity(name, prec):
    cfg, x, t, _ = _inputs(name)
    ref = oracle.velocity(oracle_model(name), x, t)
    got = host(model(name, prec).velocity(dev(x), t))
    errs = [rel_l2(got[k], ref[k]) for k in range(cfg.K)]
    assert max(errs) <= TOL[prec], errs


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("name", SMALL)
def test_stream_step_parity(name, prec):
    cfg, x, t, dt = _inputs(name)
    B = cfg.K
    z = W.z_new_for_image(cfg, 7)
    xn_ref, done_ref, v_ref = oracle.stream_step(oracle_model(name), x, t, dt, z, steady=True)
    xd = dev(x)
    done = torch.empty(cfg.latent_shape, device="cuda")
    model(name, prec).stream_step(xd, t, dt, B, dev(z), done)
    got = host(xd)
    np.testing.assert_array_equal(got[0], z)
    new = np.concatenate([got[1:], host(done)[None]])      # x'_k for k = 0..B-1
    for k in range(B):
        err = rel_l2(new[k] - x[k], dt[k] * v_ref[k])
        assert err <= TOL[prec], (k, err)


# -------------------------------------------------------- method invariants on GPU

@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("name", ["tiny_tsens", "ragged", "dh72", "dh64"])
def test_heterogeneous_batch_equals_each_sample_alone(name, prec):
    cfg, x, t, _ = _inputs(name)
    m = model(name, prec)
    full = host(m.velocity(dev(x), t))
    for k in range(cfg.K):
        alone = host(m.velocity(dev(x[k:k + 1]), t[k:k + 1]))[0]
        np.testing.assert_array_equal(full[k], alone)


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("name", SMALL)
def test_repeated_calls_are_bit_identical(name, prec):
    """No kernel depends on scheduling: the same call twice gives the same bits."""
    cfg, x, t, _ = _inputs(name)
    m = model(name, prec)
    xd = dev(x)
    first = host(m.velocity(xd, t))
    for _ in range(3):
        np.testing.assert_array_equal(host(m.velocity(xd, t)), first)


@pytest.mark.parametrize("prec", PRECS)
def test_sample_independence(prec):
    cfg, x, t, _ = _inputs("tiny_tsens")
    m = model("tiny_tsens", prec)
    v = host(m.velocity(dev(x), t))
    x2, t2 = x.copy(), t.copy()
    x2[2] += 0.5
    t2[2] = 0.1
    v2 = host(m.velocity(dev(x2), t2))
    for k in (0, 1, 3):
        np.testing.assert_array_equal(v[k], v2[k])
    assert rel_l2(v2[2], v[2]) > 1e-2


def test_tsens_negative_control_on_gpu():
    """bf16 outputs at different t must differ by far more than the tolerance (so the
    parity tests above would catch a t broadcast)."""
    cfg, x, t, _ = _inputs("tiny_tsens")
    xs = np.repeat(x[:1], cfg.K, axis=0)
    v = host(model("tiny_tsens", "bf16").velocity(dev(xs), t))
    assert min(rel_l2(v[i], v[j]) for i in range(4) for j in range(4) if i != j) >= 10 * TOL_BF16


@pytest.mark.parametrize("prec", PRECS)
def test_constant_field_stream_closed_form(prec):
    """All weights zero except the output bias c: every image leaves the pipeline as
    z + (t_end - t_start) c, bit-exact on dyadic data."""
    from paper_2511_22009_amd import Model, Precision
    from paper_2511_22009_amd.pipeline import run_images
    cfg = W.get_config("tiny")
    tens = W.make_weights(cfg, init="zero")
    rng = np.random.default_rng(12)
    c = (rng.integers(-32, 33, cfg.patch_dim) / 16.0).astype(np.float32)
    tens["b_f"] = c
    m = Model(W.write_blob(cfg, tens), Precision[prec.upper()], 4)
    grid = W.schedule(cfg)
    noise_np = lambda j: (np.round(W.z_new_for_image(cfg, j) * 256) / 256).astype(np.float32)
    imgs = run_images(m, grid, 5, lambda j: dev(noise_np(j)))
    cf = oracle.unpatchify(np.tile(c, (cfg.N, 1)), cfg.C, cfg.H, cfg.W, cfg.p)
    for i, img in enumerate(imgs):
        np.testing.assert_array_equal(host(img), noise_np(i + 1) + np.float32(grid[-1] - grid[0]) * cf)
    m.close()


def test_alg2_driver_network_call_count():
    """Eq. 7 on the GPU driver: M images take M + K - 1 network calls, the first K - 1 at
    occupancy 1 .. K - 1 with nothing finished, then M at occupancy K, each emitting one
    finished latent."""
    from paper_2511_22009_amd.pipeline import run_images
    cfg = W.get_config("tiny")
    inner = model("tiny", "bf16")

    class Counting:
        def __init__(self):
            self.calls = []

        def __getattr__(self, name):
            return getattr(inner, name)

        def stream_step(self, x, t, dt, B, z_new, x_done=None, cond=None, stream=None):
            self.calls.append((B, x_done is not None))
            return inner.stream_step(x, t, dt, B, z_new, x_done, cond, stream)

    m = Counting()
    grid = W.schedule(cfg)
    K, M = len(grid) - 1, 6
    imgs = run_images(m, grid, M, lambda j: dev(W.z_new_for_image(cfg, j)))
    assert len(imgs) == M and len(m.calls) == M + K - 1
    assert m.calls == [(b, False) for b in range(1, K)] + [(K, True)] * M
    assert all(np.isfinite(host(i)).all() for i in imgs)


@pytest.mark.parametrize("prec", PRECS)
def test_stream_equals_sequential_on_gpu(prec):
    """Alg. 2 through sf_stream_step (fill, then full) gives each image exactly what
    a one-image sampler gives (batch invariance), and matches the oracle's stream."""
    from paper_2511_22009_amd.pipeline import run_images
    cfg = W.get_config("tiny_tsens")
    m = model("tiny_tsens", prec)
    grid = W.schedule(cfg)
    M = 5
    imgs = [host(i) for i in run_images(m, grid, M, lambda j: dev(W.z_new_for_image(cfg, j)))]
    ref = oracle.run_stream(oracle_model("tiny_tsens"), grid, M, lambda j: W.z_new_for_image(cfg, j))
    for i in range(M):
        x = dev(W.z_new_for_image(cfg, i + 1)[None])
        for s in range(cfg.K):
            v = m.velocity(x, grid[s:s + 1])
            x = _euler_gpu(m, x, v, np.float32(grid[s + 1] - grid[s]))
        np.testing.assert_array_equal(imgs[i], host(x)[0])
        assert rel_l2(imgs[i], ref[i]) <= 4 * TOL[prec]


def _euler_gpu(m, x, v, dt):
    """One sample's Euler step through sf_euler_shift with a one-slot queue."""
    buf = torch.empty((2,) + tuple(x.shape[1:]), device="cuda")
    buf[0].copy_(x[0])
    done = torch.empty(tuple(x.shape[1:]), device="cuda")
    m.euler_shift(buf, v, np.float32([dt]), 1, x[0], done)
    return done[None]


# ------------------------------------------------- cross-attention and guidance

def _cfg_inputs():
    cfg = W.get_config("tiny_cfg")
    t, dt = W.slot_times(cfg)
    return cfg, W.latents(cfg, cfg.K), t, dt, W.context(cfg, cfg.K), W.null_context(cfg)


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("guided", [True, False], ids=["guided", "cond_only"])
def test_cross_attention_velocity_parity(prec, guided):
    from paper_2511_22009_amd import Cond
    cfg, x, t, _, ctx, nctx = _cfg_inputs()
    m = model("tiny_cfg", prec)
    w = cfg.guidance if guided else None
    ref = oracle.velocity(oracle_model("tiny_cfg"), x, t, ctx, nctx if guided else None, w)
    cond = Cond(dev(ctx), dev(nctx) if guided else None, cfg.guidance)
    got = host(m.velocity(dev(x), t, cond))
    errs = [rel_l2(got[k], ref[k]) for k in range(cfg.K)]
    assert max(errs) <= TOL[prec], errs


@pytest.mark.parametrize("prec", PRECS)
def test_guided_stream_step_parity(prec):
    from paper_2511_22009_amd import Cond
    cfg, x, t, dt, ctx, nctx = _cfg_inputs()
    z = W.z_new_for_image(cfg, 3)
    _, _, v_ref = oracle.stream_step(oracle_model("tiny_cfg"), x, t, dt, z, True, ctx, nctx, cfg.guidance)
    xd = dev(x)
    done = torch.empty(cfg.latent_shape, device="cuda")
    model("tiny_cfg", prec).stream_step(xd, t, dt, cfg.K, dev(z), done, Cond(dev(ctx), dev(nctx), cfg.guidance))
    got = host(xd)
    new = np.concatenate([got[1:], host(done)[None]])
    np.testing.assert_array_equal(got[0], z)
    for k in range(cfg.K):
        assert rel_l2(new[k] - x[k], dt[k] * v_ref[k]) <= TOL[prec]


def test_guidance_weight_zero_gives_unconditional_rows():
    """w = 0 must return exactly the unconditional rows (v_u + 0 (v_c - v_u) = v_u)."""
    from paper_2511_22009_amd import Cond
    cfg, x, t, _, ctx, nctx = _cfg_inputs()
    m = model("tiny_cfg", "fp32")
    v0 = host(m.velocity(dev(x), t, Cond(dev(ctx), dev(nctx), 0.0)))
    vu = host(m.velocity(dev(x), t, Cond(dev(np.repeat(nctx[None], cfg.K, 0)), None, 0.0)))
    np.testing.assert_array_equal(v0, vu)


# ------------------------------------------------- image-to-image and one-step runs

def test_noise_latent_bit_exact():
    cfg = W.get_config("tiny")
    rng = np.random.default_rng(17)
    ref = rng.standard_normal(cfg.latent_shape).astype(np.float32)
    z = rng.standard_normal(cfg.latent_shape).astype(np.float32)
    m = model("tiny", "fp32")
    for t0 in (1.0, 0.0, 0.5, 0.37):
        got = host(m.noise_latent(dev(ref), dev(z), t0))
        np.testing.assert_array_equal(got, oracle.noise_latent(ref, z, t0))


@pytest.mark.parametrize("prec", PRECS)
def test_img2img_stream_matches_oracle(prec):
    """A schedule starting at t0 = 0.5 with noised references admitted through the
    queue, against the oracle's Alg. 2 on the same noised inputs."""
    from paper_2511_22009_amd.pipeline import run_images
    cfg = W.get_config("tiny_tsens")
    grid = np.array([0.5, 0.25, 0.0], np.float32)
    refs = {j: W.latents(cfg, 1, seed=500 + j)[0] for j in range(1, 8)}
    m = model("tiny_tsens", prec)
    imgs = run_images(m, grid, 4, lambda j: dev(W.z_new_for_image(cfg, j)), references=lambda j: dev(refs[j]))
    noisy = lambda j: oracle.noise_latent(refs[j], W.z_new_for_image(cfg, j), grid[0])  # noqa: E731
    ref = oracle.run_stream(oracle_model("tiny_tsens"), grid, 4, noisy)
    for i in range(4):
        assert rel_l2(host(imgs[i]), ref[i]) <= 4 * TOL[prec]


@pytest.mark.parametrize("prec", PRECS)
def test_one_step_queue_matches_oracle(prec):
    from paper_2511_22009_amd.pipeline import run_images
    cfg = W.get_config("tiny_tsens")
    grid = np.array([1.0, 0.0], np.float32)
    imgs = run_images(model("tiny_tsens", prec), grid, 3, lambda j: dev(W.z_new_for_image(cfg, j)))
    ref = oracle.run_stream(oracle_model("tiny_tsens"), grid, 3, lambda j: W.z_new_for_image(cfg, j))
    for i in range(3):
        assert rel_l2(host(imgs[i]), ref[i]) <= TOL[prec]


# ------------------------------------------------------------------ batch limits

@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("name", ["ragged", "dh64"])
def test_max_rows_velocity_parity(name, prec):
    """The largest batch one call takes (64 network rows, the ABI's limit), every sample at
    its own t: Eq. 5's heterogeneous call against the oracle, sample by sample."""
    cfg = W.get_config(name)
    B = 64
    x = W.latents(cfg, B, seed=71)
    t = np.random.default_rng(72).uniform(0.0, 1.0, B).astype(np.float32)
    ref = oracle.velocity(oracle_model(name), x, t)
    got = host(model(name, prec, max_rows=B).velocity(dev(x), t))
    errs = [rel_l2(got[k], ref[k]) for k in range(B)]
    assert max(errs) <= TOL[prec], max(errs)


def test_gemm_k_not_multiple_of_slice_velocity_parity():
    """Width 96 (2 heads of 48, MLP 384): the QKV projection (N 288), the attention output
    projection (N 96) and fc1 (N 384) run the directly staged narrow GEMM with K = 96,
    which is not a multiple of its 64-wide K slice, so every slice's operand loads take
    the per-column K check (with K a multiple of 64 they go through resources rebased at
    each slice instead). bf16 velocity of every slot against the oracle, and each row
    alone against the batch, bit for bit."""
    from paper_2511_22009_amd import Model, Precision
    cfg = W.Config("w96", C=4, H=16, W=20, p=2, D=96, L=2, heads=2, mlp=384)
    blob = W.make_blob(cfg)
    x = W.latents(cfg, cfg.K)
    t, _ = W.slot_times(cfg)
    m = Model(blob, Precision.BF16, cfg.K)
    got = host(m.velocity(dev(x), t))
    ref = oracle.velocity(oracle.load_blob(blob), x, t)
    errs = [rel_l2(got[k], ref[k]) for k in range(cfg.K)]
    assert max(errs) <= TOL_BF16, errs
    for k in range(cfg.K):
        np.testing.assert_array_equal(got[k], host(m.velocity(dev(x[k:k + 1]), t[k:k + 1]))[0])


def test_two_query_blocks_per_wavefront_equal_one():
    """64 rows of the head-dim-48 network run attention with two 32-query blocks per
    wavefront (512 workgroups of 128 queries); four rows at a time take one block per
    wavefront. Every query is computed in the same order either way: same bits."""
    cfg = W.get_config("ragged")
    B = 64
    x = W.latents(cfg, B, seed=75)
    t = np.random.default_rng(76).uniform(0.0, 1.0, B).astype(np.float32)
    m = model("ragged", "bf16", max_rows=B)
    full = host(m.velocity(dev(x), t))
    for k0 in range(0, B, 4):
        np.testing.assert_array_equal(full[k0:k0 + 4], host(m.velocity(dev(x[k0:k0 + 4]), t[k0:k0 + 4])))


@pytest.mark.parametrize("name,prec", [("tiny", "fp32"), ("tiny", "bf16"), ("dh72", "fp32"),
                                       ("dh64", "bf16"), ("tiny_cfg", "bf16")])
def test_embed_in_modulation_launch_equals_own_launch(name, prec):
    """The patch embed shares the launch of the last adaLN projection unless per-class
    kernel times are taken; with the embed's timing on it runs as a launch of its own.
    Same bits either way, also with guidance (twice as many embedded rows as table rows)."""
    from paper_2511_22009_amd import Cond, KernelClass, Model, Precision
    from conftest import blob_for
    cfg = W.get_config(name)
    B = cfg.K
    x, t = W.latents(cfg, B, seed=81), np.random.default_rng(82).uniform(0.0, 1.0, B).astype(np.float32)
    m = Model(blob_for(name, None), Precision[prec.upper()], 2 * B)
    cond = Cond(dev(W.context(cfg, B)), dev(W.null_context(cfg)), cfg.guidance) if cfg.has_cross else None
    shared = host(m.velocity(dev(x), t, cond))
    m.timing_enable(KernelClass.EMBED, True)
    own = host(m.velocity(dev(x), t, cond))
    m.timing_enable(KernelClass.EMBED, False)
    np.testing.assert_array_equal(shared, own)
    np.testing.assert_array_equal(shared, host(m.velocity(dev(x), t, cond)))
    m.close()


@pytest.mark.parametrize("prec", PRECS)
def test_max_rows_guided_velocity_parity(prec):
    """32 text-conditioned samples with guidance fill all 64 rows (cond and uncond)."""
    from paper_2511_22009_amd import Cond
    cfg = W.get_config("tiny_cfg")
    B = 32
    x = W.latents(cfg, B, seed=73)
    t = np.random.default_rng(74).uniform(0.0, 1.0, B).astype(np.float32)
    ctx, nctx = W.context(cfg, B), W.null_context(cfg)
    ref = oracle.velocity(oracle_model("tiny_cfg"), x, t, ctx, nctx, cfg.guidance)
    m = model("tiny_cfg", prec, max_rows=2 * B)
    got = host(m.velocity(dev(x), t, Cond(dev(ctx), dev(nctx), cfg.guidance)))
    errs = [rel_l2(got[k], ref[k]) for k in range(B)]
    assert max(errs) <= TOL[prec], max(errs)


def test_batch_beyond_capacity_is_rejected():
    """A call needing more network rows than the model was loaded for fails with an error
    and writes nothing; guidance doubles the rows a sample needs."""
    from paper_2511_22009_amd import Cond, SFError
    cfg = W.get_config("tiny_cfg")
    m = model("tiny_cfg", "bf16", max_rows=4)
    x = dev(W.latents(cfg, 5))
    t = np.full(5, 0.5, np.float32)
    out = torch.full((5,) + cfg.latent_shape, 7.0, device="cuda")
    with pytest.raises(SFError):
        m.velocity(x, t, out=out)
    cond = Cond(dev(W.context(cfg, 3)), dev(W.null_context(cfg)), cfg.guidance)
    with pytest.raises(SFError):
        m.velocity(x[:3], t[:3], cond, out=out[:3])
    assert bool((host(out) == 7.0).all())
    ok = host(m.velocity(x[:2], t[:2], Cond(dev(W.context(cfg, 2)), dev(W.null_context(cfg)), cfg.guidance)))
    assert np.isfinite(ok).all()
