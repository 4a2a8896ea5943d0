"""Graph replay (sf_graph_enable): every replay of a captured stream step or velocity
call must equal the eager call bit for bit, with eager work and synchronisations in
between the replays; a change of t (or of any argument) captures a new graph."""
import numpy as np
import pytest

import workloads as W
from conftest import blob_for

pytestmark = pytest.mark.gpu

from gpu_util import dev, host, torch  # noqa: E402


def _fresh(name, prec):
    from paper_2511_22009_amd import Model, Precision
    return Model(blob_for(name), Precision[prec.upper()], 8)


@pytest.mark.parametrize("prec", ["bf16", "fp32"])
def test_stream_step_replays_equal_eager(prec):
    cfg = W.get_config("tiny_tsens")
    t, dt = W.slot_times(cfg)
    x0 = W.latents(cfg, cfg.K)
    m = _fresh("tiny_tsens", prec)
    s = torch.cuda.Stream()
    z = dev(W.z_new_for_image(cfg, 2))
    xe, de = dev(x0), torch.empty(cfg.latent_shape, device="cuda")
    m.stream_step(xe, t, dt, cfg.K, z, de, stream=s)
    s.synchronize()
    ref_x, ref_d = host(xe), host(de)
    m.graph_enable(True)
    xg, dg = dev(x0), torch.empty(cfg.latent_shape, device="cuda")
    for rep in range(4):
        with torch.cuda.stream(s):
            xg.copy_(torch.from_numpy(x0).cuda())
            dg.fill_(float("nan"))
        m.stream_step(xg, t, dt, cfg.K, z, dg, stream=s)
        s.synchronize()
        np.testing.assert_array_equal(host(xg), ref_x)
        np.testing.assert_array_equal(host(dg), ref_d)
        junk = torch.randn(1 << 16, device="cuda").sum()  # unrelated eager work between replays
        torch.cuda.synchronize()
        assert torch.isfinite(junk)
    cached, replays = m.graph_stats()
    assert cached == 1 and replays == 3
    # another t: a new graph, still equal to the eager result for that t
    t2 = (t * np.float32(0.5)).astype(np.float32)
    m.graph_enable(False)
    xe2, de2 = dev(x0), torch.empty(cfg.latent_shape, device="cuda")
    m.stream_step(xe2, t2, dt, cfg.K, z, de2, stream=s)
    s.synchronize()
    m.graph_enable(True)
    for _ in range(2):
        with torch.cuda.stream(s):
            xg.copy_(torch.from_numpy(x0).cuda())
        m.stream_step(xg, t2, dt, cfg.K, z, dg, stream=s)
        s.synchronize()
        np.testing.assert_array_equal(host(xg), host(xe2))
        np.testing.assert_array_equal(host(dg), host(de2))
    assert m.graph_stats()[0] == 1  # disabling dropped the first graph
    m.close()


def test_guided_velocity_replays_equal_eager():
    from paper_2511_22009_amd import Cond
    cfg = W.get_config("tiny_cfg")
    t, _ = W.slot_times(cfg)
    x = dev(W.latents(cfg, cfg.K))
    cond = Cond(dev(W.context(cfg, cfg.K)), dev(W.null_context(cfg)), cfg.guidance)
    m = _fresh("tiny_cfg", "bf16")
    s = torch.cuda.Stream()
    ve = torch.empty_like(x)
    m.velocity(x, t, cond, out=ve, stream=s)
    s.synchronize()
    ref = host(ve)
    m.graph_enable(True)
    vg = torch.empty_like(x)
    for _ in range(3):
        with torch.cuda.stream(s):
            vg.zero_()
        m.velocity(x, t, cond, out=vg, stream=s)
        s.synchronize()
        np.testing.assert_array_equal(host(vg), ref)
    assert m.graph_stats() == (1, 2)
    m.close()


def test_null_stream_and_timing_run_eagerly():
    """On the legacy default stream, or while a kernel class is timed, nothing is
    captured and results are unchanged."""
    from paper_2511_22009_amd import KernelClass
    cfg = W.get_config("tiny")
    t, _ = W.slot_times(cfg)
    x = dev(W.latents(cfg, cfg.K))
    m = _fresh("tiny", "bf16")
    ref = host(m.velocity(x, t))
    m.graph_enable(True)
    np.testing.assert_array_equal(host(m.velocity(x, t, stream=torch.cuda.default_stream())), ref)
    s = torch.cuda.Stream()
    m.timing_enable(KernelClass.QKV, True)
    out = m.velocity(x, t, stream=s)
    s.synchronize()
    np.testing.assert_array_equal(host(out), ref)
    m.timing_enable(KernelClass.QKV, False)
    assert m.graph_stats()[0] == 0
    m.close()


@pytest.mark.parametrize("graphs", [False, True])
def test_modulation_cache_is_bit_identical(graphs):
    """A run of stream steps whose timesteps repeat, change and come back gives the same
    bits with the modulation cache as without it, eager and graph-replayed; the cached
    table is reused exactly when the previous network call had the same timesteps."""
    cfg = W.get_config("tiny_tsens")
    t1, dt = W.slot_times(cfg)
    t2 = (t1 * np.float32(0.5)).astype(np.float32)
    seq = [t1, t1, t2, t1, t1, t1]
    x0 = W.latents(cfg, cfg.K)
    z = dev(W.z_new_for_image(cfg, 2))
    s = torch.cuda.Stream()
    runs = []
    for cache in (False, True):
        m = _fresh("tiny_tsens", "bf16")
        m.graph_enable(graphs)
        m.modulation_cache(cache)
        x, d = dev(x0), torch.empty(cfg.latent_shape, device="cuda")
        res = []
        for tt in seq:
            m.stream_step(x, tt, dt, cfg.K, z, d, stream=s)
            s.synchronize()
            res.append((host(x), host(d)))
        assert m.modulation_cache_stats() == (3 if cache else 0)
        runs.append(res)
        m.close()
    for (xa, da), (xb, db) in zip(*runs):
        np.testing.assert_array_equal(xa, xb)
        np.testing.assert_array_equal(da, db)


def test_modulation_cache_guided_and_mixed_calls():
    """With guidance (cond and uncond rows share their latent's table row) and with
    velocity calls, stream steps of another batch size and a call on another stream
    interleaved, the cached table is reused only when it is right: every call equals
    the same call on a model without the cache, bit for bit."""
    from paper_2511_22009_amd import Cond
    cfg = W.get_config("tiny_cfg")
    t, dt = W.slot_times(cfg)
    K = cfg.K
    x0 = W.latents(cfg, K)
    cond = Cond(dev(W.context(cfg, K)), dev(W.null_context(cfg)), cfg.guidance)
    z = dev(W.z_new_for_image(cfg, 3))
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    # (kind, batch, stream): velocity or stream step
    calls = [("v", K, s1), ("v", K, s1), ("step", K, s1), ("v", K - 1, s1), ("v", K - 1, s1),
             ("v", K - 1, s2), ("step", K, s1), ("step", K, s1)]
    runs = []
    for cache in (False, True):
        m = _fresh("tiny_cfg", "bf16")
        m.modulation_cache(cache)
        x = dev(x0)
        d = torch.empty(cfg.latent_shape, device="cuda")
        res = []
        for kind, b, st in calls:
            cb = Cond(cond.ctx[:b], cond.null_ctx, cond.guidance)
            if kind == "v":
                out = m.velocity(x[:b], t[:b], cb, stream=st)
            else:
                m.stream_step(x, t, dt, b, z, d, cb, stream=st)
                out = x
            st.synchronize()
            res.append(host(out))
        # reuses: call 2 (same t as call 1), call 3 (same t, a step), call 5 (same t[:K-1]),
        # call 8 (same t as call 7); not call 6 (another stream) nor call 7 (after a
        # different batch on another stream)
        assert m.modulation_cache_stats() == (4 if cache else 0)
        runs.append(res)
        m.close()
    for a, b in zip(*runs):
        np.testing.assert_array_equal(a, b)
