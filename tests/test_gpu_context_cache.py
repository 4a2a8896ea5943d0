"""GPU: the cross-attention context entries (sf_context_cache). Calls with entries
reused across calls must return the same bits as calls that project every context,
for every pattern of contexts a caller can pass: unchanged slots, Alg. 2's shift (each
context moves one slot on with its latent), a context rewritten in place, a new null
context, a call without guidance in between, and queues that shrink and grow. The
projection counts show which entries were reused."""
import numpy as np
import pytest

import oracle
import workloads as W
from conftest import blob_for, oracle_model
from helpers import TOL_BF16, TOL_FP32, rel_l2

pytestmark = pytest.mark.gpu

from gpu_util import dev, host, torch  # noqa: E402

TOL = {"fp32": TOL_FP32, "bf16": TOL_BF16}


def _fresh(prec, max_rows=8):
    from paper_2511_22009_amd import Model, Precision
    return Model(blob_for("tiny_cfg"), Precision[prec.upper()], max_rows)


def _contexts(cfg, n, seed):
    return np.stack([W.context(cfg, 1, seed=seed + i)[0] for i in range(n)])


@pytest.mark.parametrize("prec", ["bf16", "fp32"])
def test_reused_entries_give_identical_bits(prec):
    from paper_2511_22009_amd import Cond
    cfg = W.get_config("tiny_cfg")
    t, _ = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    pool = _contexts(cfg, 8, seed=50)           # distinct contexts
    null_a, null_b = W.null_context(cfg), _contexts(cfg, 1, seed=90)[0]
    plain, cached = _fresh(prec), _fresh(prec)
    cached.context_cache(True)
    assert cached.context_cache_stats() == (0, 0)
    # (slots' contexts as pool indices or arrays, null context or None, B, projections expected)
    calls = [
        ([0, 1, 2, 3], null_a, 4, 5),            # nothing known: 4 contexts + the null one
        ([0, 1, 2, 3], null_a, 4, 0),            # every slot unchanged
        ([4, 0, 1, 2], null_a, 4, 1),            # Alg. 2 shift: slots 1..3 took their neighbours' contexts
        ([4, 0, "mod", 2], null_a, 4, 1),        # slot 2 rewritten in place
        ([4, 0, "mod", 2], null_b, 4, 1),        # new null context
        ([4, 0, "mod", 2], None, 4, 0),          # no guidance: conditional rows only
        ([4, 0, "mod", 2], null_b, 4, 1),        # guidance again: the null entry was forgotten
        ([4, 0], null_b, 2, 0),                  # queue shrinks
        ([5, 4, 0], null_b, 3, 1),               # and grows with a shift (fill phase)
        ([5, 4, 0], null_b, 3, 0),
    ]
    done = 0
    for i, (slots, nctx, B, expect) in enumerate(calls):
        ctx = np.stack([pool[s] if s != "mod" else pool[1] * np.float32(0.5) for s in slots])
        cond = Cond(dev(ctx), dev(nctx) if nctx is not None else None, cfg.guidance)
        ref = host(plain.velocity(dev(x[:B]), t[:B], cond))
        got = host(cached.velocity(dev(x[:B]), t[:B], cond))
        np.testing.assert_array_equal(got, ref)
        n, proj = cached.context_cache_stats()
        assert n == i + 1
        assert proj - done == expect, (slots, B, proj - done, expect)
        done = proj
    cached.context_cache(False)
    assert cached.context_cache_stats() == (0, 0)
    plain.close()
    cached.close()


def test_context_rewritten_in_the_same_buffer_is_projected_again():
    """The lookup compares contents, not pointers: a context buffer rewritten between
    calls (same device pointer) must not reuse the old keys and values."""
    from paper_2511_22009_amd import Cond
    cfg = W.get_config("tiny_cfg")
    t, _ = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    plain, cached = _fresh("bf16"), _fresh("bf16")
    cached.context_cache(True)
    ctx = dev(_contexts(cfg, cfg.K, seed=60))
    nctx = dev(W.null_context(cfg))
    cond = Cond(ctx, nctx, cfg.guidance)
    np.testing.assert_array_equal(host(cached.velocity(dev(x), t, cond)), host(plain.velocity(dev(x), t, cond)))
    ctx[1, 3, 5] += 1.0                          # one element of slot 1's context
    np.testing.assert_array_equal(host(cached.velocity(dev(x), t, cond)), host(plain.velocity(dev(x), t, cond)))
    assert cached.context_cache_stats() == (2, cfg.K + 1 + 1)
    plain.close()
    cached.close()


def test_alg2_queue_with_reuse_matches_without():
    """Alg. 2 over six images (the queue shifts each context with its latent), graph
    replay on a side stream: finished latents bit-identical with and without reuse, and
    after the first call every step projects only the admitted image's context."""
    from paper_2511_22009_amd.pipeline import StreamQueue
    cfg = W.get_config("tiny_cfg")
    grid = W.schedule(cfg)
    K = len(grid) - 1
    M = 6
    # three noise buffers in turn and one output buffer, so full-queue steps repeat their
    # arguments and the later ones replay captured graphs while the contexts keep changing
    pool = [dev(W.z_new_for_image(cfg, j)) for j in range(3)]
    ctxs = [dev(_contexts(cfg, 1, seed=200 + j)[0]) for j in range(M + K + 1)]
    nctx = dev(W.null_context(cfg))
    torch.cuda.synchronize()
    outs = []
    for reuse in (False, True):
        m = _fresh("bf16")
        m.context_cache(reuse)
        m.graph_enable(True)
        s = torch.cuda.Stream()
        done = torch.empty(cfg.latent_shape, device="cuda")
        imgs = []
        with torch.cuda.stream(s):
            buf = torch.empty((K + 1,) + tuple(ctxs[1].shape), device="cuda")
            buf[0].copy_(ctxs[1])
            q = StreamQueue(m, grid, pool[1 % 3], buf, nctx, cfg.guidance)
            for j in range(1, M + K):
                if q.step(pool[(j + 1) % 3], done_out=done, ctx_next=ctxs[j + 1]) is not None:
                    imgs.append(done.clone())
        torch.cuda.synchronize()
        outs.append([host(i) for i in imgs[:M]])
        assert m.graph_stats()[1] > 0            # some steps were replayed
        if reuse:
            calls, proj = m.context_cache_stats()
            assert calls == M + K - 1
            # first call: its context and the null one; then one new context per step
            assert proj == 2 + (calls - 1), (calls, proj)
        m.close()
    assert len(outs[0]) == M
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("prec", ["bf16", "fp32"])
def test_guided_stream_step_with_reuse_against_oracle(prec):
    """Two identical guided stream steps with reuse on (the second reuses every entry),
    each against the oracle's step from the same state."""
    from paper_2511_22009_amd import Cond
    cfg = W.get_config("tiny_cfg")
    t, dt = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    ctx, nctx = W.context(cfg, cfg.K), W.null_context(cfg)
    z = W.z_new_for_image(cfg, 3)
    _, _, v_ref = oracle.stream_step(oracle_model("tiny_cfg"), x, t, dt, z, True, ctx, nctx, cfg.guidance)
    m = _fresh(prec)
    m.context_cache(True)
    cond = Cond(dev(ctx), dev(nctx), cfg.guidance)
    for _ in range(2):
        xd = dev(x)
        done = torch.empty(cfg.latent_shape, device="cuda")
        m.stream_step(xd, t, dt, cfg.K, dev(z), done, cond)
        got = host(xd)
        new = np.concatenate([got[1:], host(done)[None]])
        np.testing.assert_array_equal(got[0], z)
        for k in range(cfg.K):
            assert rel_l2(new[k] - x[k], dt[k] * v_ref[k]) <= TOL[prec]
    assert m.context_cache_stats() == (2, cfg.K + 1)
    m.close()


def test_network_without_cross_attention_ignores_the_switch():
    from paper_2511_22009_amd import Model, Precision
    m = Model(blob_for("tiny"), Precision.BF16, 4)
    m.context_cache(True)
    assert m.context_cache_stats() == (0, 0)
    m.close()
