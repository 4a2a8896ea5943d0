"""Pins of the oracle against things other than itself: closed forms, library
routines, brute force on tiny inputs, and special weight settings whose output is
known in closed form. CPU only."""
import math
from dataclasses import replace

import numpy as np
import pytest
import scipy.special

import oracle
import workloads as W
from workloads.configs import Config
from helpers import rel_l2

MICRO = Config("micro", C=2, H=4, W=4, p=2, D=8, L=1, heads=2, mlp=16, tdim=8, K=2,
               schedule="uniform2")
MICRO_X = replace(MICRO, name="micro_x", ctx_len=3, ctx_dim=4, has_cross=1)


def _weights(cfg, std, seed=11):
    rng = np.random.default_rng(seed)
    return {n: (rng.standard_normal(s) * std).astype(np.float32) for n, s in W.tensor_specs(cfg)}


def _model(cfg, tensors):
    return oracle.load_blob(W.write_blob(cfg, tensors))


# ----------------------------------------------------------------------------- blob

def test_blob_roundtrip_and_validation():
    cfg = W.get_config("tiny")
    tens = W.make_weights(cfg)
    blob = W.write_blob(cfg, tens)
    assert len(blob) == 64 + 4 * sum(int(np.prod(s)) for _, s in W.tensor_specs(cfg))
    m = oracle.load_blob(blob)
    assert (m.D, m.L, m.heads, m.N) == (128, 2, 4, 64)
    np.testing.assert_array_equal(m.blocks[1]["W_fc2"], tens["blk1.W_fc2"])
    np.testing.assert_array_equal(m.top["b_f"], tens["b_f"])
    with pytest.raises(ValueError):
        oracle.load_blob(blob[:-4])
    with pytest.raises(ValueError):
        oracle.load_blob(blob + b"\0\0\0\0")
    with pytest.raises(ValueError):
        oracle.load_blob(b"XFW1" + blob[4:])


# ------------------------------------------------------------------ timestep embedding

def test_timestep_embedding_at_zero():
    e = oracle.timestep_embedding(0.0, 128)
    np.testing.assert_array_equal(e, np.r_[np.ones(64), np.zeros(64)].astype(np.float32))


def test_timestep_frequency_closed_forms():
    f = oracle.timestep_frequencies(128)
    assert f[0] == np.float32(1.0)
    assert f[32] == np.float32(0.01)          # 10000^(-1/2)
    assert f[16] == np.float32(0.1)           # 10000^(-1/4)
    assert np.all(np.diff(f) < 0)


@pytest.mark.parametrize("t", [1.0, 0.75, 0.5, 0.25, 0.123, 0.9761])
def test_timestep_embedding_values(t):
    e = oracle.timestep_embedding(t, 128).astype(np.float64)
    tau = float(np.float32(1000.0) * np.float32(t))
    assert e[0] == np.float32(math.cos(tau)) and e[64] == np.float32(math.sin(tau))
    np.testing.assert_allclose(e[:64] ** 2 + e[64:] ** 2, 1.0, atol=2e-7)


# --------------------------------------------------------------- elementwise pieces

def test_layer_norm_moments():
    rng = np.random.default_rng(5)
    z = (rng.standard_normal((16, 96)) * 3 + 7).astype(np.float64)
    y = oracle.layer_norm(z)
    np.testing.assert_allclose(y.mean(axis=1), 0.0, atol=1e-12)
    var = ((z - z.mean(1, keepdims=True)) ** 2).mean(1)
    np.testing.assert_allclose((y ** 2).mean(axis=1), var / (var + 1e-6), rtol=1e-12)
    np.testing.assert_array_equal(oracle.layer_norm(np.full((2, 8), 3.5)), 0.0)


def test_gelu_and_silu():
    z = np.linspace(-8, 8, 1601)
    assert oracle.gelu_tanh(np.float64(0.0)) == 0.0 and oracle.silu(np.float64(0.0)) == 0.0
    np.testing.assert_allclose(oracle.silu(z), z * scipy.special.expit(z), rtol=1e-13, atol=1e-300)
    gelu_erf = 0.5 * z * (1 + scipy.special.erf(z / math.sqrt(2)))
    assert np.max(np.abs(oracle.gelu_tanh(z) - gelu_erf)) < 1e-3
    np.testing.assert_allclose(oracle.gelu_tanh(np.array([30.0, -30.0])), [30.0, 0.0], atol=1e-12)


# ------------------------------------------------------------------------ patchify

def test_patchify_index_map_and_roundtrip():
    cfg = W.get_config("ragged")
    x = W.latents(cfg, 1)[0]
    tok = oracle.patchify(x, cfg.p)
    gw = cfg.W // cfg.p
    for n in [0, 1, gw - 1, gw, 77, cfg.N - 1]:
        gh_, gw_ = divmod(n, gw)
        for i in range(cfg.p):
            for j in range(cfg.p):
                for c in range(cfg.C):
                    assert tok[n, (i * cfg.p + j) * cfg.C + c] == x[c, gh_ * cfg.p + i, gw_ * cfg.p + j]
    np.testing.assert_array_equal(oracle.unpatchify(tok, cfg.C, cfg.H, cfg.W, cfg.p), x)


# ----------------------------------------------------------------------- attention

def test_attention_identical_keys_returns_mean_value():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((5, 12))
    k = np.tile(rng.standard_normal((1, 12)), (7, 1))
    v = rng.standard_normal((7, 12))
    np.testing.assert_allclose(oracle.attention(q, k, v, 3), np.tile(v.mean(0), (5, 1)), rtol=1e-13)


def test_attention_one_dominant_key():
    rng = np.random.default_rng(4)
    q = np.ones((3, 4))
    k = np.zeros((6, 4)); k[2] = 200.0
    v = rng.standard_normal((6, 4))
    np.testing.assert_allclose(oracle.attention(q, k, v, 1), np.tile(v[2], (3, 1)), rtol=1e-13)


def test_attention_bruteforce():
    rng = np.random.default_rng(6)
    heads, dh, nq, nk = 3, 4, 5, 7
    q, k, v = (rng.standard_normal((n, heads * dh)) for n in (nq, nk, nk))
    out = oracle.attention(q, k, v, heads)
    for h in range(heads):
        for i in range(nq):
            s = [sum(q[i, h * dh + d] * k[j, h * dh + d] for d in range(dh)) / math.sqrt(dh) for j in range(nk)]
            mx = max(s)
            w = [math.exp(x - mx) for x in s]
            for d in range(dh):
                ref = sum(w[j] * v[j, h * dh + d] for j in range(nk)) / sum(w)
                assert abs(out[i, h * dh + d] - ref) < 1e-13


def test_linear_bruteforce():
    rng = np.random.default_rng(7)
    x, Wt, b = rng.standard_normal((3, 5)), rng.standard_normal((4, 5)), rng.standard_normal(4)
    y = oracle.dit.linear(x, Wt, b)
    for n in range(3):
        for o in range(4):
            assert abs(y[n, o] - (sum(x[n, i] * Wt[o, i] for i in range(5)) + b[o])) < 1e-13


# ------------------------------------------------------- brute-force whole network

def _bf_forward(m, x, t, ctx=None):
    """Pure-Python loops over the whole velocity network, fp64 after the input
    embedding (tau and the phases are rounded to fp32 as the network definition says)."""
    L = lambda a: np.asarray(a, dtype=np.float64).tolist()
    top = {k: L(v) for k, v in m.top.items()}
    D, P, C, dh = m.D, m.p, m.C, m.D // m.heads
    gh, gw = m.H // P, m.W // P
    N = gh * gw

    def lin(vec, Wm, b):
        return [sum(vec[i] * Wm[o][i] for i in range(len(vec))) + b[o] for o in range(len(Wm))]

    def ln(vec):
        mu = sum(vec) / len(vec)
        var = sum((z - mu) ** 2 for z in vec) / len(vec)
        return [(z - mu) / math.sqrt(var + 1e-6) for z in vec]

    def silu(z):
        return z / (1 + math.exp(-z))

    def attn(Q, K, V):
        out = [[0.0] * D for _ in Q]
        for hd in range(m.heads):
            for i, qi in enumerate(Q):
                s = [sum(qi[hd * dh + d] * kj[hd * dh + d] for d in range(dh)) / math.sqrt(dh) for kj in K]
                mx = max(s)
                w = [math.exp(z - mx) for z in s]
                Z = sum(w)
                for d in range(dh):
                    out[i][hd * dh + d] = sum(w[j] * V[j][hd * dh + d] for j in range(len(K))) / Z
        return out

    half = m.tdim // 2
    tau = float(np.float32(1000.0) * np.float32(t))
    emb_c, emb_s = [], []
    for i in range(half):
        f = float(np.float32(math.exp(-math.log(10000.0) * i / half)))
        phi = float(np.float32(tau * f))
        emb_c.append(math.cos(phi)); emb_s.append(math.sin(phi))
    emb = emb_c + emb_s
    hid = [silu(z) for z in lin(emb, top["W_t1"], top["b_t1"])]
    s = [silu(z) for z in lin(hid, top["W_t2"], top["b_t2"])]

    xl = L(x)
    h = []
    for n in range(N):
        a, b_ = divmod(n, gw)
        tok = [0.0] * (P * P * C)
        for i in range(P):
            for j in range(P):
                for c in range(C):
                    tok[(i * P + j) * C + c] = xl[c][a * P + i][b_ * P + j]
        e = lin(tok, top["W_pe"], top["b_pe"])
        h.append([e[d] + top["pos"][n][d] for d in range(D)])
    for blk in m.blocks:
        bl = {k: L(v) for k, v in blk.items()}
        mod = lin(s, bl["W_mod"], bl["b_mod"])
        sh1, sc1, g1, sh2, sc2, g2 = (mod[i * D:(i + 1) * D] for i in range(6))
        act = [[z * (1 + sc1[d]) + sh1[d] for d, z in enumerate(ln(row))] for row in h]
        qkv = [lin(row, bl["W_qkv"], bl["b_qkv"]) for row in act]
        o = attn([r[:D] for r in qkv], [r[D:2 * D] for r in qkv], [r[2 * D:] for r in qkv])
        h = [[h[n][d] + g1[d] * y for d, y in enumerate(lin(o[n], bl["W_o"], bl["b_o"]))] for n in range(N)]
        if m.has_cross:
            cl = L(ctx)
            qx = [lin(ln(row), bl["W_qx"], bl["b_qx"]) for row in h]
            kv = [lin(r, bl["W_kvx"], bl["b_kvx"]) for r in cl]
            ox = attn(qx, [r[:D] for r in kv], [r[D:] for r in kv])
            h = [[h[n][d] + y for d, y in enumerate(lin(ox[n], bl["W_ox"], bl["b_ox"]))] for n in range(N)]
        act = [[z * (1 + sc2[d]) + sh2[d] for d, z in enumerate(ln(row))] for row in h]
        for n in range(N):
            f1 = lin(act[n], bl["W_fc1"], bl["b_fc1"])
            g = [0.5 * z * (1 + math.tanh(math.sqrt(2 / math.pi) * (z + 0.044715 * z ** 3))) for z in f1]
            f2 = lin(g, bl["W_fc2"], bl["b_fc2"])
            h[n] = [h[n][d] + g2[d] * f2[d] for d in range(D)]
    fm = lin(s, top["W_fmod"], top["b_fmod"])
    shf, scf = fm[:D], fm[D:]
    v = np.zeros((C, m.H, m.W))
    for n in range(N):
        a, b_ = divmod(n, gw)
        out = lin([z * (1 + scf[d]) + shf[d] for d, z in enumerate(ln(h[n]))], top["W_f"], top["b_f"])
        for i in range(P):
            for j in range(P):
                for c in range(C):
                    v[c, a * P + i, b_ * P + j] = out[(i * P + j) * C + c]
    return v


@pytest.mark.parametrize("cfg", [MICRO, MICRO_X], ids=["self", "cross"])
@pytest.mark.parametrize("t", [1.0, 0.37])
def test_forward_matches_bruteforce(cfg, t):
    m = _model(cfg, _weights(cfg, std=0.4))
    rng = np.random.default_rng(8)
    x = rng.standard_normal(cfg.latent_shape).astype(np.float32)
    ctx = rng.standard_normal((cfg.ctx_len, cfg.ctx_dim)).astype(np.float32) if cfg.has_cross else None
    got = oracle.forward_one(m, x, t, ctx, dtype=np.float64)
    ref = _bf_forward(m, x, t, ctx)
    assert rel_l2(got, ref) < 1e-12


# --------------------------------------------------- special weights, closed forms

def test_zero_weights_give_constant_output_bias():
    cfg = W.get_config("tiny")
    tens = W.make_weights(cfg, init="zero")
    rng = np.random.default_rng(9)
    tens["b_f"] = rng.standard_normal(cfg.patch_dim).astype(np.float32)
    m = _model(cfg, tens)
    x = W.latents(cfg, 2)
    v = oracle.velocity(m, x, [0.9, 0.2])
    expect = oracle.unpatchify(np.tile(tens["b_f"], (cfg.N, 1)), cfg.C, cfg.H, cfg.W, cfg.p)
    np.testing.assert_array_equal(v[0], expect)
    np.testing.assert_array_equal(v[1], expect)


def test_zero_gates_make_blocks_identity():
    """gate1 = gate2 = 0 (chunks 2 and 5 of the block projection) turns every block
    into the identity, so the net equals the same net with no blocks."""
    cfg = W.get_config("tiny")
    tens = W.make_weights(cfg)
    D = cfg.D
    for l in range(cfg.L):
        tens[f"blk{l}.W_mod"][2 * D:3 * D] = 0; tens[f"blk{l}.b_mod"][2 * D:3 * D] = 0
        tens[f"blk{l}.W_mod"][5 * D:6 * D] = 0; tens[f"blk{l}.b_mod"][5 * D:6 * D] = 0
    m = _model(cfg, tens)
    m0 = _model(cfg, tens)
    m0.blocks, m0.L = [], 0
    x = W.latents(cfg, 1)[0]
    np.testing.assert_array_equal(oracle.forward_one(m, x, 0.6), oracle.forward_one(m0, x, 0.6))


def test_final_scale_minus_one_removes_input():
    """Final scale = -1 (second chunk) makes the head see only its shift, so v no
    longer depends on x: out = shift W_f^T + b_f for every token."""
    cfg = W.get_config("tiny")
    tens = W.make_weights(cfg)
    D = cfg.D
    tens["W_fmod"][D:] = 0
    tens["b_fmod"][D:] = -1.0
    m = _model(cfg, tens)
    xs = W.latents(cfg, 2)
    v0, v1 = oracle.forward_one(m, xs[0], 0.4, dtype=np.float64), oracle.forward_one(m, xs[1], 0.4, dtype=np.float64)
    s = oracle.dit.conditioning(m.astype(np.float64), 0.4, np.float64)
    shift = s @ m.top["W_fmod"][:D].astype(np.float64).T + m.top["b_fmod"][:D]
    tok = shift @ m.top["W_f"].astype(np.float64).T + m.top["b_f"]
    expect = oracle.unpatchify(np.tile(tok, (cfg.N, 1)), cfg.C, cfg.H, cfg.W, cfg.p)
    np.testing.assert_allclose(v0, expect, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(v1, expect, rtol=1e-12, atol=1e-14)


def test_block_scale1_minus_one_closed_form():
    """scale1 = -1 feeds every token the same attention input (shift1), so each query
    attends uniformly to identical values: the attention branch adds the constant
    gate1 * ((shift1 Wv^T + bv) Wo^T + bo). With gate2 = 0 and one block, the block
    output is h0 + that constant."""
    cfg = replace(W.get_config("tiny"), L=1)
    tens = W.make_weights(cfg)
    D = cfg.D
    tens["blk0.W_mod"][D:2 * D] = 0; tens["blk0.b_mod"][D:2 * D] = -1.0
    tens["blk0.W_mod"][5 * D:] = 0; tens["blk0.b_mod"][5 * D:] = 0
    m = _model(cfg, tens)
    x = W.latents(cfg, 1)[0].astype(np.float64)
    t = 0.3
    m64 = m.astype(np.float64)
    s = oracle.dit.conditioning(m64, t, np.float64)
    mod = s @ m64.blocks[0]["W_mod"].T + m64.blocks[0]["b_mod"]
    shift1, gate1 = mod[:D], mod[2 * D:3 * D]
    b = m64.blocks[0]
    vrow = shift1 @ b["W_qkv"][2 * D:].T + b["b_qkv"][2 * D:]
    const = gate1 * (vrow @ b["W_o"].T + b["b_o"])
    h0 = oracle.patchify(x, cfg.p) @ m64.top["W_pe"].T + m64.top["b_pe"] + m64.top["pos"]
    h1 = h0 + const
    fm = s @ m64.top["W_fmod"].T + m64.top["b_fmod"]
    out = (oracle.layer_norm(h1) * (1 + fm[D:]) + fm[:D]) @ m64.top["W_f"].T + m64.top["b_f"]
    expect = oracle.unpatchify(out, cfg.C, cfg.H, cfg.W, cfg.p)
    np.testing.assert_allclose(oracle.forward_one(m, x, t, dtype=np.float64), expect, rtol=1e-11, atol=1e-13)


def test_guidance_zero_and_one():
    cfg = W.get_config("tiny_cfg")
    m = _model(cfg, W.make_weights(cfg))
    x = W.latents(cfg, 2)
    ctx, nctx = W.context(cfg, 2), W.null_context(cfg)
    t = [0.8, 0.3]
    vu = np.stack([oracle.forward_one(m, x[k], t[k], nctx) for k in range(2)])
    vc = np.stack([oracle.forward_one(m, x[k], t[k], ctx[k]) for k in range(2)])
    np.testing.assert_array_equal(oracle.velocity(m, x, t, ctx, nctx, guidance=0.0), vu)
    np.testing.assert_allclose(oracle.velocity(m, x, t, ctx, nctx, guidance=1.0), vc, rtol=0, atol=1e-6)
    assert rel_l2(vc, vu) > 1e-3   # the context matters


# ------------------------------------------------------------------ precision check

@pytest.mark.parametrize("name", ["tiny", "tiny_tsens", "ragged", "dh72"])
def test_fp32_oracle_close_to_fp64(name):
    from conftest import oracle_model
    cfg = W.get_config(name)
    m = oracle_model(name)
    t, _ = W.slot_times(cfg)
    x = W.latents(cfg, cfg.K)
    assert rel_l2(oracle.velocity(m, x, t), oracle.velocity(m, x, t, dtype=np.float64)) < 1e-5
