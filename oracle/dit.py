"""Oracle velocity network: a DiT-style adaLN transformer F(x, t) that outputs v.

The paper (Sec. 3.2, Eq. 5) runs ONE network call over latents that each carry
their own timestep; what makes that call correct is that every sample's output
is exactly what the network gives for that sample alone at its own t. This module
therefore computes the forward one sample at a time (`forward_one`) and
`velocity` is a plain loop over samples, so the batched result equals the
per-sample result by construction.

Readings of details the paper leaves open (the paper's own network is a
noise-predicting UNet it does not describe):
  * the network sees tau = 1000 * t: Alg. 1 divides the scheduler's timesteps by a
    maximum of T_max before using them, i.e. the network's own time runs over
    [0, T_max]; T_max = 1000 here;
  * sinusoidal embedding of width tdim: frequencies f_i = 10000^(-i/half), i < half,
    evaluated in fp64 and rounded once to fp32; phases phi_i = fp32(tau * f_i);
    e = [cos(phi_0..), sin(phi_0..)]; tau and phi keep this fp32 rounding in every
    precision mode because they define the network's input;
  * timestep MLP c = W_t2 SiLU(W_t1 e + b_t1) + b_t2; every adaLN projection reads
    SiLU(c); a block's projection splits into shift1, scale1, gate1, shift2,
    scale2, gate2 (in that order, each width D); the final layer's into shift, scale;
  * LayerNorm over the width: biased variance, eps 1e-6, no affine parameters;
  * modulate(z) = LN(z) * (1 + scale) + shift;
  * block: h += gate1 * SelfAttn(modulate1(h)); [cross: h += CrossAttn(LN(h), ctx)];
           h += gate2 * MLP(modulate2(h)); MLP = fc2(GELU_tanh(fc1(.)));
  * attention: q, k, v are column thirds of one projection; head j takes columns
    j*dh..(j+1)*dh-1 of each; softmax(q k^T / sqrt(dh)) with max subtraction; no mask;
  * patchify: token n = gh*(W/p) + gw holds feature (i*p + j)*C + c from
    x[c, gh*p + i, gw*p + j]; unpatchify is its inverse;
  * guidance (rows = cond rows then uncond rows, same t): v = v_u + w (v_c - v_u).
"""
import math

import numpy as np

LN_EPS = 1e-6
T_MAX = 1000.0
MAX_PERIOD = 10000.0


def timestep_frequencies(tdim):
    """f_i = 10000^(-i/half) for i < half, computed in fp64 and rounded once to fp32."""
    half = tdim // 2
    i = np.arange(half, dtype=np.float64)
    return np.exp(-math.log(MAX_PERIOD) * i / half).astype(np.float32)


def timestep_embedding(t, tdim, dtype=np.float32):
    """Sinusoidal embedding [tdim] of one scalar time t in [0, 1] (network time 1000 t).

    Parity: pinned in tests (tau = 0 gives [1..1, 0..0]; frequency 0 is 1 so entries
    0 and half are cos(tau), sin(tau); f at i = half/2 is 10000^-0.5 = 0.01).
    """
    tau = np.float32(T_MAX) * np.float32(t)                      # fp32 product
    phi = (tau * timestep_frequencies(tdim)).astype(np.float32)  # fp32 products
    phi64 = phi.astype(np.float64)
    return np.concatenate([np.cos(phi64), np.sin(phi64)]).astype(dtype)


def silu(z):
    """SiLU(z) = z * sigmoid(z)."""
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def gelu_tanh(z):
    """tanh-approximate GELU: 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3)))."""
    return 0.5 * z * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (z + 0.044715 * z * z * z)))


def linear(x, W, b):
    """x W^T + b with W stored [out, in]."""
    return x @ W.T + b


def layer_norm(z):
    """(z - mean) / sqrt(var + eps) over the last axis; biased variance, no affine."""
    mu = z.mean(axis=-1, keepdims=True)
    d = z - mu
    var = (d * d).mean(axis=-1, keepdims=True)
    return d / np.sqrt(var + LN_EPS)


def patchify(x, p):
    """[C, H, W] -> tokens [N, p*p*C]; token gh*(W/p)+gw, feature (i*p+j)*C+c."""
    C, H, W = x.shape
    t = x.reshape(C, H // p, p, W // p, p).transpose(1, 3, 2, 4, 0)
    return t.reshape((H // p) * (W // p), p * p * C)


def unpatchify(tok, C, H, W, p):
    """Inverse of `patchify`: tokens [N, p*p*C] -> [C, H, W]."""
    t = tok.reshape(H // p, W // p, p, p, C).transpose(4, 0, 2, 1, 3)
    return t.reshape(C, H, W)


def attention(q, k, v, heads):
    """Multi-head softmax attention, no mask. q [Nq, D], k and v [Nk, D] -> [Nq, D]."""
    D = q.shape[1]
    dh = D // heads
    scale = 1.0 / math.sqrt(dh)
    out = np.empty_like(q)
    for j in range(heads):
        sl = slice(j * dh, (j + 1) * dh)
        s = (q[:, sl] @ k[:, sl].T) * scale
        s = s - s.max(axis=1, keepdims=True)
        w = np.exp(s)
        w = w / w.sum(axis=1, keepdims=True)
        out[:, sl] = w @ v[:, sl]
    return out


def conditioning(m, t, dtype=np.float32):
    """SiLU(c) [D] for one sample: the vector every adaLN projection reads."""
    e = timestep_embedding(t, m.tdim, dtype)
    hid = silu(linear(e, m.top["W_t1"], m.top["b_t1"]))
    c = linear(hid, m.top["W_t2"], m.top["b_t2"])
    return silu(c)


def modulation_table(m, t, dtype=np.float32):
    """Per-sample adaLN table [L*6D + 2D]: for each block (shift1, scale1, gate1,
    shift2, scale2, gate2), then the final (shift, scale)."""
    s = conditioning(m, t, dtype)
    parts = [linear(s, b["W_mod"], b["b_mod"]) for b in m.blocks]
    parts.append(linear(s, m.top["W_fmod"], m.top["b_fmod"]))
    return np.concatenate(parts)


def block_forward(m, b, h, s, ctx=None, trace=None):
    """One adaLN block on the residual stream h [N, D] of one sample (s = SiLU(c)).
    If `trace` is a dict, the block's intermediates are stored in it."""
    D = m.D
    mod = linear(s, b["W_mod"], b["b_mod"]).reshape(6, D)
    shift1, scale1, gate1, shift2, scale2, gate2 = mod
    a = layer_norm(h) * (1.0 + scale1) + shift1
    qkv = linear(a, b["W_qkv"], b["b_qkv"])
    q, k, v = qkv[:, :D], qkv[:, D:2 * D], qkv[:, 2 * D:]
    o = attention(q, k, v, m.heads)
    h = h + gate1 * linear(o, b["W_o"], b["b_o"])
    if trace is not None:
        trace.update(ln1=a, q=q, k=k, v=v, attn=o, h_attn=h)
    if m.has_cross:
        if ctx is None:
            raise ValueError("network has cross-attention: ctx is required")
        qx = linear(layer_norm(h), b["W_qx"], b["b_qx"])
        kv = linear(np.asarray(ctx, dtype=h.dtype), b["W_kvx"], b["b_kvx"])
        ox = attention(qx, kv[:, :D], kv[:, D:], m.heads)
        h = h + linear(ox, b["W_ox"], b["b_ox"])
        if trace is not None:
            trace.update(cross_q=qx, cross_attn=ox, h_cross=h)
    a = layer_norm(h) * (1.0 + scale2) + shift2
    f = gelu_tanh(linear(a, b["W_fc1"], b["b_fc1"]))
    h = h + gate2 * linear(f, b["W_fc2"], b["b_fc2"])
    if trace is not None:
        trace.update(ln2=a, mlp=f, h_out=h)
    return h


def residual_one(m, x, t, ctx=None, blocks=None, dtype=np.float32, trace=None):
    """Residual stream h [N, D] of ONE latent after the patch embedding and the first
    `blocks` blocks (all blocks if None); `s` = SiLU(c) is returned alongside. With a
    `trace` dict, the intermediates of the last block run are stored in it."""
    m = m if dtype == np.float32 else m.astype(dtype)
    x = np.asarray(x, dtype=dtype)
    s = conditioning(m, t, dtype)
    h = linear(patchify(x, m.p), m.top["W_pe"], m.top["b_pe"]) + m.top["pos"]
    for b in m.blocks[:blocks]:
        h = block_forward(m, b, h, s, ctx, trace)
    return h, s


def forward_one(m, x, t, ctx=None, dtype=np.float32):
    """v = F(x, t) for ONE latent x [C, H, W] at time t; ctx [ctx_len, ctx_dim] if the
    network has cross-attention. Returns v [C, H, W] in `dtype`."""
    m = m if dtype == np.float32 else m.astype(dtype)
    h, s = residual_one(m, x, t, ctx, None, dtype)
    shift, scale = linear(s, m.top["W_fmod"], m.top["b_fmod"]).reshape(2, m.D)
    out = linear(layer_norm(h) * (1.0 + scale) + shift, m.top["W_f"], m.top["b_f"])
    return unpatchify(out, m.C, m.H, m.W, m.p)


def velocity(m, x, t, ctx=None, null_ctx=None, guidance=None, dtype=np.float32):
    """Heterogeneous-t batch call (Eq. 5): v[k] = F(x[k], t[k]) for every slot k.

    x [B, C, H, W], t [B]. Without guidance, ctx (if the net has cross-attention) is
    [B, ctx_len, ctx_dim]. With guidance w, each slot is run twice, once with its own
    ctx and once with the shared null_ctx, and v = v_u + w (v_c - v_u).
    """
    B = x.shape[0]
    out = np.empty(x.shape, dtype=dtype)
    for k in range(B):
        ck = None if ctx is None else ctx[k]
        vc = forward_one(m, x[k], t[k], ck, dtype)
        if guidance is None:
            out[k] = vc
        else:
            vu = forward_one(m, x[k], t[k], null_ctx, dtype)
            out[k] = vu + dtype(guidance) * (vc - vu)
    return out
