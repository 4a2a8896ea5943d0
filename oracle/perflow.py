"""Oracle: PeRFlow's time-window conversion of a noise prediction into a velocity,
batched over heterogeneous timesteps, and the update it drives.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Follows the paper's time-window mechanism (Sec. 2, the gamma / lambda / eta equations),
the vectorized window lookup and batch parameters of Sec. 3.3 (batch velocity
parameter equation), and the batched velocity-field step (Alg. 1), in that order.

Readings (the paper leaves these open):
  * time is normalised to [0, 1] with 1 = noise (Alg. 1 divides timesteps by T_max; the
    library takes normalised t), and dt = t_next - t is negative;
  * K_w windows of equal length: window k (1-based) starts at t^s = k / K_w (its noisy
    end) and ends at t^e = (k - 1) / K_w, so the window ends in ascending order are
    (k - 1) / K_w and the lookup's mask sum gives k directly;
  * the noise schedule behind alphas_cumprod is the scaled-linear one of the latent
    diffusion models PeRFlow starts from: beta_i on a linear grid in sqrt(beta) from
    sqrt(beta_start) to sqrt(beta_end), i = 0 .. T-1, T = 1000, beta_start = 0.00085,
    beta_end = 0.012; alphas_cumprod[i] = prod_{j <= i} (1 - beta_j); a normalised time
    u reads index round(u (T - 1)) (ties to even);
  * the lookup tolerance epsilon is 1e-6;
  * all arithmetic in float64 from the float32 inputs, the new latents rounded once to
    float32.
Parity: pinned by the tests in test_oracle_perflow.py (brute-force lookup and
schedule, the lambda_s^2 - eta_s^2 = 1 identity, window-start and window-end limits,
the window-endpoint property of a step that ends on t^e).
"""
import numpy as np

from .dit import velocity

DEFAULT_T = 1000
DEFAULT_BETA_START = 0.00085
DEFAULT_BETA_END = 0.012
DEFAULT_EPS = 1e-6


def alphas_cumprod(T=DEFAULT_T, beta_start=DEFAULT_BETA_START, beta_end=DEFAULT_BETA_END):
    """Cumulative products of (1 - beta) for the scaled-linear beta schedule."""
    betas = np.linspace(np.sqrt(beta_start), np.sqrt(beta_end), T, dtype=np.float64) ** 2
    return np.cumprod(1.0 - betas)


def window_lookup(t, K_w, eps=DEFAULT_EPS):
    """Sec. 3.3: mask M_k = (t > t_k^e + eps) over the K_w window ends, k = sum_k M_k.
    Returns the 1-based window index of every timestep (at least 1)."""
    t = np.asarray(t, dtype=np.float64)
    ends = np.arange(K_w, dtype=np.float64) / K_w
    k = (t[:, None] > ends[None, :] + eps).sum(axis=1)
    return np.maximum(k, 1)


def alpha_at(abar, u):
    """alphas_cumprod read at normalised time u (index round(u (T - 1)))."""
    idx = np.rint(np.asarray(u, dtype=np.float64) * (len(abar) - 1)).astype(np.int64)
    return abar[idx]


def batch_params(t, K_w, abar, eps=DEFAULT_EPS):
    """Window bounds and the batch velocity parameters for timesteps t [B]:
    gamma = (abar(t^s) / abar(t^e))^(1/2), lambda_s = 1 / gamma,
    eta_s = -(1 - gamma^2)^(1/2) / gamma, denom = lambda_s (t - t^s) + (t^e - t),
    lambda_t = lambda_s (t^e - t^s) / denom, eta_t = eta_s (t^e - t) / denom."""
    t = np.asarray(t, dtype=np.float64)
    k = window_lookup(t, K_w, eps)
    ts = k / K_w
    te = (k - 1) / K_w
    gamma = np.sqrt(alpha_at(abar, ts) / alpha_at(abar, te))
    lam_s = 1.0 / gamma
    eta_s = -np.sqrt(1.0 - gamma ** 2) / gamma
    denom = lam_s * (t - ts) + (te - t)
    lam_t = lam_s * (te - ts) / denom
    eta_t = eta_s * (te - t) / denom
    return {"k": k, "ts": ts, "te": te, "gamma": gamma, "lam_s": lam_s, "eta_s": eta_s,
            "lam_t": lam_t, "eta_t": eta_t}


def batched_velocity_step(eps_pred, X, t, dt, K_w, abar, eps=DEFAULT_EPS):
    """Alg. 1 on normalised times: window parameters, X_pred = lambda_t X + eta_t eps,
    v = (X_pred - X) / (t^e - t), X_next = X + dt v. Returns (X_next fp32, v fp32)."""
    p = batch_params(t, K_w, abar, eps)
    shape = (-1,) + (1,) * (np.ndim(X) - 1)
    X64 = np.asarray(X, dtype=np.float64)
    E64 = np.asarray(eps_pred, dtype=np.float64)
    lam_t = p["lam_t"].reshape(shape)
    eta_t = p["eta_t"].reshape(shape)
    te_minus_t = (p["te"] - np.asarray(t, dtype=np.float64)).reshape(shape)
    x_pred = lam_t * X64 + eta_t * E64
    v = (x_pred - X64) / te_minus_t
    x_next = X64 + np.asarray(dt, dtype=np.float64).reshape(shape) * v
    return x_next.astype(np.float32), v.astype(np.float32)


def stream_step(m, x, t, dt, z_new, K_w, abar, eps=DEFAULT_EPS, steady=True, ctx=None, null_ctx=None,
                guidance=None, dtype=np.float32):
    """One stream step where the network output is read as the noise prediction and the
    update is Alg. 1's window conversion; the queue shift is that of Alg. 2 (see
    stream.stream_step). Returns (x_next, done or None, network output)."""
    e = velocity(m, x, t, ctx, null_ctx, guidance, dtype)
    xp, _ = batched_velocity_step(e, x, t, dt, K_w, abar, eps)
    z = np.asarray(z_new, dtype=np.float32)[None]
    if steady:
        return np.concatenate([z, xp[:-1]]), xp[-1].copy(), e
    return np.concatenate([z, xp]), None, e
