"""Oracle stream step: per-sample Euler update, queue shift, and the Alg. 2 driver.

Queue order follows Alg. 2: slot 0 holds the newest latent (largest t) and the last
slot the oldest; a step appends fresh noise at the front and, once the pipeline is
full, the last slot leaves as a finished sample (Sec. 3.4.1-3.4.2).
"""
import numpy as np

from .dit import velocity, forward_one


def euler(x, v, dt):
    """x'_k = x_k + dt_k * v_k for every slot k (Sec. 3.1.1 discretization; Alg. 1's
    final update). fp32 multiply, then fp32 add. dt is signed (negative when t
    runs from noise at 1 to data at 0)."""
    x = np.asarray(x)
    dt = np.asarray(dt, dtype=x.dtype).reshape((-1,) + (1,) * (x.ndim - 1))
    return x + dt * v


def stream_step(m, x, t, dt, z_new, steady=True, ctx=None, null_ctx=None, guidance=None,
                dtype=np.float32):
    """One stream step over the B slots in x [B, C, H, W] at times t [B].

    v = velocity(x, t); x'_k = x_k + dt_k v_k. Steady (full pipeline): the oldest
    slot leaves as `done`, the rest move one slot on and z_new enters slot 0, so the
    queue keeps B slots. Fill (steady=False): nothing leaves, the queue grows to B+1.
    Returns (x_next, done or None, v).
    """
    v = velocity(m, x, t, ctx, null_ctx, guidance, dtype)
    xp = euler(np.asarray(x, dtype=dtype), v, dt)
    z = np.asarray(z_new, dtype=dtype)[None]
    if steady:
        return np.concatenate([z, xp[:-1]]), xp[-1].copy(), v
    return np.concatenate([z, xp]), None, v


def run_stream(m, grid, M, noise, ctx_of=None, null_ctx=None, guidance=None, dtype=np.float32):
    """Alg. 2 over M images on the descending time grid t_0 > ... > t_S (S steps).

    Iteration j = 1 .. M+S-1 draws fresh noise for image j (`noise(j)`), forms
    P = [z_new, buffer], runs one heterogeneous-t network call on P at t[0:|P|],
    takes each sample's Euler step with dt_i = t_{i+1} - t_i, and once |P| = S emits
    the last slot as image j-S+1. `ctx_of(j)` gives image j's context when the
    network is conditioned. Returns the M finished latents in image order.
    """
    grid = np.asarray(grid, dtype=np.float32)
    S = len(grid) - 1
    dts = (grid[1:] - grid[:-1]).astype(np.float32)
    buf, ids, images = [], [], []
    for j in range(1, M + S):
        P = [np.asarray(noise(j), dtype=dtype)] + buf
        pid = [j] + ids
        n = len(P)
        ctx = None if ctx_of is None else np.stack([ctx_of(i) for i in pid])
        v = velocity(m, np.stack(P), grid[:n], ctx, null_ctx, guidance, dtype)
        Pp = euler(np.stack(P), v, dts[:n])
        if n == S:
            images.append(Pp[-1].copy())
            buf, ids = list(Pp[:-1]), pid[:-1]
        else:
            buf, ids = list(Pp), pid
    return images[:M]


def noise_latent(x_ref, z, t0):
    """The point of the straight path between a reference latent and noise at time t0
    (Sec. 2: x_t on the line from data to noise; here t = 1 is noise):
    x = (1 - t0) x_ref + t0 z, each product and the sum rounded to fp32. With a schedule
    that starts at t0 < 1, this is the latent an image-to-image run admits (the paper's
    img2img workload); t0 = 1 gives z itself."""
    t0 = np.float32(t0)
    a = np.float32(1.0) - t0
    return (a * np.asarray(x_ref, dtype=np.float32) + t0 * np.asarray(z, dtype=np.float32)).astype(np.float32)


def sequential_sample(m, z, grid, ctx=None, null_ctx=None, guidance=None, dtype=np.float32):
    """One image alone: x <- x + dt_i F(x, t_i) over the grid, from noise z."""
    grid = np.asarray(grid, dtype=np.float32)
    x = np.asarray(z, dtype=dtype)
    for i in range(len(grid) - 1):
        ck = None if ctx is None else ctx[None]
        v = velocity(m, x[None], grid[i:i + 1], ck, null_ctx, guidance, dtype)[0]
        x = euler(x[None], v[None], (grid[i + 1] - grid[i]).astype(np.float32)[None])[0]
    return x
