"""Alg. 2 (pipeline batch denoising) driven through the C ABI.

The queue lives in one device buffer of K+1 latent slots, newest first. Every call to
`step` runs one sf_stream_step: one heterogeneous-t network call over the occupied
slots, each slot's Euler step, and the shift that admits the next fresh latent at
slot 0. While the queue is filling (fewer than K slots) nothing leaves; once it is
full, every step emits one finished latent (Sec. 3.4.1-3.4.2). The host only keeps
the schedule and the occupancy; all arithmetic runs in the library's kernels.
"""
import numpy as np


class StreamQueue:
    def __init__(self, model, grid, first_latent, contexts=None, null_ctx=None, guidance=None):
        """grid: descending times t_0 > ... > t_K (K steps). first_latent: device
        [C,H,W] fp32, the noise of image 1. contexts: optional device
        [K+1, ctx_len, ctx_dim] buffer whose slot 0 holds image 1's context."""
        import torch
        self.model = model
        self.grid = np.asarray(grid, dtype=np.float32)
        self.K = len(self.grid) - 1
        self.t = self.grid[:-1].copy()
        self.dt = (self.grid[1:] - self.grid[:-1]).astype(np.float32)
        shape = tuple(first_latent.shape)
        self.x = torch.empty((self.K + 1,) + shape, dtype=torch.float32, device=first_latent.device)
        self.x[0].copy_(first_latent)
        self.n = 1
        self.contexts, self.null_ctx, self.guidance = contexts, null_ctx, guidance

    def _cond(self):
        if self.contexts is None:
            return None
        from .binding import Cond
        return Cond(self.contexts, self.null_ctx, self.guidance if self.guidance is not None else 0.0)

    def step(self, z_next, done_out=None, ctx_next=None):
        """Advance every occupied slot one step and admit z_next (device [C,H,W]).
        Returns done_out (filled with the finished latent) once the queue is full,
        else None. ctx_next is the admitted image's context when conditioned."""
        n = self.n
        full = n == self.K
        cond = self._cond()
        if full:
            if done_out is None:
                import torch
                done_out = torch.empty_like(z_next)
            self.model.stream_step(self.x, self.t[:n], self.dt[:n], n, z_next, done_out, cond)
        else:
            self.model.stream_step(self.x, self.t[:n], self.dt[:n], n, z_next, None, cond)
            self.n = n + 1
            done_out = None
        if self.contexts is not None:
            # contexts move with their latents: slot k -> k+1 (the last one leaves when
            # full), the admitted image's context enters slot 0
            kept = n - 1 if full else n
            self.contexts[1:kept + 1].copy_(self.contexts[0:kept].clone())
            self.contexts[0].copy_(ctx_next)
        return done_out


def run_images(model, grid, M, noise, contexts_of=None, null_ctx=None, guidance=None, references=None):
    """Generate M latents with Alg. 2: M + K - 1 stream steps. noise(j) gives image j's
    noise as a device tensor; contexts_of(j) its context when conditioned. With
    references(j) (image-to-image), image j enters as the straight-path point between its
    reference and its noise at grid[0] (sf_noise_latent); the grid then starts at t0 < 1."""
    import torch
    K = len(grid) - 1
    if references is not None:
        raw, t0 = noise, float(grid[0])
        noise = lambda j: model.noise_latent(references(j), raw(j), t0)  # noqa: E731
    ctx_buf = None
    if contexts_of is not None:
        c1 = contexts_of(1)
        ctx_buf = torch.empty((K + 1,) + tuple(c1.shape), dtype=torch.float32, device=c1.device)
        ctx_buf[0].copy_(c1)
    q = StreamQueue(model, grid, noise(1), ctx_buf, null_ctx, guidance)
    out = []
    for j in range(1, M + K):
        ctx_next = contexts_of(j + 1) if contexts_of is not None else None
        done = q.step(noise(j + 1), ctx_next=ctx_next)
        if done is not None:
            out.append(done)
    return out[:M]
