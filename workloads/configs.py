"""Network and stream shapes of the synthetic workloads.

Each config names a DiT-style velocity network (latent C x H x W, patch p,
width D, depth L, heads, MLP width, sinusoidal timestep width tdim, optional
cross-attention context) and a stream: K queue slots, the timestep schedule the
slots sit on, and whether classifier-free guidance doubles the network rows.
"""
from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Config:
    name: str
    C: int
    H: int
    W: int
    p: int
    D: int
    L: int
    heads: int
    mlp: int
    tdim: int = 128
    ctx_len: int = 0
    ctx_dim: int = 0
    has_cross: int = 0
    K: int = 4                  # stream slots (logical samples in flight)
    schedule: str = "uniform4"  # "uniform<S>" (S equal steps) or "irregular8"
    cfg: bool = False           # cond/uncond row pairs (needs has_cross)
    guidance: float = 7.5
    init: str = "normal"        # "normal": every tensor N(0, 0.02); "tsens": see gen.py

    @property
    def N(self) -> int:
        """Tokens per sample."""
        return (self.H // self.p) * (self.W // self.p)

    @property
    def dh(self) -> int:
        return self.D // self.heads

    @property
    def patch_dim(self) -> int:
        return self.p * self.p * self.C

    @property
    def latent_shape(self):
        return (self.C, self.H, self.W)

    @property
    def rows(self) -> int:
        """Network rows per stream step (2K under guidance)."""
        return 2 * self.K if self.cfg else self.K

    def flops_per_step(self) -> float:
        """Algorithmic (unpadded) FLOPs of one velocity-network forward over all rows.

        GEMMs count 2*M*N*K, attention 4*N^2*D per sample and block (QK^T and PV).
        The timestep MLP, adaLN projection, patch embed and output head are included.
        """
        R, N, D, L, F = self.rows, self.N, self.D, self.L, self.mlp
        per_block = 2 * N * D * (3 * D) + 2 * N * D * D + 2 * 2 * N * D * F + 4 * N * N * D
        if self.has_cross:
            per_block += 2 * N * D * D * 2 + 2 * self.ctx_len * self.ctx_dim * 2 * D + 4 * N * self.ctx_len * D
        head = 2 * N * self.patch_dim * D * 2
        tmlp = 2 * (self.tdim * D + D * D) + 2 * D * (6 * D * L + 2 * D)
        return float(R * (L * per_block + head + tmlp))

    def gemm_flops_per_step(self) -> float:
        """FLOPs of the four dense velocity-network GEMMs (QKV, out-proj, fc1, fc2) per step."""
        R, N, D, L, F = self.rows, self.N, self.D, self.L, self.mlp
        return float(R * L * (2 * N * D * 3 * D + 2 * N * D * D + 4 * N * D * F))


_TINY = Config("tiny", C=4, H=16, W=16, p=2, D=128, L=2, heads=4, mlp=512)
_S512 = Config("s512", C=4, H=64, W=64, p=2, D=768, L=12, heads=12, mlp=3072)
_S512L = Config("s512_large", C=4, H=64, W=64, p=2, D=1152, L=28, heads=16, mlp=4608)

CONFIGS = {
    # 64 tokens, width 128, 2 blocks, 4 heads; K=4 at t = 1, .75, .5, .25
    "tiny": _TINY,
    # Tiny shapes with timestep-path weights drawn at 1/fan_in variance so v depends
    # strongly on t (a t-broadcast bug cannot hide below the bf16 tolerance)
    "tiny_tsens": replace(_TINY, name="tiny_tsens", init="tsens"),
    # Tiny with a 77-token cross-attention context and cond/uncond guidance rows
    "tiny_cfg": replace(_TINY, name="tiny_cfg", ctx_len=77, ctx_dim=64, has_cross=1, cfg=True),
    # ragged shapes: 140 tokens, width 192 (head dim 48), 3 slots
    "ragged": Config("ragged", C=4, H=20, W=28, p=2, D=192, L=2, heads=4, mlp=768, K=3, schedule="uniform3"),
    # head dim 72 (as in the width-1152 nets) at a small size
    "dh72": Config("dh72", C=4, H=16, W=24, p=2, D=144, L=2, heads=2, mlp=576),
    # head dim 64 (as in the width-768 nets) with a ragged token count: 300 tokens are
    # five 64-key attention steps, the last holding 44 keys
    "dh64": Config("dh64", C=4, H=20, W=60, p=2, D=128, L=2, heads=2, mlp=512),
    # at most 32 tokens (or context tokens): a whole attention key half of 32 lies past
    # the last key. 16 tokens at head dims 32 and 72, 32 tokens at head dim 64, and the
    # Tiny guided network with contexts of 20 and 32 tokens
    "short16": Config("short16", C=4, H=8, W=8, p=2, D=128, L=2, heads=4, mlp=512),
    "short16_dh72": Config("short16_dh72", C=4, H=8, W=8, p=2, D=144, L=2, heads=2, mlp=576),
    "short32_dh64": Config("short32_dh64", C=4, H=8, W=16, p=2, D=128, L=2, heads=2, mlp=512),
    "tiny_cfg_ctx20": replace(_TINY, name="tiny_cfg_ctx20", ctx_len=20, ctx_dim=64, has_cross=1, cfg=True),
    "tiny_cfg_ctx32": replace(_TINY, name="tiny_cfg_ctx32", ctx_len=32, ctx_dim=64, has_cross=1, cfg=True),
    # 512^2 image: 4x64x64 latent, 1024 tokens, width 768, 12 blocks, 12 heads
    "s512": _S512,
    # 512^2, width 1152, 28 blocks, 16 heads; every slot at a different step
    "s512_large": _S512L,
    # 512^2 text-conditioned: cross-attention to 77x1024 context, 8-step irregular
    # schedule, 8 slots doubled to 16 cond/uncond rows
    "s512_cfg": replace(_S512, name="s512_cfg", ctx_len=77, ctx_dim=1024, has_cross=1, K=8,
                        schedule="irregular8", cfg=True),
    # 1024^2: 4x128x128 latent, 4096 tokens, width 1152, 28 blocks
    "s1024": replace(_S512L, name="s1024", H=128, W=128),
}


def get_config(name: str) -> Config:
    try:
        return CONFIGS[name]
    except KeyError:
        raise KeyError(f"unknown config {name!r}; known: {sorted(CONFIGS)}") from None
