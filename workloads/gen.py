"""Seeded generators: weights, latents, contexts and timestep schedules.

All draws use numpy's PCG64. Weight tensor i (in blob order) comes from its own
stream `default_rng([seed, i])`, drawn directly in fp32 and scaled in fp32, so the
tensors of a multi-GB blob are generated in parallel threads. Latents and contexts
are float64 normals cast to fp32. Seeds: 0 weights, 1 initial slot latents, 100+m
the fresh noise of image m, 2 the conditioning context, 3 the unconditional context,
4 the irregular schedule.
"""
import os
import struct
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .blob import HEADER_FMT, MAGIC, VERSION, header_fields, tensor_specs, write_blob

SEED_WEIGHTS = 0
SEED_LATENTS = 1
SEED_CONTEXT = 2
SEED_NULL_CONTEXT = 3
SEED_SCHEDULE = 4
SEED_IMAGE_BASE = 100


def _pos_table(cfg):
    """Fixed 2-D sin-cos position table [N, D] (half the width encodes the patch row,
    half the column; each half is [sin, cos] over D/4 geometric frequencies)."""
    gh, gw = cfg.H // cfg.p, cfg.W // cfg.p
    quarter = cfg.D // 4
    omega = 1.0 / 10000.0 ** (np.arange(quarter, dtype=np.float64) / quarter)
    rows = np.repeat(np.arange(gh, dtype=np.float64), gw)
    cols = np.tile(np.arange(gw, dtype=np.float64), gh)
    pe = np.zeros((gh * gw, cfg.D), dtype=np.float64)
    pe[:, 0 * quarter:1 * quarter] = np.sin(rows[:, None] * omega)
    pe[:, 1 * quarter:2 * quarter] = np.cos(rows[:, None] * omega)
    pe[:, 2 * quarter:3 * quarter] = np.sin(cols[:, None] * omega)
    pe[:, 3 * quarter:4 * quarter] = np.cos(cols[:, None] * omega)
    return pe.astype(np.float32)


def _std(cfg, name, shape, init):
    if init == "tsens" and name.split(".")[-1] in ("W_t1", "W_t2", "W_mod", "W_fmod"):
        return 1.0 / np.sqrt(shape[1])
    return 0.02


def _fill(cfg, specs, outs, seed, init):
    """Writes tensor i of `specs` into outs[i] (an fp32 array of its shape)."""
    def one(i):
        name, shape = specs[i]
        a = outs[i]
        if name == "pos":
            a[...] = _pos_table(cfg) if init != "zero" else 0.0
        elif init == "zero":
            a[...] = 0.0
        else:
            np.random.default_rng([seed, i]).standard_normal(out=a, dtype=np.float32)
            a *= np.float32(_std(cfg, name, shape, init))
    order = sorted(range(len(specs)), key=lambda i: -int(np.prod(specs[i][1])))
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        list(ex.map(one, order))


def make_weights(cfg, seed=SEED_WEIGHTS, init=None):
    """Random-init weights for `cfg` as a dict name -> fp32 array.

    init "normal": every tensor (weights and biases) N(0, 0.02) except the fixed
    sin-cos position table. init "tsens": as "normal", but the timestep MLP and
    every adaLN projection are drawn N(0, 1/fan_in), so v depends strongly on t.
    init "zero": all zeros (callers then set the tensors they want).
    """
    init = init or cfg.init
    specs = tensor_specs(cfg)
    outs = [np.empty(shape, np.float32) for _, shape in specs]
    _fill(cfg, specs, outs, seed, init)
    return {name: a for (name, _), a in zip(specs, outs)}


def make_blob(cfg, seed=SEED_WEIGHTS, init=None, tensors=None):
    """Blob for `cfg` (seeded weights unless `tensors` is given). The seeded blob is
    generated in place and returned as a uint8 numpy array (no copy of a multi-GB
    buffer); its bytes equal write_blob(cfg, make_weights(cfg, ...))."""
    if tensors is not None:
        return write_blob(cfg, tensors, seed=seed)
    init = init or cfg.init
    specs = tensor_specs(cfg)
    head = struct.pack(HEADER_FMT, MAGIC, VERSION, *header_fields(cfg), seed)
    total = len(head) + 4 * sum(int(np.prod(shape)) for _, shape in specs)
    buf = np.empty(total, np.uint8)  # pages are first touched by the fill threads
    buf[:len(head)] = np.frombuffer(head, np.uint8)
    outs, off = [], len(head)
    for _, shape in specs:
        n = int(np.prod(shape))
        outs.append(np.frombuffer(buf, dtype="<f4", count=n, offset=off).reshape(shape))
        off += 4 * n
    _fill(cfg, specs, outs, seed, init)
    del outs
    return buf


def latents(cfg, n, seed=SEED_LATENTS):
    """n latents [n, C, H, W] fp32 ~ N(0, 1)."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal((n,) + cfg.latent_shape).astype(np.float32)


def z_new_for_image(cfg, m):
    """The fresh noise latent [C, H, W] of image m (seed 100 + m)."""
    return latents(cfg, 1, seed=SEED_IMAGE_BASE + m)[0]


def context(cfg, n, seed=SEED_CONTEXT):
    """Conditioning contexts [n, ctx_len, ctx_dim] fp32 ~ N(0, 1)."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal((n, cfg.ctx_len, cfg.ctx_dim)).astype(np.float32)


def null_context(cfg, seed=SEED_NULL_CONTEXT):
    """The unconditional context [ctx_len, ctx_dim] shared by every uncond row."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal((cfg.ctx_len, cfg.ctx_dim)).astype(np.float32)


def schedule(cfg, seed=SEED_SCHEDULE):
    """Descending fp32 time grid t_0 = 1 > t_1 > ... > t_S = 0 with S = number of steps.

    "uniform<S>": S equal steps. "irregular8": t_1..t_7 are seven seeded U(0,1)
    draws sorted descending.
    """
    if cfg.schedule.startswith("uniform"):
        g = np.linspace(1.0, 0.0, int(cfg.schedule[len("uniform"):]) + 1)
    elif cfg.schedule == "irregular8":
        rng = np.random.default_rng(seed)
        mid = np.sort(rng.uniform(0.0, 1.0, 7))[::-1]
        g = np.concatenate([[1.0], mid, [0.0]])
    else:
        raise ValueError(cfg.schedule)
    return g.astype(np.float32)


def slot_times(cfg, seed=SEED_SCHEDULE):
    """Per-slot (t[K], dt[K]) in the full-queue steady state: slot k sits at step k.

    dt_k = fp32(t_{k+1}) - fp32(t_k), negative (t runs from noise at 1 to data at 0).
    """
    g = schedule(cfg, seed)
    if len(g) - 1 != cfg.K:
        raise ValueError(f"{cfg.name}: schedule has {len(g) - 1} steps, stream has {cfg.K} slots")
    t = g[:-1].copy()
    dt = (g[1:] - g[:-1]).astype(np.float32)
    return t, dt
