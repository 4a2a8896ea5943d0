"""Weight-blob file format (writer side).

Little-endian. A 64-byte header, then fp32 tensors back to back in a fixed order:

    magic 'SFW1' | u32 version=1 | u32 C,H,W,p,D,L,heads,mlp,tdim,ctx_len,ctx_dim,has_cross | u64 seed

    patch embed  W_pe[D, p*p*C], b_pe[D];   pos[N, D]
    timestep MLP W_t1[D, tdim], b_t1[D], W_t2[D, D], b_t2[D]
    per block    W_mod[6D, D], b_mod[6D], W_qkv[3D, D], b_qkv[3D], W_o[D, D], b_o[D],
                 (cross) W_qx[D, D], b_qx[D], W_kvx[2D, ctx_dim], b_kvx[2D], W_ox[D, D], b_ox[D],
                 W_fc1[mlp, D], b_fc1[mlp], W_fc2[D, mlp], b_fc2[D]
    final        W_fmod[2D, D], b_fmod[2D], W_f[p*p*C, D], b_f[p*p*C]

Linear weights are stored [out, in]. The oracle and the HIP library each parse
this layout with their own reader; the format is the only thing they share.
"""
import struct

import numpy as np

MAGIC = b"SFW1"
VERSION = 1
HEADER_FMT = "<4sI12IQ"
HEADER_SIZE = struct.calcsize(HEADER_FMT)
assert HEADER_SIZE == 64


def tensor_specs(cfg):
    """Ordered (name, shape) list of every tensor in a blob for `cfg`."""
    D, P, F = cfg.D, cfg.patch_dim, cfg.mlp
    specs = [("W_pe", (D, P)), ("b_pe", (D,)), ("pos", (cfg.N, D)),
             ("W_t1", (D, cfg.tdim)), ("b_t1", (D,)), ("W_t2", (D, D)), ("b_t2", (D,))]
    for l in range(cfg.L):
        specs += [(f"blk{l}.W_mod", (6 * D, D)), (f"blk{l}.b_mod", (6 * D,)),
                  (f"blk{l}.W_qkv", (3 * D, D)), (f"blk{l}.b_qkv", (3 * D,)),
                  (f"blk{l}.W_o", (D, D)), (f"blk{l}.b_o", (D,))]
        if cfg.has_cross:
            specs += [(f"blk{l}.W_qx", (D, D)), (f"blk{l}.b_qx", (D,)),
                      (f"blk{l}.W_kvx", (2 * D, cfg.ctx_dim)), (f"blk{l}.b_kvx", (2 * D,)),
                      (f"blk{l}.W_ox", (D, D)), (f"blk{l}.b_ox", (D,))]
        specs += [(f"blk{l}.W_fc1", (F, D)), (f"blk{l}.b_fc1", (F,)),
                  (f"blk{l}.W_fc2", (D, F)), (f"blk{l}.b_fc2", (D,))]
    specs += [("W_fmod", (2 * D, D)), ("b_fmod", (2 * D,)), ("W_f", (P, D)), ("b_f", (P,))]
    return specs


def header_fields(cfg):
    return (cfg.C, cfg.H, cfg.W, cfg.p, cfg.D, cfg.L, cfg.heads, cfg.mlp, cfg.tdim,
            cfg.ctx_len, cfg.ctx_dim, cfg.has_cross)


def write_blob(cfg, tensors, seed=0):
    """Serialise `tensors` (name -> array) for `cfg` into blob bytes."""
    parts = [struct.pack(HEADER_FMT, MAGIC, VERSION, *header_fields(cfg), seed)]
    for name, shape in tensor_specs(cfg):
        a = np.ascontiguousarray(tensors[name], dtype="<f4")
        if a.shape != tuple(shape):
            raise ValueError(f"{name}: shape {a.shape}, expected {shape}")
        parts.append(a.tobytes())
    return b"".join(parts)
