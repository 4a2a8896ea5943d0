"""Oracle-side reader of the weight blob (independent of the library's C++ reader).

Layout: 64-byte little-endian header (magic 'SFW1', u32 version 1, twelve u32 shape
fields C,H,W,p,D,L,heads,mlp,tdim,ctx_len,ctx_dim,has_cross, u64 seed), then fp32
tensors in a fixed order, linear weights stored [out, in].
"""
import struct
from dataclasses import dataclass, field

import numpy as np

_FIELDS = ("C", "H", "W", "p", "D", "L", "heads", "mlp", "tdim", "ctx_len", "ctx_dim", "has_cross")


@dataclass
class OracleModel:
    C: int
    H: int
    W: int
    p: int
    D: int
    L: int
    heads: int
    mlp: int
    tdim: int
    ctx_len: int
    ctx_dim: int
    has_cross: int
    seed: int
    top: dict = field(default_factory=dict)      # non-block tensors
    blocks: list = field(default_factory=list)   # per-block dicts

    @property
    def N(self):
        return (self.H // self.p) * (self.W // self.p)

    @property
    def dh(self):
        return self.D // self.heads

    def astype(self, dtype):
        """Copy with every tensor cast to `dtype` (fp64 self-check runs)."""
        m = OracleModel(**{k: getattr(self, k) for k in _FIELDS}, seed=self.seed)
        m.top = {k: v.astype(dtype) for k, v in self.top.items()}
        m.blocks = [{k: v.astype(dtype) for k, v in b.items()} for b in self.blocks]
        return m


def load_blob(blob: bytes) -> OracleModel:
    if len(blob) < 64:
        raise ValueError("blob shorter than its header")
    magic, version, *dims, seed = struct.unpack_from("<4sI12IQ", blob, 0)
    if magic != b"SFW1" or version != 1:
        raise ValueError("bad magic or version")
    m = OracleModel(**dict(zip(_FIELDS, dims)), seed=seed)
    D, P, F = m.D, m.p * m.p * m.C, m.mlp
    off = 64

    def take(shape):
        nonlocal off
        n = int(np.prod(shape))
        if off + 4 * n > len(blob):
            raise ValueError("blob truncated")
        a = np.frombuffer(blob, dtype="<f4", count=n, offset=off).reshape(shape).astype(np.float32)
        off += 4 * n
        return a

    t = m.top
    t["W_pe"], t["b_pe"], t["pos"] = take((D, P)), take((D,)), take((m.N, D))
    t["W_t1"], t["b_t1"], t["W_t2"], t["b_t2"] = take((D, m.tdim)), take((D,)), take((D, D)), take((D,))
    for _ in range(m.L):
        b = {}
        b["W_mod"], b["b_mod"] = take((6 * D, D)), take((6 * D,))
        b["W_qkv"], b["b_qkv"] = take((3 * D, D)), take((3 * D,))
        b["W_o"], b["b_o"] = take((D, D)), take((D,))
        if m.has_cross:
            b["W_qx"], b["b_qx"] = take((D, D)), take((D,))
            b["W_kvx"], b["b_kvx"] = take((2 * D, m.ctx_dim)), take((2 * D,))
            b["W_ox"], b["b_ox"] = take((D, D)), take((D,))
        b["W_fc1"], b["b_fc1"] = take((F, D)), take((F,))
        b["W_fc2"], b["b_fc2"] = take((D, F)), take((D,))
        m.blocks.append(b)
    t["W_fmod"], t["b_fmod"], t["W_f"], t["b_f"] = take((2 * D, D)), take((2 * D,)), take((P, D)), take((P,))
    if off != len(blob):
        raise ValueError(f"blob has {len(blob) - off} trailing bytes")
    return m
