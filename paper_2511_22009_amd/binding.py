"""ctypes binding of the C ABI declared in include/streamflow.h.

Argument marshalling only: shapes, dtypes and devices are checked, pointers and host
scalars are handed to the library, and errors come back as SFError. Tensors are torch
CUDA tensors; streams default to torch's current stream on the tensor's device.
"""
import ctypes
import enum
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_NAME = "libstreamflow.so"

SF_MAX_ROWS = 64


class Precision(enum.IntEnum):
    BF16 = 0
    FP32 = 1


class KernelClass(enum.IntEnum):
    TEMB = 0
    EMBED = 1
    LN = 2
    QKV = 3
    ATTN = 4
    PROJ = 5
    FC1 = 6
    FC2 = 7
    CROSS = 8
    HEAD = 9
    EULER = 10


class Buffer(enum.IntEnum):
    H = 0
    ACT = 1
    Q = 2
    K = 3
    VT = 4
    ATTN = 5
    MLP = 6
    TABLE = 7


class _PeRFlow(ctypes.Structure):
    _fields_ = [("windows", ctypes.c_int), ("train_steps", ctypes.c_int), ("beta_start", ctypes.c_float),
                ("beta_end", ctypes.c_float), ("eps", ctypes.c_double)]


class SFError(RuntimeError):
    def __init__(self, code, where):
        self.code = code
        msg = _lib().sf_strerror(code).decode() if _LIB is not None else str(code)
        super().__init__(f"{where}: {msg} (code {code})")


class _Cond(ctypes.Structure):
    _fields_ = [("ctx", ctypes.c_void_p), ("null_ctx", ctypes.c_void_p), ("guidance", ctypes.c_float)]


class _Info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in
                ("C", "H", "W", "p", "D", "L", "heads", "mlp", "tdim", "ctx_len", "ctx_dim", "has_cross",
                 "tokens", "mod_width", "precision", "max_rows")] + \
               [("weight_bytes", ctypes.c_size_t), ("workspace_bytes", ctypes.c_size_t),
                ("vt_ld", ctypes.c_int), ("vt_key_perm", ctypes.c_int)]


_LIB = None
_P = ctypes.c_void_p
_I = ctypes.c_int
_SIGS = {
    "sf_load_weights": (_I, [ctypes.c_void_p, ctypes.c_size_t, _I, _I, ctypes.POINTER(_P)]),
    "sf_free": (None, [_P]),
    "sf_strerror": (ctypes.c_char_p, [_I]),
    "sf_get_info": (_I, [_P, ctypes.POINTER(_Info)]),
    "sf_velocity": (_I, [_P, _P, _P, _I, _P, _P, _P]),
    "sf_stream_step": (_I, [_P, _P, _P, _P, _I, _P, _P, _P, _P]),
    "sf_euler_shift": (_I, [_P, _P, _P, _P, _I, _P, _P, _P]),
    "sf_modulation": (_I, [_P, _P, _I, _P, _P]),
    "sf_modulation_noalloc": (_I, [_P, _P, _I, _P, _P]),
    "sf_residual": (_I, [_P, _P, _P, _I, _P, _I, _P, _P]),
    "sf_debug_read": (_I, [_P, _I, _P, ctypes.c_size_t, _P]),
    "sf_attention": (_I, [_P, _P, _P, _P, _P, _I, _P]),
    "sf_timing_enable": (_I, [_P, _I, _I]),
    "sf_timing_read": (_I, [_P, _I, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_long)]),
    "sf_graph_enable": (_I, [_P, _I]),
    "sf_noise_latent": (_I, [_P, _P, _P, ctypes.c_float, _P, _P]),
    "sf_set_scheduler": (_I, [_P, ctypes.POINTER(_PeRFlow)]),
    "sf_scheduler_shift": (_I, [_P, _P, _P, _P, _P, _I, _P, _P, _P]),
    "sf_graph_stats": (_I, [_P, ctypes.POINTER(_I), ctypes.POINTER(ctypes.c_long)]),
    "sf_modulation_cache": (_I, [_P, _I]),
    "sf_modulation_cache_stats": (_I, [_P, ctypes.POINTER(ctypes.c_long)]),
    "sf_context_cache": (_I, [_P, _I]),
    "sf_context_cache_stats": (_I, [_P, ctypes.POINTER(ctypes.c_long), ctypes.POINTER(ctypes.c_long)]),
}


def lib_path():
    return os.path.join(_HERE, _LIB_NAME)


def library_symbols():
    return sorted(_SIGS)


def load_library():
    """Load libstreamflow.so; raises if it has not been built (there is no fallback)."""
    global _LIB
    if _LIB is None:
        path = lib_path()
        if not os.path.exists(path):
            raise ImportError(f"{path} is missing: build it with `python -m paper_2511_22009_amd.build` "
                              "(or __graft_entry__.build()); there is no CPU fallback")
        L = ctypes.CDLL(path)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = L
    return _LIB


_lib = load_library


def _check(rc, where):
    if rc != 0:
        raise SFError(rc, where)


def _host_f32(vals, n, what):
    a = np.ascontiguousarray(np.asarray(vals, dtype=np.float32).reshape(-1))
    if a.shape[0] != n:
        raise ValueError(f"{what}: expected {n} values, got {a.shape[0]}")
    return a


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


class Cond:
    """Conditioning for a network with cross-attention.

    ctx: device fp32 [B, ctx_len, ctx_dim]; null_ctx: device fp32 [ctx_len, ctx_dim] or
    None (no guidance); guidance: w in v = v_u + w (v_c - v_u)."""

    def __init__(self, ctx, null_ctx=None, guidance=7.5):
        self.ctx, self.null_ctx, self.guidance = ctx, null_ctx, float(guidance)

    def _struct(self):
        return _Cond(self.ctx.data_ptr(), self.null_ctx.data_ptr() if self.null_ctx is not None else None,
                     self.guidance)

    @property
    def guided(self):
        return self.null_ctx is not None


class Model:
    """A loaded velocity network (weights + workspace on the current HIP device)."""

    def __init__(self, blob, precision=Precision.BF16, max_rows=8):
        """`blob`: the weight blob as bytes or any writable buffer (bytearray, numpy)."""
        L = load_library()
        h = ctypes.c_void_p()
        if isinstance(blob, bytes):
            ptr, n = ctypes.cast(ctypes.c_char_p(blob), ctypes.c_void_p), len(blob)
        else:
            mv = memoryview(blob).cast("B")
            n = mv.nbytes
            ptr = ctypes.cast((ctypes.c_char * n).from_buffer(mv), ctypes.c_void_p)
        _check(L.sf_load_weights(ptr, n, int(precision), int(max_rows), ctypes.byref(h)),
               "sf_load_weights")
        self._h = h
        info = _Info()
        _check(L.sf_get_info(h, ctypes.byref(info)), "sf_get_info")
        self.info = {n: getattr(info, n) for n, _ in _Info._fields_}
        self.latent_shape = (info.C, info.H, info.W)

    # -- helpers ---------------------------------------------------------------------
    def _stream(self, stream):
        import torch
        s = stream if stream is not None else torch.cuda.current_stream()
        return ctypes.c_void_p(s.cuda_stream)

    def _latents(self, x, n, what, writable=False):
        import torch
        if not isinstance(x, torch.Tensor) or not x.is_cuda:
            raise TypeError(f"{what}: expected a CUDA tensor")
        if x.dtype != torch.float32 or not x.is_contiguous():
            raise TypeError(f"{what}: expected contiguous float32")
        if tuple(x.shape[-3:]) != self.latent_shape or x.numel() < n * int(np.prod(self.latent_shape)):
            raise ValueError(f"{what}: shape {tuple(x.shape)} does not hold {n} latents of {self.latent_shape}")
        return ctypes.c_void_p(x.data_ptr())

    def _cond(self, cond, B):
        if cond is None:
            return None, None
        c = cond._struct()
        return ctypes.byref(c), c

    # -- C ABI -------------------------------------------------------------------------
    def velocity(self, x, t, cond=None, out=None, stream=None):
        import torch
        B = x.shape[0]
        tt = _host_f32(t, B, "t")
        if out is None:
            out = torch.empty_like(x)
        cref, keep = self._cond(cond, B)
        _check(load_library().sf_velocity(self._h, self._latents(x, B, "x"), _ptr(tt), B, cref,
                                          self._latents(out, B, "v"), self._stream(stream)), "sf_velocity")
        return out

    def stream_step(self, x, t, dt, B, z_new, x_done=None, cond=None, stream=None):
        tt, dd = _host_f32(t, B, "t"), _host_f32(dt, B, "dt")
        cref, keep = self._cond(cond, B)
        need = B if x_done is not None else B + 1
        done = self._latents(x_done, 1, "x_done") if x_done is not None else None
        _check(load_library().sf_stream_step(self._h, self._latents(x, need, "x"), _ptr(tt), _ptr(dd), B, cref,
                                             self._latents(z_new, 1, "z_new"), done, self._stream(stream)),
               "sf_stream_step")

    def euler_shift(self, x, v, dt, B, z_new, x_done=None, stream=None):
        dd = _host_f32(dt, B, "dt")
        need = B if x_done is not None else B + 1
        done = self._latents(x_done, 1, "x_done") if x_done is not None else None
        _check(load_library().sf_euler_shift(self._h, self._latents(x, need, "x"), self._latents(v, B, "v"),
                                             _ptr(dd), B, self._latents(z_new, 1, "z_new"), done,
                                             self._stream(stream)), "sf_euler_shift")

    def modulation(self, t, out=None, stream=None):
        import torch
        tt = np.ascontiguousarray(np.asarray(t, dtype=np.float32).reshape(-1))
        B = tt.shape[0]
        if out is None:
            out = torch.empty((B, self.info["mod_width"]), dtype=torch.float32, device="cuda")
        if out.dtype != torch.float32 or not out.is_contiguous() or out.numel() < B * self.info["mod_width"]:
            raise ValueError("table: expected contiguous float32 [B, mod_width]")
        _check(load_library().sf_modulation(self._h, _ptr(tt), B, ctypes.c_void_p(out.data_ptr()),
                                            self._stream(stream)), "sf_modulation")
        return out

    def modulation_noalloc(self, t, out, stream=None):
        """sf_modulation_noalloc: the table of `modulation`, computed with the library's
        fixed scratch array (no device allocation); `out` is required."""
        tt = np.ascontiguousarray(np.asarray(t, dtype=np.float32).reshape(-1))
        B = tt.shape[0]
        import torch
        if out.dtype != torch.float32 or not out.is_contiguous() or out.numel() < B * self.info["mod_width"]:
            raise ValueError("table: expected contiguous float32 [B, mod_width]")
        _check(load_library().sf_modulation_noalloc(self._h, _ptr(tt), B, ctypes.c_void_p(out.data_ptr()),
                                                    self._stream(stream)), "sf_modulation_noalloc")
        return out

    def residual(self, x, t, blocks, cond=None, stream=None):
        import torch
        B = x.shape[0]
        tt = _host_f32(t, B, "t")
        rows = 2 * B if (cond is not None and cond.guided) else B
        out = torch.empty((rows, self.info["tokens"], self.info["D"]), dtype=torch.float32, device=x.device)
        cref, keep = self._cond(cond, B)
        _check(load_library().sf_residual(self._h, self._latents(x, B, "x"), _ptr(tt), B, cref, int(blocks),
                                          ctypes.c_void_p(out.data_ptr()), self._stream(stream)), "sf_residual")
        return out

    def debug_read(self, buffer, shape, stream=None):
        """Copy an internal buffer (see sf_debug_read) into a new fp32 tensor of `shape`."""
        import torch
        fp32 = buffer in (Buffer.H, Buffer.TABLE) or self.info["precision"] == int(Precision.FP32)
        out = torch.empty(shape, dtype=torch.float32 if fp32 else torch.bfloat16, device="cuda")
        _check(load_library().sf_debug_read(self._h, int(buffer), ctypes.c_void_p(out.data_ptr()),
                                            out.numel() * out.element_size(), self._stream(stream)),
               "sf_debug_read")
        return out.float()

    def attention(self, q, k, vT, stream=None):
        """The model's self-attention on caller tensors (see sf_attention): q, k
        [rows, heads, N, dh], vT [rows, heads, dh, vt_ld] in the compute type (bf16 in
        bf16 mode, else float32), contiguous, on the GPU. Returns o [rows, N, D]."""
        import torch
        inf = self.info
        rows = q.shape[0]
        dt = torch.float32 if inf["precision"] == int(Precision.FP32) else torch.bfloat16
        dh = inf["D"] // inf["heads"]
        want = {"q": (q, (rows, inf["heads"], inf["tokens"], dh)), "k": (k, (rows, inf["heads"], inf["tokens"], dh)),
                "vT": (vT, (rows, inf["heads"], dh, inf["vt_ld"]))}
        for name, (ten, shape) in want.items():
            if tuple(ten.shape) != shape or ten.dtype != dt or not ten.is_cuda or not ten.is_contiguous():
                raise ValueError(f"{name}: expected contiguous {dt} {shape} on the GPU")
        o = torch.empty((rows, inf["tokens"], inf["D"]), dtype=dt, device=q.device)
        _check(load_library().sf_attention(self._h, ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()),
                                           ctypes.c_void_p(vT.data_ptr()), ctypes.c_void_p(o.data_ptr()), rows,
                                           self._stream(stream)), "sf_attention")
        return o

    def set_scheduler(self, windows=4, train_steps=1000, beta_start=0.00085, beta_end=0.012, eps=1e-6):
        """Read the network output as a noise prediction and update with PeRFlow's time
        windows (see sf_set_scheduler)."""
        p = _PeRFlow(int(windows), int(train_steps), float(beta_start), float(beta_end), float(eps))
        _check(load_library().sf_set_scheduler(self._h, ctypes.byref(p)), "sf_set_scheduler")

    def clear_scheduler(self):
        _check(load_library().sf_set_scheduler(self._h, None), "sf_set_scheduler")

    def scheduler_shift(self, x, out, t, dt, B, z_new, x_done=None, stream=None):
        """The update + shift of a stream step for a given network output `out`."""
        tt, dd = _host_f32(t, B, "t"), _host_f32(dt, B, "dt")
        need = B if x_done is not None else B + 1
        done = self._latents(x_done, 1, "x_done") if x_done is not None else None
        _check(load_library().sf_scheduler_shift(self._h, self._latents(x, need, "x"), self._latents(out, B, "out"),
                                                 _ptr(tt), _ptr(dd), B, self._latents(z_new, 1, "z_new"), done,
                                                 self._stream(stream)), "sf_scheduler_shift")

    def noise_latent(self, x_ref, z, t0, out=None, stream=None):
        """out = (1 - t0) x_ref + t0 z: the admitted latent of an image-to-image run."""
        import torch
        if out is None:
            out = torch.empty_like(z)
        _check(load_library().sf_noise_latent(self._h, self._latents(x_ref, 1, "x_ref"), self._latents(z, 1, "z"),
                                              float(t0), self._latents(out, 1, "out"), self._stream(stream)),
               "sf_noise_latent")
        return out

    def graph_enable(self, on=True):
        """Capture each distinct velocity / stream-step call into a HIP graph and replay it
        on identical calls (needs a non-default stream; see sf_graph_enable)."""
        _check(load_library().sf_graph_enable(self._h, 1 if on else 0), "sf_graph_enable")

    def graph_stats(self):
        cached, replays = ctypes.c_int(), ctypes.c_long()
        _check(load_library().sf_graph_stats(self._h, ctypes.byref(cached), ctypes.byref(replays)), "sf_graph_stats")
        return cached.value, replays.value

    def modulation_cache(self, on=True):
        """Skip the per-sample conditioning launches when a call's timesteps equal the
        previous network call's on the same stream (see sf_modulation_cache)."""
        _check(load_library().sf_modulation_cache(self._h, 1 if on else 0), "sf_modulation_cache")

    def modulation_cache_stats(self):
        skips = ctypes.c_long()
        _check(load_library().sf_modulation_cache_stats(self._h, ctypes.byref(skips)), "sf_modulation_cache_stats")
        return skips.value

    def context_cache(self, on=True):
        """Keep the cross-attention context entries across calls, reusing an entry whose
        context is bitwise unchanged (see sf_context_cache). Waits for the device."""
        _check(load_library().sf_context_cache(self._h, 1 if on else 0), "sf_context_cache")

    def context_cache_stats(self):
        """(calls through the entry lookup, context entries projected by them)."""
        calls, projected = ctypes.c_long(0), ctypes.c_long(0)
        _check(load_library().sf_context_cache_stats(self._h, ctypes.byref(calls), ctypes.byref(projected)),
               "sf_context_cache_stats")
        return calls.value, projected.value

    def timing_enable(self, kc, on=True):
        _check(load_library().sf_timing_enable(self._h, int(kc), 1 if on else 0), "sf_timing_enable")

    def timing_read(self, kc):
        ms, n = ctypes.c_double(), ctypes.c_long()
        _check(load_library().sf_timing_read(self._h, int(kc), ctypes.byref(ms), ctypes.byref(n)), "sf_timing_read")
        return ms.value, n.value

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            load_library().sf_free(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
