"""The C ABI without a GPU: the library loads, exports every declared entry point,
and rejects bad arguments and malformed blobs on the host before any HIP call."""
import ctypes
import os
import re
import struct

import pytest

import workloads as W
from paper_2511_22009_amd import binding, load_library

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "streamflow.h")).read()
    return sorted(set(re.findall(r"^\s*(?:int|void|const char\*)\s+(sf_\w+)\s*\(", src, re.M)))


def test_every_declared_symbol_is_exported_and_bound():
    L = load_library()
    names = _declared()
    assert "sf_stream_step" in names and "sf_velocity" in names and "sf_load_weights" in names
    for n in names:
        assert hasattr(L, n), n
    assert sorted(binding.library_symbols()) == names


def _load(blob, prec=0, max_rows=4):
    h = ctypes.c_void_p()
    rc = load_library().sf_load_weights(blob, len(blob) if blob is not None else 0, prec, max_rows, ctypes.byref(h))
    assert not h.value  # never a handle on failure
    return rc


@pytest.fixture(scope="module")
def tiny_blob():
    return bytes(W.make_blob(W.get_config("tiny")))


def test_load_rejects_bad_arguments(tiny_blob):
    L = load_library()
    assert L.sf_load_weights(None, 0, 0, 4, ctypes.byref(ctypes.c_void_p())) == -1
    assert L.sf_load_weights(tiny_blob, len(tiny_blob), 0, 4, None) == -1
    assert _load(tiny_blob, prec=2) == -1
    assert _load(tiny_blob, max_rows=0) == -1
    assert _load(tiny_blob, max_rows=65) == -1


def test_load_rejects_malformed_blobs(tiny_blob):
    assert _load(b"SFW1") == -2                                  # shorter than the header
    assert _load(b"XFW1" + tiny_blob[4:]) == -2                  # magic
    assert _load(tiny_blob[:4] + struct.pack("<I", 2) + tiny_blob[8:]) == -2   # version
    assert _load(tiny_blob[:-4]) == -2                           # truncated
    assert _load(tiny_blob + b"\0" * 4) == -2                    # trailing bytes
    hdr = bytearray(tiny_blob[:64])
    struct.pack_into("<I", hdr, 8 + 4 * 3, 3)                    # p = 3 does not divide H = 16
    assert _load(bytes(hdr) + tiny_blob[64:]) == -2


def test_load_rejects_unsupported_shapes():
    from dataclasses import replace
    cfg = replace(W.get_config("tiny"), D=132, heads=4)          # head dim 33: not a multiple of 8
    assert _load(bytes(W.make_blob(cfg))) == -6
    cfg = replace(W.get_config("tiny"), D=256, heads=1, mlp=512)  # head dim 256 > 128
    assert _load(bytes(W.make_blob(cfg))) == -6


def test_calls_reject_null_handle_and_arguments():
    L = load_library()
    t = (ctypes.c_float * 4)(1, 0.75, 0.5, 0.25)
    dummy = ctypes.c_void_p(16)
    assert L.sf_velocity(None, dummy, t, 4, None, dummy, None) == -3
    assert L.sf_graph_enable(None, 1) == -3
    assert L.sf_modulation_cache(None, 1) == -3
    assert L.sf_modulation_cache_stats(None, None) == -3
    assert L.sf_set_scheduler(None, None) == -3
    assert L.sf_noise_latent(None, dummy, dummy, 0.5, dummy, None) == -3
    assert L.sf_stream_step(None, dummy, t, t, 4, None, dummy, None, None) == -3
    assert L.sf_euler_shift(None, dummy, dummy, t, 4, dummy, None, None) == -3
    assert L.sf_modulation(None, t, 4, dummy, None) == -3
    assert L.sf_residual(None, dummy, t, 4, None, 0, dummy, None) == -3
    assert L.sf_attention(None, dummy, dummy, dummy, dummy, 1, None) == -3
    assert L.sf_timing_enable(None, 0, 1) == -3
    assert L.sf_get_info(None, None) == -3
    L.sf_free(None)


def test_strerror_texts():
    L = load_library()
    texts = {c: L.sf_strerror(c).decode() for c in range(-6, 1)}
    assert texts[0] == "ok" and len(set(texts.values())) == 7
    assert L.sf_strerror(-99).decode() == "unknown status code"


def test_load_rejects_rows_whose_operands_pass_the_offset_range():
    """The bf16 kernels address activations with 32-bit byte offsets: a load whose
    largest operand (rows x tokens x MLP width, bf16) would reach 2^31 bytes is refused
    on the host, from the header alone. At 1024^2 (4096 tokens, MLP 4608) 64 rows are
    2.4 GB; the loader never gets to read past the 64-byte header it is given."""
    import numpy as np
    from workloads.blob import HEADER_FMT, MAGIC, VERSION, header_fields, tensor_specs
    cfg = W.get_config("s1024")
    head = struct.pack(HEADER_FMT, MAGIC, VERSION, *header_fields(cfg), 0)
    nbytes = len(head) + 4 * sum(int(np.prod(s)) for _, s in tensor_specs(cfg))
    assert 64 * cfg.N * cfg.mlp * 2 >= 0x7ffffff0
    h = ctypes.c_void_p()
    rc = load_library().sf_load_weights(head, nbytes, 0, 64, ctypes.byref(h))
    assert rc == -6 and not h.value
