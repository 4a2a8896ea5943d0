"""Host-side input generators: the in-place blob equals the serialised weight dict,
draws are reproducible, and their statistics are the stated ones."""
import struct

import numpy as np
import pytest

import workloads as W


@pytest.mark.parametrize("init", [None, "tsens", "zero"])
@pytest.mark.parametrize("name", ["tiny", "tiny_cfg", "ragged"])
def test_blob_in_place_equals_serialised_weights(name, init):
    cfg = W.get_config(name)
    blob = W.make_blob(cfg, init=init)
    assert bytes(blob) == W.write_blob(cfg, W.make_weights(cfg, init=init))
    assert bytes(W.make_blob(cfg, init=init)) == bytes(blob)          # reproducible


def test_blob_header_and_size():
    cfg = W.get_config("ragged")
    blob = W.make_blob(cfg)
    magic, version, *dims, seed = struct.unpack_from(W.blob.HEADER_FMT, blob, 0)
    assert magic == b"SFW1" and version == 1 and seed == 0
    assert tuple(dims) == W.blob.header_fields(cfg)
    assert len(blob) == 64 + 4 * sum(int(np.prod(s)) for _, s in W.tensor_specs(cfg))


def test_weight_statistics():
    cfg = W.get_config("s512")
    w = W.make_weights(W.get_config("tiny"))
    assert all(a.dtype == np.float32 for a in w.values())
    big = W.make_weights(cfg)["blk0.W_fc1"]                          # 3072 x 768 draws
    assert abs(float(big.mean())) < 1e-4 and abs(float(big.std()) - 0.02) < 1e-4
    ts = W.make_weights(W.get_config("tiny"), init="tsens")
    assert abs(float(ts["blk0.W_mod"].std()) - 1 / np.sqrt(128)) < 0.01 / np.sqrt(128) * 10
    assert abs(float(ts["blk0.W_fc1"].std()) - 0.02) < 2e-3
    # distinct tensors come from distinct streams
    assert not np.array_equal(w["blk0.W_o"], w["blk1.W_o"])


def test_slot_times_descend_with_negative_steps():
    for name in ("tiny", "s512", "s512_cfg"):
        cfg = W.get_config(name)
        t, dt = W.slot_times(cfg)
        assert t.dtype == np.float32 and dt.dtype == np.float32 and len(t) == cfg.K
        assert t[0] == 1.0 and np.all(dt < 0) and np.all(np.diff(t) < 0)
        g = W.schedule(cfg)
        np.testing.assert_array_equal(dt, (g[1:] - g[:-1]).astype(np.float32))
