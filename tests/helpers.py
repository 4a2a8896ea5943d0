"""Small test helpers (no method arithmetic)."""
import numpy as np


def rel_l2(a, b):
    """||a - b||_2 / ||b||_2 accumulated in fp64."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(b.ravel()), 1e-300))


def rel_l2_per_sample(a, b):
    return [rel_l2(a[k], b[k]) for k in range(a.shape[0])]


# Tolerances on relative L2 per sample and per step (v, and the update x' - x).
TOL_BF16 = 2e-2
TOL_FP32 = 1e-4


def bf16_round(a):
    """fp32 -> bf16 with round-to-nearest-even (the kernels' conversion), returned as
    fp32 values. NaN and inf are not expected in the test data."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def elementwise_ratio(got, ref, rel, floor):
    """max over elements of |got - ref| / (rel |ref| + floor rms(ref)): <= 1 when every
    element is within `rel` of itself plus `floor` of the tensor's rms (fp64)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref)))
    return float(np.max(np.abs(got - ref) / (rel * np.abs(ref) + floor * rms)))
