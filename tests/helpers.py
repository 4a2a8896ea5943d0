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
