"""bench.py on the host: the one-GPU contract and the work figures its roofline divides
by (no GPU needed)."""
import os
import subprocess
import sys

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0
    assert "one GPU" in r.stdout + r.stderr


def test_class_work_is_the_algorithmic_flop_count():
    """Per-launch FLOPs of the 512^2 width-768 step (4 rows x 1024 tokens), written out:
    2 M K N per projection, 4 N^2 D per row for attention (scores and P.V)."""
    import bench
    from paper_2511_22009_amd import KernelClass as KC
    cfg = W.get_config("s512")
    assert (cfg.N, cfg.D, cfg.mlp, cfg.rows) == (1024, 768, 3072, 4)
    want = {
        KC.QKV: 14_495_514_624,   # 2 * 4096 * 768 * 2304
        KC.PROJ: 4_831_838_208,   # 2 * 4096 * 768 * 768
        KC.FC1: 19_327_352_832,   # 2 * 4096 * 768 * 3072
        KC.FC2: 19_327_352_832,   # 2 * 4096 * 3072 * 768
        KC.ATTN: 12_884_901_888,  # 4 * 4 * 1024^2 * 768
    }
    for kc, flops in want.items():
        assert bench.class_work(cfg, kc, cfg.rows) == flops, kc
