"""Host-side parts of bench.py: the flop count it divides by, and the one-GPU contract."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


@pytest.mark.parametrize("B,S,H,d_c", [(1, 16384, 16, 512), (2, 777, 3, 64), (1, 1, 1, 32)])
def test_step_flops_match_the_oracle_count(B, S, H, d_c):
    import bench
    from oracle.laga import algorithmic_flops
    assert bench.step_flops(B, S, H, d_c, 192, 128, 256) == pytest.approx(
        algorithmic_flops(B, S, H, d_c, 192, 128, 256), rel=1e-12)


def test_benchmark_workload_is_4329_gflop():
    import bench
    import laga_inputs as LI
    assert abs(bench.flops(LI.WORKLOADS[bench.WORKLOAD]) / 1e9 - 4329.3) < 0.05


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)
