"""bench.py's host-side contract (no GPU): more than one GPU is refused with a
message and exit status 2 before anything touches a device; --envs applies to
the sampled workloads only; the algorithmic-work figures it prices the
roofline with match the MLP shapes."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120, cwd=ROOT)


@pytest.mark.parametrize("n", ["2", "8"])
def test_more_than_one_gpu_is_refused(n):
    r = _bench("--gpus", n, "--no-cpu-baseline")
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout.strip() == ""


@pytest.mark.parametrize("wl", ["matrix", "iter", "feature"])
def test_envs_only_for_sampled_workloads(wl):
    r = _bench("--workload", wl, "--envs", "100", "--no-cpu-baseline")
    assert r.returncode == 2
    assert "--envs" in r.stderr


def test_policy_flops_per_frame():
    sys.path.insert(0, ROOT)
    import bench
    # 2 flops per multiply-add over the three layers
    assert bench.policy_flops_per_frame([256, 512, 512, 18]) == 804_864
    assert bench.policy_flops_per_frame([512, 512, 512, 18]) == 1_067_008
    assert bench.policy_flops_per_frame([75, 256, 256, 5]) == 172_032
    assert bench.policy_flops_per_frame([24, 64, 64, 3]) == 11_648
