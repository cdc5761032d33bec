"""bench.py's JSON line on the GPU: one short pursuit run in a child process,
every field the line promises present and consistent (metric and unit, one
GPU, the timed steps, the roofline of the grouped forward)."""
import json
import os
import subprocess
import sys

import pytest

from gpu_helpers import say

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_bench_json_line():
    say("[bench] pursuit, 2 timed fills, child process")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "pursuit",
                        "--steps", "2", "--warmup", "1", "--no-cpu-baseline", "--fill-only"],
                       capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    d = json.loads(r.stdout.strip().splitlines()[-1])
    assert d["metric"].startswith("agent-frames/s") and d["unit"] == "agent-frames/s"
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1
    assert d["value"] > 0 and d["ms_per_step"] > 0
    assert d["higher_is_better"] is True and d["scaling"] == "weak"
    assert d["vs_baseline"] is None and d["dtype"] == "bf16"
    assert d["config"]["workload"] == "pursuit"
    # agent-frames per fill / fill time = value (live frames: pursuit ends
    # episodes at capture, so at most n_envs * 2 * H)
    assert d["value"] * d["ms_per_step"] / 1e3 <= 16384 * 2 * 100 * 1.0001
    rf = d["roofline"]
    assert rf["bound"] == "mfma" and rf["unit"] == "TFLOP/s" and rf["peak"] == 2500.0
    assert 0 < rf["frac"] < 1 and abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3
    assert "traffic" in rf
