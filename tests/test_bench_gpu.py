"""bench.py end to end on the GPU (small workloads): the JSON line and the optional passes.

Regression: the --cold loop runs the attention kernel on its own after the cached-means
selection has reused the workspace; it must build the plan again first."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(*args):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                       timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    return json.loads(r.stdout.strip().splitlines()[-1])


def test_bench_tiny_with_cold_and_dense():
    d = run_bench("--workload", "tiny", "--steps", "3", "--warmup", "1", "--no-cpu-baseline", "--cold",
                  "--clock-warmup-ms", "20")
    assert d["config"]["workload"] == "tiny" and d["n_gpus"] == 1 and d["steps"] == 3
    assert d["cold_attn_run_ms"] is not None and d["cold_attn_run_ms"] > 0
    assert d["dense_attn_ms"] is not None and d["select_cached_same_mask"] is True
    assert d["roofline"]["bound"] == "mfma" and d["roofline"]["achieved"] > 0
