"""Host-side parts of bench.py: the one-GPU guard, the kernel-source digest that keys the
traffic record, the traffic lookup, and the oracle CPU baseline on the tiny workload."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
from oracle import la_oracle as O
from paper_2605_31158_amd.workloads import WORKLOADS, make_inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_code_digest_ignores_comments_and_blank_space():
    a = "int f(int x) {\n  return x + 1;  // add one\n}\n"
    b = "/* header */\nint f(int x)   {\n\n  return x + 1;\n}"
    c = "int f(int x) {\n  return x + 2;\n}\n"
    assert bench.code_digest(a) == bench.code_digest(b)
    assert bench.code_digest(a) != bench.code_digest(c)


def test_traffic_record_matches_only_its_kernel_source():
    path = os.path.join(ROOT, "profiles", "traffic_attn_fwd_480p_window.json")
    rec = json.load(open(path))
    assert bench.traffic_from_profile("attn_fwd", "480p_window", rec["src_digest"], 0.0) == rec["hbm_bytes_per_launch"]
    assert bench.traffic_from_profile("attn_fwd", "480p_window", "0" * 16, 0.0) is None
    assert bench.traffic_from_profile("attn_fwd", "no_such_workload", rec["src_digest"], 0.0) is None
    # the calibrated bytes are the counters over the copy-kernel factors
    kib = rec["fetch_kib_per_launch"] / rec["read_factor"] + rec["write_kib_per_launch"] / rec["write_factor"]
    assert rec["hbm_bytes_per_launch"] == pytest.approx(kib * 1024)


def test_cpu_baseline_on_tiny():
    wl = WORKLOADS["tiny"]
    inp = make_inputs(wl)
    mask = O.select_blocks(inp["q"], inp["k"], wl.block, tau=wl.tau, n_text=wl.n_text)["mask"]
    out = bench.cpu_baseline(wl, inp, mask, target_s=0.2)
    assert out["kind"] == "oracle" and out["unit"] == "TFLOP/s"
    assert out["value"] > 0 and out["cores"] >= 1
    assert "heads" in out["sample"]
    assert np.isfinite(out["value"])


@pytest.mark.parametrize("Lq,Lk,block", [(256, 1024, 64), (200, 1000, 64), (300, 1100, 128)])
def test_kept_flop_count_matches_oracle(Lq, Lk, block):
    rng = np.random.default_rng(7)
    NQ, NK = -(-Lq // block), -(-Lk // block)
    mask = (rng.random((2, 3, NQ, NK)) < 0.3).astype(np.uint8)
    assert bench.kept_flop_count(mask, Lq, Lk, block, 128) == O.kept_flops(mask, Lq, Lk, block, 128)
