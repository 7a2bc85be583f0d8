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


def test_kept_flop_count_3d_matches_oracle_sets():
    from paper_2605_31158_amd.workloads import WORKLOADS_3D
    wl = WORKLOADS_3D["tiny_3d"]
    L = O.layout_3d(wl.n_text, wl.T_ctx, wl.T_q, wl.Hs, wl.Ws, wl.bt, wl.bh, wl.bw, wl.block)
    rng = np.random.default_rng(3)
    NQ, NK = len(L["qsets"]), len(L["ksets"])
    mask = (rng.random((1, 2, NQ, NK)) < 0.4).astype(np.uint8)
    want = 0
    for h in range(2):
        for i in range(NQ):
            kept = np.nonzero(mask[0, h, i])[0]
            want += 4 * wl.d * L["qsets"][i].size * sum(L["ksets"][m].size for m in kept)
    qv = [s.size for s in L["qsets"]]
    kv = [s.size for s in L["ksets"]]
    assert bench.kept_flop_count_3d(mask, qv, kv, wl.d) == want


def test_cpu_baseline_3d_on_tiny():
    from paper_2605_31158_amd.workloads import WORKLOADS_3D, make_inputs_3d
    wl = WORKLOADS_3D["tiny_3d"]
    inp = make_inputs_3d(wl)
    L = O.layout_3d(wl.n_text, wl.T_ctx, wl.T_q, wl.Hs, wl.Ws, wl.bt, wl.bh, wl.bw, wl.block)
    sel = O.select_blocks_sets(inp["q"], inp["k"], L["qsets"], L["ksets"], L["forced"], tau=wl.tau)
    qv = [s.size for s in L["qsets"]]
    kv = [s.size for s in L["ksets"]]
    out = bench.cpu_baseline_3d(wl, inp, sel["mask"], qv, kv, target_s=0.2)
    assert out["kind"] == "oracle" and out["value"] > 0 and "heads" in out["sample"]


def test_prep_bytes_3d_counts_every_slot():
    from paper_2605_31158_amd.workloads import WORKLOADS_3D
    wl = WORKLOADS_3D["480p_3d"]
    # 16 heads; 52 query blocks; 3 text + 312 context + 52 chunk key blocks of 128 slots, d = 128
    assert bench.prep_bytes_3d(wl, "q") == 16 * (6240 * 256 + 52 * 128 * 256 + 52 * 512)
    assert bench.prep_bytes_3d(wl, "kv") == 16 * (2 * 43980 * 256 + 2 * 367 * 128 * 256 + 367 * 512)
