#!/usr/bin/env python3
"""Benchmark of the AR block-sparse attention hot path on one MI355X.

A step is one pass of the whole path over one synthetic batch already resident in HBM:
la_select_blocks (pool Q, pool+score historical K, select and compact) followed by the three
steps of la_sparse_attn_fwd over the kept blocks (plan, run, merge), each called through its own
entry point so that HIP events on the launch stream can time every stage.  Prints ONE JSON line.

The K timed steps carry HIP events only around the attention kernel (the run stage), for its
roofline: every event record costs the GPU about 3 us, which with one event per stage added 4 % to
a 480P step.  The per-stage times come from K more steps, with an event between every two stages.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

NAME may also be a 3-D block workload (480p_3d, 720p_3d, tiny_3d): then a step is the 3-D path
(Q-Prep, KV-Prep, selection from the pooled means, attention, Untile Scatter).

Before the W warm-up steps the step is repeated for --clock-warmup-ms of wall time (200 ms by
default, reported as clock_warmup): the GPU's clock ramps up over the first milliseconds of work,
and without this the timed steps of the short workloads would partly run before it has.

value = kept-block TFLOP/s of the whole step (kept FLOPs / step time).  The line also
carries the per-kernel split, the dense baseline (same attention kernel, every block
kept), the roofline of the attention kernel (la_sparse_attn_run launches exactly that one
kernel, so its event time is the kernel's launch duration) and the fp64 oracle's CPU rate.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
HBM_PEAK_GBS = 8000.0              # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1, help="GPUs (one only: the path runs on one GPU)")
    ap.add_argument("--steps", type=int, default=50, help="timed steps (selection + attention per step)")
    ap.add_argument("--warmup", type=int, default=10, help="untimed steps before the timed ones")
    ap.add_argument("--workload", default="720p",
                    help="named synthetic workload, default the largest single-GPU one (1-D: tiny, 480p_window, "
                         "480p_memory, 720p, 720p_causal, "
                         "480p_long, 480p_long_dense; 3-D: tiny_3d, 480p_3d, 720p_3d)")
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip timing the fp64 oracle on the host")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense (every block kept) reference run")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU time of the oracle sample")
    ap.add_argument("--cold", action="store_true",
                    help="also time the attention run with the caches flushed (512 MiB written between calls)")
    ap.add_argument("--profile-only", action="store_true",
                    help="run warmup + steps of the sparse path only (for rocprofv3), print the JSON anyway")
    ap.add_argument("--clock-warmup-ms", type=float, default=200.0,
                    help="before the warm-up steps, repeat the step for this much wall time so that the timed "
                         "steps run at the GPU's steady clock (0: off; off with --profile-only)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 256 MiB device-to-device copy (reference for HBM byte counters)")
    return ap.parse_args()


def code_digest(text: str) -> str:
    """Digest of C/C++ source text with comments and blank space removed: a change of the code
    changes it, a change of a comment does not."""
    import re
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return hashlib.sha256(" ".join(text.split()).encode()).hexdigest()[:16]


def src_digest(*names) -> str:
    """code_digest of the named kernel sources (paper_2605_31158_amd/csrc), concatenated."""
    text = ""
    for n in names:
        with open(os.path.join(ROOT, "paper_2605_31158_amd", "csrc", n)) as f:
            text += f.read() + "\n"
    return code_digest(text)


def traffic_from_profile(kernel_tag: str, workload: str, digest: str, launches_bytes: float):
    """HBM bytes per launch measured by rocprofv3 PMC runs of the current kernel source, or None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel_tag}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("src_digest") != digest:
        return None
    return rec.get("hbm_bytes_per_launch")


def clock_warmup(stages, ms: float):
    """Repeats the step (the bound calls in order) until `ms` of wall time have passed; returns
    (steps, elapsed ms).  The first milliseconds of GPU work in a process run up to ~13 % slower
    (the clock ramps up), which would otherwise bias the short workloads' timed steps."""
    import torch
    if ms <= 0:
        return 0, 0.0
    n, t0 = 0, time.perf_counter()
    while (time.perf_counter() - t0) * 1e3 < ms:
        for _ in range(8):
            for f in stages:
                f()
        n += 8
        torch.cuda.synchronize()
    return n, round((time.perf_counter() - t0) * 1e3, 1)


def timed_steps(stages, run_index: int, stream, K: int):
    """The timed region: K steps between two device synchronisations, HIP events only around stage
    run_index (the attention kernel).  Returns (wall ms per step, event ms of that stage per step)."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for it in range(K):
        for j, f in enumerate(stages):
            if j == run_index:
                ev[it][0].record(stream)
            f()
            if j == run_index:
                ev[it][1].record(stream)
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / K
    return ms_step, np.array([a.elapsed_time(b) for a, b in ev])


def stage_times(stages, stream, K: int):
    """K more steps with a HIP event between every two stages: ms per stage, [K, len(stages)]."""
    import torch
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)] for _ in range(K)]
    torch.cuda.synchronize()
    for it in range(K):
        ev[it][0].record(stream)
        for j, f in enumerate(stages):
            f()
            ev[it][j + 1].record(stream)
    torch.cuda.synchronize()
    return np.array([[ev[i][j].elapsed_time(ev[i][j + 1]) for j in range(len(stages))] for i in range(K)])


def kept_flop_count(mask_np, Lq: int, Lk: int, block: int, d: int) -> int:
    """4 d x (valid query rows x valid keys) summed over the kept (query block, key block) pairs:
    the two matrix products over kept blocks."""
    NQ, NK = mask_np.shape[-2], mask_np.shape[-1]
    rows = np.minimum(np.arange(1, NQ + 1) * block, Lq) - np.arange(NQ) * block
    keys = np.minimum(np.arange(1, NK + 1) * block, Lk) - np.arange(NK) * block
    kept = mask_np.reshape(-1, NQ, NK).astype(np.int64)
    return int(4 * d * (kept * rows[:, None] * keys[None, :]).sum())


def cpu_baseline(wl, inp, mask_np, target_s: float):
    """The fp64 oracle on the host, head after head (selection of the head, then fp64 attention of
    its query blocks on the GPU's mask) until about target_s seconds have passed; rate in kept
    TFLOP/s over the heads done."""
    from oracle import la_oracle as O
    threads = None
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        threads = max((i.get("num_threads", 1) for i in info), default=1)
    except Exception:
        pass
    F = wl.frame_tokens if wl.causal_frames else 0
    flops = 0
    blocks = 0
    t0 = time.perf_counter()
    heads = 0
    passes = 0
    while True:      # whole passes over the heads until about target_s of work is done
        for b in range(wl.B):
            for h in range(wl.H):
                O.select_blocks(inp["q"][b:b + 1, h:h + 1], inp["k"][b:b + 1, h:h + 1], wl.block, tau=wl.tau,
                                n_text=wl.n_text)
                for i0 in range(0, wl.nq, 8):
                    rows = [(b, h, r) for r in range(i0, min(i0 + 8, wl.nq))]
                    O.attention_rows(inp["q"], inp["k"], inp["v"], mask_np, wl.block, rows, frame_tokens=F)
                    for _, _, r in rows:
                        lo, hi = r * wl.block, min((r + 1) * wl.block, wl.Lq)
                        nk = sum(min((m + 1) * wl.block, wl.Lk) - m * wl.block for m in np.nonzero(mask_np[b, h, r])[0])
                        flops += 4 * wl.d * (hi - lo) * nk
                    blocks += len(rows)
                heads += 1
                if time.perf_counter() - t0 > target_s:
                    break
            if time.perf_counter() - t0 > target_s:
                break
        passes += 1
        if time.perf_counter() - t0 > target_s:
            break
    t_total = time.perf_counter() - t0
    return {"value": round(flops / t_total / 1e12, 5), "unit": "TFLOP/s", "cores": threads or os.cpu_count(),
            "kind": "oracle",
            "sample": f"{heads} heads ({passes} pass(es) over the {wl.B * wl.H} heads) of {wl.name}: fp64 selection of each head and fp64 attention of "
                      f"its {blocks // max(heads, 1)} query blocks on the GPU's mask; {flops / 1e9:.1f} GFLOP kept in "
                      f"{t_total:.1f} s; os.cpu_count()={os.cpu_count()}, "
                      f"affinity={len(os.sched_getaffinity(0))}"}


def device_info(dev) -> dict:
    """Name, architecture, compute units and memory of the device, and the HIP version torch uses."""
    import torch
    p = torch.cuda.get_device_properties(dev)
    return {"name": p.name, "arch": getattr(p, "gcnArchName", None), "cus": p.multi_processor_count,
            "mem_gib": round(p.total_memory / 2**30, 1), "hip": torch.version.hip}


def calibration_copy(dev):
    """Three plain 256 MiB device copies: the known byte count the PMC byte counters are scaled by."""
    import torch
    src = torch.empty(256 << 20, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def kept_flop_count_3d(mask_np, qvalid, kvalid, d: int) -> int:
    """kept_flop_count for blocks with padding: 4 d x (valid query tokens of the block) x (valid
    keys of the kept key blocks), summed over the kept (query block, key block) pairs."""
    NQ, NK = mask_np.shape[-2], mask_np.shape[-1]
    kept = mask_np.reshape(-1, NQ, NK).astype(np.int64)
    q = np.asarray(qvalid, np.int64)
    k = np.asarray(kvalid, np.int64)
    return int(4 * d * (kept * q[:, None] * k[None, :]).sum())


def prep_bytes_3d(wl, which: str) -> int:
    """Algorithmic HBM bytes of one prep launch set: the valid tokens read once, every block-major
    slot written once (bf16), the block means written (fp32).  which: "q", "kv" or "kv_chunk"."""
    BH, d, blk = wl.B * wl.H, wl.d, wl.block
    per_frame = -(-wl.Hs // wl.bh) * -(-wl.Ws // wl.bw)
    NQ = -(-wl.T_q // wl.bt) * per_frame
    NC = -(-wl.T_ctx // wl.bt) * per_frame
    NT = -(-wl.n_text // blk)
    if which == "q":
        return BH * (wl.Lq * d * 2 + NQ * blk * d * 2 + NQ * d * 4)
    if which == "kv":
        return BH * (2 * wl.Lk * d * 2 + 2 * (NT + NC + NQ) * blk * d * 2 + (NT + NC + NQ) * d * 4)
    return BH * (2 * wl.Lq * d * 2 + 2 * NQ * blk * d * 2 + NQ * d * 4)


def cpu_baseline_3d(wl, inp, mask_np, qvalid, kvalid, target_s: float):
    """The fp64 oracle on the host for the 3-D layout, head after head (selection of the head over
    the block sets, then fp64 attention of its query blocks on the GPU's mask) until about
    target_s seconds have passed; rate in kept TFLOP/s (valid tokens) over the heads done."""
    from oracle import la_oracle as O
    L = O.layout_3d(wl.n_text, wl.T_ctx, wl.T_q, wl.Hs, wl.Ws, wl.bt, wl.bh, wl.bw, wl.block)
    rule = dict(tau=wl.tau) if wl.tau is not None else dict(topk_r=wl.topk_r)
    flops = heads = blocks = 0
    t0 = time.perf_counter()
    NQ = len(L["qsets"])
    while time.perf_counter() - t0 <= target_s:
        for b in range(wl.B):
            for h in range(wl.H):
                O.select_blocks_sets(inp["q"][b:b + 1, h:h + 1], inp["k"][b:b + 1, h:h + 1], L["qsets"], L["ksets"],
                                     L["forced"], **rule)
                rows = [(b, h, i) for i in range(NQ)]
                O.attention_sets_rows(inp["q"], inp["k"], inp["v"], L["qsets"], L["ksets"], mask_np, rows)
                flops += kept_flop_count_3d(mask_np[b:b + 1, h:h + 1], qvalid, kvalid, wl.d)
                blocks += NQ
                heads += 1
                if time.perf_counter() - t0 > target_s:
                    break
            if time.perf_counter() - t0 > target_s:
                break
    t_total = time.perf_counter() - t0
    threads = None
    try:
        import threadpoolctl
        threads = max((i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()), default=1)
    except Exception:
        pass
    return {"value": round(flops / t_total / 1e12, 5), "unit": "TFLOP/s", "cores": threads or os.cpu_count(),
            "kind": "oracle",
            "sample": f"{heads} heads of {wl.name}: fp64 selection of each head over the 3-D block sets and fp64 "
                      f"attention of its {NQ} query blocks on the GPU's mask; {flops / 1e9:.1f} GFLOP kept in "
                      f"{t_total:.1f} s; os.cpu_count()={os.cpu_count()}, affinity={len(os.sched_getaffinity(0))}"}


def main_3d(args, wl):
    """The 3-D block path: Q-Prep, KV-Prep, selection from the pooled means, attention (plan, run,
    merge) over the block-major buffers, Untile Scatter; the attention kernel timed with HIP events
    in the timed steps, every stage in a second loop."""
    import torch
    from paper_2605_31158_amd import la
    from paper_2605_31158_amd.workloads import make_inputs_3d

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t_gen = time.perf_counter()
    inp = make_inputs_3d(wl)
    g = {x: la.bf16_from_bits(inp[x], dev) for x in "qkv"}
    t_gen = time.perf_counter() - t_gen
    B, H, d, blk = wl.B, wl.H, wl.d, wl.block
    grid = la.grid3d(B, H, d, wl.n_text, wl.T_ctx, wl.T_q, wl.Hs, wl.Ws, wl.bt, wl.bh, wl.bw, blk)
    shape = la.grid3d_shape(grid)
    qv, kv = la.grid3d_valid(grid)
    NQ, NK = shape.Lq // blk, shape.Lk // blk
    M = (shape.Lk - shape.Lq - shape.n_text) // blk
    keep_blocks = None if wl.tau is not None else int(math.floor(wl.topk_r * M))
    ws = torch.empty(max(la.workspace_bytes(shape), 256), dtype=torch.uint8, device=dev)
    q_t = torch.empty((B, H, shape.Lq, d), dtype=torch.bfloat16, device=dev)
    k_t = torch.empty((B, H, shape.Lk, d), dtype=torch.bfloat16, device=dev)
    v_t = torch.empty_like(k_t)
    qbar = torch.empty((B, H, NQ, d), dtype=torch.float32, device=dev)
    kbar = torch.empty((B, H, NK, d), dtype=torch.float32, device=dev)
    mask = torch.empty((B, H, NQ, NK), dtype=torch.uint8, device=dev)
    counts = torch.empty((B, H, NQ), dtype=torch.int32, device=dev)
    idx = torch.empty((B, H, NQ, NK), dtype=torch.int32, device=dev)
    kvalid = torch.from_numpy(kv).to(dev)
    o_t = torch.empty_like(q_t)
    o = torch.empty_like(g["q"])
    stream = torch.cuda.current_stream(dev)
    stages = la.bind_3d(grid, g["q"], g["k"], g["v"], q_t, k_t, v_t, qbar, kbar, mask, counts, idx, kvalid, o_t,
                        None, o, None, ws, tau=wl.tau, keep_blocks=keep_blocks)
    names = ("prep_q", "prep_kv", "select", "attn_plan", "attn_run", "attn_merge", "untile")
    if args.calibrate_copy:
        calibration_copy(dev)
    cw = clock_warmup(stages, 0.0 if args.profile_only else args.clock_warmup_ms)
    for _ in range(args.warmup):
        for f in stages:
            f()
    torch.cuda.synchronize()
    K = args.steps
    ms_step, t_run = timed_steps(stages, names.index("attn_run"), stream, K)
    st_ms = stage_times(stages, stream, K)
    t = {n: float(np.mean(st_ms[:, j])) for j, n in enumerate(names)}
    t["attn_run"] = float(np.mean(t_run))

    mask_np = mask.cpu().numpy()
    kept_flops = float(kept_flop_count_3d(mask_np, qv, kv, d))
    dense_flops = float(kept_flop_count_3d(np.ones_like(mask_np), qv, kv, d))
    rho = kept_flops / dense_flops

    def time_calls(calls, n):
        for _ in range(2):
            for f in calls:
                f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(n):
            for f in calls:
                f()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    # the chunk's K/V only (text and context regions kept from an earlier call)
    chunk_kv = la.bind_3d(grid, g["q"], g["k"], g["v"], q_t, k_t, v_t, qbar, kbar, mask, counts, idx, kvalid, o_t,
                          None, o, None, ws, tau=wl.tau, keep_blocks=keep_blocks, parts=la.LA_PART_CHUNK)[1]
    chunk_kv_ms = time_calls([chunk_kv], max(3, min(K, 10)))
    dense_ms = None
    if not args.no_dense and not args.profile_only:
        dmask = torch.ones_like(mask)
        dcounts, didx = la.mask_to_list(dmask, blk, shape.Lq, shape.Lk, d)
        dsteps = la.bind_3d(grid, g["q"], g["k"], g["v"], q_t, k_t, v_t, qbar, kbar, dmask, dcounts, didx, kvalid,
                            o_t, None, o, None, ws, tau=1.0)[3:6]
        dense_ms = time_calls(dsteps, max(3, min(K, 10)))
        del dmask, dcounts, didx, dsteps

    att_ms = t["attn_plan"] + t["attn_run"] + t["attn_merge"]
    run_ms = t["attn_run"]
    value = kept_flops / (ms_step * 1e-3) / 1e12
    achieved = kept_flops / (run_ms * 1e-3) / 1e12
    bq, bkv, bkc = prep_bytes_3d(wl, "q"), prep_bytes_3d(wl, "kv"), prep_bytes_3d(wl, "kv_chunk")
    digest = src_digest("attn.hip")
    out = {
        "metric": "sparse AR attention kept-block TFLOP/s (3-D blocks: prep + select + sparse attention + untile "
                  "per call)",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "clock_warmup": {"steps": cw[0], "ms": cw[1]},
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "B": B, "H": H, "d": d, "n_text": wl.n_text, "T_ctx": wl.T_ctx,
                   "T_q": wl.T_q, "latent": [wl.Hs, wl.Ws], "block3d": [wl.bt, wl.bh, wl.bw], "block": blk,
                   "tau": wl.tau, "topk_r": wl.topk_r, "keep_blocks": keep_blocks, "seed": wl.seed},
        **{f"{n}_ms": round(t[n], 4) for n in names},
        "prep_kv_chunk_ms": round(chunk_kv_ms, 4),
        "prep_q_gbs": round(bq / (t["prep_q"] * 1e-3) / 1e9, 1),
        "prep_kv_gbs": round(bkv / (t["prep_kv"] * 1e-3) / 1e9, 1),
        "prep_kv_chunk_gbs": round(bkc / (chunk_kv_ms * 1e-3) / 1e9, 1),
        "untile_gbs": round(B * H * wl.Lq * d * 4 / (t["untile"] * 1e-3) / 1e9, 1),
        "attn_ms": round(att_ms, 4),
        "keep_ratio": round(rho, 5),
        "padded_slot_fraction_q": round(1 - float(qv.sum()) / (NQ * blk), 4),
        "kept_tflop": round(kept_flops / 1e12, 5),
        "attn_run_tflops": round(achieved, 2),
        "attn_run_pct_mfma_peak": round(100 * achieved / MFMA_BF16_PEAK_TFLOPS, 2),
        "dense_attn_ms": None if dense_ms is None else round(dense_ms, 4),
        "speedup_vs_dense": None if dense_ms is None else round(dense_ms / (t["select"] + att_ms), 3),
        "ideal_speedup": round(1.0 / rho, 3),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
                     "traffic": traffic_from_profile("attn_fwd", wl.name, digest, kept_flops),
                     "kernel": f"attn_fwd_kernel<{d}>", "src_digest": digest},
        "gpu": device_info(dev),
        "gen_s": round(t_gen, 2),
    }
    # latent dynamics (Sec. 3.1) once per AR step: a chunk latent of 4 frames of 30x52 tokens x 64
    # values (fp32), and a 256 Mi-value pair that shows the kernel's bandwidth
    mse = {}
    for label, nval in (("chunk", wl.T_q * wl.Hs * wl.Ws * 64), ("256Mi", 1 << 28)):
        za = torch.randn(nval, device=dev)
        zb = torch.randn(nval, device=dev)
        mws = torch.empty(la.LATENT_MSE_WS_BYTES, dtype=torch.uint8, device=dev)
        mout = torch.empty(1, dtype=torch.float64, device=dev)
        ms = time_calls([lambda: la.latent_mse(za, zb, ws=mws, out=mout)], 20)
        mse[label] = {"values": nval, "us": round(ms * 1e3, 2), "gbs": round(2 * 4 * nval / (ms * 1e-3) / 1e9, 1)}
        del za, zb
    out["latent_mse"] = mse
    if not args.no_cpu_baseline and not args.profile_only:
        out["cpu_baseline"] = cpu_baseline_3d(wl, inp, mask_np, qv, kv, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (one GPU's share of the "
              "heads is the unit of work). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2605_31158_amd import la
    from paper_2605_31158_amd.workloads import WORKLOADS, WORKLOADS_3D, make_inputs

    if args.workload in WORKLOADS_3D:
        return main_3d(args, WORKLOADS_3D[args.workload])
    wl = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t_gen = time.perf_counter()
    inp = make_inputs(wl)
    g = {x: la.bf16_from_bits(inp[x], dev) for x in "qkv"}
    t_gen = time.perf_counter() - t_gen
    B, H, Lq, d = wl.B, wl.H, wl.Lq, wl.d
    NQ, NK = wl.nq, wl.nk
    F = wl.frame_tokens if wl.causal_frames else 0
    shape = la.make_shape(B, H, Lq, wl.Lk, d, wl.block, wl.n_text, F)
    ws = torch.empty(max(la.workspace_bytes(shape), 256), dtype=torch.uint8, device=dev)
    mask = torch.empty((B, H, NQ, NK), dtype=torch.uint8, device=dev)
    counts = torch.empty((B, H, NQ), dtype=torch.int32, device=dev)
    idx = torch.empty((B, H, NQ, NK), dtype=torch.int32, device=dev)
    o = torch.empty_like(g["q"])
    stream = torch.cuda.current_stream(dev)
    # the calls with their arguments marshalled once, so that the host stays ahead of the GPU
    select = la.bind_select(g["q"], g["k"], wl.block, wl.tau, mask, counts, idx, ws, n_text=wl.n_text)
    plan, run, merge = la.bind_attn_steps(g["q"], g["k"], g["v"], counts, idx, wl.block, o, ws, n_text=wl.n_text,
                                          frame_tokens=F)
    stages = (select, plan, run, merge)

    if args.calibrate_copy:
        calibration_copy(dev)
    cw = clock_warmup(stages, 0.0 if args.profile_only else args.clock_warmup_ms)
    for _ in range(args.warmup):
        for f in stages:
            f()
    torch.cuda.synchronize()
    K = args.steps
    ms_step, t_run = timed_steps(stages, 2, stream, K)
    st_ms = stage_times(stages, stream, K)
    t_sel, t_plan, t_run_b, t_merge = (st_ms[:, j] for j in range(4))
    t_att = t_plan + t_run_b + t_merge

    mask_np = mask.cpu().numpy()
    kept_flops = float(kept_flop_count(mask_np, Lq, wl.Lk, wl.block, d))
    dense_flops = 4.0 * B * H * Lq * wl.Lk * d
    rho = kept_flops / dense_flops

    # dense baseline: the same attention steps over every key block
    dense_ms = None
    if not args.no_dense and not args.profile_only:
        dmask = torch.ones_like(mask)
        dcounts, didx = la.mask_to_list(dmask, wl.block, Lq, wl.Lk, d)
        dsteps = la.bind_attn_steps(g["q"], g["k"], g["v"], dcounts, didx, wl.block, o, ws, n_text=wl.n_text,
                                    frame_tokens=F)
        for _ in range(2):
            for f in dsteps:
                f()
        torch.cuda.synchronize()
        nd = max(3, min(K, 10))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(nd):
            for f in dsteps:
                f()
        e1.record(stream)
        torch.cuda.synchronize()
        dense_ms = e0.elapsed_time(e1) / nd
        del dmask, dcounts, didx, dsteps

    # selection of a denoising step with the context's key means kept from an earlier call (the
    # paper pools K once, when it enters the KV buffer): pool Q, then select from the means
    kbar = la.pool_blocks(g["k"], wl.block, "k", shape)
    qbar = torch.empty((B, H, NQ, d), dtype=torch.float32, device=dev)
    cmask, ccounts, cidx = torch.empty_like(mask), torch.empty_like(counts), torch.empty_like(idx)
    cached = la.bind_select_cached(g["q"], wl.block, wl.tau, kbar, qbar, cmask, ccounts, cidx, ws, wl.Lk,
                                   n_text=wl.n_text)
    for _ in range(2):
        for f in cached:
            f()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(K):
        for f in cached:
            f()
    e1.record(stream)
    torch.cuda.synchronize()
    sel_cached_ms = e0.elapsed_time(e1) / K
    cached_same = bool(torch.equal(cmask, mask) and torch.equal(ccounts, counts))
    del kbar, qbar, cmask, ccounts, cidx

    # cold caches: a 512 MiB write between calls evicts the L2s and the 256 MB MALL
    cold_run_ms = None
    if args.cold and not args.profile_only:
        scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
        # the selections above used the workspace that holds the attention plan: plan again
        plan()
        torch.cuda.synchronize()
        ts = []
        for _ in range(max(3, min(K, 10))):
            scratch.fill_(1)
            c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            c0.record(stream)
            run()
            c1.record(stream)
            torch.cuda.synchronize()
            ts.append(c0.elapsed_time(c1))
        cold_run_ms = float(np.median(ts))
        del scratch

    sel_ms = float(np.mean(t_sel))
    att_ms = float(np.mean(t_att))
    run_ms = float(np.mean(t_run))
    value = kept_flops / (ms_step * 1e-3) / 1e12
    achieved = kept_flops / (run_ms * 1e-3) / 1e12
    hbm_sel_bytes = 2.0 * B * H * (Lq + (wl.Lk - Lq - wl.n_text)) * d + mask_np.size * (1 + 4) + counts.numel() * 4
    digest = src_digest("attn.hip")
    traffic = traffic_from_profile("attn_fwd", wl.name, digest, kept_flops)

    out = {
        "metric": "sparse AR attention kept-block TFLOP/s (select + sparse attention per call)",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "clock_warmup": {"steps": cw[0], "ms": cw[1]},
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "B": B, "H": H, "d": d, "Lq": Lq, "Lk": wl.Lk, "block": wl.block,
                   "tau": wl.tau, "frame_causal": bool(F), "seed": wl.seed},
        "select_ms": round(sel_ms, 4),
        "attn_ms": round(att_ms, 4),
        "attn_ms_p10_p90": [round(float(np.percentile(t_att, 10)), 4), round(float(np.percentile(t_att, 90)), 4)],
        "attn_plan_ms": round(float(np.mean(t_plan)), 4),
        "attn_run_ms": round(run_ms, 4),
        "attn_merge_ms": round(float(np.mean(t_merge)), 4),
        "keep_ratio": round(rho, 5),
        "kept_tflop": round(kept_flops / 1e12, 5),
        "attn_tflops": round(kept_flops / (att_ms * 1e-3) / 1e12, 2),
        "attn_run_tflops": round(achieved, 2),
        "attn_run_pct_mfma_peak": round(100 * achieved / MFMA_BF16_PEAK_TFLOPS, 2),
        "select_gbs": round(hbm_sel_bytes / (sel_ms * 1e-3) / 1e9, 1),
        "select_pct_hbm_peak": round(100 * hbm_sel_bytes / (sel_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 1),
        "median_ms": {"select": round(float(np.median(t_sel)), 4), "attn": round(float(np.median(t_att)), 4),
                      "attn_run": round(float(np.median(t_run)), 4)},
        "cold_attn_run_ms": None if cold_run_ms is None else round(cold_run_ms, 4),
        "dense_attn_ms": None if dense_ms is None else round(dense_ms, 4),
        "dense_tflops": None if dense_ms is None else round(dense_flops / (dense_ms * 1e-3) / 1e12, 2),
        "speedup_vs_dense": None if dense_ms is None else round(dense_ms / (sel_ms + att_ms), 3),
        "ideal_speedup": round(1.0 / rho, 3),
        "select_cached_kmeans_ms": round(sel_cached_ms, 4),
        "select_cached_same_mask": cached_same,
        "speedup_vs_dense_cached_kmeans": None if dense_ms is None else round(dense_ms / (sel_cached_ms + att_ms), 3),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
                     "traffic": traffic, "kernel": f"attn_fwd_kernel<{d}>", "src_digest": digest},
        "gpu": device_info(dev),
        "gen_s": round(t_gen, 2),
    }
    if not args.no_cpu_baseline and not args.profile_only:
        out["cpu_baseline"] = cpu_baseline(wl, inp, mask_np, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
