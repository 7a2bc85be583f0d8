"""Seeded random 3-D block layouts through the whole 3-D path against the fp64 oracle.

Each case draws a latent grid (frame height and width, context and chunk frame counts), a
block shape bt x bh x bw that fits in the block's slots (not necessarily filling them), text
tokens, head dim and a selection rule; the GPU runs Q-Prep, KV-Prep, selection from the pooled
means, attention with the padding masked and Untile Scatter.  The mask is checked against the
oracle's block-set selection and every output row against the oracle's attention on the
GPU's mask.  The cases are fixed by the seed below.
"""
import numpy as np
import pytest

from oracle import la_oracle as O
from paper_2605_31158_amd.workloads import Workload3D, make_inputs_3d
from helpers import say, tau32, check_list, check_selection
from test_3d_gpu import layout_of, run_path, rule_args, compare_rows

pytestmark = pytest.mark.gpu


def _draw_cases(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for c in range(n):
        block = int(rng.choice([64, 128]))
        while True:
            bt, bh, bw = int(rng.choice([1, 2, 4])), int(rng.choice([1, 2, 4, 8])), int(rng.choice([1, 2, 4, 8, 16]))
            if bt * bh * bw <= block and bt * bh * bw >= block // 4:
                break
        d = int(rng.choice([64, 128]))
        n_text = int(rng.choice([0, int(rng.integers(1, 2 * block + 1))]))
        tau, topk_r = (float(rng.uniform(0.3, 0.99)), None) if rng.random() < 0.5 else (None, float(rng.uniform(0, 1)))
        out.append(Workload3D(f"r{c}", int(rng.integers(1, 3)), int(rng.integers(1, 3)), d, n_text,
                              int(rng.integers(0, 6)), int(rng.integers(1, 4)), int(rng.integers(1, 25)),
                              int(rng.integers(1, 41)), bt, bh, bw, block, 5000 + c, int(rng.integers(0, 4)),
                              int(rng.integers(0, 3)), tau=tau, topk_r=topk_r))
    return out


CASES = _draw_cases(30, 20261203)


def _case_id(wl):
    rule = f"tau{wl.tau:.2f}" if wl.tau is not None else f"r{wl.topk_r:.2f}"
    return (f"{wl.name}-B{wl.B}H{wl.H}-d{wl.d}-t{wl.n_text}-T{wl.T_ctx}+{wl.T_q}-{wl.Hs}x{wl.Ws}-"
            f"{wl.bt}x{wl.bh}x{wl.bw}in{wl.block}-{rule}")


@pytest.mark.parametrize("wl", CASES, ids=[_case_id(w) for w in CASES])
def test_random_3d_path(wl):
    say(f"[random-3d] {_case_id(wl)}")
    inp = make_inputs_3d(wl)
    L = layout_of(wl)
    M = int((~L["forced"]).sum())
    gargs, oargs = rule_args(wl, M)
    o, lse, mask, counts, idx = run_path(wl, inp, **gargs)
    sel = O.select_blocks_sets(inp["q"], inp["k"], L["qsets"], L["ksets"], L["forced"], **oargs)
    check_selection(mask, sel)
    check_list(mask, counts, idx)
    rows = [(b, h, i) for b in range(wl.B) for h in range(wl.H) for i in range(len(L["qsets"]))]
    compare_rows(o, lse, inp, L, mask, rows, _case_id(wl))
