"""The attention schedule checker (helpers.check_schedule) on schedules built by the rule the
library states, and on planted mistakes it must reject.  CPU only: the GPU tests run the same
checker on the plans the library builds."""
import numpy as np
import pytest

from helpers import check_schedule


def model_schedule(P, ucount, demote=True):
    """A schedule built by the stated rule: whole units in R = (U - P/4) / P rounds, XCD-major
    (workgroup l = x P/8 + c takes unit x R P/8 + r P/8 + c in round r, if that unit has at most
    T / (P R) tiles), the other units after them in unit order, and shares of the rest sized by
    the quotas max(0, ceil(T/P) - round tiles).  demote=False keeps long units in the rounds
    (a planted mistake)."""
    uc = np.asarray(ucount, np.int64)
    U = uc.size
    n = np.maximum(1, uc)
    T = int(n.sum())
    R = (U - P // 4) // P if U > P // 4 else 0
    PX = P // 8
    thr = max(1, T // (P * R)) if R > 0 else 0
    in_r = np.zeros(U, bool)
    in_r[:R * P] = (n[:R * P] <= thr) | (not demote)
    ts = np.zeros(U + 1, np.int64)
    dp = np.zeros(P + 1, np.int64)
    pos = 0
    for lam in range(P):
        dp[lam] = pos
        for r in range(R):
            u = (lam // PX) * R * PX + r * PX + lam % PX
            if in_r[u]:
                ts[u] = pos
                pos += n[u]
    dp[P] = Tdp = pos
    for u in np.nonzero(~in_r)[0]:
        ts[u] = pos
        pos += n[u]
    ts[U] = T
    q = np.maximum(0, -(-T // P) - np.diff(dp))
    Q = int(q.sum())
    qa = np.concatenate([[0], np.cumsum(q)[:-1]])
    sk = np.zeros(P + 1, np.int64)
    sk[:P] = Tdp + ((T - Tdp) * qa // Q if Q > 0 else 0)
    sk[P] = T
    return {"P": P, "U": U, "tstart": ts, "ucount": uc, "dp_start": dp, "sk_start": sk}


def cases():
    rng = np.random.default_rng(5)
    out = []
    # two rounds on 256 workgroups: short units, some long (demoted) and some empty
    uc = rng.integers(1, 40, size=640)
    uc[rng.choice(640, 20, replace=False)] = 2000
    uc[rng.choice(640, 20, replace=False)] = 0
    out.append(("rounds+long+empty", 256, uc))
    out.append(("no rounds", 256, rng.integers(0, 300, size=60)))
    out.append(("P=8 many rounds", 8, rng.integers(1, 9, size=100)))
    out.append(("equal units", 64, np.full(400, 25)))
    return out


@pytest.mark.parametrize("case", cases(), ids=[c[0] for c in cases()])
def test_rule_schedules_pass(case):
    _, P, uc = case
    s = model_schedule(P, uc)
    info = check_schedule(s)
    assert info["T"] == int(np.maximum(1, uc).sum())
    assert info["max_load"] <= -(-info["T"] // P)


def _mutants(s):
    """Planted mistakes: (name, mutated schedule)."""
    P, U = s["P"], s["U"]
    out = []
    n = np.maximum(1, s["ucount"])
    # two consecutive units of one round range swap places
    dp = s["dp_start"]
    lam = int(np.argmax(np.diff(dp)))
    if dp[lam + 1] > dp[lam]:
        inside = [u for u in range(U) if dp[lam] <= s["tstart"][u] < dp[lam + 1]]
        inside.sort(key=lambda u: s["tstart"][u])
        if len(inside) >= 2 and n[inside[0]] != n[inside[1]]:
            m = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in s.items()}
            a, b = inside[0], inside[1]
            m["tstart"][b] = m["tstart"][a]
            m["tstart"][a] = m["tstart"][b] + n[b]
            out.append(("swapped round units", m))
    # a round boundary moved by one tile
    if P > 1 and dp[1] > 0:
        m = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in s.items()}
        m["dp_start"][1] -= 1
        out.append(("round boundary inside a unit", m))
    # one share takes the next workgroup's share too
    sk = s["sk_start"]
    l2 = int(np.argmax(np.diff(sk)))
    if l2 + 2 <= P:
        m = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in s.items()}
        m["sk_start"][l2 + 1] = m["sk_start"][l2 + 2]
        out.append(("overloaded share", m))
    # two units' ranges overlap
    m = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in s.items()}
    u = int(np.argmax(m["tstart"][:U]))
    m["tstart"][u] -= 1
    out.append(("overlapping units", m))
    return out


@pytest.mark.parametrize("case", cases(), ids=[c[0] for c in cases()])
def test_planted_mistakes_fail(case):
    _, P, uc = case
    s = model_schedule(P, uc)
    muts = _mutants(s)
    assert len(muts) >= 2
    for name, m in muts:
        with pytest.raises(AssertionError):
            check_schedule(m)


def test_long_unit_left_in_rounds_fails():
    # a unit longer than T / (P R) must not be run whole in the rounds
    rng = np.random.default_rng(6)
    P = 8
    uc = rng.integers(1, 5, size=40)
    uc[3] = 500
    check_schedule(model_schedule(P, uc))
    with pytest.raises(AssertionError):
        check_schedule(model_schedule(P, uc, demote=False))


def test_row_tiles_bounds():
    # a head's unit tiles between its longest list and the sum of its lists
    s = model_schedule(8, np.array([3, 4, 5, 6] * 10))
    rows = np.array([[6, 5, 4, 3]] * 10)     # 10 heads of 4 query blocks, 4 units each
    check_schedule(s, row_tiles=rows)
    with pytest.raises(AssertionError):
        check_schedule(s, row_tiles=rows * 10)
