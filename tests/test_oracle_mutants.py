"""Plant plausible mistakes in a copy of the oracle and check that the pins catch each one.

The mistakes are planted in the CPU oracle only (a source copy built in memory); the
real oracle module is never modified.
"""
import inspect
import types

import pytest

import test_oracle as T
from oracle import la_oracle

MUTANTS = {
    "score without 1/sqrt(d)": ("/ math.sqrt(d)", "/ 1.0"),
    "score with d instead of sqrt(d)": ("/ math.sqrt(d)", "/ d"),
    "ascending score order": ("np.lexsort((pos, -s_row))", "np.lexsort((pos, s_row))"),
    "ties go to the higher index": ("np.lexsort((pos, -s_row))", "np.lexsort((-pos, -s_row))"),
    "strict tau crossing": ("if cum[r] >= tau:", "if cum[r] > tau:"),
    "one block too many": ("kstar = r + 1\n", "kstar = min(r + 2, M)\n"),
    "pool divides by the block size": ("out[..., i, :] = total / (hi - lo)", "out[..., i, :] = total / block"),
    "pool drops the last token": ("for t in range(lo, hi):", "for t in range(lo, hi - 1):"),
    "chunk block overlap test": ("if hi > chunk_start:", "if lo >= chunk_start:"),
    "text ignored": ("if lo < n_text:", "if False:"),
    "frame-causal strict": ("(chunk_pos // frame_tokens) <= (t // frame_tokens)",
                            "(chunk_pos // frame_tokens) < (t // frame_tokens)"),
    "lse without the max": ("lse[has] = mx[has] + np.log(den[has])", "lse[has] = np.log(den[has])"),
    "transposed attention operand": ("logits = (qb @ kc.T) * scale", "logits = (kc @ qb.T).T * scale * 1.0001"),
    "softmax without normalisation": ("return e / e.sum(axis=-1, keepdims=True)", "return e"),
    "top-k off by one": ("kstar = max(0, min(kstar, M))", "kstar = max(0, min(kstar + 1, M))"),
    "bf16 decode shift": ("astype(np.uint32) << 16", "astype(np.uint32) << 15"),
    "kept flops drops factor": ("return int(4 * d *", "return int(2 * d *"),
    # the ambiguity band (which mask differences the GPU comparison forgives)
    "band: tie clause needs three": ("if near.sum() > 1:", "if near.sum() > 2:"),
    "band: tie clause dropped": ("                flag |= near\n", "                pass\n"),
    "band: crossing margin sign": ('if sel["tau"] - before <= tol:', 'if before - sel["tau"] <= tol:'),
    "band: crossing margin from C_k*": ("before = cum[kstar - 2] if kstar >= 2 else 0.0", "before = cum[kstar - 1]"),
    "band: first-dropped clause flags the last kept": ("flag[order[kstar]] = True", "flag[order[kstar - 1]] = True"),
    "band: first-dropped margin from C_k*-1": ('cum[kstar - 1] - sel["tau"] <= tol', 'cum[kstar - 2] - sel["tau"] <= tol'),
    "band: top-k gap test inverted": ("if lo_kept - hi_dropped <= tol:", "if lo_kept - hi_dropped > tol:"),
    "band: top-k window without tol": ("flag |= (sr >= hi_dropped - tol) & (sr <= lo_kept + tol)",
                                       "flag |= (sr >= hi_dropped) & (sr <= lo_kept)"),
    "band: candidates not mapped to blocks": ("amb[b, h, i, hist[flag]] = True", "amb[b, h, i, np.nonzero(flag)[0]] = True"),
    "band: tolerance 1e-3": ("def ambiguous_blocks(sel: Dict[str, object], tol: float = 1e-4)",
                             "def ambiguous_blocks(sel: Dict[str, object], tol: float = 1e-3)"),
    "band: tau >= 1 not exempt": ('            if sel["tau"] >= 1.0:\n                continue\n', ""),
}


def _build(old, new):
    src = inspect.getsource(la_oracle)
    assert src.count(old) >= 1, old
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, monkeypatch):
    old, new = MUTANTS[name]
    mutant = _build(old, new)
    monkeypatch.setattr(T, "O", mutant)
    caught = []
    for pin in T.ALL_PINS:
        try:
            pin()
        except Exception:          # an assertion or a crash both reveal the mistake
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake: {name}"
