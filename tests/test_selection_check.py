"""The acceptance rule for GPU selections (tests/selection_check.py) on the
CPU: it accepts the oracle's own set and a swap at a cut narrower than 1e-4,
and rejects the plausible mistakes of a selection kernel -- a forced row
dropped, an extra or a missing row, a swap across a wide cut, a row outside
its prompt, rows out of order."""
import numpy as np
import pytest

from oracle import selection as osel
from selection_check import check_selection


def _case():
    # two prompts of 40 rows; candidates 0..35 of each, rows 36..39 live;
    # row 0 of each prompt is a forced (seam) candidate with a low deviation,
    # row 1 a forced candidate with the highest one
    T = 80
    cu = np.array([0, 40, 80], np.int32)
    rng = np.random.default_rng(3)
    d = rng.uniform(0.0, 1.0, T).astype(np.float32)
    cand = np.zeros(T, bool)
    forced = np.zeros(T, bool)
    for lo in (0, 40):
        cand[lo:lo + 36] = True
        forced[lo + 36:lo + 40] = True
        forced[lo] = forced[lo + 1] = True
        d[lo] = 0.001
        d[lo + 1] = 0.999
    k = np.array([6, 6])
    # prompt 1: the 6th and 7th ranked candidates 2e-5 apart (a narrow cut)
    order = osel.top_k(d, [r for r in range(40, 80) if cand[r]], 36)
    d[order[6]] = np.float32(d[order[5]] - np.float32(2e-5))
    return d, cand, forced, cu, k


def _ref(d, cand, forced, cu, k):
    return osel.select(d, cand, forced, cu, k)


def test_accepts_the_oracle_set_and_a_narrow_swap():
    d, cand, forced, cu, k = _case()
    rows, cur = _ref(d, cand, forced, cu, k)
    assert check_selection(rows, cur, d, cand, forced, cu, k) == 0
    order = osel.top_k(d, [r for r in range(40, 80) if cand[r]], 36)
    swapped = np.sort(np.concatenate([rows[rows != order[5]], [order[6]]])).astype(np.int32)
    assert check_selection(swapped, cur, d, cand, forced, cu, k) == 1


@pytest.mark.parametrize("mistake", ["drop_forced", "extra", "missing", "wide_swap",
                                     "outside", "order", "narrow_swap_prompt0"])
def test_rejects_mistakes(mistake):
    d, cand, forced, cu, k = _case()
    rows, cur = _ref(d, cand, forced, cu, k)
    rows, cur = rows.copy(), cur.copy()
    o0 = osel.top_k(d, [r for r in range(0, 40) if cand[r]], 36)
    o1 = osel.top_k(d, [r for r in range(40, 80) if cand[r]], 36)
    if mistake == "drop_forced":            # live row 39 of prompt 1 left out
        rows = rows[rows != 79]
        cur[2] -= 1
    elif mistake == "extra":                # one more candidate in prompt 1 (narrow cut)
        rows = np.sort(np.concatenate([rows, [o1[6]]]))
        cur[2] += 1
    elif mistake == "missing":              # the 6th of prompt 1 dropped (narrow cut)
        rows = rows[rows != o1[5]]
        cur[2] -= 1
    elif mistake == "wide_swap":            # prompt 1: 5th ranked for the 8th
        rows = np.sort(np.concatenate([rows[rows != o1[4]], [o1[7]]]))
    elif mistake == "outside":              # a row of prompt 1 reported in prompt 0
        rows = rows.copy()
        rows[cur[1] - 1] = 45
    elif mistake == "order":
        rows = rows.copy()
        rows[[0, 1]] = rows[[1, 0]]
    elif mistake == "narrow_swap_prompt0":  # prompt 0's cut is wide: no swap allowed
        rows = np.sort(np.concatenate([rows[rows != o0[5]], [o0[6]]]))
    with pytest.raises(AssertionError):
        check_selection(rows.astype(np.int32), cur, d, cand, forced, cu, k)
