"""Acceptance rule for a selection computed on the GPU from its own
deviations (Alg. 2 step 3 with Alg. 1 windows and live rows).

Both sides rank on float32 deviations, but the GPU's deviations come from its
own float64 sums and can differ from the oracle's in the last float32 bit, so
near-equal candidates at the top-k cut can swap.  Per prompt b:

* if the oracle's k-th / (k+1)-th margin exceeds 1e-4 (or there is no cut:
  k = 0 or every candidate taken), the GPU's rows must equal the oracle's;
* otherwise the set must still be a valid top-k under the oracle's
  deviations up to the band: every forced row (live rows, seam windows) is
  selected; the selected rows that are not forced are candidates, each with
  a deviation >= delta_(k) - 1e-4, and every candidate left out has one
  <= delta_(k) + 1e-4; the top-k's remaining k_b - (non-forced rows) members
  are forced candidates, which must cover every forced candidate above
  delta_(k) + 1e-4 and may use only those at or above delta_(k) - 1e-4.

Always: rows ascending and unique inside each prompt, inside the prompt's
rows, and ``cu_rows`` consistent.
"""
import numpy as np

from oracle import selection as osel

BAND = 1e-4


def check_selection(g_rows, g_cu, delta_ref32, candidate, forced, cu_seqlens, k_per_seq,
                    where=""):
    """Assert the rule for one set; returns the number of prompts whose rows
    differ from the oracle's inside the band."""
    g_rows = np.asarray(g_rows)
    g_cu = np.asarray(g_cu)
    d = np.asarray(delta_ref32, np.float32)
    candidate = np.asarray(candidate, bool)
    forced = np.asarray(forced, bool)
    B = len(cu_seqlens) - 1
    assert len(g_cu) == B + 1 and g_cu[0] == 0 and g_cu[-1] == len(g_rows), f"{where}: cu_rows"
    assert np.all(np.diff(g_cu) >= 0), f"{where}: cu_rows not monotone"
    r_rows, r_cu = osel.select(d, candidate, forced, cu_seqlens, k_per_seq)
    margins = osel.kth_margin(d, candidate, cu_seqlens, k_per_seq)
    n_band = 0
    for b in range(B):
        lo, hi = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        S = g_rows[g_cu[b]:g_cu[b + 1]]
        R = r_rows[r_cu[b]:r_cu[b + 1]]
        assert np.all(np.diff(S) > 0), f"{where} prompt {b}: rows not ascending"
        assert np.all((S >= lo) & (S < hi)), f"{where} prompt {b}: a row outside the prompt"
        if np.array_equal(S, R):
            continue
        assert margins[b] <= BAND, \
            f"{where} prompt {b}: rows differ from the oracle's with margin {margins[b]}"
        sel = np.zeros(hi - lo, bool)
        sel[S - lo] = True
        f_b, c_b, d_b = forced[lo:hi], candidate[lo:hi], d[lo:hi].astype(np.float64)
        assert np.all(sel[f_b]), f"{where} prompt {b}: a forced row is missing"
        free = sel & ~f_b
        assert np.all(c_b[free]), f"{where} prompt {b}: a selected row is neither forced nor a candidate"
        cand_rows = [r for r in range(lo, hi) if candidate[r]]
        k = min(int(k_per_seq[b]), len(cand_rows))
        kth = float(d[osel.top_k(d, cand_rows, k)[-1]])
        # the top-k also holds k - n_free forced candidates: every one ranked
        # clearly above the cut, and none ranked clearly below it
        n_free = int(free.sum())
        fc = d_b[f_b & c_b]
        must, may = int(np.sum(fc > kth + BAND)), int(np.sum(fc >= kth - BAND))
        assert must <= k - n_free <= may, \
            f"{where} prompt {b}: {n_free} non-forced rows for k = {k} " \
            f"(forced candidates: {must} above the band, {may} within or above)"
        assert np.all(d_b[free] >= kth - BAND), f"{where} prompt {b}: a selected row below the band"
        assert np.all(d_b[c_b & ~sel] <= kth + BAND), f"{where} prompt {b}: a left-out row above the band"
        n_band += 1
    return n_band
