"""Row selection: which query rows are recomputed.

* CacheBlendRecompute step 3 (paper Alg. 2): the top floor(rho * n) rows by
  deviation, rho ~ 0.15 (Sec. 1, Sec. 4.6).
* SelectiveRecompute (Alg. 1): the rows around every chunk seam are
  recomputed.
* Live rows -- rows of chunks with no cache hit and the attention-sink rows
  (Sec. 4.1) -- are always computed.

Readings:
* candidates are the rows of cached (hit) chunks; n_b counts the candidates of
  prompt b and k_b = floor(rho * n_b) with rho = rho_num / rho_den in integers;
* order is deviation descending, then row ascending (the lower row wins a
  tie); -0.0 equals +0.0; NaN ranks below every number, -inf included;
* the decision is taken on the float32 value of the deviation;
* seams are the chunk starts p > 0 of a prompt (sink rows count as content
  before the first chunk); the window of a seam is rows
  [max(0, p - seam_left), min(T_b, p + seam_right)) of that prompt, kept only
  where they are candidates (Alg. 1 is seam_left = 16, seam_right = 0);
* top-k runs over all candidates, seam rows included, and is then united with
  the forced rows (live rows and seam windows);
* output: the selected rows of every prompt, ascending.
"""
import math

import numpy as np


def forced_rows(cu_seqlens, hit_row, chunk_starts, seam_left: int, seam_right: int) -> np.ndarray:
    """bool [T]: live rows plus seam-window candidate rows."""
    hit_row = np.asarray(hit_row, dtype=bool)
    forced = ~hit_row
    for b in range(len(cu_seqlens) - 1):
        lo, hi = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        T_b = hi - lo
        for p in chunk_starts[b]:
            p = int(p)
            if p <= 0:
                continue
            a, e = max(0, p - seam_left), min(T_b, p + seam_right)
            for r in range(lo + a, lo + e):
                if hit_row[r]:
                    forced[r] = True
    return forced


def k_per_prompt(cu_seqlens, candidate, rho_num: int, rho_den: int) -> np.ndarray:
    ks = []
    for b in range(len(cu_seqlens) - 1):
        n = int(np.count_nonzero(candidate[int(cu_seqlens[b]):int(cu_seqlens[b + 1])]))
        ks.append((rho_num * n) // rho_den)
    return np.asarray(ks, dtype=np.int64)


def probe_gate(cu_seqlens, candidate, k_per_seq, min_num: int, min_den: int):
    """Threshold-activated probe (Sec. 7.4, "Limitations": the probe pass costs
    time in proportion to the cached tokens and can be skipped when the cache
    hit ratio is below a minimum).

    Readings: the hit ratio of prompt b is n_b / T_b, its candidate (cached)
    rows over all its rows; the probe runs for prompt b iff n_b > 0 and
    n_b * min_den >= min_num * T_b (integers, so the comparison is exact); a
    prompt without the probe has no deviation to rank, so its top-k is empty
    (k_b = 0) and only its forced rows -- live rows and seam windows, i.e.
    SelectiveRecompute alone -- are recomputed.

    Returns (k_per_seq with the skipped prompts' k set to 0, bool [B] probed).
    """
    k = np.array(k_per_seq, dtype=np.int64, copy=True)
    probed = np.zeros(len(cu_seqlens) - 1, dtype=bool)
    for b in range(len(cu_seqlens) - 1):
        lo, hi = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        n = int(np.count_nonzero(candidate[lo:hi]))
        probed[b] = n > 0 and n * min_den >= min_num * (hi - lo)
        if not probed[b]:
            k[b] = 0
    return k, probed


def _rank_key(value: float, row: int):
    """Sort key: numbers by value descending (-0 as +0), then NaN; row ascending
    within equal keys."""
    v = float(value)
    if math.isnan(v):
        return (1, 0.0, row)
    if v == 0.0:
        v = 0.0
    return (0, -v, row)


def top_k(delta32, rows, k: int):
    """The first ``k`` of ``rows`` in (delta desc, row asc) order."""
    order = sorted((int(r) for r in rows), key=lambda r: _rank_key(delta32[r], r))
    return order[:k]


def select(delta32, candidate, forced, cu_seqlens, k_per_seq):
    """One selection set.  ``delta32`` float32 [T].

    Returns (rows int32 ascending over all prompts, cu_rows int32 [B+1])."""
    delta32 = np.asarray(delta32, dtype=np.float32)
    out, cu = [], [0]
    for b in range(len(cu_seqlens) - 1):
        lo, hi = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        cand = [r for r in range(lo, hi) if candidate[r]]
        chosen = set(top_k(delta32, cand, int(k_per_seq[b])))
        chosen.update(r for r in range(lo, hi) if forced[r])
        sel = sorted(chosen)
        out.extend(sel)
        cu.append(cu[-1] + len(sel))
    return np.asarray(out, dtype=np.int32), np.asarray(cu, dtype=np.int32)


def kth_margin(delta32, candidate, cu_seqlens, k_per_seq):
    """Per prompt: |delta_(k) - delta_(k+1)| of the candidate ranking, i.e. how
    far the cut of the top-k lies from the next candidate.

    inf when k is 0 or every candidate is taken (there is no cut to move).
    The ordering rule decides cuts the subtraction cannot measure: a cut
    between a number and NaN (NaN ranks below every number) is as wide as it
    gets (inf); two equal values -- -0 and +0, or the same infinity -- are a
    tie (0), settled by row order alone."""
    out = []
    for b in range(len(cu_seqlens) - 1):
        lo, hi = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        cand = [r for r in range(lo, hi) if candidate[r]]
        order = top_k(delta32, cand, len(cand))
        k = int(k_per_seq[b])
        if k == 0 or k >= len(order):
            out.append(math.inf)
            continue
        a, c = float(delta32[order[k - 1]]), float(delta32[order[k]])
        if math.isnan(a) or math.isnan(c):
            out.append(0.0 if (math.isnan(a) and math.isnan(c)) else math.inf)
        elif a == c:
            out.append(0.0)
        else:
            out.append(abs(a - c))
    return np.asarray(out)
