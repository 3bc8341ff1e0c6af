"""The whole stitched-prefill path on the CPU, step by step (oracle).

stitch (Sec. 4.3 / 3.2 / 4.5) -> deviation (Alg. 2 step 2) -> selection
(Alg. 2 step 3, Alg. 1 windows, live rows) -> patch (Alg. 2 step 4) ->
attention of the selected rows (Eq. 2).
"""
import time
from dataclasses import dataclass

import numpy as np

from . import attention, deviation, selection, stitch


@dataclass
class PathResult:
    cache_k: np.ndarray     # stitched, before the patch (uint16 [L'][Hkv][T][d])
    cache_v: np.ndarray
    delta: np.ndarray       # float64 [sets][T]
    rows: list              # per set: int32 ascending
    cu_rows: list           # per set: int32 [B+1]
    out: dict               # layer index (within populated) -> float64 [n][Hq][d]
    out_rows: dict          # layer index -> the rows ``out`` covers


def selection_inputs(w, s):
    candidate = s.hit_row.copy()
    forced = selection.forced_rows(s.cu_seqlens, s.hit_row, s.chunk_starts, w.seam_left, w.seam_right)
    k = selection.k_per_prompt(s.cu_seqlens, candidate, w.rho_num, w.rho_den)
    return candidate, forced, k


def run(w, s, pop, attend_layers=None, attend_rows=None, timings=None) -> PathResult:
    """``attend_rows``: optional callable(layer_index, selected_rows) -> the
    subset of rows to evaluate attention on (rows are independent, so a
    subset is exact for the rows it holds).  ``timings``: optional dict that
    receives the wall time in seconds of each stage ("stitch",
    "deviation_select", "patch_attention")."""
    clock = time.perf_counter
    t0 = clock()
    ck, cv = pop.cache_k.copy(), pop.cache_v.copy()
    stitch.stitch_into(ck, cv, pop.pool, pop.chunks, pop.cos, pop.sin, "bf16")
    t1 = clock()
    delta = deviation.deviation(ck, pop.k_fresh, per_layer=w.per_layer)
    d32 = delta.astype(np.float32)
    candidate, forced, k = selection_inputs(w, s)
    rows, cus = [], []
    for si in range(d32.shape[0]):
        r, cu = selection.select(d32[si], candidate, forced, s.cu_seqlens, k)
        rows.append(r)
        cus.append(cu)
    t2 = clock()
    out, out_rows = {}, {}
    Lp = ck.shape[0]
    layers = range(Lp) if attend_layers is None else attend_layers
    for i in layers:
        sel = rows[i if w.per_layer else 0]
        kp = attention.patch(ck[i], pop.k_fresh[i], sel)
        vp = attention.patch(cv[i], pop.v_fresh[i], sel)
        ev = sel if attend_rows is None else attend_rows(i, sel)
        out[i] = attention.attend_rows(pop.q[i], kp, vp, ev, s.cu_seqlens)
        out_rows[i] = np.asarray(ev, dtype=np.int32)
    t3 = clock()
    if timings is not None:
        timings.update(stitch=t1 - t0, deviation_select=t2 - t1, patch_attention=t3 - t2)
    return PathResult(cache_k=ck, cache_v=cv, delta=delta, rows=rows, cu_rows=cus,
                      out=out, out_rows=out_rows)
