"""GPU parity of kvb_stitch_deviation (stitch fused with the per-layer K
deviation of the stitched rows) against the oracle and the unfused calls.

* stitch outputs (K, V): bit-identical to kvb_stitch and to the oracle's
  stitch;
* delta at every stitched row and layer: within one float32 ulp of the
  oracle's per-layer K deviation (float64) rounded to float32;
* rows outside the stitched chunks (sinks, cache misses): delta untouched;
* fresh keys equal to the stitched cache: delta exactly 0 on every stitched row;
* selection on the fused deltas: the oracle's rows, or a valid top-k inside
  the 1e-4 band at the cut (``selection_check``).
"""
import sys

import numpy as np
import pytest
import torch

import kvb_workload as kw
from oracle import deviation as odev
from oracle import populate as opop, selection as osel, stitch as ostitch
from selection_check import check_selection

pytestmark = pytest.mark.gpu

CASES = {
    "tiny": kw.WORKLOADS["tiny"],
    "qwen_1l": kw.WORKLOADS["qwen_1l"],
    "int4_2l": kw.scaled(kw.WORKLOADS["qwen_36l_8k"], n_layers=2, chunks_per_prompt=9),
    "sinks_seams_2l": kw.scaled(kw.WORKLOADS["long_32k"], n_layers=2, chunks_per_prompt=7),
    "batched_small": kw.scaled(kw.WORKLOADS["batched_mixed"], n_prompts=3, chunks_per_prompt=5),
    "prefix_hits_2l": kw.scaled(kw.WORKLOADS["qwen_36l_8k"], n_layers=2, chunks_per_prompt=7,
                                placement="prefix_hits", hit_chunks=3, seam_left=16,
                                seam_right=16),
    # one sink row per prompt and three prompts of 641 rows: every chunk starts
    # at an odd row and t_total is not a multiple of 4 (the deviations of a
    # token quad are not 16-byte aligned)
    "sink1_3p": kw.scaled(kw.WORKLOADS["long_32k"], n_layers=2, n_prompts=3, chunks_per_prompt=5,
                          n_sinks=1),
    # the smallest key-statistic group the API takes (4 tokens): 32 groups of
    # scales and zeros per head, the largest set the fused kernel stages
    "kgroup4_2l": kw.scaled(kw.WORKLOADS["qwen_36l_8k"], n_layers=2, chunks_per_prompt=5,
                            k_group=4),
    # nothing cached: the fused call is a no-op (no row is written)
    "cold_2l": kw.scaled(kw.WORKLOADS["qwen_36l_8k"], n_layers=2, chunks_per_prompt=3,
                         placement="prefix_hits", hit_chunks=0, seam_left=16, seam_right=16),
}
UNTOUCHED = -7.0  # delta sentinel for rows the fused call must not write


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _np16(t):
    return t.detach().cpu().numpy().view(np.uint16)


def _ulp32(x):
    return np.spacing(np.abs(np.asarray(x, np.float32)))


@pytest.mark.parametrize("name", list(CASES))
def test_stitch_deviation(name):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21362_amd import pipeline

    w = CASES[name]
    s = kw.structure(w)
    _say(f"[stitch_deviation] {name}: L={w.n_layers} T={w.t_total}")
    dev = pipeline.populate(w, s)
    ref = opop.populate(w, s)
    hit = s.hit_row
    L, T = w.n_layers, w.t_total

    # unfused stitch, for bitwise comparison
    pu = pipeline.buffers(dev)
    pipeline.stitch(dev, pu)
    # fused call
    pf = pipeline.buffers(dev)
    pf.delta = torch.full((L, T), UNTOUCHED, dtype=torch.float32, device="cuda")
    pipeline.stitch_deviation(dev, pf)
    torch.cuda.synchronize()
    for a, b, nm in ((pu.k_cache, pf.k_cache, "K"), (pu.v_cache, pf.v_cache, "V")):
        assert torch.equal(a, b), f"{name}: fused {nm} differs from kvb_stitch"

    # oracle: stitch, then the per-layer K deviation
    ck, cv = ref.cache_k.copy(), ref.cache_v.copy()
    ostitch.stitch_into(ck, cv, ref.pool, ref.chunks, ref.cos, ref.sin, "bf16")
    assert np.array_equal(_np16(pf.k_cache), ck) and np.array_equal(_np16(pf.v_cache), cv)
    rd32 = odev.deviation(ck, ref.k_fresh, per_layer=True).astype(np.float32)
    gd = pf.delta.cpu().numpy()
    assert np.all(np.abs(gd[:, hit].astype(np.float64) - rd32[:, hit]) <= _ulp32(rd32[:, hit])), \
        f"{name}: fused deviation beyond 1 ulp"
    assert np.all(gd[:, ~hit] == UNTOUCHED), f"{name}: a row outside the chunks was written"
    same = float(np.mean(gd[:, hit] == rd32[:, hit])) if hit.any() else 1.0
    _say(f"[stitch_deviation] {name}: {same:.6f} of stitched rows bit-equal to the oracle; "
         f"{int((~hit).sum())} live rows untouched")

    # selection on the fused deltas (live rows are never candidates)
    if w.per_layer or L == 1:
        forced = osel.forced_rows(s.cu_seqlens, hit, s.chunk_starts, w.seam_left, w.seam_right)
        kseq = osel.k_per_prompt(s.cu_seqlens, hit, w.rho_num, w.rho_den)
        pipeline.select(dev, pf)
        torch.cuda.synchronize()
        rows, cu = pf.rows.cpu().numpy(), pf.cu_rows.cpu().numpy()
        for li in range(L):
            ref_d = rd32[li].copy()
            ref_d[~hit] = UNTOUCHED
            n_band = check_selection(rows[li, : cu[li, -1]], cu[li], ref_d, hit, forced,
                                     s.cu_seqlens, kseq, where=f"{name} layer {li}")
            if n_band:
                _say(f"[stitch_deviation] {name} layer {li}: {n_band} prompts differ inside "
                     f"the band")


@pytest.mark.parametrize("name", ["tiny", "int4_2l", "sink1_3p"])
def test_identical_rows_give_zero(name):
    """Fresh keys set to the stitched cache: every stitched row has delta = 0
    exactly (dot and both norms are summed in one order)."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21362_amd import pipeline

    w = CASES[name]
    s = kw.structure(w)
    dev = pipeline.populate(w, s)
    pb = pipeline.buffers(dev)
    pipeline.stitch(dev, pb)
    torch.cuda.synchronize()
    dev.k_fresh.copy_(pb.k_cache)
    pb.delta = torch.full((w.n_layers, w.t_total), UNTOUCHED, dtype=torch.float32, device="cuda")
    pipeline.stitch_deviation(dev, pb)
    torch.cuda.synchronize()
    gd = pb.delta.cpu().numpy()
    assert np.all(gd[:, s.hit_row] == 0.0), f"{name}: identical rows do not give delta = 0"
    assert np.all(gd[:, ~s.hit_row] == UNTOUCHED), f"{name}: a live row's delta was written"
