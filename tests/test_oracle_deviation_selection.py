"""Pins of the oracle's deviation (Alg. 2 step 2) and selection (Alg. 2 step
3, Alg. 1 windows, live rows): closed forms of the cosine, scipy's cosine
distance, brute-force ranking with numpy's lexsort, constructed ties, the
special cases k = 0 / k = n, and closed-form seam-set sizes."""
import numpy as np
import pytest
from scipy.spatial import distance

import kvb_workload as kw
from oracle import deviation, numerics, selection


def _bf16(x):
    return numerics.f32_to_bf16_bits(np.asarray(x, np.float32))


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape).astype(np.float32)


def test_identical_rows_give_exactly_zero():
    a = _bf16(_rand((2, 2, 300, 128), 0) * 7)
    assert np.all(deviation.deviation(a, a) == 0.0)
    assert np.all(deviation.deviation(a, a, a, a, per_layer=False) == 0.0)


def test_closed_forms():
    a = _rand((1, 2, 200, 128), 1)
    ka = _bf16(a)
    assert np.all(deviation.deviation(ka, _bf16(-a)) == 2.0)              # cos = -1
    assert np.all(deviation.deviation(ka, _bf16(2 * a)) == 0.0)           # exact power-of-two scale
    d3 = deviation.deviation(ka, _bf16(3 * a))
    assert np.all(np.abs(d3) <= 1e-5)                                     # bf16 rounding of 3a
    e = np.zeros((1, 2, 4, 128), np.float32)
    f = np.zeros_like(e)
    e[..., 0] = 1.0
    f[..., 1] = 5.0                                                       # orthogonal
    assert np.all(deviation.deviation(_bf16(e), _bf16(f)) == 1.0)
    z = np.zeros_like(e)
    assert np.all(deviation.deviation(_bf16(z), _bf16(z)) == 0.0)         # both zero: cos 1
    assert np.all(deviation.deviation(_bf16(z), _bf16(f)) == 1.0)         # one zero: cos 0


def test_matches_scipy_cosine_distance_and_symmetry():
    a, b = _bf16(_rand((3, 2, 50, 64), 2)), _bf16(_rand((3, 2, 50, 64), 3))
    d = deviation.deviation(a, b)
    fa, fb = numerics.bf16_bits_to_f32(a).astype(np.float64), numerics.bf16_bits_to_f32(b).astype(np.float64)
    for l in range(3):
        for t in range(50):
            ref = np.mean([distance.cosine(fa[l, h, t], fb[l, h, t]) for h in range(2)])
            assert abs(d[l, t] - ref) < 1e-14
    assert np.array_equal(d, deviation.deviation(b, a))
    assert np.all((d >= 0) & (d <= 2))


def test_all_layer_mean_is_mean_of_per_layer():
    a, b = _bf16(_rand((4, 2, 30, 64), 4)), _bf16(_rand((4, 2, 30, 64), 5))
    per = deviation.deviation(a, b, per_layer=True)
    allm = deviation.deviation(a, b, per_layer=False)
    assert np.allclose(allm[0], per.mean(axis=0), rtol=0, atol=1e-15)
    kv = deviation.deviation(a, b, a, b)
    assert np.allclose(kv, per, atol=1e-15)       # V equal to K: same mean


def _brute_select(d32, candidate, forced, cu, k):
    """numpy lexsort ranking: primary key -delta (with -0 -> +0, NaN last),
    secondary key row."""
    rows, cus = [], [0]
    for b in range(len(cu) - 1):
        lo, hi = cu[b], cu[b + 1]
        cand = np.nonzero(candidate[lo:hi])[0] + lo
        v = d32[cand].astype(np.float64) + 0.0
        v = np.where(np.isnan(v), -np.inf, v)
        order = cand[np.lexsort((cand, -v))]
        sel = np.union1d(order[: k[b]], np.nonzero(forced[lo:hi])[0] + lo)
        rows.extend(sel.tolist())
        cus.append(len(rows))
    return np.array(rows, np.int32), np.array(cus, np.int32)


@pytest.mark.parametrize("levels", [0, 3, 17])
def test_selection_matches_brute_force_with_ties(levels):
    T, B = 2048, 4
    cu = np.arange(B + 1, dtype=np.int32) * (T // B)
    rng = np.random.default_rng(levels)
    candidate = rng.random(T) < 0.7
    forced = (~candidate) | (rng.random(T) < 0.05)
    d = kw.deviation_draw(1, T, seed=levels, n_levels=levels)[0]
    d[5] = np.nan
    k = selection.k_per_prompt(cu, candidate, 15, 100)
    r, c = selection.select(d, candidate, forced, cu, k)
    rb, cb = _brute_select(d, candidate, forced, cu, k)
    assert np.array_equal(r, rb) and np.array_equal(c, cb)
    assert np.all(np.diff(r) > 0)


def test_lower_row_wins_ties_and_signed_zero():
    d = np.array([1.0, 0.5, 1.0, 0.5, 1.0, -0.0, 0.0, 0.0], np.float32)
    assert selection.top_k(d, range(8), 2) == [0, 2]
    assert selection.top_k(d, range(8), 4) == [0, 2, 4, 1]
    assert selection.top_k(d, [7, 6, 5], 2) == [5, 6]        # -0 ties +0, lower row first


def test_nan_ranks_below_every_number():
    d = np.array([np.nan, -np.inf, 0.25, np.nan, np.inf, -1.0], np.float32)
    assert selection.top_k(d, range(6), 6) == [4, 2, 5, 1, 0, 3]
    assert selection.top_k(d, range(6), 4) == [4, 2, 5, 1]


def test_k_zero_and_k_all():
    T = 300
    cu = np.array([0, T], np.int32)
    candidate = np.ones(T, bool)
    candidate[:10] = False
    forced = ~candidate
    d = kw.deviation_draw(1, T, seed=9)[0]
    r, _ = selection.select(d, candidate, forced, cu, [0])
    assert np.array_equal(r, np.arange(10))
    r, _ = selection.select(d, candidate, forced, cu, [int(candidate.sum())])
    assert np.array_equal(r, np.arange(T))


@pytest.mark.parametrize("name,expect_forced,expect_k", [
    ("tiny", 0, [76]),
    ("qwen_1l", 31 * 32, [614]),
    ("qwen_36l_8k", 0, [1228]),
    ("long_32k", 4 + 16 + 255 * 32, [4915]),
])
def test_seam_set_and_k_closed_forms(name, expect_forced, expect_k):
    w = kw.WORKLOADS[name]
    s = kw.structure(w)
    f = selection.forced_rows(s.cu_seqlens, s.hit_row, s.chunk_starts, w.seam_left, w.seam_right)
    assert int(f.sum()) == expect_forced
    k = selection.k_per_prompt(s.cu_seqlens, s.hit_row, w.rho_num, w.rho_den)
    assert k.tolist() == expect_k


def test_batched_live_rows_and_k():
    w = kw.WORKLOADS["batched_mixed"]
    s = kw.structure(w)
    f = selection.forced_rows(s.cu_seqlens, s.hit_row, s.chunk_starts, 0, 0)
    for b in range(16):
        lo, hi = s.cu_seqlens[b], s.cu_seqlens[b + 1]
        assert int(f[lo:hi].sum()) == 1024 and int(s.hit_row[lo:hi].sum()) == 1024
    assert selection.k_per_prompt(s.cu_seqlens, s.hit_row, 15, 100).tolist() == [153] * 16


def test_alg1_one_sided_window():
    """Alg. 1: rows [p - R, p) before each seam, R = 16."""
    cu = np.array([0, 512], np.int32)
    hit = np.ones(512, bool)
    f = selection.forced_rows(cu, hit, [np.array([0, 128, 256, 384])], 16, 0)
    expect = np.zeros(512, bool)
    for p in (128, 256, 384):
        expect[p - 16:p] = True
    assert np.array_equal(f, expect)


def test_kth_margin_hand_worked():
    """The margin at the top-k cut, worked by hand on values that are exact in
    float32: prompt 0 ranks its five candidates 0.875 (row 1), 0.875 (row 2),
    0.75, 0.5, 0.125 -- row 5 is live and its 0.8 must not enter; prompt 1
    ranks 0.375, -0.0 (row 8) = +0.0 (row 9), then NaN; prompt 2 two +inf then
    1; prompt 3 2, then two NaN."""
    inf = float("inf")
    d = np.array([0.5, 0.875, 0.875, 0.125, 0.75, 0.8,
                  np.nan, 0.375, -0.0, 0.0,
                  np.inf, np.inf, 1.0,
                  np.nan, np.nan, 2.0], np.float32)
    cu = np.array([0, 6, 10, 13, 16], np.int32)
    cand = np.ones(16, bool)
    cand[5] = False

    def m(ks):
        return selection.kth_margin(d, cand, cu, ks).tolist()

    assert m([1, 1, 1, 1]) == [0.0, 0.375, 0.0, inf]      # equal values tie; number | NaN is wide
    assert m([2, 2, 2, 2]) == [0.125, 0.0, inf, 0.0]      # -0 ties +0; inf | 1; NaN | NaN ties
    assert m([3, 3, 0, 0]) == [0.25, inf, inf, inf]       # k = 0: no cut
    assert m([4, 4, 3, 3]) == [0.375, inf, inf, inf]      # k = every candidate: no cut
    assert m([5, 9, 9, 9]) == [inf, inf, inf, inf]        # prompt 0 has 5 candidates
