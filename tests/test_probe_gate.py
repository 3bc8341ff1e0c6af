"""Threshold-activated probe (Sec. 7.4): the oracle's gate pinned by exact
rational comparison, and the library's host gate against the oracle."""
from fractions import Fraction

import numpy as np
import pytest

import kvb_workload as kw
from oracle import selection as osel
from paper_2608_21362_amd import kvb


def _layout(rng, n_seqs):
    lens = rng.integers(0, 40, size=n_seqs)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    cand = rng.random(int(cu[-1])) < rng.random()
    return cu, cand


def test_exact_ratio_rule_on_tiny_layouts():
    rng = np.random.default_rng(0)
    for _ in range(300):
        cu, cand = _layout(rng, int(rng.integers(1, 6)))
        k = rng.integers(0, 9, size=len(cu) - 1)
        num, den = int(rng.integers(0, 12)), int(rng.integers(1, 12))
        gk, probed = osel.probe_gate(cu, cand, k, num, den)
        for b in range(len(cu) - 1):
            n = int(cand[cu[b]:cu[b + 1]].sum())
            t = int(cu[b + 1] - cu[b])
            want = n > 0 and Fraction(n, t) >= Fraction(num, den)
            assert probed[b] == want
            assert gk[b] == (k[b] if want else 0)


def test_special_thresholds():
    cu = np.array([0, 10, 10, 30, 34], np.int32)        # prompt 1 is empty
    cand = np.zeros(34, bool)
    cand[2:7] = True                                      # prompt 0: 5 of 10
    cand[10:30] = True                                    # prompt 2: all 20
    k = np.array([3, 4, 5, 6])
    # threshold 0: every prompt with a candidate is probed
    gk, p = osel.probe_gate(cu, cand, k, 0, 1)
    assert list(p) == [True, False, True, False] and list(gk) == [3, 0, 5, 0]
    # equality probes: 5/10 reaches 1/2
    gk, p = osel.probe_gate(cu, cand, k, 1, 2)
    assert list(p) == [True, False, True, False]
    gk, p = osel.probe_gate(cu, cand, k, 51, 100)
    assert list(p) == [False, False, True, False] and list(gk) == [0, 0, 5, 0]
    # above 1: nothing is probed
    gk, p = osel.probe_gate(cu, cand, k, 101, 100)
    assert not p.any() and not gk.any()


def test_gated_selection_is_seams_and_live_rows():
    """A skipped prompt's selection is its forced rows alone: the
    SelectiveRecompute-only variant (rho = 0)."""
    w = kw.scaled(kw.WORKLOADS["qwen_1l"], n_prompts=3, chunks_per_prompt=5,
                  placement="ramp_hits", seam_left=16, seam_right=16)
    s = kw.structure(w)
    forced = osel.forced_rows(s.cu_seqlens, s.hit_row, s.chunk_starts, 16, 16)
    k = osel.k_per_prompt(s.cu_seqlens, s.hit_row, 15, 100)
    gk, probed = osel.probe_gate(s.cu_seqlens, s.hit_row, k, 1, 1)
    assert not probed.any()
    delta = np.random.default_rng(1).random(w.t_total).astype(np.float32)
    rows, _ = osel.select(delta, s.hit_row, forced, s.cu_seqlens, gk)
    assert np.array_equal(rows, np.flatnonzero(forced))


def test_ramp_placement():
    w = kw.scaled(kw.WORKLOADS["qwen_1l"], n_prompts=4, chunks_per_prompt=6,
                  placement="ramp_hits")
    s = kw.structure(w)
    per = [int(s.hit_row[s.cu_seqlens[b]:s.cu_seqlens[b + 1]].sum()) // 128 for b in range(4)]
    assert per == [0, 1, 3, 4]


def test_library_gate_matches_oracle():
    rng = np.random.default_rng(2)
    for _ in range(200):
        cu, cand = _layout(rng, int(rng.integers(1, 8)))
        flags = np.where(cand, kvb.KVB_ROW_CANDIDATE, kvb.KVB_ROW_FORCED).astype(np.uint8)
        k = rng.integers(0, 9, size=len(cu) - 1).astype(np.int32)
        num, den = int(rng.integers(0, 12)), int(rng.integers(1, 12))
        gk, n = kvb.kvb_probe_gate(cu, flags, k, num, den)
        rk, rp = osel.probe_gate(cu, cand, k, num, den)
        assert np.array_equal(gk, rk) and n == int(rp.sum())


@pytest.mark.parametrize("kwargs", [
    dict(min_den=0), dict(min_num=-1), dict(cu_seqlens=np.array([1, 4], np.int32)),
    dict(cu_seqlens=np.array([0, 4, 2], np.int32)),
])
def test_library_gate_rejects(kwargs):
    args = dict(cu_seqlens=np.array([0, 4], np.int32), row_flags=np.ones(4, np.uint8),
                k_per_seq=np.zeros(len(kwargs.get("cu_seqlens", [0, 4])) - 1, np.int32),
                min_num=1, min_den=2)
    args.update(kwargs)
    with pytest.raises(kvb.KvbError) as e:
        kvb.kvb_probe_gate(**args)
    assert e.value.status == kvb.KVB_EINVAL
