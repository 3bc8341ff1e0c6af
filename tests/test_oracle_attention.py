"""Pins of the oracle's patch (Alg. 2 step 4) and sparse-query causal GQA
attention (Eq. 2): dense brute force, torch's scaled_dot_product_attention
(float64, GQA), the full-recompute special case, and closed-form invariants."""
import numpy as np
import pytest
import torch

import kvb_workload as kw
from oracle import attention, numerics, path, populate


def _data(T, Hq, Hkv, d, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    q = numerics.f32_to_bf16_bits(rng.standard_normal((T, Hq, d)).astype(np.float32) * scale)
    k = numerics.f32_to_bf16_bits(rng.standard_normal((Hkv, T, d)).astype(np.float32) * scale)
    v = numerics.f32_to_bf16_bits(rng.standard_normal((Hkv, T, d)).astype(np.float32) * 3)
    return q, k, v


@pytest.mark.parametrize("Hq,Hkv", [(4, 2), (8, 1), (2, 2)])
def test_sparse_rows_match_dense_brute_force(Hq, Hkv):
    T, d = 96, 32
    q, k, v = _data(T, Hq, Hkv, d, 0, scale=2.0)
    cu = np.array([0, 40, 96], np.int32)
    rows = np.array([0, 3, 39, 40, 41, 70, 95], np.int32)
    ours = attention.attend_rows(q, k, v, rows, cu)
    ref = attention.full_causal_reference(q, k, v, cu)[rows]
    assert np.max(np.abs(ours - ref)) < 1e-12


def test_matches_torch_sdpa_gqa_float64():
    T, Hq, Hkv, d = 80, 8, 2, 64
    q, k, v = _data(T, Hq, Hkv, d, 1, scale=1.5)
    f = lambda x: torch.from_numpy(numerics.bf16_bits_to_f32(x).astype(np.float64))
    tq = f(q).permute(1, 0, 2)[None]      # [1][Hq][T][d]
    tk, tv = f(k)[None], f(v)[None]       # [1][Hkv][T][d]
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True, enable_gqa=True)
    ref = ref[0].permute(1, 0, 2).numpy()
    ours = attention.attend_rows(q, k, v, np.arange(T), np.array([0, T]))
    assert np.max(np.abs(ours - ref)) < 1e-12


def test_first_row_is_its_value_and_zero_query_is_mean():
    T, Hq, Hkv, d = 50, 4, 2, 32
    q, k, v = _data(T, Hq, Hkv, d, 2)
    cu = np.array([0, 20, 50], np.int32)
    o = attention.attend_rows(q, k, v, [0, 20], cu)
    vf = numerics.bf16_bits_to_f32(v).astype(np.float64)
    for n, t in enumerate((0, 20)):
        for h in range(Hq):
            assert np.array_equal(o[n, h], vf[(h * Hkv) // Hq, t])
    qz = np.zeros_like(q)
    o = attention.attend_rows(qz, k, v, [30], cu)
    for h in range(Hq):
        assert np.allclose(o[0, h], vf[(h * Hkv) // Hq, 20:31].mean(axis=0), atol=1e-14)


def test_future_rows_and_shared_key_shift_do_not_matter():
    T, Hq, Hkv, d = 64, 4, 2, 32
    q, k, v = _data(T, Hq, Hkv, d, 3)
    cu = np.array([0, T], np.int32)
    base = attention.attend_rows(q, k, v, [30], cu)
    k2, v2 = k.copy(), v.copy()
    k2[:, 31:] = 0x3F80
    v2[:, 31:] = 0x4000
    assert np.array_equal(attention.attend_rows(q, k2, v2, [30], cu), base)
    # the same vector added to every key shifts every score of a row equally
    kf = numerics.bf16_bits_to_f32(k).astype(np.float64)
    w = np.random.default_rng(4).standard_normal(d)
    shifted = attention.attend_rows(q, kf + w, v, [30], cu)
    assert np.max(np.abs(shifted - base)) < 1e-10


def test_every_row_selected_equals_full_prefill():
    """FULL_RECOMPUTE as the special case rho = 1: with every row selected the
    patched cache is the fresh K/V and the sparse attention is the full causal
    prefill over it (Table 1's baseline mode)."""
    w = kw.scaled(kw.WORKLOADS["tiny"], rho_num=1, rho_den=1)
    s = kw.structure(w)
    pop = populate.populate(w, s)
    r = path.run(w, s, pop)
    assert np.array_equal(r.rows[0], np.arange(w.t_total))
    full = attention.full_causal_reference(pop.q[0], pop.k_fresh[0], pop.v_fresh[0], s.cu_seqlens)
    assert np.max(np.abs(r.out[0] - full)) < 1e-12


def test_patch_copies_selected_rows_only():
    rng = np.random.default_rng(5)
    cache = rng.integers(0, 65535, (2, 40, 8)).astype(np.uint16)
    fresh = rng.integers(0, 65535, (2, 40, 8)).astype(np.uint16)
    rows = np.array([1, 7, 39])
    out = attention.patch(cache, fresh, rows)
    assert np.array_equal(out[:, rows], fresh[:, rows])
    keep = np.setdiff1d(np.arange(40), rows)
    assert np.array_equal(out[:, keep], cache[:, keep])


def test_planted_deviation_is_recovered_on_tiny():
    """Sanity (not parity): the 76 most-deviated rows of the tiny workload are
    all among its 102 rows with planted deviation."""
    w = kw.WORKLOADS["tiny"]
    s = kw.structure(w)
    pop = populate.populate(w, s)
    r = path.run(w, s, pop)
    assert len(r.rows[0]) == 76
    assert np.all(pop.noise_rows[0][r.rows[0]])
