"""Pins of the oracle's KIVI quantisation (Eq. 7) and stitch (Sec. 4.3 with
the Sec. 3.2 position correction): hand-worked cases, the round-trip error
bound of Eq. 7, and the end-to-end property that a stitched key equals the
key rotated at its new position up to the quantisation error."""
import json
import os

import numpy as np
import pytest

import kvb_workload as kw
from oracle import kivi, numerics, populate, rope, stitch

GOLD = os.path.join(os.path.dirname(__file__), "golden", "kivi_eq7_hand.json")


def test_hand_worked_eq7():
    g = json.load(open(GOLD))
    c = g["keys_b4"]
    codes, scale, zero = kivi.quantise_keys(np.array(c["x"]), c["bits"], c["k_group"])
    assert codes.tolist() == c["codes"]
    assert np.array_equal(scale, np.array(c["scale"], np.float32))
    assert np.array_equal(zero, np.array(c["zero"], np.float32))
    c = g["keys_b8_tie"]
    codes, _, _ = kivi.quantise_keys(np.array(c["x"]), c["bits"], c["k_group"])
    assert codes.tolist() == c["codes"]
    c = g["values_b8"]
    codes, _, _ = kivi.quantise_values(np.array(c["x"]), c["bits"], c["v_group"])
    assert codes.tolist() == c["codes"]
    c = g["int4_packing"]
    assert kivi.pack(np.array(c["codes"]), 4).tolist() == c["bytes"]


@pytest.mark.parametrize("bits,gk,gv", [(8, 128, 128), (4, 32, 32), (8, 128, 64)])
def test_roundtrip_error_bound(bits, gk, gv):
    """|x - (code*scale + zero)| <= scale/2, plus the float32 rounding of the
    stored scale (<= 2^-24 * (max-min)) and zero (<= 2^-24 |min|), plus the
    float64 evaluation."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, 128, 128)) * np.exp(rng.uniform(np.log(0.1), np.log(10), (1, 1, 128)))
    for quant, deq, g in ((kivi.quantise_keys, kivi.dequantise_keys, gk),
                          (kivi.quantise_values, kivi.dequantise_values, gv)):
        codes, scale, zero = quant(x, bits, g)
        assert codes.max() <= (1 << bits) - 1
        back = deq(codes, scale, zero, g)
        axis = -2 if quant is kivi.quantise_keys else -1
        s64 = np.repeat(scale.astype(np.float64), g, axis=axis)
        z64 = np.repeat(np.abs(zero.astype(np.float64)), g, axis=axis)
        rng_ = s64 * ((1 << bits) - 1)
        bound = s64 / 2 + 2.0**-24 * rng_ * 1.01 + 2.0**-24 * z64 + 1e-15 * (np.abs(x) + z64)
        assert np.all(np.abs(back - x) <= bound)


def test_group_extremes_map_to_code_range():
    rng = np.random.default_rng(6)
    x = rng.standard_normal((2, 128, 64))
    for bits in (4, 8):
        codes, _, _ = kivi.quantise_keys(x, bits, 32)
        g = codes.reshape(2, 4, 32, 64)
        assert np.all(g.min(axis=2) == 0) and np.all(g.max(axis=2) == (1 << bits) - 1)
        # monotone in x within a group
        xs = x.reshape(2, 4, 32, 64)
        order = np.argsort(xs, axis=2)
        assert np.all(np.diff(np.take_along_axis(g, order, axis=2).astype(int), axis=2) >= 0)


def test_pack_unpack_roundtrip():
    rng = np.random.default_rng(7)
    for bits in (4, 8):
        c = rng.integers(0, 1 << bits, size=(5, 128)).astype(np.uint8)
        assert np.array_equal(kivi.unpack(kivi.pack(c, bits), bits), c)


def _small(name, **kw_):
    w = kw.scaled(kw.WORKLOADS[name], **kw_)
    return w, kw.structure(w)


@pytest.mark.parametrize("name,changes", [
    ("tiny", {}),
    ("qwen_1l", dict(chunks_per_prompt=4, seam_left=16, seam_right=16)),
    ("qwen_36l_8k", dict(n_layers=2, chunks_per_prompt=3)),
    ("long_32k", dict(n_layers=1, chunks_per_prompt=3)),
])
def test_stitched_key_is_key_at_new_position(name, changes):
    """End to end through populate (rotate at src, quantise) and stitch
    (dequantise, rotate by Delta): each stitched key row is within the
    rotated quantisation error of the raw key rotated at its new position;
    each stitched value row is the plain dequantisation, unrotated."""
    w, s = _small(name, **changes)
    pop = populate.populate(w, s, with_q=False)
    k, v = stitch.stitch_values(pop.pool, pop.chunks, pop.cos, pop.sin)
    C, d = w.chunk_len, w.head_dim
    for l in range(w.n_layers):
        dr = kw.layer_draws(w, s, l, with_q=False)
        for c in range(pop.chunks.shape[0]):
            new_pos = int(pop.chunks[c, 3]) + np.arange(C)
            ref = rope.apply_at_positions(dr.k_pool_raw[c], new_pos, w.rope_theta, dtype=np.float64)
            scale = np.repeat(pop.pool["k_scale"][c, l].astype(np.float64), w.k_group, axis=-2)
            # |R(x - x_hat)| = |x - x_hat| <= |scale/2| per channel, plus float32 tables
            bound = 0.5 * np.linalg.norm(scale, axis=-1) * 1.001 + 1e-5 * np.linalg.norm(ref, axis=-1)
            err = np.linalg.norm(k[c, l] - ref, axis=-1)
            assert np.all(err <= bound)
            vdq = kivi.dequantise_values(kivi.unpack(pop.pool["v_codes"][c, l], w.bits),
                                         pop.pool["v_scale"][c, l], pop.pool["v_zero"][c, l], w.v_group)
            assert np.array_equal(v[c, l], vdq)


def test_zero_delta_reduces_to_dequantisation():
    w, s = _small("tiny")
    pop = populate.populate(w, s, with_q=False)
    chunks = pop.chunks.copy()
    chunks[:, 3] = chunks[:, 1]          # place every chunk at its cached position
    c, sn = rope.angle_table(w.rope_theta, w.head_dim, chunks[:, 3] - chunks[:, 1])
    k, _ = stitch.stitch_values(pop.pool, chunks, c, sn)
    for i in range(chunks.shape[0]):
        plain = kivi.dequantise_keys(kivi.unpack(pop.pool["k_codes"][i], w.bits),
                                     pop.pool["k_scale"][i], pop.pool["k_zero"][i], w.k_group)
        assert np.array_equal(k[i], plain)


def test_stitch_into_writes_hit_rows_only_and_bf16_is_rne_of_f32():
    w, s = _small("batched_mixed", n_prompts=2, chunks_per_prompt=4)
    pop = populate.populate(w, s, with_q=False)
    ck, cv = pop.cache_k.copy(), pop.cache_v.copy()
    stitch.stitch_into(ck, cv, pop.pool, pop.chunks, pop.cos, pop.sin, "bf16")
    live = ~s.hit_row
    assert np.array_equal(ck[:, :, live], pop.k_fresh[:, :, live])
    assert not np.any(ck[:, :, s.hit_row] == populate.SENTINEL_BF16)
    f32k = np.zeros(ck.shape, np.float32)
    f32v = np.zeros(cv.shape, np.float32)
    stitch.stitch_into(f32k, f32v, pop.pool, pop.chunks, pop.cos, pop.sin, "f32")
    assert np.array_equal(numerics.f32_to_bf16_bits(f32k)[:, :, s.hit_row], ck[:, :, s.hit_row])
