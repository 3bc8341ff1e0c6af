"""Oracle-side preparation of the path's inputs from the seeded raw draws.

This is the cache-population side of the method (paper Sec. 4.7 ``warm``:
forward pass, KV sliced per chunk, quantised per Sec. 4.5) and the model's own
RoPE (Eq. 3), written here independently of the HIP library:

* cached chunk keys are rotated at their original positions src + u and
  quantised (Eq. 7, keys per channel); cached values are quantised per token;
* probe-pass keys and queries are rotated at their row's position in the
  prompt and stored as bfloat16, probe-pass values likewise (not rotated);
* live rows (miss chunks, sinks) enter the cache directly with their fresh
  keys and values; rows of cached chunks start as a sentinel that the stitch
  must overwrite.

Rotation and quantisation arithmetic is float64 (see ``rope`` and ``kivi``).
"""
from dataclasses import dataclass

import numpy as np

from . import importance, kivi, numerics, rope

SENTINEL_BF16 = np.uint16(0xFFFF)  # a NaN pattern no stitched value can take


@dataclass
class Populated:
    pool: dict            # pool layout arrays for the populated layers
    chunks: np.ndarray    # int32 [P][4] = pool_idx, src_pos, dst_row, dst_pos
    cos: np.ndarray       # float32 [P][d/2] rotation table of Delta = dst - src
    sin: np.ndarray
    k_fresh: np.ndarray   # uint16 [L'][Hkv][T][d]
    v_fresh: np.ndarray
    q: np.ndarray         # uint16 [L'][T][Hq][d] (None when not drawn)
    cache_k: np.ndarray   # uint16 [L'][Hkv][T][d]: live rows filled, hit rows sentinel
    cache_v: np.ndarray
    noise_rows: list      # per populated layer, bool [T]
    layers: list
    importance: np.ndarray = None  # float64 [P]: chunk importance over the populated layers


def _rotate_pool_keys(k_pool_raw, src_pos, theta):
    P, H, C, d = k_pool_raw.shape
    pos = (np.asarray(src_pos, dtype=np.int64)[:, None] + np.arange(C)[None, :])  # [P][C]
    uniq, inv = np.unique(pos.reshape(-1), return_inverse=True)
    c, s = rope.angle_table(theta, d, uniq)
    c = c[inv].reshape(P, 1, C, d // 2)
    s = s[inv].reshape(P, 1, C, d // 2)
    return rope.rotate(k_pool_raw, c, s)


def populate(w, s, layers=None, draws_fn=None, with_q=True) -> Populated:
    """``w``/``s`` from ``kvb_workload``; ``draws_fn(layer)`` returns that
    layer's ``LayerDraws``."""
    import kvb_workload as kw  # the shared seeded generator (no method arithmetic)

    layers = list(range(w.n_layers)) if layers is None else list(layers)
    if draws_fn is None:
        def draws_fn(l):
            return kw.layer_draws(w, s, l, with_q=with_q)
    P, H, C, d, T = s.n_pool, w.n_kv_heads, w.chunk_len, w.head_dim, w.t_total
    Lp = len(layers)
    cb = d * w.bits // 8
    pool = dict(
        bits=w.bits, k_group=w.k_group, v_group=w.v_group,
        k_codes=np.zeros((P, Lp, H, C, cb), np.uint8),
        v_codes=np.zeros((P, Lp, H, C, cb), np.uint8),
        k_scale=np.zeros((P, Lp, H, C // w.k_group, d), np.float32),
        k_zero=np.zeros((P, Lp, H, C // w.k_group, d), np.float32),
        v_scale=np.zeros((P, Lp, H, C, d // w.v_group), np.float32),
        v_zero=np.zeros((P, Lp, H, C, d // w.v_group), np.float32),
    )
    k_fresh = np.zeros((Lp, H, T, d), np.uint16)
    v_fresh = np.zeros((Lp, H, T, d), np.uint16)
    q = np.zeros((Lp, T, w.n_q_heads, d), np.uint16) if with_q else None
    pos = s.positions()
    noise = []
    imp = np.zeros(P, np.float64)
    for i, l in enumerate(layers):
        dr = draws_fn(l)
        noise.append(dr.noise_rows)
        if P:
            k_rot = _rotate_pool_keys(dr.k_pool_raw, s.src_pos, w.rope_theta)
            imp += importance.layer_share(k_rot[:, None], Lp)
            kc, ks, kz = kivi.quantise_keys(k_rot, w.bits, w.k_group)
            vc, vs, vz = kivi.quantise_values(dr.v_pool_raw, w.bits, w.v_group)
            pool["k_codes"][:, i] = kivi.pack(kc, w.bits)
            pool["v_codes"][:, i] = kivi.pack(vc, w.bits)
            pool["k_scale"][:, i], pool["k_zero"][:, i] = ks, kz
            pool["v_scale"][:, i], pool["v_zero"][:, i] = vs, vz
        k_fresh[i] = numerics.to_bf16_bits_via_f32(
            rope.apply_at_positions(dr.k_raw, pos, w.rope_theta, axis=-2))
        v_fresh[i] = numerics.f32_to_bf16_bits(dr.v_raw)
        if with_q:
            q[i] = numerics.to_bf16_bits_via_f32(
                rope.apply_at_positions(dr.q_raw, pos, w.rope_theta, axis=0))
    hit = s.hit_row
    cache_k = np.where(hit[None, None, :, None], SENTINEL_BF16, k_fresh).astype(np.uint16)
    cache_v = np.where(hit[None, None, :, None], SENTINEL_BF16, v_fresh).astype(np.uint16)
    chunks = np.stack([np.arange(P), s.src_pos, s.dst_row, s.dst_pos], axis=1).astype(np.int32)
    cos, sin = rope.angle_table(w.rope_theta, d, s.dst_pos.astype(np.int64) - s.src_pos)
    return Populated(pool=pool, chunks=chunks, cos=cos, sin=sin, k_fresh=k_fresh,
                     v_fresh=v_fresh, q=q, cache_k=cache_k, cache_v=cache_v,
                     noise_rows=noise, layers=layers, importance=imp)
