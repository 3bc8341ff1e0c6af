"""Stitch: assemble cached chunks into one prompt cache at their new positions.

Paper Sec. 4.3 (CHUNK_REUSE: matched chunks' KV concatenated in prompt order),
Sec. 3.2 (a key cached at position t needs R^Delta to be reused at t + Delta)
and Sec. 4.5 (cached chunks are stored KIVI-quantised).

For every chunk descriptor c = (pool slot p, cached position src, destination
row r0, new position dst), layer l, kv head h and token u of the chunk:

  K[l][h][r0 + u] = R^(dst - src) ( code_k * scale_k + zero_k )
  V[l][h][r0 + u] =                 code_v * scale_v + zero_v

with key statistics of token group floor(u / Gk) and value statistics of
channel group floor(j / Gv).  Values are not rotated: Eq. 3 rotates queries
and keys only.  The rotation uses the float32 table row of chunk c (computed
by ``rope.angle_table`` from Delta = dst - src).  Arithmetic is float64
(product and sum each rounded once, no fused multiply-add); the stored result
is float32 (RNE) or bfloat16 (float64 -> float32 -> bfloat16, each RNE).
"""
import numpy as np

from . import kivi, numerics, rope


def stitch_values(pool, chunks, cos, sin, layers=None):
    """Float64 stitched rows.

    ``pool``: dict with k_codes, k_scale, k_zero, v_codes, v_scale, v_zero in
    the pool layout ([P][L][Hkv][C][...]) and ints bits, k_group, v_group.
    ``chunks``: int array [n][4] = (pool_idx, src_pos, dst_row, dst_pos).
    ``cos``/``sin``: [n][d/2] float32 rotation table, row c for chunk c.

    Returns (k, v): float64 [n][len(layers)][Hkv][C][d] in descriptor order.
    """
    bits, gk, gv = pool["bits"], pool["k_group"], pool["v_group"]
    L = pool["k_codes"].shape[1]
    layers = list(range(L)) if layers is None else list(layers)
    chunks = np.asarray(chunks)
    ks, vs = [], []
    for c in range(chunks.shape[0]):
        p = int(chunks[c, 0])
        kc = kivi.unpack(pool["k_codes"][p, layers], bits)
        vc = kivi.unpack(pool["v_codes"][p, layers], bits)
        x = kivi.dequantise_keys(kc, pool["k_scale"][p, layers], pool["k_zero"][p, layers], gk)
        ks.append(rope.rotate(x, cos[c], sin[c]))
        vs.append(kivi.dequantise_values(vc, pool["v_scale"][p, layers], pool["v_zero"][p, layers], gv))
    return np.stack(ks), np.stack(vs)


def stitch_into(cache_k, cache_v, pool, chunks, cos, sin, out_dtype: str, layers=None):
    """Write the stitched rows into caches [len(layers)][Hkv][T][d].

    ``out_dtype`` "f32": caches are float32 arrays; "bf16": caches hold uint16
    bfloat16 bit patterns.  Rows outside the chunks are left untouched; with no
    chunk (nothing cached) nothing is written."""
    if np.asarray(chunks).shape[0] == 0:
        return
    k, v = stitch_values(pool, chunks, cos, sin, layers)
    C = k.shape[3]
    for c in range(k.shape[0]):
        r0 = int(chunks[c, 2])
        for dst, src in ((cache_k, k[c]), (cache_v, v[c])):
            if out_dtype == "f32":
                dst[:, :, r0:r0 + C, :] = src.astype(np.float32)
            elif out_dtype == "bf16":
                dst[:, :, r0:r0 + C, :] = numerics.to_bf16_bits_via_f32(src)
            else:
                raise ValueError(out_dtype)
