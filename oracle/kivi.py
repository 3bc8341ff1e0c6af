"""KIVI asymmetric quantisation of cached chunks (paper Sec. 4.5, Eq. 7).

Eq. 7 (keys): code = round( (k - min) / (max - min) * (2^b - 1) ), with the
minimum and maximum taken per channel over tokens.  Values use the same scheme
per token, over channels.  b is 8 or 4.

Readings (the paper fixes neither group sizes nor storage):
* keys: one (min, max) per (pool slot, layer, kv head, group of Gk consecutive
  tokens of the chunk, channel);
* values: one (min, max) per (pool slot, layer, kv head, token, group of Gv
  consecutive channels);
* round is round-half-to-even; codes are clamped to [0, 2^b - 1]; a group with
  max == min gets scale 0 and codes 0;
* stored statistics are float32: scale = (max - min) / (2^b - 1), zero = min,
  each rounded once from float64; dequantised value = code * scale + zero;
* int4 codes are packed two per byte along the channel axis, the even channel
  in the low nibble.

All arithmetic here is float64; inputs may be float32 or float64.
"""
import numpy as np


def _quantise_groups(x, axis_group, bits):
    """``x`` float64 with the group members on axis ``axis_group``.
    Returns codes (same shape, uint8), scale, zero (group axis reduced, kept as size 1)."""
    levels = float((1 << bits) - 1)
    mn = x.min(axis=axis_group, keepdims=True)
    mx = x.max(axis=axis_group, keepdims=True)
    rng = mx - mn
    flat = rng == 0.0
    safe = np.where(flat, 1.0, rng)
    t = (x - mn) / safe
    code = np.rint(t * levels)
    code = np.clip(code, 0.0, levels)
    code = np.where(flat, 0.0, code)
    scale = np.where(flat, 0.0, rng / levels)
    return code.astype(np.uint8), scale.astype(np.float32), mn.astype(np.float32)


def quantise_keys(k, bits: int, k_group: int):
    """Keys [..., C, d] (C tokens of a chunk).  Per-channel statistics over
    groups of ``k_group`` tokens.

    Returns codes [..., C, d] uint8 (unpacked), scale / zero [..., C/Gk, d] float32.
    """
    k = np.asarray(k, dtype=np.float64)
    *lead, C, d = k.shape
    g = k.reshape(*lead, C // k_group, k_group, d)
    code, scale, zero = _quantise_groups(g, -2, bits)
    return (code.reshape(*lead, C, d), scale.reshape(*lead, C // k_group, d),
            zero.reshape(*lead, C // k_group, d))


def quantise_values(v, bits: int, v_group: int):
    """Values [..., C, d].  Per-token statistics over groups of ``v_group``
    channels.  Returns codes [..., C, d] uint8, scale / zero [..., C, d/Gv]."""
    v = np.asarray(v, dtype=np.float64)
    *lead, C, d = v.shape
    g = v.reshape(*lead, C, d // v_group, v_group)
    code, scale, zero = _quantise_groups(g, -1, bits)
    return (code.reshape(*lead, C, d), scale.reshape(*lead, C, d // v_group),
            zero.reshape(*lead, C, d // v_group))


def pack(codes, bits: int) -> np.ndarray:
    """Unpacked codes [..., d] -> stored bytes [..., d*bits/8]."""
    codes = np.asarray(codes, dtype=np.uint8)
    if bits == 8:
        return codes.copy()
    if np.any(codes > 15):
        raise ValueError("int4 code out of range")
    return (codes[..., 0::2] | (codes[..., 1::2] << 4)).astype(np.uint8)


def unpack(stored, bits: int) -> np.ndarray:
    """Stored bytes [..., d*bits/8] -> codes [..., d]."""
    stored = np.asarray(stored, dtype=np.uint8)
    if bits == 8:
        return stored.copy()
    out = np.empty(stored.shape[:-1] + (stored.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = stored & 0x0F
    out[..., 1::2] = stored >> 4
    return out


def dequantise_keys(codes, scale, zero, k_group: int) -> np.ndarray:
    """code * scale + zero in float64 (key statistics per Gk tokens)."""
    s = np.repeat(np.asarray(scale, np.float64), k_group, axis=-2)
    z = np.repeat(np.asarray(zero, np.float64), k_group, axis=-2)
    return np.asarray(codes, np.float64) * s + z


def dequantise_values(codes, scale, zero, v_group: int) -> np.ndarray:
    s = np.repeat(np.asarray(scale, np.float64), v_group, axis=-1)
    z = np.repeat(np.asarray(zero, np.float64), v_group, axis=-1)
    return np.asarray(codes, np.float64) * s + z
