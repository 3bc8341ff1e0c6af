"""Storage-format conversions used by the oracle (test infrastructure only).

bfloat16 is the upper 16 bits of an IEEE binary32.  Rounding binary32 to
bfloat16 is round-to-nearest, ties to even on the 16 dropped bits.  NaN stays
NaN (quiet), infinities stay infinite.
"""
import numpy as np


def f32_to_bf16_bits(x) -> np.ndarray:
    """Round float32 values to bfloat16 (RNE); returns the uint16 bit patterns."""
    x = np.asarray(x, dtype=np.float32)
    shape = x.shape
    x = x.reshape(-1)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        r[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return r.reshape(shape)


def bf16_bits_to_f32(b) -> np.ndarray:
    b = np.asarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def to_bf16_bits_via_f32(x64) -> np.ndarray:
    """float64 -> float32 (RNE) -> bfloat16 (RNE), the storage rule of every
    bfloat16 tensor the path writes from a float64 value."""
    return f32_to_bf16_bits(np.asarray(x64, dtype=np.float64).astype(np.float32))


def bf16_round(x) -> np.ndarray:
    """Values of float32 ``x`` after rounding to bfloat16, as float32."""
    return bf16_bits_to_f32(f32_to_bf16_bits(x))
