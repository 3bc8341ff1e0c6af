"""Rotary position embedding and the position correction R^Delta.

Paper, Sec. 3.2 / Eq. 3: q'_t = R^t q_t, k'_t = R^t k_t, and
q'_s . k'_t = q_s^T R^(t-s) k_t.  A key cached at position t carries R^t; reused
at position t + Delta it needs R^Delta applied on top (the "RoPE position
collision" example of Sec. 3.2).

Readings (the paper names only "R_theta^t"):
* channel pairing is the HuggingFace ``rotate_half`` one used by the Qwen2
  models the paper runs: channel i pairs with channel i + d/2, i < d/2, with
  angle p * omega_i and omega_i = theta^(-2i/d);
* rotation tables are computed in float64 with the C library's ``cos``/``sin``
  (Python's ``math`` module) and rounded once to float32; they are the form in
  which the tables enter the path;
* a rotation is applied in float64 arithmetic:
  y_i = x_i c_i - x_{i+d/2} s_i,  y_{i+d/2} = x_{i+d/2} c_i + x_i s_i
  (each product and the sum rounded once, no fused multiply-add).
"""
import math

import numpy as np


def inv_freq(theta: float, head_dim: int) -> np.ndarray:
    """omega_i = theta^(-2i/d), i < d/2, float64."""
    return np.array([math.pow(theta, -(2.0 * i) / head_dim) for i in range(head_dim // 2)],
                    dtype=np.float64)


def angle_table(theta: float, head_dim: int, offsets, dtype=np.float32):
    """cos / sin of offset * omega_i for every offset (a1: the per-chunk Delta
    table when ``offsets`` are Delta = new position - cached position).

    Returns two arrays [n][d/2]; float64 trig rounded once to ``dtype``.
    """
    w = inv_freq(theta, head_dim)
    offsets = [int(o) for o in np.asarray(offsets).reshape(-1)]
    c = np.empty((len(offsets), head_dim // 2), dtype=np.float64)
    s = np.empty_like(c)
    for n, o in enumerate(offsets):
        for i in range(head_dim // 2):
            a = float(o) * float(w[i])
            c[n, i] = math.cos(a)
            s[n, i] = math.sin(a)
    return c.astype(dtype), s.astype(dtype)


def rotate(x, cos, sin) -> np.ndarray:
    """Apply the rotation given by per-vector tables.

    ``x`` [..., d]; ``cos``/``sin`` broadcastable to [..., d/2].  Returns
    float64.  Tables of float32 are promoted exactly to float64.
    """
    x = np.asarray(x, dtype=np.float64)
    h = x.shape[-1] // 2
    c = np.asarray(cos, dtype=np.float64)
    s = np.asarray(sin, dtype=np.float64)
    lo, hi = x[..., :h], x[..., h:]
    out = np.empty_like(x)
    out[..., :h] = lo * c - hi * s
    out[..., h:] = hi * c + lo * s
    return out


_TABLES = {}


def _cached_table(theta, d, uniq, dtype):
    key = (float(theta), int(d), np.dtype(dtype).str, uniq.tobytes())
    if key not in _TABLES:
        if len(_TABLES) > 16:
            _TABLES.clear()
        _TABLES[key] = angle_table(theta, d, uniq, dtype=dtype)
    return _TABLES[key]


def apply_at_positions(x, positions, theta: float, axis: int = -2, dtype=np.float32) -> np.ndarray:
    """RoPE at absolute positions (Eq. 3): the vectors at index n along
    ``axis`` of ``x`` [..., d] are rotated by R^positions[n].  Returns float64."""
    x = np.asarray(x)
    positions = np.asarray(positions, dtype=np.int64).reshape(-1)
    d = x.shape[-1]
    uniq, inv = np.unique(positions, return_inverse=True)
    c, s = _cached_table(theta, d, uniq, dtype)
    c, s = c[inv], s[inv]
    ax = axis % x.ndim
    shape = [1] * x.ndim
    shape[ax] = positions.shape[0]
    shape[-1] = d // 2
    return rotate(x, c.reshape(shape), s.reshape(shape))
