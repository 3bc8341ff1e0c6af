"""Patch and sparse-query causal attention.

* Patch, CacheBlendRecompute step 4 (paper Alg. 2): the cache rows of the
  selected rows are replaced by the probe-pass K~, V~ (keys and values, every
  kv head).
* Attention (Sec. 3.1, Eq. 2): for a query row t of prompt b and query head h,
  O = softmax( q . K_{<=t}^T / sqrt(d) ) V_{<=t}, over the rows
  cu_seqlens[b] .. t of the same prompt (inclusive).

Readings: grouped-query attention maps query head h to kv head
floor(h * Hkv / Hq); queries are already rotated at their positions; only the
selected rows are computed (the forward on live / recomputed tokens of
Sec. 4.7); the cache read is the patched one.  Arithmetic is float64 over the
exact float64 images of the bfloat16 inputs; softmax subtracts the row maximum.
"""
import numpy as np

from .numerics import bf16_bits_to_f32


def patch(cache, fresh, rows) -> np.ndarray:
    """Copy of ``cache`` [Hkv][T][d] with rows ``rows`` taken from ``fresh``."""
    out = np.array(cache, copy=True)
    rows = np.asarray(rows, dtype=np.int64)
    out[:, rows, :] = np.asarray(fresh)[:, rows, :]
    return out


def attend_rows(q, k, v, rows, cu_seqlens, scale=None) -> np.ndarray:
    """One layer.  ``q`` [T][Hq][d], ``k``/``v`` [Hkv][T][d] as bfloat16 bits
    (uint16) or float arrays.  Returns float64 [len(rows)][Hq][d]."""
    q = _f64(q)
    k = _f64(k)
    v = _f64(v)
    T, Hq, d = q.shape
    Hkv = k.shape[0]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    group = [np.array([h for h in range(Hq) if (h * Hkv) // Hq == g]) for g in range(Hkv)]
    out = np.empty((len(rows), Hq, d), dtype=np.float64)
    for n, t in enumerate(np.asarray(rows, dtype=np.int64)):
        b = int(np.searchsorted(cu, t, side="right") - 1)
        lo = int(cu[b])
        for g in range(Hkv):
            hs = group[g]
            # one score row per query head of the group, over keys lo..t
            s = (q[t, hs, :] @ k[g, lo:t + 1, :].T) * scale
            p = np.exp(s - s.max(axis=1, keepdims=True))
            out[n, hs, :] = (p @ v[g, lo:t + 1, :]) / p.sum(axis=1, keepdims=True)
    return out


def full_causal_reference(q, k, v, cu_seqlens, scale=None) -> np.ndarray:
    """Brute force for small inputs: the whole masked T x T score matrix per
    head, dense softmax, no per-row loop.  Returns float64 [T][Hq][d]."""
    q = _f64(q)
    k = _f64(k)
    v = _f64(v)
    T, Hq, d = q.shape
    Hkv = k.shape[0]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    prompt = np.searchsorted(cu, np.arange(T), side="right") - 1
    allowed = (np.arange(T)[None, :] <= np.arange(T)[:, None]) & (prompt[None, :] == prompt[:, None])
    out = np.empty((T, Hq, d))
    for h in range(Hq):
        g = (h * Hkv) // Hq
        s = (q[:, h, :] @ k[g].T) * scale
        s = np.where(allowed, s, -np.inf)
        e = np.exp(s - s.max(axis=1, keepdims=True))
        out[:, h, :] = (e / e.sum(axis=1, keepdims=True)) @ v[g]
    return out


def _f64(x):
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return bf16_bits_to_f32(x).astype(np.float64)
    return x.astype(np.float64)
