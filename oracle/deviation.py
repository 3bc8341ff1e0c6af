"""Per-token deviation, CacheBlendRecompute step 2 (paper Alg. 2):

  delta_t = 1 - 1/(|layers| * H) * sum_{l,h} cos( K_t^(l,h), K~_t^(l,h) )

between the stitched cache K and the probe-pass keys K~.

Readings:
* H is the number of KV heads (the cache holds Hkv heads under grouped-query
  attention);
* with ``per_layer`` each layer gets its own delta (one selection per layer);
  otherwise the mean runs over every layer, as Alg. 2 writes it;
* optionally the values enter with equal weight (both value tensors given);
* cos(a, b) = dot(a, b) / sqrt(|a|^2 |b|^2) in float64 over the exact float64
  images of the bfloat16 inputs; when |a|^2 |b|^2 == 0 the cosine is 1 if both
  vectors are zero and 0 otherwise.

Returns float64 [n_sets][T]; selection uses its float32 rounding.
"""
import numpy as np

from .numerics import bf16_bits_to_f32


def cosine(a, b) -> np.ndarray:
    """Row-wise cosine over the last axis, float64."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    dot = np.einsum("...i,...i->...", a, b)
    na = np.einsum("...i,...i->...", a, a)
    nb = np.einsum("...i,...i->...", b, b)
    den = na * nb
    zero = den == 0.0
    safe = np.where(zero, 1.0, den)
    c = dot / np.sqrt(safe)
    both_zero = (na == 0.0) & (nb == 0.0)
    return np.where(zero, np.where(both_zero, 1.0, 0.0), c)


def deviation(k_cache, k_fresh, v_cache=None, v_fresh=None, per_layer=True) -> np.ndarray:
    """``k_cache``/``k_fresh`` uint16 bfloat16 bits [L][Hkv][T][d] (values likewise or None)."""
    if (v_cache is None) != (v_fresh is None):
        raise ValueError("give both value tensors or neither")
    terms = [cosine(bf16_bits_to_f32(k_cache), bf16_bits_to_f32(k_fresh))]  # [L][Hkv][T]
    if v_cache is not None:
        terms.append(cosine(bf16_bits_to_f32(v_cache), bf16_bits_to_f32(v_fresh)))
    cos = np.stack(terms, axis=2)           # [L][Hkv][n_tensors][T]
    L, H, n_t, T = cos.shape
    if per_layer:
        total = cos.reshape(L, H * n_t, T).sum(axis=1)
        return 1.0 - total / float(H * n_t)
    total = cos.reshape(L * H * n_t, T).sum(axis=0)
    return (1.0 - total / float(L * H * n_t))[None, :]
