"""Chunk importance for the cache manager's eviction order (paper Sec. 4.4,
"Memory Management and Eviction", the importance equation).

importance(C) = 1 / (L * H * |C|) * sum over layers l, kv heads h and tokens t
of the chunk of || k_t^(l,h) ||_2: the mean Euclidean norm of the chunk's
cached key vectors.

Reading (the paper does not say which copy of the keys): the keys as the chunk
is cached, i.e. rotated at the chunk's original positions and before KIVI
quantisation.  The rotation preserves norms, so the position does not matter.

Test infrastructure only: the library's kernels never call this module.
Float64 throughout.
"""
import numpy as np


def chunk_importance(k_cached):
    """``k_cached``: float [P][L][H][C][d] -> float64 [P]."""
    k = np.asarray(k_cached, dtype=np.float64)
    norms = np.sqrt(np.sum(k * k, axis=-1))  # [P][L][H][C]
    return norms.mean(axis=(1, 2, 3))


def layer_share(k_layers, n_layers_total):
    """Contribution of some layers to the importance: ``k_layers`` float
    [P][L'][H][C][d] holds L' of the ``n_layers_total`` layers; the shares of
    disjoint layer sets add up to ``chunk_importance`` of all layers."""
    k = np.asarray(k_layers, dtype=np.float64)
    P, Lp, H, C, _ = k.shape
    norms = np.sqrt(np.sum(k * k, axis=-1))
    return norms.sum(axis=(1, 2, 3)) / (n_layers_total * H * C)
