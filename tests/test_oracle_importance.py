"""Pins of the oracle's chunk importance (Sec. 4.4 importance equation)."""
import numpy as np

from oracle import importance, rope


def test_constant_vectors_closed_form():
    # every key = c * (1, ..., 1): norm |c| sqrt(d)
    P, L, H, C, d = 3, 2, 2, 8, 64
    c = np.array([0.5, -2.0, 3.25])
    k = np.ones((P, L, H, C, d)) * c[:, None, None, None, None]
    np.testing.assert_allclose(importance.chunk_importance(k), np.abs(c) * np.sqrt(d), rtol=1e-15)


def test_unit_basis_vectors():
    # keys that are standard basis vectors have norm 1 whatever the channel
    rng = np.random.default_rng(0)
    P, L, H, C, d = 2, 3, 2, 5, 16
    k = np.zeros((P, L, H, C, d))
    idx = rng.integers(0, d, size=(P, L, H, C))
    np.put_along_axis(k, idx[..., None], 1.0, axis=-1)
    assert np.array_equal(importance.chunk_importance(k), np.ones(P))


def test_scale_equivariance_and_order():
    rng = np.random.default_rng(1)
    k = rng.standard_normal((4, 2, 2, 16, 32))
    base = importance.chunk_importance(k)
    for a in (3.0, -0.25):
        np.testing.assert_allclose(importance.chunk_importance(a * k), abs(a) * base, rtol=1e-13)
    # doubling one chunk's keys doubles its importance and leaves the others
    k2 = k.copy()
    k2[1] *= 2.0
    imp2 = importance.chunk_importance(k2)
    np.testing.assert_allclose(imp2[1], 2.0 * base[1], rtol=1e-13)
    np.testing.assert_array_equal(np.delete(imp2, 1), np.delete(base, 1))


def test_rotation_invariance():
    # RoPE at any positions preserves every key's norm (float64 tables: a
    # rotation up to rounding), so the importance of the cached keys does not
    # depend on where the chunk was cached
    rng = np.random.default_rng(2)
    P, L, H, C, d = 2, 2, 2, 16, 64
    k = rng.standard_normal((P, L, H, C, d))
    c1, s1 = rope.angle_table(1e6, d, np.arange(C) + 100, dtype=np.float64)
    c2, s2 = rope.angle_table(1e6, d, np.arange(C) + 31000, dtype=np.float64)
    r1 = rope.rotate(k, c1[None, None, None], s1[None, None, None])
    r2 = rope.rotate(k, c2[None, None, None], s2[None, None, None])
    np.testing.assert_allclose(importance.chunk_importance(r1), importance.chunk_importance(k),
                               rtol=1e-12)
    np.testing.assert_allclose(importance.chunk_importance(r2), importance.chunk_importance(k),
                               rtol=1e-12)


def test_layer_shares_add_up():
    rng = np.random.default_rng(3)
    P, L, H, C, d = 3, 5, 2, 8, 32
    k = rng.standard_normal((P, L, H, C, d))
    total = sum(importance.layer_share(k[:, [l]], L) for l in range(L))
    np.testing.assert_allclose(total, importance.chunk_importance(k), rtol=1e-13)
