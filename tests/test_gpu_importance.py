"""GPU parity of kvb_chunk_importance (Sec. 4.4 importance equation) from fewer
key vectors per chunk and call than the workgroup takes in one round (128,
eight lanes each) to many rounds (9,216), both head sizes, float32 and
float64 keys.  Against the oracle's mean
key norm (double sums in another order: relative 1e-12), the same eviction
order, bit-identical results on a repeated call, and accumulation over calls
equal to one call over all layers up to rounding."""
import sys

import numpy as np
import pytest
import torch

from oracle import importance as oimp

pytestmark = pytest.mark.gpu

SHAPES = [  # (chunks, layers per call, kv heads, head dim, dtype)
    (5, 1, 1, 128, np.float64),   # 128 vectors: one round of 1024 lanes
    (7, 1, 2, 64, np.float32),    # 256 vectors: two rounds
    (3, 2, 2, 128, np.float32),   # 512 vectors
    (4, 4, 2, 128, np.float64),   # 1024 vectors
    (2, 36, 2, 128, np.float32),  # 9216 vectors: 72 rounds
    (3, 3, 1, 64, np.float64),    # 384 vectors, d = 64
]


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"P{s[0]}_L{s[1]}_H{s[2]}_d{s[3]}_{np.dtype(s[4]).name}")
def test_importance_shapes(shape):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21362_amd import kvb

    P, L, H, d, dt = shape
    _say(f"[importance] P={P} L={L} H={H} d={d} {np.dtype(dt).name}")
    rng = np.random.default_rng(P * 1000 + L * 10 + H)
    scales = np.exp(rng.uniform(np.log(0.1), np.log(10.0), size=d))
    k = (rng.standard_normal((P, L, H, 128, d)) * scales).astype(dt)
    pool = kvb.pool_layout(L, H, d, 8, 128, d)
    kin = torch.from_numpy(k).cuda()
    kdt = kvb.KVB_F64 if dt == np.float64 else kvb.KVB_F32
    imp = torch.zeros(P, dtype=torch.float64, device="cuda")
    kvb.kvb_chunk_importance(pool, P, L, kdt, kin, imp)
    imp2 = torch.zeros_like(imp)
    kvb.kvb_chunk_importance(pool, P, L, kdt, kin, imp2)
    torch.cuda.synchronize()
    g, g2 = imp.cpu().numpy(), imp2.cpu().numpy()
    assert np.array_equal(g.view(np.uint64), g2.view(np.uint64)), "not deterministic"
    r = oimp.chunk_importance(k)
    np.testing.assert_allclose(g, r, rtol=1e-12, atol=0)
    assert np.array_equal(np.argsort(g, kind="stable"), np.argsort(r, kind="stable"))
    if L > 1:
        # layer by layer adds up to the same value
        acc = torch.zeros_like(imp)
        for l in range(L):
            kvb.kvb_chunk_importance(pool, P, 1, kdt, torch.from_numpy(
                np.ascontiguousarray(k[:, l:l + 1])).cuda(), acc)
        torch.cuda.synchronize()
        np.testing.assert_allclose(acc.cpu().numpy(), r, rtol=1e-12, atol=0)
