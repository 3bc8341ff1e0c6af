"""kvb_select_noalloc (staging in the library's static device scratch, no
workspace) against kvb_select with a caller workspace: bit-identical rows and
row offsets on two calls in a row, the second on a smaller batch, so the
second call runs on scratch the first one left behind."""
import sys

import numpy as np
import pytest
import torch

import kvb_workload as kw
from oracle import selection as osel

pytestmark = pytest.mark.gpu


def _batch(lens, n_sets, seed):
    rng = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T, B = int(cu[-1]), len(lens)
    cand = rng.random(T) < 0.8
    forced = (~cand) | (rng.random(T) < 0.05)
    flags = (cand.astype(np.uint8) | (forced.astype(np.uint8) << 1)).astype(np.uint8)
    delta = kw.deviation_draw(n_sets, T, seed=seed, n_levels=7)
    ks = np.array([osel.k_per_prompt(cu, cand, 15 + 5 * si, 100) for si in range(n_sets)],
                  np.int32)
    return cu, T, B, flags, delta, ks


def test_select_noalloc_matches_select_twice():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21362_amd import kvb

    for lens, n_sets, seed in (([3000, 1, 4096, 777, 2500], 4, 1),   # larger first
                               ([900, 1200], 2, 2)):                  # then smaller
        cu, T, B, flags, delta, ks = _batch(lens, n_sets, seed)
        print(f"[noalloc] T={T} prompts={B} sets={n_sets}", file=sys.stderr, flush=True)
        d_cu = torch.from_numpy(cu).cuda()
        d_delta = torch.from_numpy(delta).cuda()
        d_flags = torch.from_numpy(flags).cuda()
        d_k = torch.from_numpy(ks).cuda()
        outs = []
        for noalloc in (False, True):
            rows = torch.full((n_sets, T), -1, dtype=torch.int32, device="cuda")
            cur = torch.full((n_sets, B + 1), -1, dtype=torch.int32, device="cuda")
            if noalloc:
                kvb.kvb_select_noalloc(n_sets, T, d_cu, B, d_delta, d_flags, d_k, rows, cur)
            else:
                wsb = kvb.kvb_select_workspace_bytes(n_sets, T, B)
                ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
                kvb.kvb_select(n_sets, T, d_cu, B, d_delta, d_flags, d_k, rows, cur, ws, wsb)
            torch.cuda.synchronize()
            outs.append((rows.cpu().numpy(), cur.cpu().numpy()))
        (r0, c0), (r1, c1) = outs
        assert np.array_equal(c0, c1)
        for si in range(n_sets):
            assert np.array_equal(r0[si, : c0[si, -1]], r1[si, : c1[si, -1]]), si
            # and both equal the oracle's selection on the same deviations
            cand = (flags & 1) != 0
            forced = (flags & 2) != 0
            rr, rc = osel.select(delta[si], cand, forced, cu, ks[si])
            assert np.array_equal(c1[si], rc) and np.array_equal(r1[si, : rc[-1]], rr), si
