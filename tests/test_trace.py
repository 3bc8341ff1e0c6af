"""The synthetic request trace: its request mix (host side) and one short run
through the path on the GPU."""
import collections

import numpy as np
import pytest

from paper_2608_21362_amd import trace


def test_request_mix_follows_the_buckets():
    reqs = trace.make_requests(4000, seed=3)
    counts = collections.Counter(r[0] for r in reqs)
    paper = {label: n for label, _, _, n in trace.BUCKETS}
    total = sum(paper.values())
    for label, n in paper.items():
        # binomial standard deviation at n = 4000 is under 0.008
        assert abs(counts[label] / len(reqs) - n / total) < 0.03, label
    for label, chunks, hits in reqs:
        lo, hi = next((b[1], b[2]) for b in trace.BUCKETS if b[0] == label)
        assert -(-lo // 128) <= chunks <= -(-hi // 128)
        assert 0 <= hits <= chunks


def test_reuse_is_bimodal_with_the_paper_mean():
    reqs = trace.make_requests(4000, seed=4)
    reuse = np.array([h / c for _, c, h in reqs])
    cold = reuse == 0
    # one request in four is cold; single-chunk warm requests can round to 0 too
    assert 0.22 < cold.mean() < 0.30
    warm = reuse[~cold]
    assert warm.min() >= 0.25 and warm.max() <= 1.0
    assert abs(reuse.mean() - 0.364) < 0.03


def test_same_seed_same_trace():
    assert trace.make_requests(50, 9) == trace.make_requests(50, 9)
    assert trace.make_requests(50, 9) != trace.make_requests(50, 10)


@pytest.mark.gpu
def test_trace_runs_on_the_gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    results, summary = trace.run(n_requests=4, seed=1, n_layers=2,
                                 log=lambda m: print(m, flush=True))
    assert summary["requests"] == 4 and len(results) == 4
    for r in results:
        assert r["ms"] > 0
        hit_rows = 128 * r["cached_chunks"]
        # every live row is recomputed, and at most all rows
        assert r["tokens"] - hit_rows <= r["selected_rows"] <= r["tokens"]
    assert summary["tokens_per_s"] > 0
    # graph replays of every request reproduce its eager outputs bit for bit
    assert summary["graph_replays_equal_eager"]


@pytest.mark.gpu
def test_trace_with_probe_threshold():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    # a threshold above 100 % skips every deviation pass: only forced rows
    results, summary = trace.run(n_requests=3, seed=2, n_layers=1, probe_min_pct=101,
                                 log=lambda m: print(m, flush=True))
    assert summary["probed"] == 0 and summary["graph_replays_equal_eager"]
    for r in results:
        assert r["selected_rows"] <= r["tokens"]


@pytest.mark.gpu
def test_trace_requests_match_the_oracle():
    """Two requests of a trace, run with the calls the trace times (fused
    stitch + deviation, selection, patch of every layer, one attention call
    per layer), against the oracle on the same draws: a short warm request
    (3-4 chunks, whole-tile attention launch) and a long one (at least 20
    chunks, balanced ranges).  Stitch bit-exact, deviation within one float32 ulp,
    selection by the band rule, patch bit-exact on the GPU's rows, attention
    on every selected row of both layers within 2e-2 + 1e-2 |ref|."""
    import sys

    import torch

    import kvb_workload as kw
    from oracle import attention as oatt
    from oracle import deviation as odev
    from oracle import numerics, populate as opop, selection as osel, stitch as ostitch
    from paper_2608_21362_amd import pipeline
    from selection_check import check_selection

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    seed, n_layers = 0, 2
    reqs = trace.make_requests(12, seed)
    short = next(i for i, (_, c, h) in enumerate(reqs) if 3 <= c <= 4 and 0 < h < c)
    long_ = next(i for i, (_, c, h) in enumerate(reqs) if c >= 20 and 0 < h < c)
    for i in (short, long_):
        _, chunks, hits = reqs[i]
        w = trace.request_workload(i, chunks, hits, seed, n_layers)
        s = kw.structure(w)
        draws = trace.request_draws(w, s)
        print(f"[trace-oracle] request {i}: {chunks} chunks, {hits} cached, T={w.t_total}",
              file=sys.stderr, flush=True)
        di = pipeline.populate(w, s, draws_fn=draws)
        pb = pipeline.buffers(di)
        pipeline.stitch(di, pb)
        torch.cuda.synchronize()
        st_k, st_v = pb.k_cache.cpu().numpy().view(np.uint16), pb.v_cache.cpu().numpy().view(np.uint16)
        trace.request_calls(di, pb)
        torch.cuda.synchronize()
        ref = opop.populate(w, s, draws_fn=draws)
        ck, cv = ref.cache_k.copy(), ref.cache_v.copy()
        ostitch.stitch_into(ck, cv, ref.pool, ref.chunks, ref.cos, ref.sin, "bf16")
        assert np.array_equal(st_k, ck) and np.array_equal(st_v, cv), f"request {i}: stitch"
        hit = s.hit_row
        rd32 = odev.deviation(ck, ref.k_fresh, per_layer=True).astype(np.float32)
        gd = pb.delta.cpu().numpy()
        assert np.all(np.abs(gd[:, hit].astype(np.float64) - rd32[:, hit])
                      <= np.spacing(np.abs(rd32[:, hit]))), f"request {i}: deviation"
        forced = osel.forced_rows(s.cu_seqlens, hit, s.chunk_starts, w.seam_left, w.seam_right)
        kseq = osel.k_per_prompt(s.cu_seqlens, hit, w.rho_num, w.rho_den)
        rows, cu = pb.rows.cpu().numpy(), pb.cu_rows.cpu().numpy()
        out = pb.out.cpu().numpy().view(np.uint16)
        kc, vc = pb.k_cache.cpu().numpy().view(np.uint16), pb.v_cache.cpu().numpy().view(np.uint16)
        for li in range(n_layers):
            d_ref = rd32[li].copy()
            d_ref[~hit] = 0.0
            g_rows = rows[li, : cu[li, -1]]
            check_selection(g_rows, cu[li], d_ref, hit, forced, s.cu_seqlens, kseq,
                            where=f"request {i} layer {li}")
            pk = oatt.patch(ck[li], ref.k_fresh[li], g_rows)
            pv = oatt.patch(cv[li], ref.v_fresh[li], g_rows)
            assert np.array_equal(kc[li], pk) and np.array_equal(vc[li], pv), f"request {i}: patch"
            refo = oatt.attend_rows(ref.q[li], pk, pv, g_rows, s.cu_seqlens)
            got = numerics.bf16_bits_to_f32(out[li][g_rows]).astype(np.float64)
            err = np.abs(got - refo)
            ratio = float(np.max(err / (2e-2 + 1e-2 * np.abs(refo))))
            print(f"[trace-oracle] request {i} layer {li}: {len(g_rows)} rows, max err/tol "
                  f"{ratio:.3f}", file=sys.stderr, flush=True)
            assert ratio <= 1.0, f"request {i} layer {li}: attention error/tolerance {ratio:.3f}"
