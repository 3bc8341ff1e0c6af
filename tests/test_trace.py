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
