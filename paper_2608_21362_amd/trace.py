"""A synthetic request trace shaped like the paper's workload, run through the
path one request at a time.

The paper's benchmark (Sec. 6, "Workload") is 1,000 prompts whose shared
context documents fall in four length buckets (0-500, 500-1K, 1K-2K and 2K+
tokens: 218, 210, 204 and 368 prompts), answered in groups that reuse the same
context: the first request of a group finds nothing cached, the following
ones reuse most of the context (the per-request reuse distribution is bimodal,
near zero and around 30-50 %, mean 36.4 %).  The paper's data and model weights
are not available; this trace keeps only those shapes:

* context lengths drawn uniformly inside the buckets (the open 2K+ bucket is
  taken as 2K-3.4K, the longest context the paper mentions), with the bucket
  sizes as weights, rounded up to whole 128-token chunks;
* one request in four is cold (no chunk cached); a warm request finds a
  leading run of its chunks cached at random original offsets, the run's length
  drawn uniformly between 32 % and 65 % of the chunks (mean reuse about 36 %
  over the trace);
* the 36-layer Qwen2.5-3B attention shape, int4 KIVI chunks (groups of 32),
  16-row seam windows on both sides of every chunk boundary and rho = 0.15.

Each request runs the same calls as the benchmark's step: the fused stitch +
deviation (when anything is cached), the selection, and one attention call
per layer; a cold request therefore recomputes every row (its rows are all
live).  The time of a request is the device time of those calls (HIP events);
the model's own layers, which the paper's time-to-first-token includes, are
not part of this path.  Each request is timed eagerly and as a captured HIP
graph replay; the replay's outputs are compared with the eager ones and its
time is the request's time when they are equal.  Values are seeded synthetic draws (one layer's draw is
reused for every layer: only the shapes matter for the timing).

    python -m paper_2608_21362_amd.trace [--requests 40] [--seed 0] [--probe-min PCT]

prints one line per request and a JSON summary (per-bucket mean and p90 time,
tokens per second over the trace, mean reuse).
"""
import argparse
import json
import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

BUCKETS = [  # (label, lowest, highest context tokens, prompts in the paper's benchmark)
    ("0-500", 1, 500, 218),
    ("500-1K", 500, 1000, 210),
    ("1K-2K", 1000, 2000, 204),
    ("2K+", 2000, 3400, 368),
]
COLD_FRACTION = 0.25
WARM_REUSE = (0.32, 0.65)


def make_requests(n, seed):
    """[(bucket label, chunks, cached leading chunks)] for ``n`` requests."""
    rng = np.random.default_rng([seed, 7])
    weights = np.array([b[3] for b in BUCKETS], dtype=np.float64)
    picks = rng.choice(len(BUCKETS), size=n, p=weights / weights.sum())
    out = []
    for k in picks:
        label, lo, hi, _ = BUCKETS[k]
        tokens = int(rng.integers(lo, hi + 1))
        chunks = max(1, math.ceil(tokens / 128))
        if rng.random() < COLD_FRACTION:
            hits = 0
        else:
            hits = int(round(rng.uniform(*WARM_REUSE) * chunks))
        out.append((label, chunks, min(hits, chunks)))
    return out


def request_workload(i, chunks, hits, seed, n_layers=36, probe_min_pct=0):
    """The workload of request ``i`` of a trace drawn with ``seed``: one prompt
    of ``chunks`` chunks whose first ``hits`` were cached."""
    import kvb_workload as kw

    return kw.Workload(
        name=f"request{i}", n_layers=n_layers, n_q_heads=16, n_kv_heads=2, head_dim=128,
        rope_theta=1e6, bits=4, k_group=32, v_group=32, n_prompts=1,
        chunks_per_prompt=chunks, placement="prefix_hits", hit_chunks=hits,
        seam_left=16, seam_right=16, probe_min_num=probe_min_pct, probe_min_den=100,
        seed=seed * 100003 + i)


def request_draws(w, s):
    """A request's values: one layer's seeded draw, reused for every layer."""
    import kvb_workload as kw

    draw = kw.layer_draws(w, s, 0)
    return lambda l: draw


def request_calls(di, pb):
    """The calls one request makes: the fused stitch + deviation when anything
    is cached and probed (the stitch alone when nothing is probed), the
    selection, the patch of every layer, then one attention call per layer."""
    from paper_2608_21362_amd import pipeline

    if di.n_pool and di.n_probed:
        pipeline.stitch_deviation(di, pb)
    elif di.n_pool:
        pipeline.stitch(di, pb)
    pipeline.select(di, pb)
    pipeline.patch(di, pb)
    for li in range(di.n_layers):
        pipeline.attn_layer(di, pb, li)


def run(n_requests=40, seed=0, n_layers=36, probe_min_pct=0, log=print):
    """Run the trace; ``probe_min_pct`` > 0 turns on the threshold-activated
    probe (Sec. 7.4): a request with fewer cached rows than that percentage
    skips the deviation pass and recomputes its seams and live rows only."""
    import torch

    import kvb_workload as kw
    from paper_2608_21362_amd import pipeline

    assert torch.cuda.is_available(), "the trace needs a GPU"
    stream = torch.cuda.current_stream()
    results = []
    for i, (label, chunks, hits) in enumerate(make_requests(n_requests, seed)):
        w = request_workload(i, chunks, hits, seed, n_layers, probe_min_pct)
        s = kw.structure(w)
        di = pipeline.populate(w, s, draws_fn=request_draws(w, s))
        pb = pipeline.buffers(di)

        def request():
            request_calls(di, pb)

        def timed(fn):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            torch.cuda.synchronize()
            return a.elapsed_time(b)

        request()  # warm-up (first launch of each shape)
        torch.cuda.synchronize()
        eager_ms = float(np.median([timed(request) for _ in range(3)]))
        outs = (pb.k_cache, pb.v_cache, pb.delta, pb.rows, pb.cu_rows, pb.out)
        ref = [t.clone() for t in outs]
        # the request's launches captured once and replayed back to back, as a
        # serving loop would run a captured prefill (small requests are
        # launch-bound when run eagerly)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            request()
        graph.replay()
        torch.cuda.synchronize()
        graph_ms = float(np.median([timed(graph.replay) for _ in range(3)]))
        same = all(torch.equal(a, b) for a, b in zip(ref, outs))
        del graph
        ms = graph_ms if same else eager_ms
        rows = int(pb.cu_rows[0, -1].item())
        results.append(dict(bucket=label, tokens=w.t_total, cached_chunks=hits, chunks=chunks,
                            selected_rows=rows, ms=ms, eager_ms=eager_ms, graph_ms=graph_ms,
                            graph_same=same, probed=bool(di.n_probed)))
        log(f"[trace] request {i:3d} bucket {label:6s} tokens {w.t_total:5d} cached "
            f"{hits:2d}/{chunks:2d} chunks, {rows:5d} rows recomputed per layer: {ms:7.3f} ms "
            f"({'graph' if same else 'eager, graph replay differed'}; eager {eager_ms:.3f} ms)")
        del di, pb
    summary = {"requests": len(results), "layers": n_layers, "seed": seed,
               "probe_min_pct": probe_min_pct,
               "probed": sum(r["probed"] for r in results)}
    tok = sum(r["tokens"] for r in results)
    tot_ms = sum(r["ms"] for r in results)
    summary["tokens_per_s"] = tok / (tot_ms * 1e-3)
    summary["tokens_per_s_eager"] = tok / (sum(r["eager_ms"] for r in results) * 1e-3)
    summary["graph_replays_equal_eager"] = all(r["graph_same"] for r in results)
    summary["mean_reuse"] = float(np.mean([r["cached_chunks"] / r["chunks"] for r in results]))
    per = {}
    for label, *_ in BUCKETS:
        ms = [r["ms"] for r in results if r["bucket"] == label]
        if ms:
            per[label] = {"n": len(ms), "mean_ms": float(np.mean(ms)),
                          "p90_ms": float(np.percentile(ms, 90))}
    summary["buckets"] = per
    cold = [r["ms"] for r in results if r["cached_chunks"] == 0]
    warm = [r["ms"] for r in results if r["cached_chunks"] > 0]
    summary["cold_mean_ms"] = float(np.mean(cold)) if cold else None
    summary["warm_mean_ms"] = float(np.mean(warm)) if warm else None
    return results, summary


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--requests", type=int, default=40)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--layers", type=int, default=36)
    ap.add_argument("--probe-min", type=int, default=0,
                    help="minimum cached-row percentage for the deviation probe (0: always)")
    args = ap.parse_args()
    _, summary = run(args.requests, args.seed, args.layers, args.probe_min,
                     log=lambda m: print(m, file=sys.stderr, flush=True))
    print(json.dumps(summary), flush=True)


if __name__ == "__main__":
    main()
