"""The path captured in a HIP graph: replays give the eager step's results.

The step (stitch, deviation + selection, one attention call per layer) is run
eagerly once and its outputs kept; the same step is then captured in a graph
and replayed several times, with eager work that resets every output and a
synchronisation before every replay.  Every replay must reproduce the eager
outputs bit for bit: the calls are deterministic (no atomics decide a value
or an order) and record no memset into the graph.
"""
import sys

import pytest
import torch

import kvb_workload as kw

pytestmark = pytest.mark.gpu

CASES = [
    # workload, populated layers (None = all), one patch of every layer then a
    # call per layer (the bench's configuration) or a patch inside every call
    ("qwen_1l", None, True),
    ("qwen_36l_8k", [0, 1, 2], True),
    ("batched_mixed", None, True),
    ("qwen_1l", None, False),
]


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.mark.parametrize("name,layers,split", CASES,
                         ids=[c[0] + ("" if c[2] else "_patch_per_layer") for c in CASES])
def test_graph_replays_match_eager(name, layers, split):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21362_amd import pipeline

    w = kw.WORKLOADS[name]
    s = kw.structure(w)
    gl = list(range(w.n_layers)) if layers is None else list(layers)
    _say(f"[graph] {name}: layers {gl}")
    di = pipeline.populate(w, s, layers=gl)
    pb = pipeline.buffers(di)

    def step():
        pipeline.stitch(di, pb)
        pipeline.deviation_topk(di, pb)
        if split:
            pipeline.patch(di, pb)
            for i in range(di.n_layers):
                pipeline.attn_layer(di, pb, i)
        else:
            for i in range(di.n_layers):
                pipeline.sparse_attn_layer(di, pb, i)

    outputs = lambda: (pb.k_cache, pb.v_cache, pb.v_cache_f16, pb.delta, pb.rows,  # noqa: E731
                       pb.cu_rows, pb.out)
    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outputs()]

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for r in range(4):
        # eager work between replays: every output back to its state before
        # the first step (the harness-written live rows in the cache, the
        # untouched-row markers elsewhere), then an eager stitch
        pb.k_cache.copy_(di.cache_init_k)
        pb.v_cache.copy_(di.cache_init_v)
        pb.v_cache_f16.zero_()
        pb.delta.zero_()
        pb.rows.fill_(-1)
        pb.cu_rows.zero_()
        pb.out.fill_(torch.tensor(pipeline.SENTINEL, dtype=torch.int32).to(torch.int16).item())
        pipeline.stitch(di, pb)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        names = ("k_cache", "v_cache", "v_cache_f16", "delta", "rows", "cu_rows", "out")
        for nm, a, b in zip(names, ref, outputs()):
            assert torch.equal(a, b), f"{name}: replay {r}: {nm} differs from the eager step"
        _say(f"[graph] {name}: replay {r} matches the eager step")
    del graph
