"""Patch once, then attention layer by layer.

Alg. 2 takes the rows it patches from the probe pass (every layer, before the
selection) and patches before the repair forward runs, so a caller may patch
every layer with one ``kvb_patch`` call (which also builds each layer's work
plan) and then make one ``kvb_sparse_attn_layer`` call per layer.  That split
must give exactly what one ``kvb_sparse_attn`` call per layer gives: caches,
fp16 shadow and outputs bit for bit.  The per-layer ``kvb_sparse_attn`` path is
checked against the oracle at these sizes elsewhere, and the small parity cases
run the split path against the oracle directly.

The cases cover both launch shapes of the attention kernel (balanced key
ranges whose cut tiles are merged by the combine kernel, and one whole tile
per workgroup, which the 32K workload takes), one row set shared by every
layer, d = 64 with two query heads per kv head, a cold batch (every row live)
and a batch with no probed prompt.  A graph of the split step replays to the
eager result.
"""
import sys

import numpy as np
import pytest
import torch

import kvb_workload as kw

pytestmark = pytest.mark.gpu

CASES = [
    # name, workload, GPU-populated layers (None = all)
    ("tiny", kw.WORKLOADS["tiny"], None),
    ("batched_mixed", kw.WORKLOADS["batched_mixed"], None),
    ("shared_rows_3l", kw.scaled(kw.WORKLOADS["qwen_36l_8k"], n_layers=3, chunks_per_prompt=4,
                                 per_layer=False, seam_left=16, seam_right=0), None),
    ("cold_2l", kw.scaled(kw.WORKLOADS["qwen_36l_8k"], n_layers=2, chunks_per_prompt=3,
                          placement="prefix_hits", hit_chunks=0, seam_left=16, seam_right=16),
     None),
    ("probe_off_3p", kw.scaled(kw.WORKLOADS["qwen_36l_8k"], n_layers=1, n_prompts=3,
                               chunks_per_prompt=5, placement="ramp_hits", seam_left=16,
                               probe_min_num=1, probe_min_den=1), None),
    ("qwen_36l_8k", kw.WORKLOADS["qwen_36l_8k"], [0, 1, 17, 35]),
    ("long_32k", kw.WORKLOADS["long_32k"], [0]),
]


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _setup(w, layers):
    from paper_2608_21362_amd import pipeline

    s = kw.structure(w)
    gl = list(range(w.n_layers)) if layers is None else list(layers)
    di = pipeline.populate(w, s, layers=gl)
    pb = pipeline.buffers(di)
    pipeline.stitch(di, pb)
    if di.n_probed:
        pipeline.deviation_topk(di, pb)
    else:
        pipeline.select(di, pb)
    torch.cuda.synchronize()
    return di, pb


def _reset(di, pb, stitched):
    from paper_2608_21362_amd import pipeline

    for t, v in zip((pb.k_cache, pb.v_cache, pb.v_cache_f16), stitched):
        t.copy_(v)
    pb.out.fill_(torch.tensor(pipeline.SENTINEL, dtype=torch.int32).to(torch.int16).item())


@pytest.mark.parametrize("name,w,layers", CASES, ids=[c[0] for c in CASES])
def test_split_equals_per_layer_calls(name, w, layers):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21362_amd import pipeline

    _say(f"[split] {name}: layers {layers if layers is not None else 'all'}")
    di, pb = _setup(w, layers)
    stitched = [t.clone() for t in (pb.k_cache, pb.v_cache, pb.v_cache_f16)]
    outputs = lambda: (pb.k_cache, pb.v_cache, pb.v_cache_f16, pb.out)  # noqa: E731
    names = ("k_cache", "v_cache", "v_cache_f16", "out")

    _reset(di, pb, stitched)
    for i in range(di.n_layers):
        pipeline.sparse_attn_layer(di, pb, i)
    torch.cuda.synchronize()
    ref = [t.clone() for t in outputs()]
    n_rows = pb.cu_rows[:, -1].cpu().numpy()
    _say(f"[split] {name}: per-layer calls done, selected rows per set {n_rows.min()}..{n_rows.max()}")

    for rep in range(2):
        _reset(di, pb, stitched)
        pipeline.patch(di, pb)
        for i in range(di.n_layers):
            pipeline.attn_layer(di, pb, i)
        torch.cuda.synchronize()
        for nm, a, b in zip(names, ref, outputs()):
            assert torch.equal(a, b), f"{name}: split path, run {rep}: {nm} differs"
        _say(f"[split] {name}: split path run {rep} equals the per-layer calls")
    # an output row is written exactly when it is selected
    rows = pb.rows.cpu().numpy()
    cu = pb.cu_rows.cpu().numpy()
    sentinel = torch.tensor(pipeline.SENTINEL, dtype=torch.int32).to(torch.int16).item()
    for i in range(di.n_layers):
        si = i if w.per_layer else 0
        sel = np.zeros(w.t_total, dtype=bool)
        sel[rows[si, : cu[si, -1]]] = True
        o = pb.out[i].cpu().numpy().reshape(w.t_total, -1)
        untouched = np.all(o == sentinel, axis=1)
        assert np.array_equal(untouched, ~sel), f"{name} layer {i}: written rows != selected rows"


def test_split_graph_replays_match_eager():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21362_amd import pipeline

    w = kw.WORKLOADS["qwen_36l_8k"]
    _say("[split] graph: qwen_36l_8k layers 0..3")
    di, pb = _setup(w, [0, 1, 2, 3])
    stitched = [t.clone() for t in (pb.k_cache, pb.v_cache, pb.v_cache_f16)]

    def step():
        pipeline.patch(di, pb)
        for i in range(di.n_layers):
            pipeline.attn_layer(di, pb, i)

    outputs = lambda: (pb.k_cache, pb.v_cache, pb.v_cache_f16, pb.out)  # noqa: E731
    _reset(di, pb, stitched)
    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outputs()]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for r in range(3):
        _reset(di, pb, stitched)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for nm, a, b in zip(("k_cache", "v_cache", "v_cache_f16", "out"), ref, outputs()):
            assert torch.equal(a, b), f"graph replay {r}: {nm} differs from the eager step"
        _say(f"[split] graph replay {r} matches the eager step")
    del graph
