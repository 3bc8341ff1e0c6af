"""Benchmark of the stitched-prefill path on one MI355X.

One step = one pass of the whole path over one batch of a workload, by
default one 8K-token prompt of the 36-layer Qwen2.5-3B-shaped workload
(16 query / 2 KV heads, d = 128, int4 KIVI pool with 64 cached chunks at
random original offsets, 15 % per-layer recompute):

    kvb_stitch_deviation (all layers, one launch: dequantise + re-rotate the
                          cached chunks and the per-layer K deviation of the
                          stitched rows)
    kvb_select           (all layers, one launch)
    kvb_patch            (all layers: the patch and the attention plans in one
                          launch, then the fp16 copy of every layer's V)
    kvb_sparse_attn_layer x 36 (one call per layer, as a model runs its layers)

captured once in a HIP graph and replayed.  Inputs are resident in HBM before
the timed region.  Prints one JSON line.

``roofline`` covers the dominant call, the per-layer attention: algorithmic
flops per call / its average duration from HIP events on the stream it runs
on; "traffic" is the per-call HBM bytes from the committed rocprofv3 counter
summary when it was taken on the current kernel sources.  ``rooflines`` adds
the same figures for the bandwidth-bound calls (stitch, deviation, fused
stitch + deviation) on the method's own bytes, timed with the Infinity Cache
flushed; the fp16 copy of V that the patch call builds for the attention
(its P.V operand, not part of the method) is reported as an overhead.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--attn-all-layers] [--no-cpu-baseline]
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 / fp16 MFMA
METRIC = "stitched-prefill tokens/s + HBM GB/s / MFMA util, Qwen2.5-3B shape 8K ctx"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic(w, s, rows_per_set, cu_rows_per_set):
    """Algorithmic work of one step: the bytes each bandwidth-bound call must
    move for the method itself, and the attention's flops.

    Stitch (Eq. 7 dequantisation and the Sec. 3.2 re-rotation): the codes and
    statistics it reads and the bf16 K and V rows it writes.  Deviation (Alg. 2
    step 2): the stitched and fresh K rows it reads (bf16) and the deviation it
    writes.  Fused stitch + deviation: the stitch's bytes plus the fresh K rows
    of the stitched chunks and their deviations.  The fp16 copy of V built for
    the attention's P.V operand (the patched V cache read, the copy written)
    is not the method's work: its bytes are returned separately.  Attention
    (Eq. 2): 4 d Hq flops per (selected query row, visible key): QK^T and PV."""
    L, H, d, C, T, Hq = w.n_layers, w.n_kv_heads, w.head_dim, w.chunk_len, w.t_total, w.n_q_heads
    P = s.n_pool
    cb = d * w.bits // 8
    codes = 2 * P * L * H * C * cb
    stats = P * L * H * (C // w.k_group) * d * 8 + P * L * H * C * (d // w.v_group) * 8
    stitch_out = 2 * P * L * H * C * d * 2
    shadow = 2 * L * H * T * d * 2
    n_sets = rows_per_set.shape[0]
    fresh_k = P * L * H * C * d * 2
    b = {
        "stitch": codes + stats + stitch_out,
        "deviation": 2 * L * H * T * d * 2 + n_sets * T * 4,
        "stitch_deviation": codes + stats + stitch_out + fresh_k + L * P * C * 4,
        "shadow": shadow,
    }
    # bytes read of each (the rest is written), for the practical ceilings
    reads = {"stitch": codes + stats, "deviation": 2 * L * H * T * d * 2,
             "stitch_deviation": codes + stats + fresh_k}
    pos = s.positions().astype(np.int64)
    flops_per_layer = []
    for l in range(L):
        si = l if w.per_layer else 0
        r = rows_per_set[si, : cu_rows_per_set[si, -1]]
        flops_per_layer.append(4.0 * d * Hq * float(np.sum(pos[r] + 1)))
    return b, reads, np.array(flops_per_layer)


def committed_traffic(workload, key="traffic_bytes_per_launch"):
    """Per-launch HBM bytes of the attention call from the committed counter
    summary, if it was taken on the current kernel sources (else None).  The
    summary's ``traffic_bytes_per_launch`` covers attention + combine (one
    kvb_sparse_attn_layer call), ``traffic_bytes_per_launch_with_patch`` adds
    the patch (one per-layer kvb_sparse_attn call)."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", f"sparse_attn_{workload}_traffic.md")
    if not os.path.exists(path):
        return None, "no committed counter summary"
    text = open(path).read()
    m_b = re.search(r"^" + key + r":\s*([0-9.eE+]+)", text, re.M)
    m_h = re.search(r"^kernel_sources_sha256:\s*([0-9a-f]+)", text, re.M)
    if not m_h:
        return None, "summary lacks the source-hash line"
    if not m_b:
        return None, f"summary holds no {key} figure (no counters for this call grouping)"
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    if h.hexdigest() != m_h.group(1):
        return None, "attention sources changed since the counters were taken"
    return float(m_b.group(1)), "rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated"


KERNEL_SOURCES = ("paper_2608_21362_amd/csrc/sparse_attn.hip", "paper_2608_21362_amd/csrc/kvb_device.h")


def cpu_host():
    """The host the oracle runs on: core count, CPU model, OMP_NUM_THREADS."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"os_cpu_count": os.cpu_count(), "cpu_model": model,
            "OMP_NUM_THREADS": os.environ.get("OMP_NUM_THREADS")}


def cpu_baseline(w, s, n_layers_sample, attn_rows_sample=0):
    """The oracle as it stands on the first ``n_layers_sample`` layers of the
    same workload, stage by stage (stitch; deviation + selection; patch +
    attention), scaled to the whole step linearly in layers.  With
    ``attn_rows_sample`` > 0 the attention is evaluated on that many selected
    rows per layer, spread evenly over the set (rows are independent), and
    scaled by the ratio of visible keys (sum of pi(t) + 1) over all selected
    rows to that over the sample; such a figure is labelled extrapolated."""
    from threadpoolctl import threadpool_info

    from oracle import path as opath
    from oracle import populate as opop

    layers = list(range(n_layers_sample))
    pop = opop.populate(w, s, layers=layers)
    pos = s.positions().astype(np.int64)
    work = {}

    def sampler(i, sel):
        sel = np.asarray(sel)
        pick = sel
        if attn_rows_sample and len(sel) > attn_rows_sample:
            pick = sel[np.linspace(0, len(sel) - 1, attn_rows_sample).astype(np.int64)]
        work[i] = (float(np.sum(pos[sel] + 1)), float(np.sum(pos[pick] + 1)))
        return pick

    tm = {}
    t0 = time.perf_counter()
    opath.run(w, s, pop, attend_rows=sampler, timings=tm)
    dt = time.perf_counter() - t0
    scale = w.n_layers / n_layers_sample
    attn_ratio = (sum(a for a, _ in work.values()) / sum(b for _, b in work.values())
                  if work else 1.0)
    stages = {"stitch_s": tm["stitch"] * scale,
              "deviation_select_s": tm["deviation_select"] * scale,
              "patch_attention_s": tm["patch_attention"] * scale * attn_ratio}
    per_step = sum(stages.values())
    blas = [i.get("num_threads", 1) for i in threadpool_info()]
    extrapolated = attn_ratio > 1.0
    sample = (f"{n_layers_sample} of {w.n_layers} layers, stitch, deviation, selection and "
              f"patch in full, attention on "
              + (f"{attn_rows_sample} evenly spread selected rows per layer (scaled by visible "
                 f"keys x{attn_ratio:.1f}: extrapolated)" if extrapolated
                 else "every selected row")
              + f"; {dt:.1f} s of CPU time; scaled to {w.n_layers} layers")
    return {
        "value": w.t_total / per_step, "unit": "tokens/s",
        "cores": int(max(blas) if blas else 1), "kind": "oracle",
        "sample": sample, "seconds": dt, "stages_per_step": stages,
        "attention_extrapolated": extrapolated, "host": cpu_host(),
    }


def measure_ceilings(torch):
    """Practical ceilings on this device, next to the published peaks: a loop of
    back-to-back bf16 32x32x16 matrix products in the attention kernel's launch
    shape (no memory traffic), streaming read and copy kernels (16-byte
    accesses) and torch's fill as the write stream, over 1 GiB.  Best of three
    timed runs after one warm-up."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2608_21362_amd", "lib", "libkvb_ceiling.so"))
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.kvb_ceiling_mfma.argtypes = [i32, i32, vp, vp]
    lib.kvb_ceiling_read.argtypes = [vp, i64, i32, vp, vp]
    lib.kvb_ceiling_copy.argtypes = [vp, vp, i64, i32, vp]
    stream = torch.cuda.current_stream()
    sh = ctypes.c_void_p(stream.cuda_stream)
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count

    def best(fn, reps=3):
        fn()
        times = []
        for _ in range(reps):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b) * 1e-3)
        return min(times)

    def check(rc):
        if rc != 0:
            raise RuntimeError(f"ceiling kernel launch failed ({rc})")

    n_wg, iters = 2 * n_cu, 4000
    sink = torch.empty(n_wg * 256, dtype=torch.float32, device="cuda")
    t = best(lambda: check(lib.kvb_ceiling_mfma(n_wg, iters, vp(sink.data_ptr()), sh)))
    mfma_tflops = n_wg * 4 * iters * 8 * 32768 / t / 1e12
    nbytes = 1 << 30
    buf = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    rsink = torch.empty(8 * n_cu * 256, dtype=torch.int32, device="cuda")
    t = best(lambda: check(lib.kvb_ceiling_read(vp(buf.data_ptr()), nbytes, 8 * n_cu,
                                                 vp(rsink.data_ptr()), sh)))
    read_gbs = nbytes / t / 1e9
    half = nbytes // 2
    t = best(lambda: check(lib.kvb_ceiling_copy(vp(buf.data_ptr()), vp(buf.data_ptr() + half),
                                                 half, 8 * n_cu, sh)))
    copy_gbs = 2 * half / t / 1e9
    t = best(lambda: buf.fill_(3))
    write_gbs = nbytes / t / 1e9
    del buf, rsink, sink
    return {"mfma_bf16_TFLOPs": mfma_tflops, "read_GBps": read_gbs, "write_GBps": write_gbs,
            "copy_GBps": copy_gbs,
            "note": "measured on this device: bf16 32x32x16 products on 8 independent "
                    "accumulators per wave, 2 workgroups of 256 per CU; streaming 16-byte "
                    "read of 1 GiB, torch fill of 1 GiB (write), copy of 512 MiB (read + "
                    "write bytes).  A kernel's practical ceiling is its bytes over "
                    "read_bytes / read_GBps + written_bytes / write_GBps"}


def practical_frac(gbs, total_bytes, read_bytes, ceil):
    """Achieved GB/s over the time-additive ceiling at the kernel's byte mix."""
    w = total_bytes - read_bytes
    t = read_bytes / ceil["read_GBps"] + w / ceil["write_GBps"]
    return gbs / (total_bytes / t)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen_36l_8k")
    ap.add_argument("--attn-all-layers", action="store_true",
                    help="one attention launch for all layers (ceiling variant)")
    ap.add_argument("--patch-per-layer", action="store_true",
                    help="patch inside every per-layer kvb_sparse_attn call instead of one "
                         "kvb_patch of every layer before the per-layer calls")
    ap.add_argument("--unfused", action="store_true",
                    help="separate stitch and deviation + selection calls instead of the fused "
                         "stitch + deviation call followed by selection")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=24,
                    help="layers of the oracle timed for cpu_baseline (scaled to the whole step)")
    ap.add_argument("--cpu-attn-rows", type=int, default=0,
                    help="evaluate the oracle's attention on this many selected rows per layer "
                         "and scale by visible keys (0: every selected row)")
    ap.add_argument("--flush-mb", type=int, default=512)
    ap.add_argument("--calibrate-copy-mb", type=int, default=0,
                    help="also run one plain device copy of this size (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the path runs on a single MI355X and no "
              "multi-GPU variant is built (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    import kvb_workload as kw
    from paper_2608_21362_amd import pipeline

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = kw.WORKLOADS[args.workload]
    s = kw.structure(w)
    log(f"[bench] workload {w.name}: L={w.n_layers} T={w.t_total} chunks={s.n_pool} "
        f"bits={w.bits}; populating on the GPU")
    t0 = time.time()
    di = pipeline.populate(w, s, progress=lambda i, n: log(f"[bench] populated {i}/{n} layers")
                           if i % 6 == 0 or i == n else None)
    pb = pipeline.buffers(di, attn_all_layers=args.attn_all_layers)
    torch.cuda.synchronize()
    log(f"[bench] inputs resident ({time.time() - t0:.1f} s)")

    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    L = di.n_layers

    fused = not args.unfused
    patch_once = not args.patch_per_layer and not args.attn_all_layers
    a0 = 4 if patch_once else 3  # event index after which the attention calls start

    def step(rec=None):
        if rec is not None:
            rec[0].record(stream)
        if fused:
            pipeline.stitch_deviation(di, pb)
        else:
            pipeline.stitch(di, pb)
        if rec is not None:
            rec[1].record(stream)
        if fused:
            pipeline.select(di, pb)
        else:
            pipeline.deviation_topk(di, pb)
        if rec is not None:
            rec[2].record(stream)
        if args.attn_all_layers:
            pipeline.sparse_attn_all(di, pb)
            if rec is not None:
                rec[3].record(stream)
        elif patch_once:
            # Alg. 2 step 4 for every layer, then the repair forward's
            # attention layer by layer
            pipeline.patch(di, pb)
            if rec is not None:
                rec[3].record(stream)
            for i in range(L):
                pipeline.attn_layer(di, pb, i)
                if rec is not None:
                    rec[4 + i].record(stream)
        else:
            for i in range(L):
                pipeline.sparse_attn_layer(di, pb, i)
                if rec is not None:
                    rec[3 + i].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (pb.k_cache, pb.v_cache, pb.delta, pb.rows, pb.cu_rows, pb.out)]

    # Headline: the whole step (stitch, deviation + selection, the attention
    # calls) captured once in a HIP graph and replayed, so the per-layer
    # launches run back to back as a model's captured forward would run them
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        graph.replay()
    torch.cuda.synchronize()
    g0, g1 = ev(), ev()
    g0.record(stream)
    for _ in range(args.steps):
        graph.replay()
    g1.record(stream)
    torch.cuda.synchronize()
    ms_step_graph = g0.elapsed_time(g1) / args.steps
    graph_same = all(torch.equal(a, b) for a, b in
                     zip(ref, (pb.k_cache, pb.v_cache, pb.delta, pb.rows, pb.cu_rows, pb.out)))
    if not graph_same:
        log("[bench] graph replay differs from the eager step: reporting the eager time")
    del graph

    # Eager steps with HIP events around every call: per-kernel times and the
    # attention call's duration for the roofline
    n_ev = a0 + (1 if args.attn_all_layers else L)
    recs = [[ev() for _ in range(n_ev)] for _ in range(args.steps)]
    start, stop = ev(), ev()
    torch.cuda.synchronize()
    start.record(stream)
    for k in range(args.steps):
        step(recs[k])
    stop.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    ms_step_eager = total_ms / args.steps
    ms_step = ms_step_graph if graph_same else ms_step_eager
    st_ms = np.mean([r[0].elapsed_time(r[1]) for r in recs])
    dv_ms = np.mean([r[1].elapsed_time(r[2]) for r in recs])
    pt_ms = float(np.mean([r[2].elapsed_time(r[3]) for r in recs])) if patch_once else None
    at_ms = np.array([[r[a0 - 1 + j].elapsed_time(r[a0 + j]) for j in range(n_ev - a0)]
                      for r in recs])
    attn_ms_launch = float(at_ms.mean())
    attn_p10, attn_p50, attn_p90 = (float(np.percentile(at_ms, p)) for p in (10, 50, 90))

    rows = pb.rows.cpu().numpy()
    cu = pb.cu_rows.cpu().numpy()
    nbytes, nreads, flops = algorithmic(w, s, rows, cu)
    attn_flops_launch = float(flops.mean()) if not args.attn_all_layers else float(flops.sum())
    attn_tflops = attn_flops_launch / (attn_ms_launch * 1e-3) / 1e12

    # stitch and deviation bandwidth with the 256 MiB Infinity Cache flushed
    # between reps: a read of a larger buffer leaves only clean lines, so the
    # timed call neither hits its inputs in the cache nor pays for another
    # kernel's write-back
    flush = torch.ones(args.flush_mb << 18, dtype=torch.float32, device="cuda")
    flushed = {"stitch": [], "deviation_topk": [], "deviation": [], "stitch_deviation": [],
               "patch": [], "patch_no_copy": []}
    calls = {"stitch": lambda: pipeline.stitch(di, pb),
             "deviation_topk": lambda: pipeline.deviation_topk(di, pb),
             "deviation": lambda: pipeline.deviation(di, pb),
             "stitch_deviation": lambda: pipeline.stitch_deviation(di, pb),
             "patch": lambda: pipeline.patch(di, pb),
             "patch_no_copy": lambda: pipeline.patch(di, pb, f16_copy=False)}
    for _ in range(5):
        # flush, then the timed call right behind it on the same stream (no
        # host synchronisation in between, so the interval holds no idle
        # launch latency)
        for name, fn in calls.items():
            flush.sum()
            a, b = ev(), ev()
            a.record(stream)
            fn()
            b.record(stream)
            torch.cuda.synchronize()
            flushed[name].append(a.elapsed_time(b))
    fl_ms = {k: float(np.median(v)) for k, v in flushed.items()}
    # chunk importance (cache population, Sec. 4.4; not part of the step): fp32
    # keys of every pool chunk and layer, cache flushed before each repetition
    from paper_2608_21362_amd import kvb as _kvb
    P = di.n_pool
    k_pool = torch.randn((P, L, w.n_kv_heads, w.chunk_len, w.head_dim), dtype=torch.float32,
                         device="cuda")
    imp = torch.zeros(P, dtype=torch.float64, device="cuda")
    imp_f = []
    for _ in range(5):
        flush.sum()
        a, b = ev(), ev()
        a.record(stream)
        _kvb.kvb_chunk_importance(di.pool, P, L, _kvb.KVB_F32, k_pool, imp)
        b.record(stream)
        torch.cuda.synchronize()
        imp_f.append(a.elapsed_time(b))
    imp_bytes = k_pool.numel() * 4 + P * 8
    imp_gbs = imp_bytes / (np.median(imp_f) * 1e-3) / 1e9
    del k_pool, imp
    del flush

    log("[bench] practical ceilings")
    ceil = measure_ceilings(torch)
    if args.calibrate_copy_mb:
        src = torch.ones(args.calibrate_copy_mb << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    traffic, traffic_note = (
        (None, "") if args.attn_all_layers else
        committed_traffic(w.name, "traffic_bytes_per_launch" if patch_once
                          else "traffic_bytes_per_launch_with_patch"))
    def bw(name, key):
        """Roofline figures of a bandwidth-bound call on the method's bytes."""
        by = nbytes[key]
        ms = fl_ms[name]
        gbs = by / (ms * 1e-3) / 1e9
        return {"bound": "hbm", "bytes": int(by), "us": ms * 1e3, "achieved": gbs,
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
                "frac_of_practical": practical_frac(gbs, by, nreads[key], ceil),
                "timing": "median of 5 flushed calls (HIP events)"}

    rooflines = {
        "stitch": bw("stitch", "stitch"),
        "deviation": bw("deviation", "deviation"),
        "stitch_deviation": bw("stitch_deviation", "stitch_deviation"),
    }
    copy_us = (fl_ms["patch"] - fl_ms["patch_no_copy"]) * 1e3
    shadow_overhead = {
        "bytes": int(nbytes["shadow"]),
        "what": "fp16 copy of every layer's V (the attention's P.V operand), built by the "
                "patch call from the patched bf16 V cache: V read, copy written",
        "patch_us_with": fl_ms["patch"] * 1e3, "patch_us_without": fl_ms["patch_no_copy"] * 1e3,
        "us": copy_us,
        "GBps": nbytes["shadow"] / (copy_us * 1e-6) / 1e9 if copy_us > 0 else None,
    }
    tokens_per_step = w.t_total
    result = {
        "metric": METRIC,
        "value": tokens_per_step / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded draws with the workload's shapes and distributions)",
        "config": {
            "workload": w.name, "layers": w.n_layers, "prompt_tokens": w.t_total,
            "q_heads": w.n_q_heads, "kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
            "kivi_bits": w.bits, "k_group": w.k_group, "v_group": w.v_group,
            "cached_chunks": s.n_pool, "recompute": f"{w.rho_num}/{w.rho_den} per layer",
            "attention_launches": ("one patch of every layer, then one call per layer" if patch_once
                                   else "patch and attention per layer" if not args.attn_all_layers
                                   else "one for all layers"),
            "stitch_and_deviation": "fused (kvb_stitch_deviation, then kvb_select)" if fused
            else "separate (kvb_stitch, then kvb_deviation_topk)",
            "step_timing": "HIP graph replay" if graph_same else "eager (graph replay differed)",
            "parallelism": "single GPU",
        },
        "roofline": {
            "kernel": ("kvb_sparse_attn_layer call per layer (attention and combine kernels)"
                       if patch_once else
                       "kvb_sparse_attn call per layer (patch, attention and combine kernels)"
                       if not args.attn_all_layers else
                       "kvb_sparse_attn call for all layers (patch, attention and combine kernels)"),
            "bound": "mfma", "achieved": attn_tflops, "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": attn_tflops / MFMA_BF16_PEAK_TFLOPS, "traffic": traffic,
            "traffic_note": traffic_note,
            "flops_per_launch": attn_flops_launch, "ms_per_launch": attn_ms_launch,
            "ms_per_launch_p10_p50_p90": [attn_p10, attn_p50, attn_p90],
            "timing": "HIP events around each call in eager steps",
            "frac_of_measured_ceiling": attn_tflops / ceil["mfma_bf16_TFLOPs"],
        },
        "rooflines": rooflines,
        "shadow_overhead": shadow_overhead,
        "ceilings": ceil,
        "kernels": {
            "ms_per_step_eager": ms_step_eager, "ms_per_step_graph": ms_step_graph,
            ("stitch_deviation_ms" if fused else "stitch_ms"): float(st_ms),
            ("select_ms" if fused else "deviation_topk_ms"): float(dv_ms),
            "patch_ms": pt_ms,
            "sparse_attn_ms_per_step": float(at_ms.sum(axis=1).mean()),
            "deviation_topk_ms_flushed": fl_ms["deviation_topk"],
            "select_ms_flushed": fl_ms["deviation_topk"] - fl_ms["deviation"],
            "chunk_importance_GBps_flushed": imp_gbs,
            "chunk_importance_hbm_frac": imp_gbs / HBM_PEAK_GBS,
            "chunk_importance_bytes": int(imp_bytes),
            "chunk_importance_frac_of_practical": practical_frac(
                imp_gbs, imp_bytes, imp_bytes - P * 8, ceil),
            "selected_rows_per_layer": float(np.mean(cu[:, -1])),
        },
    }
    if not args.no_cpu_baseline:
        n_cpu = min(args.cpu_layers, w.n_layers)
        log(f"[bench] cpu baseline: oracle on {n_cpu} layers"
            + (f", attention on {args.cpu_attn_rows} rows per layer" if args.cpu_attn_rows else ""))
        result["cpu_baseline"] = cpu_baseline(w, s, n_cpu, args.cpu_attn_rows)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
