"""Device-side driver of the stitched-prefill path on one MI355X.

Builds the path's inputs in HBM from the seeded raw draws of ``kvb_workload``
with the library's own population kernels (RoPE at absolute positions, KIVI
quantisation), then runs the path through the C ABI:

    kvb_stitch_deviation (or kvb_stitch, then kvb_deviation_topk)
      -> kvb_select -> kvb_patch (every layer) -> kvb_sparse_attn_layer (per layer)

(``run_path`` can also attend all layers in one kvb_sparse_attn call, or patch
inside a kvb_sparse_attn call per layer.)

torch provides device memory, copies and the stream; every step of the path
runs in libkvb's HIP kernels.
"""
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
import torch

import kvb_workload as kw

from . import kvb

SENTINEL = 0xFFFF  # bf16 NaN pattern: rows a kernel must overwrite start as this


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


@dataclass
class DeviceInputs:
    w: kw.Workload
    s: kw.Structure
    layers: List[int]
    pool: kvb.kvb_pool_layout
    n_pool: int
    k_codes: torch.Tensor
    k_scale: torch.Tensor
    k_zero: torch.Tensor
    v_codes: torch.Tensor
    v_scale: torch.Tensor
    v_zero: torch.Tensor
    chunks: torch.Tensor        # int32 [P][4]
    rope_cos: torch.Tensor      # f32 [P][d/2]
    rope_sin: torch.Tensor
    k_fresh: torch.Tensor       # bf16 bits as int16 [L][Hkv][T][d]
    v_fresh: torch.Tensor
    q: Optional[torch.Tensor]   # [L][T][Hq][d]
    cache_init_k: torch.Tensor  # live rows fresh, hit rows SENTINEL
    cache_init_v: torch.Tensor
    cu_seqlens: torch.Tensor
    row_flags: torch.Tensor
    k_per_set: torch.Tensor     # int32 [n_sets][B]
    max_rows: int
    max_seq_len: int
    host_flags: np.ndarray = field(default=None)
    host_k: np.ndarray = field(default=None)
    importance: Optional[torch.Tensor] = None  # f64 [P]: chunk importance (Sec. 4.4)
    n_probed: int = 0  # prompts whose deviation pass runs (threshold-activated probe)

    @property
    def n_layers(self):
        return len(self.layers)

    @property
    def n_sets(self):
        return self.n_layers if self.w.per_layer else 1


def populate(w: kw.Workload, s: kw.Structure, layers=None, with_q=True, draws_fn=None,
             progress=None, q_layers=None) -> DeviceInputs:
    """Upload the raw draws and build pool / fresh tensors on the GPU.
    ``progress(i, n)``, if given, is called after each populated layer.
    ``q_layers`` (layer ids), if given, limits the query draws to those layers;
    the queries of the other layers are zero (their attention still runs, on
    uniform scores)."""
    layers = list(range(w.n_layers)) if layers is None else list(layers)
    if draws_fn is None:
        def draws_fn(l):
            return kw.layer_draws(w, s, l, with_q=with_q and (q_layers is None or l in q_layers))
    L, H, C, d, T, Hq = len(layers), w.n_kv_heads, w.chunk_len, w.head_dim, w.t_total, w.n_q_heads
    P = s.n_pool
    pool = kvb.pool_layout(L, H, d, w.bits, w.k_group, w.v_group, C)
    cb = d * w.bits // 8
    dev = dict(device="cuda")
    k_codes = torch.zeros((P, L, H, C, cb), dtype=torch.uint8, **dev)
    v_codes = torch.zeros_like(k_codes)
    k_scale = torch.zeros((P, L, H, C // w.k_group, d), dtype=torch.float32, **dev)
    k_zero = torch.zeros_like(k_scale)
    v_scale = torch.zeros((P, L, H, C, d // w.v_group), dtype=torch.float32, **dev)
    v_zero = torch.zeros_like(v_scale)
    k_fresh = torch.empty((L, H, T, d), dtype=torch.int16, **dev)
    v_fresh = torch.empty_like(k_fresh)
    q = None
    if with_q:
        q = (torch.empty if q_layers is None else torch.zeros)((L, T, Hq, d), dtype=torch.int16, **dev)

    pos = s.positions()
    max_pos = int(max(int(pos.max()) + 1, (int(s.src_pos.max()) + C) if P else 0))
    tc, ts = kvb.kvb_rope_delta_table(w.rope_theta, d, np.arange(max_pos, dtype=np.int32))
    tab_c, tab_s = _dev(tc), _dev(ts)
    pos_d = _dev(pos.astype(np.int32))
    u_d = _dev(np.arange(C, dtype=np.int32))
    outer_src = _dev(np.repeat(s.src_pos.astype(np.int32), H)) if P else None
    k_rot = torch.empty((P, H, C, d), dtype=torch.float64, **dev) if P else None
    importance = torch.zeros(max(P, 1), dtype=torch.float64, **dev)
    for i, l in enumerate(layers):
        dr = draws_fn(l)
        if P:
            kp = _dev(dr.k_pool_raw)
            vp = _dev(dr.v_pool_raw)
            kvb.kvb_rope_rows(d, P * H, C, 1, kp, u_d, outer_src, tab_c, tab_s, max_pos,
                              kvb.KVB_F64, k_rot)
            kvb.kvb_kivi_quantize(pool, P, i, 1, kvb.KVB_F64, k_rot, vp.double(), k_codes,
                                  k_scale, k_zero, v_codes, v_scale, v_zero)
            kvb.kvb_chunk_importance(pool, P, 1, kvb.KVB_F64, k_rot, importance)
        kr = _dev(dr.k_raw)
        kvb.kvb_rope_rows(d, H, T, 1, kr, pos_d, None, tab_c, tab_s, max_pos, kvb.KVB_BF16,
                          k_fresh[i])
        vr = _dev(dr.v_raw)
        kvb.kvb_rope_rows(d, H, T, 1, vr, None, None, None, None, 0, kvb.KVB_BF16, v_fresh[i])
        if with_q and dr.q_raw is not None:
            qr = _dev(dr.q_raw)
            kvb.kvb_rope_rows(d, 1, T, Hq, qr, pos_d, None, tab_c, tab_s, max_pos, kvb.KVB_BF16,
                              q[i])
        torch.cuda.synchronize()
        if progress is not None:
            progress(i + 1, len(layers))
    chunks_np = np.stack([np.arange(P), s.src_pos, s.dst_row, s.dst_pos], axis=1).astype(np.int32)
    rc, rs = kvb.kvb_rope_delta_table(w.rope_theta, d, (s.dst_pos - s.src_pos).astype(np.int32))
    hit = torch.from_numpy(s.hit_row).cuda()
    sentinel = torch.tensor(SENTINEL, dtype=torch.int32).to(torch.int16).cuda()
    cache_k = torch.where(hit[None, None, :, None], sentinel, k_fresh)
    cache_v = torch.where(hit[None, None, :, None], sentinel, v_fresh)
    flags, kseq = kvb.kvb_row_flags(s.cu_seqlens, w.n_sinks, C, chunks_np, w.seam_left,
                                    w.seam_right, w.rho_num, w.rho_den)
    kseq, n_probed = kvb.kvb_probe_gate(s.cu_seqlens, flags, kseq, w.probe_min_num,
                                        w.probe_min_den)
    n_sets = L if w.per_layer else 1
    forced = (flags & kvb.KVB_ROW_FORCED) != 0
    bound = 0
    for b in range(len(s.cu_seqlens) - 1):
        lo, hi = int(s.cu_seqlens[b]), int(s.cu_seqlens[b + 1])
        bound += int(kseq[b]) + int(forced[lo:hi].sum())
    max_rows = min(bound, T)
    max_seq_len = int(np.max(np.diff(s.cu_seqlens)))
    return DeviceInputs(
        w=w, s=s, layers=layers, pool=pool, n_pool=P, k_codes=k_codes, k_scale=k_scale,
        k_zero=k_zero, v_codes=v_codes, v_scale=v_scale, v_zero=v_zero,
        chunks=_dev(chunks_np), rope_cos=_dev(rc), rope_sin=_dev(rs), k_fresh=k_fresh,
        v_fresh=v_fresh, q=q, cache_init_k=cache_k, cache_init_v=cache_v,
        cu_seqlens=_dev(s.cu_seqlens.astype(np.int32)), row_flags=_dev(flags),
        k_per_set=_dev(np.tile(kseq[None, :], (n_sets, 1)).astype(np.int32)),
        max_rows=max_rows, max_seq_len=max_seq_len, host_flags=flags, host_k=kseq,
        importance=importance[:P], n_probed=n_probed)


@dataclass
class PathBuffers:
    k_cache: torch.Tensor
    v_cache: torch.Tensor
    v_cache_f16: torch.Tensor  # fp16 copy of the patched v_cache (kvb_patch builds it)
    delta: torch.Tensor
    rows: torch.Tensor
    cu_rows: torch.Tensor
    out: torch.Tensor
    sel_ws: torch.Tensor
    attn_ws: torch.Tensor
    sel_ws_bytes: int
    attn_ws_bytes: int
    attn_ws_bytes_all: int = 0
    plans: torch.Tensor = None  # per-layer attention plans written by kvb_patch
    plans_bytes: int = 0
    v_status: torch.Tensor = None  # uint32 word: set when a V value does not fit fp16


def buffers(di: DeviceInputs, out_dtype=kvb.KVB_BF16, attn_all_layers=False) -> PathBuffers:
    w, T, L = di.w, di.w.t_total, di.n_layers
    B = len(di.s.cu_seqlens) - 1
    sel_bytes = kvb.kvb_select_workspace_bytes(di.n_sets, T, B)
    per_layer_ws = kvb.kvb_sparse_attn_workspace_bytes(1, w.n_q_heads, w.n_kv_heads, w.head_dim, T,
                                                       B, di.max_seq_len, di.max_rows, 1)
    all_ws = kvb.kvb_sparse_attn_workspace_bytes(L, w.n_q_heads, w.n_kv_heads, w.head_dim, T, B,
                                                 di.max_seq_len, di.max_rows, 1)
    attn_bytes = max(per_layer_ws, all_ws if attn_all_layers else 0)
    plans_bytes = kvb.kvb_attn_plans_bytes(L, w.n_q_heads, w.n_kv_heads, w.head_dim, T, B,
                                           di.max_seq_len, di.max_rows)
    odt = torch.int16 if out_dtype == kvb.KVB_BF16 else torch.float32
    out = torch.full((L, T, w.n_q_heads, w.head_dim), -1, dtype=odt, device="cuda")
    if out_dtype == kvb.KVB_BF16:
        out.fill_(torch.tensor(SENTINEL, dtype=torch.int32).to(torch.int16).item())
    else:
        out.fill_(float("nan"))
    return PathBuffers(
        k_cache=di.cache_init_k.clone(), v_cache=di.cache_init_v.clone(),
        v_cache_f16=torch.zeros((L, w.n_kv_heads, T, w.head_dim), dtype=torch.int16,
                                device="cuda"),
        delta=torch.zeros((di.n_sets, T), dtype=torch.float32, device="cuda"),
        rows=torch.full((di.n_sets, T), -1, dtype=torch.int32, device="cuda"),
        cu_rows=torch.zeros((di.n_sets, B + 1), dtype=torch.int32, device="cuda"),
        out=out,
        sel_ws=torch.empty(max(sel_bytes, 16), dtype=torch.uint8, device="cuda"),
        attn_ws=torch.empty(max(attn_bytes, 16), dtype=torch.uint8, device="cuda"),
        sel_ws_bytes=sel_bytes, attn_ws_bytes=per_layer_ws, attn_ws_bytes_all=all_ws,
        plans=torch.empty(max(plans_bytes, 16), dtype=torch.uint8, device="cuda"),
        plans_bytes=plans_bytes,
        v_status=torch.zeros(4, dtype=torch.int32, device="cuda"))


def stitch(di: DeviceInputs, pb: PathBuffers, out_dtype=kvb.KVB_BF16, k_out=None, v_out=None,
           stream=None):
    """Stitch into pb's bf16 cache, or into ``k_out`` / ``v_out`` of ``out_dtype``."""
    kvb.kvb_stitch(di.pool, di.n_pool, di.k_codes, di.k_scale, di.k_zero, di.v_codes, di.v_scale,
                   di.v_zero, di.chunks, di.n_pool, di.rope_cos, di.rope_sin, di.w.t_total,
                   out_dtype, pb.k_cache if k_out is None else k_out,
                   pb.v_cache if v_out is None else v_out, stream)


def stitch_deviation(di: DeviceInputs, pb: PathBuffers, stream=None):
    """Stitch (bf16 cache) fused with the per-layer deviation of the stitched
    rows."""
    kvb.kvb_stitch_deviation(di.pool, di.n_pool, di.k_codes, di.k_scale, di.k_zero, di.v_codes,
                             di.v_scale, di.v_zero, di.chunks, di.n_pool, di.rope_cos,
                             di.rope_sin, di.w.t_total, pb.k_cache, pb.v_cache, di.k_fresh,
                             pb.delta, stream)


def select(di: DeviceInputs, pb: PathBuffers, stream=None):
    """Row selection on pb.delta."""
    kvb.kvb_select(di.n_sets, di.w.t_total, di.cu_seqlens, len(di.s.cu_seqlens) - 1, pb.delta,
                   di.row_flags, di.k_per_set, pb.rows, pb.cu_rows, pb.sel_ws, pb.sel_ws_bytes,
                   stream)


def deviation(di: DeviceInputs, pb: PathBuffers, stream=None):
    """Deviation of the stitched K against the fresh K only (no selection)."""
    w = di.w
    kvb.kvb_deviation(di.n_layers, w.n_kv_heads, w.head_dim, w.t_total, pb.k_cache, di.k_fresh,
                      None, None, w.per_layer, pb.delta, stream)


def deviation_topk(di: DeviceInputs, pb: PathBuffers, stream=None):
    w = di.w
    kvb.kvb_deviation_topk(di.n_layers, w.n_kv_heads, w.head_dim, w.t_total, di.cu_seqlens,
                           len(di.s.cu_seqlens) - 1, pb.k_cache, di.k_fresh, None, None,
                           w.per_layer, di.row_flags, di.k_per_set, pb.delta, pb.rows, pb.cu_rows,
                           pb.sel_ws, pb.sel_ws_bytes, stream)


def sparse_attn_layer(di: DeviceInputs, pb: PathBuffers, i: int, out_dtype=kvb.KVB_BF16,
                      stream=None):
    """Attention of populated layer index ``i`` (one launch; a model runs these in layer order)."""
    w, T = di.w, di.w.t_total
    B = len(di.s.cu_seqlens) - 1
    si = i if w.per_layer else 0
    kvb.kvb_sparse_attn(1, w.n_q_heads, w.n_kv_heads, w.head_dim, T, di.cu_seqlens, B,
                        di.max_seq_len, pb.rows[si], pb.cu_rows[si], 0, di.max_rows, di.q[i],
                        di.k_fresh[i], di.v_fresh[i], pb.k_cache[i], pb.v_cache[i],
                        pb.v_cache_f16[i], 1.0 / float(np.sqrt(w.head_dim)), out_dtype, pb.out[i],
                        pb.attn_ws, pb.attn_ws_bytes, stream, v_status=pb.v_status)


def patch(di: DeviceInputs, pb: PathBuffers, stream=None, f16_copy=True):
    """Alg. 2 step 4 for every populated layer in one launch, which also builds
    the per-layer attention plans that ``attn_layer`` reads, then (unless
    ``f16_copy`` is False) the fp16 copy of the patched V cache, with the fp16
    range status word."""
    w, T = di.w, di.w.t_total
    B = len(di.s.cu_seqlens) - 1
    kvb.kvb_patch(di.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, T, di.cu_seqlens, B,
                  di.max_seq_len, pb.rows, pb.cu_rows, int(w.per_layer), di.max_rows,
                  di.k_fresh, di.v_fresh, pb.k_cache, pb.v_cache,
                  pb.v_cache_f16 if f16_copy else None, pb.plans, pb.plans_bytes, stream,
                  v_status=pb.v_status if f16_copy else None)


def attn_layer(di: DeviceInputs, pb: PathBuffers, i: int, out_dtype=kvb.KVB_BF16, stream=None):
    """Attention of populated layer ``i`` over the cache ``patch`` left (the
    repair forward's per-layer launch: attention and the merge of cut tiles)."""
    w, T = di.w, di.w.t_total
    B = len(di.s.cu_seqlens) - 1
    kvb.kvb_sparse_attn_layer(i, di.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, T,
                              di.cu_seqlens, B, di.max_seq_len, pb.rows, pb.cu_rows,
                              int(w.per_layer), di.max_rows, di.q, pb.k_cache, pb.v_cache_f16,
                              pb.plans, pb.plans_bytes, 1.0 / float(np.sqrt(w.head_dim)),
                              out_dtype, pb.out, pb.attn_ws, pb.attn_ws_bytes, stream)


def sparse_attn_all(di: DeviceInputs, pb: PathBuffers, out_dtype=kvb.KVB_BF16, stream=None):
    """Attention of every populated layer in one launch."""
    w, T = di.w, di.w.t_total
    B = len(di.s.cu_seqlens) - 1
    kvb.kvb_sparse_attn(di.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, T, di.cu_seqlens, B,
                        di.max_seq_len, pb.rows, pb.cu_rows, int(w.per_layer), di.max_rows, di.q,
                        di.k_fresh, di.v_fresh, pb.k_cache, pb.v_cache, pb.v_cache_f16,
                        1.0 / float(np.sqrt(w.head_dim)), out_dtype, pb.out, pb.attn_ws,
                        pb.attn_ws_bytes_all, stream, v_status=pb.v_status)


def run_path(di: DeviceInputs, pb: PathBuffers, attn_all_layers=False, out_dtype=kvb.KVB_BF16,
             stream=None, patch_once=True):
    """One pass of the whole path over the batch.  With no prompt above the
    probe threshold the deviation pass is skipped (every top-k is empty).
    Attention: one launch for every layer (attn_all_layers), or layer by layer,
    after one patch of every layer (patch_once) or with a patch per layer."""
    stitch(di, pb, stream=stream)
    if di.n_probed:
        deviation_topk(di, pb, stream=stream)
    else:
        select(di, pb, stream=stream)
    if attn_all_layers:
        sparse_attn_all(di, pb, out_dtype, stream)
    elif patch_once:
        patch(di, pb, stream=stream)
        for i in range(di.n_layers):
            attn_layer(di, pb, i, out_dtype, stream)
    else:
        for i in range(di.n_layers):
            sparse_attn_layer(di, pb, i, out_dtype, stream)
