"""Python binding of libkvb (ctypes): the C entry points under the same names.

Argument marshalling only -- every step of the path runs in the HIP kernels of
``lib/libkvb.so``.  Device tensors are torch tensors (torch supplies device
memory and the current stream); host helpers take and return numpy arrays.
Importing this module fails loudly when the library has not been built.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "lib", "libkvb.so")

KVB_OK, KVB_EINVAL, KVB_EUNSUPPORTED, KVB_EHIP = 0, 1, 2, 3
KVB_BF16, KVB_F32, KVB_F64 = 0, 1, 2
KVB_ROW_CANDIDATE, KVB_ROW_FORCED = 1, 2

_STATUS = {0: "KVB_OK", 1: "KVB_EINVAL", 2: "KVB_EUNSUPPORTED", 3: "KVB_EHIP"}


class KvbError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status
        self.message = message


class kvb_pool_layout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("n_layers", "n_kv_heads", "head_dim", "chunk_len", "bits", "k_group", "v_group")]


class kvb_chunk(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("pool_idx", "src_pos", "dst_row", "dst_pos")]


_i32, _i64, _f32, _f64, _vp, _sz = (ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                    ctypes.c_double, ctypes.c_void_p, ctypes.c_size_t)

_SIGS = {
    "kvb_abi_version": (ctypes.c_int, []),
    "kvb_last_error": (ctypes.c_char_p, []),
    "kvb_rope_delta_table": (_i32, [_f64, _i32, _vp, _i32, _vp, _vp]),
    "kvb_row_flags": (_i32, [_i32, _vp, _i32, _i32, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp]),
    "kvb_probe_gate": (_i32, [_i32, _vp, _vp, _i32, _i32, _vp, _vp]),
    "kvb_rope_rows": (_i32, [_i32, _i64, _i64, _i64, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp]),
    "kvb_kivi_quantize": (_i32, [ctypes.POINTER(kvb_pool_layout), _i32, _i32, _i32, _i32, _vp, _vp,
                                 _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "kvb_chunk_importance": (_i32, [ctypes.POINTER(kvb_pool_layout), _i32, _i32, _i32, _vp, _vp,
                                    _vp]),
    "kvb_stitch": (_i32, [ctypes.POINTER(kvb_pool_layout), _i32, _vp, _vp, _vp, _vp, _vp, _vp,
                          _vp, _i32, _vp, _vp, _i64, _i32, _vp, _vp, _vp]),
    "kvb_stitch_deviation": (_i32, [ctypes.POINTER(kvb_pool_layout), _i32, _vp, _vp, _vp, _vp,
                                    _vp, _vp, _vp, _i32, _vp, _vp, _i64, _vp, _vp, _vp, _vp,
                                    _vp]),
    "kvb_deviation": (_i32, [_i32, _i32, _i32, _i64, _vp, _vp, _vp, _vp, _i32, _vp, _vp]),
    "kvb_select_workspace_bytes": (_sz, [_i32, _i64, _i32]),
    "kvb_select": (_i32, [_i32, _i64, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "kvb_select_noalloc": (_i32, [_i32, _i64, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
    "kvb_select_noalloc_max_bytes": (_sz, []),
    "kvb_deviation_topk": (_i32, [_i32, _i32, _i32, _i64, _vp, _i32, _vp, _vp, _vp, _vp, _i32,
                                  _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "kvb_sparse_attn_workspace_bytes": (_sz, [_i32, _i32, _i32, _i32, _i64, _i32, _i32, _i32,
                                              _i32]),
    "kvb_sparse_attn": (_i32, [_i32, _i32, _i32, _i32, _i64, _vp, _i32, _i32, _vp, _vp, _i32,
                               _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _f32, _i32, _vp, _vp,
                               _sz, _vp]),
    "kvb_attn_plans_bytes": (_sz, [_i32, _i32, _i32, _i32, _i64, _i32, _i32, _i32]),
    "kvb_patch": (_i32, [_i32, _i32, _i32, _i32, _i64, _vp, _i32, _i32, _vp, _vp, _i32, _i32,
                         _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "kvb_sparse_attn_layer": (_i32, [_i32, _i32, _i32, _i32, _i32, _i64, _vp, _i32, _i32, _vp,
                                     _vp, _i32, _i32, _vp, _vp, _vp, _vp, _sz, _f32, _i32, _vp,
                                     _vp, _sz, _vp]),
}


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2608_21362_amd.build` (hipcc, gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGS.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()
EXPORTED = tuple(_SIGS)


def library():
    return _lib


def _check(status: int):
    if status != KVB_OK:
        raise KvbError(status, _lib.kvb_last_error().decode())


def _p(t):
    """Device (or host) address of a torch tensor / numpy array, 0 for None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def pool_layout(n_layers, n_kv_heads, head_dim, bits, k_group, v_group, chunk_len=128):
    return kvb_pool_layout(n_layers, n_kv_heads, head_dim, chunk_len, bits, k_group, v_group)


# ---- host helpers -------------------------------------------------------------

def kvb_abi_version() -> int:
    return _lib.kvb_abi_version()


def kvb_rope_delta_table(theta: float, head_dim: int, delta):
    delta = np.ascontiguousarray(delta, dtype=np.int32).reshape(-1)
    n = delta.shape[0]
    c = np.empty((n, head_dim // 2), np.float32)
    s = np.empty((n, head_dim // 2), np.float32)
    _check(_lib.kvb_rope_delta_table(theta, head_dim, _p(delta), n, _p(c), _p(s)))
    return c, s


def kvb_row_flags(cu_seqlens, n_sinks, chunk_len, chunks, seam_left, seam_right, rho_num, rho_den):
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    ch = np.ascontiguousarray(chunks, dtype=np.int32).reshape(-1, 4)
    n_seqs = cu.shape[0] - 1
    flags = np.empty(int(cu[-1]), np.uint8)
    k = np.empty(n_seqs, np.int32)
    _check(_lib.kvb_row_flags(n_seqs, _p(cu), n_sinks, chunk_len, _p(ch), ch.shape[0], seam_left,
                              seam_right, rho_num, rho_den, _p(flags), _p(k)))
    return flags, k


def kvb_probe_gate(cu_seqlens, row_flags, k_per_seq, min_num, min_den):
    """Returns (k_per_seq with skipped prompts at 0, number of probed prompts)."""
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    fl = np.ascontiguousarray(row_flags, dtype=np.uint8)
    k = np.array(k_per_seq, dtype=np.int32, copy=True)
    n = np.zeros(1, np.int32)
    _check(_lib.kvb_probe_gate(cu.shape[0] - 1, _p(cu), _p(fl), min_num, min_den, _p(k), _p(n)))
    return k, int(n[0])


# ---- population ---------------------------------------------------------------

def kvb_rope_rows(head_dim, n_outer, n_rows, n_inner, x, row_pos, outer_pos, table_cos,
                  table_sin, table_len, out_dtype, out, stream=None):
    _check(_lib.kvb_rope_rows(head_dim, n_outer, n_rows, n_inner, _p(x), _p(row_pos),
                              _p(outer_pos), _p(table_cos), _p(table_sin), table_len, out_dtype,
                              _p(out), _stream(stream)))


def kvb_kivi_quantize(pool, n_pool, first_layer, n_in, in_dtype, k_in, v_in, k_codes, k_scale,
                      k_zero, v_codes, v_scale, v_zero, stream=None):
    _check(_lib.kvb_kivi_quantize(ctypes.byref(pool), n_pool, first_layer, n_in, in_dtype,
                                  _p(k_in), _p(v_in), _p(k_codes), _p(k_scale), _p(k_zero),
                                  _p(v_codes), _p(v_scale), _p(v_zero), _stream(stream)))


# ---- the hot path -------------------------------------------------------------

def kvb_chunk_importance(pool, n_pool, n_in, in_dtype, k_in, importance, stream=None):
    _check(_lib.kvb_chunk_importance(ctypes.byref(pool), n_pool, n_in, in_dtype, _p(k_in),
                                     _p(importance), _stream(stream)))


def kvb_stitch(pool, n_pool, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero, chunks,
               n_chunks, rope_cos, rope_sin, t_total, out_dtype, k_cache, v_cache, stream=None):
    _check(_lib.kvb_stitch(ctypes.byref(pool), n_pool, _p(k_codes), _p(k_scale), _p(k_zero),
                           _p(v_codes), _p(v_scale), _p(v_zero), _p(chunks), n_chunks,
                           _p(rope_cos), _p(rope_sin), t_total, out_dtype, _p(k_cache),
                           _p(v_cache), _stream(stream)))


def kvb_stitch_deviation(pool, n_pool, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero,
                         chunks, n_chunks, rope_cos, rope_sin, t_total, k_cache, v_cache,
                         k_fresh, delta, stream=None):
    _check(_lib.kvb_stitch_deviation(ctypes.byref(pool), n_pool, _p(k_codes), _p(k_scale),
                                     _p(k_zero), _p(v_codes), _p(v_scale), _p(v_zero), _p(chunks),
                                     n_chunks, _p(rope_cos), _p(rope_sin), t_total, _p(k_cache),
                                     _p(v_cache), _p(k_fresh), _p(delta), _stream(stream)))


def kvb_deviation(n_layers, n_kv_heads, head_dim, t_total, k_cache, k_fresh, v_cache, v_fresh,
                  per_layer, delta, stream=None):
    _check(_lib.kvb_deviation(n_layers, n_kv_heads, head_dim, t_total, _p(k_cache), _p(k_fresh),
                              _p(v_cache), _p(v_fresh), int(per_layer), _p(delta),
                              _stream(stream)))


def kvb_select_workspace_bytes(n_sets, t_total, n_seqs) -> int:
    return _lib.kvb_select_workspace_bytes(n_sets, t_total, n_seqs)


def kvb_select(n_sets, t_total, cu_seqlens, n_seqs, delta, row_flags, k_per_seq, rows, cu_rows,
               workspace, workspace_bytes, stream=None):
    _check(_lib.kvb_select(n_sets, t_total, _p(cu_seqlens), n_seqs, _p(delta), _p(row_flags),
                           _p(k_per_seq), _p(rows), _p(cu_rows), _p(workspace), workspace_bytes,
                           _stream(stream)))


def kvb_select_noalloc(n_sets, t_total, cu_seqlens, n_seqs, delta, row_flags, k_per_seq, rows,
                       cu_rows, stream=None):
    _check(_lib.kvb_select_noalloc(n_sets, t_total, _p(cu_seqlens), n_seqs, _p(delta),
                                   _p(row_flags), _p(k_per_seq), _p(rows), _p(cu_rows),
                                   _stream(stream)))


def kvb_select_noalloc_max_bytes():
    return int(_lib.kvb_select_noalloc_max_bytes())


def kvb_deviation_topk(n_layers, n_kv_heads, head_dim, t_total, cu_seqlens, n_seqs, k_cache,
                       k_fresh, v_cache, v_fresh, per_layer, row_flags, k_per_seq, delta, rows,
                       cu_rows, workspace, workspace_bytes, stream=None):
    _check(_lib.kvb_deviation_topk(n_layers, n_kv_heads, head_dim, t_total, _p(cu_seqlens), n_seqs,
                                   _p(k_cache), _p(k_fresh), _p(v_cache), _p(v_fresh),
                                   int(per_layer), _p(row_flags), _p(k_per_seq), _p(delta),
                                   _p(rows), _p(cu_rows), _p(workspace), workspace_bytes,
                                   _stream(stream)))


def kvb_sparse_attn_workspace_bytes(n_layers, n_q_heads, n_kv_heads, head_dim, t_total, n_seqs,
                                    max_seq_len, max_rows, v_f16_given) -> int:
    return _lib.kvb_sparse_attn_workspace_bytes(n_layers, n_q_heads, n_kv_heads, head_dim, t_total,
                                                n_seqs, max_seq_len, max_rows, int(v_f16_given))


def kvb_sparse_attn(n_layers, n_q_heads, n_kv_heads, head_dim, t_total, cu_seqlens, n_seqs,
                    max_seq_len, rows, cu_rows, rows_per_layer, max_rows, q, k_fresh, v_fresh,
                    k_cache, v_cache, v_cache_f16, softmax_scale, out_dtype, out, workspace,
                    workspace_bytes, stream=None, v_status=None):
    _check(_lib.kvb_sparse_attn(n_layers, n_q_heads, n_kv_heads, head_dim, t_total,
                                _p(cu_seqlens), n_seqs, max_seq_len, _p(rows), _p(cu_rows),
                                int(rows_per_layer), max_rows, _p(q), _p(k_fresh), _p(v_fresh),
                                _p(k_cache), _p(v_cache), _p(v_cache_f16), _p(v_status),
                                float(softmax_scale), out_dtype, _p(out), _p(workspace),
                                workspace_bytes, _stream(stream)))


def kvb_attn_plans_bytes(n_layers, n_q_heads, n_kv_heads, head_dim, t_total, n_seqs, max_seq_len,
                         max_rows) -> int:
    return _lib.kvb_attn_plans_bytes(n_layers, n_q_heads, n_kv_heads, head_dim, t_total, n_seqs,
                                     max_seq_len, max_rows)


def kvb_patch(n_layers, n_q_heads, n_kv_heads, head_dim, t_total, cu_seqlens, n_seqs,
              max_seq_len, rows, cu_rows, rows_per_layer, max_rows, k_fresh, v_fresh, k_cache,
              v_cache, v_cache_f16, plans, plans_bytes, stream=None, v_status=None):
    _check(_lib.kvb_patch(n_layers, n_q_heads, n_kv_heads, head_dim, t_total, _p(cu_seqlens),
                          n_seqs, max_seq_len, _p(rows), _p(cu_rows), int(rows_per_layer),
                          max_rows, _p(k_fresh), _p(v_fresh), _p(k_cache), _p(v_cache),
                          _p(v_cache_f16), _p(v_status), _p(plans), plans_bytes,
                          _stream(stream)))


def kvb_sparse_attn_layer(layer, n_layers, n_q_heads, n_kv_heads, head_dim, t_total, cu_seqlens,
                          n_seqs, max_seq_len, rows, cu_rows, rows_per_layer, max_rows, q,
                          k_cache, v_cache_f16, plans, plans_bytes, softmax_scale, out_dtype,
                          out, workspace, workspace_bytes, stream=None):
    _check(_lib.kvb_sparse_attn_layer(layer, n_layers, n_q_heads, n_kv_heads, head_dim, t_total,
                                      _p(cu_seqlens), n_seqs, max_seq_len, _p(rows), _p(cu_rows),
                                      int(rows_per_layer), max_rows, _p(q), _p(k_cache),
                                      _p(v_cache_f16), _p(plans), plans_bytes,
                                      float(softmax_scale), out_dtype, _p(out), _p(workspace),
                                      workspace_bytes, _stream(stream)))
