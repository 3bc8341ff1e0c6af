"""The C ABI on the CPU: the library loads and exports every entry point the
header declares; host helpers agree with the oracle; every argument check
fires before any HIP call.  Nothing here launches a kernel on a GPU: tests
that would reach a launch skip when a device is present."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import kvb_workload as kw
from oracle import rope, selection

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "kvb.h")
kvb = pytest.importorskip("paper_2608_21362_amd.kvb")

NO_GPU = torch.cuda.device_count() == 0
FAKE = 0x10000  # never dereferenced: validation rejects the call first


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kvb_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared()
    assert len(names) >= 13
    lib = ctypes.CDLL(kvb.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(names) == sorted(kvb.EXPORTED)
    assert kvb.kvb_abi_version() == 7


def test_ceiling_library_loads():
    """The benchmark's practical-ceiling kernels build into their own library
    and export their three entry points (no compute call here)."""
    import os

    path = os.path.join(os.path.dirname(kvb.LIB_PATH), "libkvb_ceiling.so")
    lib = ctypes.CDLL(path)
    for n in ("kvb_ceiling_mfma", "kvb_ceiling_read", "kvb_ceiling_copy"):
        assert hasattr(lib, n), n
    # argument checks reject before any launch
    lib.kvb_ceiling_mfma.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    assert lib.kvb_ceiling_mfma(0, 10, ctypes.c_void_p(FAKE), None) == -1
    lib.kvb_ceiling_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                     ctypes.c_void_p, ctypes.c_void_p]
    assert lib.kvb_ceiling_read(ctypes.c_void_p(FAKE), 24, 8, ctypes.c_void_p(FAKE), None) == -1


@pytest.mark.parametrize("theta,d", [(1e4, 64), (1e6, 128)])
def test_rope_table_matches_oracle_bitwise(theta, d):
    delta = np.array([0, 1, -1, 1000, -32767, 32767, 12345, -5], np.int32)
    c, s = kvb.kvb_rope_delta_table(theta, d, delta)
    oc, os_ = rope.angle_table(theta, d, delta)
    assert np.array_equal(c, oc) and np.array_equal(s, os_)


@pytest.mark.parametrize("name", kw.ORDER)
def test_row_flags_match_oracle(name):
    w = kw.WORKLOADS[name]
    s = kw.structure(w)
    chunks = np.stack([np.arange(s.n_pool), s.src_pos, s.dst_row, s.dst_pos], 1)
    flags, k = kvb.kvb_row_flags(s.cu_seqlens, w.n_sinks, w.chunk_len, chunks, w.seam_left,
                                 w.seam_right, w.rho_num, w.rho_den)
    forced = selection.forced_rows(s.cu_seqlens, s.hit_row, s.chunk_starts, w.seam_left, w.seam_right)
    assert np.array_equal((flags & 1) != 0, s.hit_row)
    assert np.array_equal((flags & 2) != 0, forced)
    assert np.array_equal(k, selection.k_per_prompt(s.cu_seqlens, s.hit_row, w.rho_num, w.rho_den))


def test_host_helper_errors():
    with pytest.raises(kvb.KvbError) as e:
        kvb.kvb_rope_delta_table(-1.0, 64, [0])
    assert e.value.status == kvb.KVB_EINVAL
    with pytest.raises(kvb.KvbError):
        kvb.kvb_row_flags([0, 10], 0, 128, [[0, 0, 0, 0]], 0, 0, 15, 100)  # chunk past the rows
    with pytest.raises(kvb.KvbError):
        kvb.kvb_row_flags([0, 256], 0, 128, [[0, 0, 0, 0]], 0, 0, 15, 0)


def test_workspace_functions_are_pure():
    a = kvb.kvb_select_workspace_bytes(36, 8192, 1)
    assert a == 0 and kvb.kvb_select_workspace_bytes(1, 32768, 16) > 32768 * 4
    x = kvb.kvb_sparse_attn_workspace_bytes(1, 16, 2, 128, 8192, 1, 8192, 1228, 0)
    assert x == kvb.kvb_sparse_attn_workspace_bytes(1, 16, 2, 128, 8192, 1, 8192, 1228, 0) and x > 0
    # the fp16 copy of V (unless the caller passes it), the work
    # decomposition and the partial records
    y = kvb.kvb_sparse_attn_workspace_bytes(36, 16, 2, 128, 8192, 1, 8192, 1228, 0)
    y16 = kvb.kvb_sparse_attn_workspace_bytes(36, 16, 2, 128, 8192, 1, 8192, 1228, 1)
    assert y > 36 * 2 * 8192 * 128 * 2 and y % 256 == 0
    assert y - y16 >= 36 * 2 * 8192 * 128 * 2 and y16 > 0
    assert kvb.kvb_sparse_attn_workspace_bytes(1, 16, 3, 128, 8192, 1, 8192, 1228, 0) == 0


def _pool(**kw_):
    base = dict(n_layers=1, n_kv_heads=2, head_dim=128, bits=8, k_group=128, v_group=128)
    base.update(kw_)
    return kvb.pool_layout(**base)


def _stitch(**over):
    args = dict(pool=_pool(), n_pool=1, k_codes=FAKE, k_scale=FAKE, k_zero=FAKE, v_codes=FAKE,
                v_scale=FAKE, v_zero=FAKE, chunks=FAKE, n_chunks=1, rope_cos=FAKE, rope_sin=FAKE,
                t_total=128, out_dtype=kvb.KVB_BF16, k_cache=FAKE, v_cache=FAKE, stream=0)
    args.update(over)
    kvb.kvb_stitch(**args)


@pytest.mark.parametrize("over,status", [
    (dict(pool=_pool(bits=2)), kvb.KVB_EUNSUPPORTED),
    (dict(pool=_pool(head_dim=96, v_group=32)), kvb.KVB_EUNSUPPORTED),
    (dict(pool=_pool(chunk_len=64, k_group=64)), kvb.KVB_EUNSUPPORTED),
    (dict(pool=_pool(k_group=48)), kvb.KVB_EINVAL),
    (dict(pool=_pool(v_group=48)), kvb.KVB_EINVAL),
    (dict(k_codes=None), kvb.KVB_EINVAL),
    (dict(v_cache=FAKE + 4), kvb.KVB_EINVAL),
    (dict(t_total=0), kvb.KVB_EINVAL),
    (dict(t_total=2**31), kvb.KVB_EINVAL),
    (dict(out_dtype=kvb.KVB_F64), kvb.KVB_EINVAL),
    (dict(rope_cos=None), kvb.KVB_EINVAL),
    (dict(n_pool=0), kvb.KVB_EINVAL),                  # chunks listed with an empty pool
    (dict(n_pool=-1, n_chunks=0), kvb.KVB_EINVAL),
    (dict(n_pool=0, n_chunks=0, k_cache=None), kvb.KVB_EINVAL),
])
def test_stitch_rejects(over, status):
    with pytest.raises(kvb.KvbError) as e:
        _stitch(**over)
    assert e.value.status == status


def test_empty_pool_is_a_no_op():
    """A cold prompt: nothing cached, no chunks, NULL pool arrays.  Both stitch
    entry points return before any device work (no GPU needed)."""
    empty = dict(n_pool=0, n_chunks=0, k_codes=None, k_scale=None, k_zero=None, v_codes=None,
                 v_scale=None, v_zero=None, chunks=None, rope_cos=None, rope_sin=None)
    _stitch(**empty)
    _stitch_dev(**empty)


def _stitch_dev(**over):
    args = dict(pool=_pool(), n_pool=1, k_codes=FAKE, k_scale=FAKE, k_zero=FAKE, v_codes=FAKE,
                v_scale=FAKE, v_zero=FAKE, chunks=FAKE, n_chunks=1, rope_cos=FAKE, rope_sin=FAKE,
                t_total=128, k_cache=FAKE, v_cache=FAKE, k_fresh=FAKE, delta=FAKE, stream=0)
    args.update(over)
    kvb.kvb_stitch_deviation(**args)


@pytest.mark.parametrize("over,status", [
    (dict(pool=_pool(bits=2)), kvb.KVB_EUNSUPPORTED),
    (dict(pool=_pool(head_dim=96, v_group=32)), kvb.KVB_EUNSUPPORTED),
    (dict(k_fresh=None), kvb.KVB_EINVAL),
    (dict(delta=None), kvb.KVB_EINVAL),
    (dict(delta=FAKE + 4), kvb.KVB_EINVAL),
    (dict(k_cache=FAKE + 2), kvb.KVB_EINVAL),
    (dict(t_total=0), kvb.KVB_EINVAL),
    (dict(rope_sin=None), kvb.KVB_EINVAL),
    (dict(n_pool=0), kvb.KVB_EINVAL),
    (dict(n_pool=0, n_chunks=0, delta=None), kvb.KVB_EINVAL),
])
def test_stitch_deviation_rejects(over, status):
    with pytest.raises(kvb.KvbError) as e:
        _stitch_dev(**over)
    assert e.value.status == status


def _dev_args(**over):
    args = dict(n_layers=1, n_kv_heads=2, head_dim=128, t_total=64, k_cache=FAKE, k_fresh=FAKE,
                v_cache=None, v_fresh=None, per_layer=1, delta=FAKE, stream=0)
    args.update(over)
    return args


@pytest.mark.parametrize("over,status", [
    (dict(v_cache=FAKE), kvb.KVB_EINVAL),            # exactly one value tensor
    (dict(head_dim=80), kvb.KVB_EUNSUPPORTED),
    (dict(n_kv_heads=3), kvb.KVB_EUNSUPPORTED),
    (dict(n_kv_heads=32), kvb.KVB_EUNSUPPORTED),
    (dict(n_layers=0), kvb.KVB_EINVAL),
    (dict(k_fresh=None), kvb.KVB_EINVAL),
    (dict(delta=FAKE + 8), kvb.KVB_EINVAL),
])
def test_deviation_rejects(over, status):
    with pytest.raises(kvb.KvbError) as e:
        kvb.kvb_deviation(**_dev_args(**over))
    assert e.value.status == status


def test_select_rejects_small_workspace_and_nulls():
    need = kvb.kvb_select_workspace_bytes(2, 1000, 4)
    with pytest.raises(kvb.KvbError) as e:
        kvb.kvb_select(2, 1000, FAKE, 4, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need - 1, 0)
    assert e.value.status == kvb.KVB_EINVAL
    with pytest.raises(kvb.KvbError):
        kvb.kvb_select(2, 1000, None, 4, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need, 0)
    with pytest.raises(kvb.KvbError):
        kvb.kvb_select(0, 1000, FAKE, 4, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need, 0)


def _attn(**over):
    args = dict(n_layers=1, n_q_heads=16, n_kv_heads=2, head_dim=128, t_total=4096,
                cu_seqlens=FAKE, n_seqs=1, max_seq_len=4096, rows=FAKE, cu_rows=FAKE,
                rows_per_layer=0, max_rows=600, q=FAKE, k_fresh=FAKE, v_fresh=FAKE,
                k_cache=FAKE, v_cache=FAKE, v_cache_f16=None, softmax_scale=0.088,
                out_dtype=kvb.KVB_BF16, out=FAKE,
                workspace=FAKE, workspace_bytes=0, stream=0)
    args.update(over)
    if "workspace_bytes" not in over:
        args["workspace_bytes"] = kvb.kvb_sparse_attn_workspace_bytes(
            args["n_layers"], args["n_q_heads"], args["n_kv_heads"], max(args["head_dim"], 1),
            args["t_total"], max(args["n_seqs"], 1), max(args["max_seq_len"], 1), args["max_rows"],
            args["v_cache_f16"] is not None)
    kvb.kvb_sparse_attn(**args)


@pytest.mark.parametrize("over,status", [
    (dict(n_kv_heads=3), kvb.KVB_EINVAL),
    (dict(n_q_heads=24, n_kv_heads=4), kvb.KVB_EUNSUPPORTED),   # group of 6 does not divide 32
    (dict(n_q_heads=128, n_kv_heads=2), kvb.KVB_EUNSUPPORTED),  # group of 64
    (dict(head_dim=256), kvb.KVB_EUNSUPPORTED),
    (dict(workspace_bytes=1), kvb.KVB_EINVAL),
    (dict(q=None), kvb.KVB_EINVAL),
    (dict(out=FAKE + 2), kvb.KVB_EINVAL),
    (dict(max_seq_len=5000), kvb.KVB_EINVAL),
    (dict(max_rows=5000), kvb.KVB_EINVAL),
    (dict(softmax_scale=0.0), kvb.KVB_EINVAL),
    (dict(out_dtype=7), kvb.KVB_EINVAL),
    (dict(v_cache_f16=FAKE + 2), kvb.KVB_EINVAL),
    (dict(v_status=FAKE + 2), kvb.KVB_EINVAL),          # status word not 4-byte aligned
])
def test_sparse_attn_rejects(over, status):
    with pytest.raises(kvb.KvbError) as e:
        _attn(**over)
    assert e.value.status == status


def _plans_bytes(a):
    return kvb.kvb_attn_plans_bytes(a["n_layers"], a["n_q_heads"], a["n_kv_heads"],
                                    max(a["head_dim"], 1), a["t_total"], max(a["n_seqs"], 1),
                                    max(a["max_seq_len"], 1), a["max_rows"])


def _patch(**over):
    args = dict(n_layers=4, n_q_heads=16, n_kv_heads=2, head_dim=128, t_total=4096,
                cu_seqlens=FAKE, n_seqs=1, max_seq_len=4096, rows=FAKE, cu_rows=FAKE,
                rows_per_layer=1, max_rows=600, k_fresh=FAKE, v_fresh=FAKE, k_cache=FAKE,
                v_cache=FAKE, v_cache_f16=FAKE, plans=FAKE, plans_bytes=None, stream=0)
    args.update(over)
    if args["plans_bytes"] is None:
        args["plans_bytes"] = _plans_bytes(args)
    kvb.kvb_patch(**args)


def _attn_layer(**over):
    args = dict(layer=2, n_layers=4, n_q_heads=16, n_kv_heads=2, head_dim=128, t_total=4096,
                cu_seqlens=FAKE, n_seqs=1, max_seq_len=4096, rows=FAKE, cu_rows=FAKE,
                rows_per_layer=1, max_rows=600, q=FAKE, k_cache=FAKE, v_cache_f16=FAKE,
                plans=FAKE, plans_bytes=None, softmax_scale=0.088, out_dtype=kvb.KVB_BF16,
                out=FAKE, workspace=FAKE, workspace_bytes=None, stream=0)
    args.update(over)
    if args["plans_bytes"] is None:
        args["plans_bytes"] = _plans_bytes(args)
    if args["workspace_bytes"] is None:
        args["workspace_bytes"] = kvb.kvb_sparse_attn_workspace_bytes(
            1, args["n_q_heads"], args["n_kv_heads"], max(args["head_dim"], 1), args["t_total"],
            max(args["n_seqs"], 1), max(args["max_seq_len"], 1), args["max_rows"], 1)
    kvb.kvb_sparse_attn_layer(**args)


def test_plans_bytes_is_pure_and_per_layer():
    one = kvb.kvb_attn_plans_bytes(1, 16, 2, 128, 8192, 1, 8192, 1228)
    assert one > 0 and one % 256 == 0
    assert kvb.kvb_attn_plans_bytes(36, 16, 2, 128, 8192, 1, 8192, 1228) == 36 * one
    assert kvb.kvb_attn_plans_bytes(1, 16, 3, 128, 8192, 1, 8192, 1228) == 0
    assert kvb.kvb_attn_plans_bytes(0, 16, 2, 128, 8192, 1, 8192, 1228) == 0


@pytest.mark.parametrize("over,status", [
    (dict(n_kv_heads=3), kvb.KVB_EINVAL),
    (dict(n_q_heads=24, n_kv_heads=4), kvb.KVB_EUNSUPPORTED),
    (dict(head_dim=256), kvb.KVB_EUNSUPPORTED),
    (dict(plans_bytes=16), kvb.KVB_EINVAL),
    (dict(plans=FAKE + 2), kvb.KVB_EINVAL),
    (dict(k_fresh=None), kvb.KVB_EINVAL),
    (dict(v_cache=FAKE + 2), kvb.KVB_EINVAL),
    (dict(rows=None), kvb.KVB_EINVAL),
    (dict(max_rows=5000), kvb.KVB_EINVAL),
    (dict(v_cache_f16=FAKE + 2), kvb.KVB_EINVAL),
    (dict(v_status=FAKE + 1), kvb.KVB_EINVAL),
    (dict(v_cache_f16=None, v_status=FAKE), kvb.KVB_EINVAL),  # a status needs the fp16 copy of V
])
def test_patch_rejects(over, status):
    with pytest.raises(kvb.KvbError) as e:
        _patch(**over)
    assert e.value.status == status


@pytest.mark.parametrize("over,status", [
    (dict(layer=4), kvb.KVB_EINVAL),
    (dict(layer=-1), kvb.KVB_EINVAL),
    (dict(n_kv_heads=3), kvb.KVB_EINVAL),
    (dict(n_q_heads=128, n_kv_heads=2), kvb.KVB_EUNSUPPORTED),
    (dict(v_cache_f16=None), kvb.KVB_EINVAL),
    (dict(plans=None), kvb.KVB_EINVAL),
    (dict(plans_bytes=16), kvb.KVB_EINVAL),
    (dict(workspace_bytes=1), kvb.KVB_EINVAL),
    (dict(workspace=None), kvb.KVB_EINVAL),
    (dict(q=FAKE + 2), kvb.KVB_EINVAL),
    (dict(softmax_scale=float("nan")), kvb.KVB_EINVAL),
    (dict(out_dtype=7), kvb.KVB_EINVAL),
])
def test_sparse_attn_layer_rejects(over, status):
    with pytest.raises(kvb.KvbError) as e:
        _attn_layer(**over)
    assert e.value.status == status


def test_patch_and_layer_without_rows_are_no_ops():
    """max_rows = 0: nothing to patch or attend; without an fp16 copy of V to
    build both calls return before any device work (so they succeed here, with
    no GPU)."""
    _patch(max_rows=0, v_cache_f16=None)
    _attn_layer(max_rows=0)


def test_chunk_importance_rejects():
    with pytest.raises(kvb.KvbError) as e:
        kvb.kvb_chunk_importance(_pool(), 1, 1, kvb.KVB_BF16, FAKE, FAKE, 0)
    assert e.value.status == kvb.KVB_EINVAL
    with pytest.raises(kvb.KvbError):
        kvb.kvb_chunk_importance(_pool(), 1, 2, kvb.KVB_F64, FAKE, FAKE, 0)  # n_in > n_layers
    with pytest.raises(kvb.KvbError):
        kvb.kvb_chunk_importance(_pool(), 1, 1, kvb.KVB_F64, None, FAKE, 0)
    with pytest.raises(kvb.KvbError):
        kvb.kvb_chunk_importance(_pool(), 1, 1, kvb.KVB_F64, FAKE, FAKE + 8, 0)
    with pytest.raises(kvb.KvbError) as e:
        kvb.kvb_chunk_importance(_pool(head_dim=96, v_group=32), 1, 1, kvb.KVB_F64, FAKE, FAKE, 0)
    assert e.value.status == kvb.KVB_EUNSUPPORTED


def test_population_rejects():
    with pytest.raises(kvb.KvbError) as e:
        kvb.kvb_rope_rows(96, 1, 1, 1, FAKE, FAKE, None, FAKE, FAKE, 10, kvb.KVB_BF16, FAKE, 0)
    assert e.value.status == kvb.KVB_EUNSUPPORTED
    with pytest.raises(kvb.KvbError):
        kvb.kvb_rope_rows(64, 1, 1, 1, FAKE, FAKE, None, FAKE, None, 10, kvb.KVB_BF16, FAKE, 0)
    with pytest.raises(kvb.KvbError):
        kvb.kvb_kivi_quantize(_pool(), 1, 1, 1, kvb.KVB_F64, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                              FAKE, FAKE, 0)  # layers out of range


@pytest.mark.skipif(not NO_GPU, reason="would launch on a real device")
def test_valid_call_without_device_reports_hip_error():
    """In a container with no GPU a call that passes validation fails in the HIP
    runtime and reports KVB_EHIP with a message."""
    with pytest.raises(kvb.KvbError) as e:
        kvb.kvb_deviation(**_dev_args())
    assert e.value.status == kvb.KVB_EHIP and e.value.message


def test_select_noalloc_rejects_sizes_beyond_its_scratch():
    """The allocation-free selection refuses, before any HIP call, a batch
    whose staging would not fit its static scratch, and checks its pointers
    like kvb_select."""
    lib = kvb.library()
    cap = kvb.kvb_select_noalloc_max_bytes()
    assert cap == 16 << 20
    # 2 prompts: staging = sets x rows x 4 bytes (+ counts) > cap
    t_big = cap // 4 + 1
    st = lib.kvb_select_noalloc(1, t_big, FAKE, 2, FAKE, FAKE, FAKE, FAKE, FAKE, None)
    assert st == kvb.KVB_EINVAL and b"scratch" in lib.kvb_last_error()
    st = lib.kvb_select_noalloc(8, cap // 32, FAKE, 2, FAKE, FAKE, FAKE, FAKE, FAKE, None)
    assert st == kvb.KVB_EINVAL
    st = lib.kvb_select_noalloc(1, 1000, FAKE, 2, None, FAKE, FAKE, FAKE, FAKE, None)
    assert st == kvb.KVB_EINVAL
    st = lib.kvb_select_noalloc(0, 1000, FAKE, 2, FAKE, FAKE, FAKE, FAKE, FAKE, None)
    assert st == kvb.KVB_EINVAL
