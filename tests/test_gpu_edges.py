"""Edge cases of the stitch, the deviation, the selection and the attention
through the C ABI, on generator-drawn inputs: out-of-range chunk descriptors;
zero and negative-zero vectors, identical rows, values in the deviation,
all-layer deviation; ragged batches with empty prompts, one-row prompts and
prompts with no selected row, both head sizes, the fp16 copy of V in a
caller buffer or in the workspace; the fp16 range flag.  Stitch bit-exact;
deviation within one float32 ulp of the oracle; selection bit-exact; patch
and the fp16 copy of V bit-exact; attention within
|o - o_ref| <= 2e-2 + 1e-2 |o_ref|; rows that are not selected never written."""
import sys

import numpy as np
import pytest
import torch

from oracle import attention as oatt
from oracle import deviation as odev
from oracle import numerics, selection as osel

pytestmark = pytest.mark.gpu
ATOL, RTOL = 2e-2, 1e-2


def _f16_of_bf16(bits):
    """fp16 bit patterns of bf16 values (numpy's float32 -> float16, RNE;
    magnitudes past fp16's range become infinities, as on the device)."""
    with np.errstate(over="ignore"):
        return numerics.bf16_bits_to_f32(bits).astype(np.float16).view(np.uint16)
LENS = [0, 37, 0, 129, 1, 640, 0, 255, 3]


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bf16(rng, shape, scale=1.0):
    return numerics.f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))


def test_select_empty_and_tiny_prompts():
    _need_gpu()
    from paper_2608_21362_amd import kvb

    rng = np.random.default_rng(3)
    cu = np.concatenate([[0], np.cumsum(LENS)]).astype(np.int32)
    T, B, n_sets = int(cu[-1]), len(LENS), 2
    cand = rng.random(T) < 0.7
    forced = (~cand) | (rng.random(T) < 0.03)
    flags = (cand.astype(np.uint8) * kvb.KVB_ROW_CANDIDATE) | (forced.astype(np.uint8) * kvb.KVB_ROW_FORCED)
    delta = rng.random((n_sets, T)).astype(np.float32)
    ks = np.stack([osel.k_per_prompt(cu, cand, 15, 100), osel.k_per_prompt(cu, cand, 60, 100)])
    ks = ks.astype(np.int32)
    ws_bytes = kvb.kvb_select_workspace_bytes(n_sets, T, B)
    d_rows = torch.full((n_sets, T), -1, dtype=torch.int32, device="cuda")
    d_cur = torch.zeros((n_sets, B + 1), dtype=torch.int32, device="cuda")
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
    kvb.kvb_select(n_sets, T, torch.from_numpy(cu).cuda(), B, torch.from_numpy(delta).cuda(),
                   torch.from_numpy(flags).cuda(), torch.from_numpy(ks).cuda(), d_rows, d_cur, ws,
                   ws_bytes)
    torch.cuda.synchronize()
    g_rows, g_cu = d_rows.cpu().numpy(), d_cur.cpu().numpy()
    for si in range(n_sets):
        r_rows, r_cu = osel.select(delta[si], cand, forced, cu, ks[si])
        assert np.array_equal(g_cu[si], r_cu), si
        assert np.array_equal(g_rows[si, : r_cu[-1]], r_rows), si
        # empty prompts own no rows of the list
        for b in np.flatnonzero(np.diff(cu) == 0):
            assert g_cu[si, b] == g_cu[si, b + 1]


@pytest.mark.parametrize("hq,hkv,d,shadow,split", [(16, 2, 128, True, False),
                                                  (16, 2, 128, False, False),
                                                  (4, 2, 64, True, False),
                                                  (8, 8, 64, False, False),
                                                  (16, 2, 128, True, True),
                                                  (4, 2, 64, True, True)])
def test_attention_ragged_with_empty_prompts(hq, hkv, d, shadow, split):
    """split: kvb_patch, then kvb_sparse_attn_layer (instead of one kvb_sparse_attn)."""
    _need_gpu()
    from paper_2608_21362_amd import kvb

    _say(f"[edges] attention Hq={hq} Hkv={hkv} d={d} shadow={shadow} split={split}")
    rng = np.random.default_rng(hq * 100 + d + shadow)
    cu = np.concatenate([[0], np.cumsum(LENS)]).astype(np.int32)
    T, B = int(cu[-1]), len(LENS)
    q = _bf16(rng, (T, hq, d))
    kc, vc = _bf16(rng, (hkv, T, d)), _bf16(rng, (hkv, T, d), 2.0)
    kf, vf = _bf16(rng, (hkv, T, d)), _bf16(rng, (hkv, T, d), 2.0)
    # selected rows: about a third of each prompt, none of the 129-row prompt,
    # the one-row prompt's row, the whole 3-row prompt
    rows = []
    for b in range(B):
        lo, hi = int(cu[b]), int(cu[b + 1])
        if hi - lo in (0, 129):
            continue
        if hi - lo <= 3:
            rows.extend(range(lo, hi))
        else:
            rows.extend(sorted(rng.choice(np.arange(lo, hi), size=(hi - lo) // 3, replace=False)))
    rows = np.asarray(rows, dtype=np.int32)
    cu_rows = np.searchsorted(rows, cu).astype(np.int32)
    max_seq = int(np.max(np.diff(cu)))
    dk, dv = torch.from_numpy(kc.view(np.int16)).cuda(), torch.from_numpy(vc.view(np.int16)).cuda()
    # shadow: the call builds the fp16 copy of V into a caller buffer (filled
    # with NaN patterns first; else into its workspace); a range status word
    # rides along
    v16 = None
    if shadow:
        v16 = torch.full((hkv, T, d), 0x7E00, dtype=torch.int16, device="cuda")
    status = torch.zeros(4, dtype=torch.int32, device="cuda")
    out = torch.full((T, hq, d), -1, dtype=torch.int16, device="cuda")
    wsb = kvb.kvb_sparse_attn_workspace_bytes(1, hq, hkv, d, T, B, max_seq, len(rows), int(shadow))
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
    dcu, drows, dcur = (torch.from_numpy(x).cuda() for x in (cu, rows, cu_rows))
    dq = torch.from_numpy(q.view(np.int16)).cuda()
    dkf, dvf = torch.from_numpy(kf.view(np.int16)).cuda(), torch.from_numpy(vf.view(np.int16)).cuda()
    if split:
        pbytes = kvb.kvb_attn_plans_bytes(1, hq, hkv, d, T, B, max_seq, len(rows))
        plans = torch.empty(max(pbytes, 16), dtype=torch.uint8, device="cuda")
        kvb.kvb_patch(1, hq, hkv, d, T, dcu, B, max_seq, drows, dcur, 0, len(rows), dkf, dvf, dk,
                      dv, v16, plans, pbytes, v_status=status if shadow else None)
        kvb.kvb_sparse_attn_layer(0, 1, hq, hkv, d, T, dcu, B, max_seq, drows, dcur, 0, len(rows),
                                  dq, dk, v16, plans, pbytes, 1.0 / np.sqrt(d), kvb.KVB_BF16, out,
                                  ws, wsb)
    else:
        kvb.kvb_sparse_attn(1, hq, hkv, d, T, dcu, B, max_seq, drows, dcur, 0, len(rows), dq, dkf,
                            dvf, dk, dv, v16, 1.0 / np.sqrt(d), kvb.KVB_BF16, out, ws, wsb,
                            v_status=status)
    torch.cuda.synchronize()
    pk, pv = oatt.patch(kc, kf, rows), oatt.patch(vc, vf, rows)
    assert np.array_equal(dk.cpu().numpy().view(np.uint16), pk)
    assert np.array_equal(dv.cpu().numpy().view(np.uint16), pv)
    if shadow:
        assert np.array_equal(v16.cpu().numpy().view(np.uint16), _f16_of_bf16(pv))
    assert int(status[0].item()) == 0
    ref = oatt.attend_rows(q, pk, pv, rows, cu)
    o = out.cpu().numpy().view(np.uint16)
    got = numerics.bf16_bits_to_f32(o[rows]).astype(np.float64)
    err = np.abs(got - ref)
    _say(f"[edges] rows {len(rows)} max|err| {err.max():.3e}")
    assert np.all(err <= ATOL + RTOL * np.abs(ref))
    others = np.setdiff1d(np.arange(T), rows)
    assert np.all(o[others] == 0xFFFF), "a row that was not selected was written"


@pytest.mark.parametrize("with_v,per_layer,d", [(False, True, 128), (True, True, 128),
                                                (True, False, 64), (False, False, 128)])
def test_deviation_zero_rows_and_values(with_v, per_layer, d):
    """kvb_deviation alone: planted rows where both vectors are zero (cosine 1),
    one of them is zero (cosine 0), -0 entries, identical rows (delta 0 exactly
    per term), with the values entering or not, per layer or over all layers:
    within one float32 ulp of the oracle."""
    _need_gpu()
    from paper_2608_21362_amd import kvb

    rng = np.random.default_rng(d + 2 * with_v + per_layer)
    L, H, T = 3, 2, 700
    kc, kf = _bf16(rng, (L, H, T, d)), _bf16(rng, (L, H, T, d))
    vc, vf = _bf16(rng, (L, H, T, d), 3.0), _bf16(rng, (L, H, T, d), 3.0)
    kf[:, :, 10:20] = kc[:, :, 10:20]           # identical rows
    kc[:, :, 30:35] = 0                          # both zero
    kf[:, :, 30:35] = 0
    kc[:, :, 40:45] = 0                          # cache zero only
    kf[:, :, 50:55] = 0x8000                     # fresh -0 only
    kc[1, 0, 60] = 0                             # a zero in one layer and head only
    vc[:, :, 70:72] = 0
    vf[:, :, 70:72] = 0
    n_sets = L if per_layer else 1
    delta = torch.full((n_sets, T), -5.0, dtype=torch.float32, device="cuda")
    t = lambda a: torch.from_numpy(a.view(np.int16)).cuda()  # noqa: E731
    kvb.kvb_deviation(L, H, d, T, t(kc), t(kf), t(vc) if with_v else None,
                      t(vf) if with_v else None, int(per_layer), delta)
    torch.cuda.synchronize()
    ref = odev.deviation(kc, kf, vc if with_v else None, vf if with_v else None,
                         per_layer=per_layer).astype(np.float32)
    got = delta.cpu().numpy()
    ulp = np.spacing(np.abs(ref))
    assert np.all(np.abs(got.astype(np.float64) - ref) <= ulp)
    if not with_v:
        assert np.all(got[:, 10:20] == 0.0) and np.all(got[:, 30:35] == 0.0)
        assert np.all(got[:, 40:45] == 1.0) and np.all(got[:, 50:55] == 1.0)


def test_stitch_skips_out_of_range_descriptors():
    """Descriptors whose pool slot or destination rows fall outside the arrays
    are skipped (nothing written); the valid ones in the same list are stitched
    bit-exact with the oracle."""
    _need_gpu()
    import kvb_workload as kw
    from oracle import populate as opop, stitch as ostitch
    from paper_2608_21362_amd import kvb, pipeline

    # half of the chunks are misses: the bad descriptors point at live rows,
    # which no valid descriptor writes, so a write there would show
    w = kw.scaled(kw.WORKLOADS["batched_mixed"], n_prompts=2, chunks_per_prompt=4)
    s = kw.structure(w)
    dev = pipeline.populate(w, s)
    ref = opop.populate(w, s)
    P, T = s.n_pool, w.t_total
    good = ref.chunks.copy()
    live = [r for r in range(0, T, 128) if not s.hit_row[r]]
    assert len(live) >= 2
    bad = np.array([[P, 0, live[0], 0], [-1, 0, live[1], 128], [0, 0, T - 64, 0],
                    [1, 0, -128, 0]], dtype=np.int32)
    chunks = np.concatenate([bad[:2], good, bad[2:]])
    cos = np.concatenate([ref.cos[:2] * 0, ref.cos, ref.cos[:2] * 0]).astype(np.float32)
    sin = np.concatenate([ref.sin[:2] * 0, ref.sin, ref.sin[:2] * 0]).astype(np.float32)
    pb = pipeline.buffers(dev)
    kvb.kvb_stitch(dev.pool, P, dev.k_codes, dev.k_scale, dev.k_zero, dev.v_codes, dev.v_scale,
                   dev.v_zero, torch.from_numpy(chunks).cuda(), len(chunks),
                   torch.from_numpy(np.ascontiguousarray(cos)).cuda(),
                   torch.from_numpy(np.ascontiguousarray(sin)).cuda(), T, kvb.KVB_BF16,
                   pb.k_cache, pb.v_cache, None)
    torch.cuda.synchronize()
    ck, cv = ref.cache_k.copy(), ref.cache_v.copy()
    ostitch.stitch_into(ck, cv, ref.pool, ref.chunks, ref.cos, ref.sin, "bf16")
    assert np.array_equal(pb.k_cache.cpu().numpy().view(np.uint16), ck)
    assert np.array_equal(pb.v_cache.cpu().numpy().view(np.uint16), cv)


@pytest.mark.parametrize("where", ["patched", "stitched"])
def test_fp16_range_flag(where):
    """A V value fp16 cannot hold (|v| = 1e5: 99840 in bf16) in a patched row
    or in a row the patch leaves alone sets the status word of kvb_patch; the
    same cache without it leaves the word at 0."""
    _need_gpu()
    from paper_2608_21362_amd import kvb

    rng = np.random.default_rng(5)
    hq, hkv, d, T = 16, 2, 128, 300
    cu = np.array([0, T], np.int32)
    kc, vc = _bf16(rng, (hkv, T, d)), _bf16(rng, (hkv, T, d))
    kf, vf = _bf16(rng, (hkv, T, d)), _bf16(rng, (hkv, T, d))
    rows = np.arange(0, T, 3, dtype=np.int32)
    cu_rows = np.array([0, len(rows)], np.int32)
    for planted in (False, True):
        vc2, vf2 = vc.copy(), vf.copy()
        if planted:
            big = numerics.f32_to_bf16_bits(np.array([1e5], np.float32))[0]
            if where == "patched":
                vf2[1, rows[7], 5] = big
            else:
                vc2[0, 4, 17] = big  # row 4 is not selected
        dk, dv = (torch.from_numpy(x.view(np.int16)).cuda() for x in (kc, vc2))
        dkf, dvf = (torch.from_numpy(x.view(np.int16)).cuda() for x in (kf, vf2))
        v16 = torch.zeros((hkv, T, d), dtype=torch.int16, device="cuda")
        status = torch.zeros(4, dtype=torch.int32, device="cuda")
        pbytes = kvb.kvb_attn_plans_bytes(1, hq, hkv, d, T, 1, T, len(rows))
        plans = torch.empty(max(pbytes, 16), dtype=torch.uint8, device="cuda")
        dcu, drows, dcur = (torch.from_numpy(x).cuda() for x in (cu, rows, cu_rows))
        kvb.kvb_patch(1, hq, hkv, d, T, dcu, 1, T, drows, dcur, 0, len(rows), dkf, dvf, dk, dv,
                      v16, plans, pbytes, v_status=status)
        torch.cuda.synchronize()
        flag = int(status[0].item())
        _say(f"[fp16-range] {where} planted={planted}: flag {flag}")
        assert flag == (1 if planted else 0)
        assert np.all(status.cpu().numpy()[1:] == 0)


@pytest.mark.parametrize("call", ["patch", "sparse_attn"])
def test_fp16_copy_without_selected_rows(call):
    """max_rows = 0 (no prompt selects a row): nothing is patched or attended,
    but a caller-kept fp16 copy of V is still rebuilt from the V cache, and a
    value fp16 cannot hold still sets the status word; the caches are left
    alone."""
    _need_gpu()
    from paper_2608_21362_amd import kvb

    rng = np.random.default_rng(9)
    L, hq, hkv, d, T = 2, 8, 2, 64, 200
    cu = np.array([0, 120, T], np.int32)
    kc, vc = _bf16(rng, (L, hkv, T, d)), _bf16(rng, (L, hkv, T, d), scale=3.0)
    vc[1, 1, 150, 7] = numerics.f32_to_bf16_bits(np.array([-1e5], np.float32))[0]
    dk, dv = (torch.from_numpy(x.view(np.int16)).cuda() for x in (kc, vc))
    dkf, dvf = (torch.from_numpy(_bf16(rng, (L, hkv, T, d)).view(np.int16)).cuda() for _ in range(2))
    dq = torch.from_numpy(_bf16(rng, (L, T, hq, d)).view(np.int16)).cuda()
    rows = torch.full((T,), -1, dtype=torch.int32, device="cuda")
    cu_rows = torch.zeros(3, dtype=torch.int32, device="cuda")
    dcu = torch.from_numpy(cu).cuda()
    v16 = torch.full((L, hkv, T, d), 0x7E00, dtype=torch.int16, device="cuda")
    status = torch.zeros(4, dtype=torch.int32, device="cuda")
    if call == "patch":
        pbytes = kvb.kvb_attn_plans_bytes(L, hq, hkv, d, T, 2, 120, 0)
        plans = torch.empty(max(pbytes, 16), dtype=torch.uint8, device="cuda")
        kvb.kvb_patch(L, hq, hkv, d, T, dcu, 2, 120, rows, cu_rows, 0, 0, dkf, dvf, dk, dv, v16,
                      plans, pbytes, v_status=status)
    else:
        out = torch.full((L, T, hq, d), -1, dtype=torch.int16, device="cuda")
        wsb = kvb.kvb_sparse_attn_workspace_bytes(L, hq, hkv, d, T, 2, 120, 0, 1)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
        kvb.kvb_sparse_attn(L, hq, hkv, d, T, dcu, 2, 120, rows, cu_rows, 0, 0, dq, dkf, dvf, dk,
                            dv, v16, 1.0 / np.sqrt(d), kvb.KVB_BF16, out, ws, wsb,
                            v_status=status)
        torch.cuda.synchronize()
        assert np.all(out.cpu().numpy() == -1), "an output row was written"
    torch.cuda.synchronize()
    assert np.array_equal(dk.cpu().numpy().view(np.uint16), kc)
    assert np.array_equal(dv.cpu().numpy().view(np.uint16), vc)
    assert np.array_equal(v16.cpu().numpy().view(np.uint16), _f16_of_bf16(vc))
    assert int(status[0].item()) == 1
