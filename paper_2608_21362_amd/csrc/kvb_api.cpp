// C entry points of libkvb: host-side validation, error reporting and the
// host-only helpers.  Every check here runs before the first HIP call, so a
// bad argument is reported the same way with or without a GPU.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <string>
#include <vector>

#include "kvb.h"
#include "kvb_internal.h"

namespace {

thread_local std::string g_err;

kvb_status fail(kvb_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

kvb_status ok() {
  g_err.clear();
  return KVB_OK;
}

kvb_status hip_status(hipError_t e, const char* where) {
  if (e != hipSuccess) return fail(KVB_EHIP, "%s: %s", where, hipGetErrorString(e));
  return ok();
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define REQUIRE(cond, ...) \
  do {                     \
    if (!(cond)) return fail(KVB_EINVAL, __VA_ARGS__); \
  } while (0)
#define REQUIRE_PTR(p) REQUIRE((p) != nullptr, "%s is NULL", #p)
#define REQUIRE_ALIGNED(p) REQUIRE(aligned16(p), "%s is not 16-byte aligned", #p)

kvb_status check_head_dim(int32_t d) {
  if (d != 64 && d != 128) return fail(KVB_EUNSUPPORTED, "head_dim %d: built for 64 and 128", d);
  return KVB_OK;
}

kvb_status check_pool(const kvb_pool_layout* p) {
  REQUIRE_PTR(p);
  REQUIRE(p->n_layers > 0 && p->n_kv_heads > 0 && p->head_dim > 0 && p->chunk_len > 0 &&
              p->k_group > 0 && p->v_group > 0,
          "pool layout has a non-positive size");
  if (kvb_status s = check_head_dim(p->head_dim)) return s;
  if (p->chunk_len != 128) return fail(KVB_EUNSUPPORTED, "chunk_len %d: built for 128", p->chunk_len);
  if (p->bits != 4 && p->bits != 8) return fail(KVB_EUNSUPPORTED, "bits %d: built for 4 and 8", p->bits);
  REQUIRE(p->chunk_len % p->k_group == 0, "k_group %d does not divide chunk_len %d", p->k_group,
          p->chunk_len);
  REQUIRE(p->head_dim % p->v_group == 0, "v_group %d does not divide head_dim %d", p->v_group,
          p->head_dim);
  if (p->k_group % 4 != 0) return fail(KVB_EUNSUPPORTED, "k_group %d: must be a multiple of 4", p->k_group);
  if (p->v_group % 16 != 0) return fail(KVB_EUNSUPPORTED, "v_group %d: must be a multiple of 16", p->v_group);
  return KVB_OK;
}

}  // namespace

extern "C" {

int kvb_abi_version(void) { return 7; }

const char* kvb_last_error(void) { return g_err.c_str(); }

kvb_status kvb_rope_delta_table(double theta, int32_t head_dim, const int32_t* delta, int32_t n,
                                float* cos_out, float* sin_out) {
  REQUIRE(n >= 0, "n < 0");
  REQUIRE(head_dim > 0 && head_dim % 2 == 0, "head_dim %d must be even and positive", head_dim);
  REQUIRE(theta > 0.0, "theta must be positive");
  if (n == 0) return ok();
  REQUIRE_PTR(delta);
  REQUIRE_PTR(cos_out);
  REQUIRE_PTR(sin_out);
  const int half = head_dim / 2;
  std::vector<double> w(half);
  for (int i = 0; i < half; ++i) w[i] = pow(theta, -(2.0 * i) / head_dim);
  for (int32_t k = 0; k < n; ++k) {
    const double dlt = (double)delta[k];
    for (int i = 0; i < half; ++i) {
      const double a = dlt * w[i];
      cos_out[(size_t)k * half + i] = (float)cos(a);
      sin_out[(size_t)k * half + i] = (float)sin(a);
    }
  }
  return ok();
}

kvb_status kvb_row_flags(int32_t n_seqs, const int32_t* cu_seqlens, int32_t n_sinks,
                         int32_t chunk_len, const kvb_chunk* chunks, int32_t n_chunks,
                         int32_t seam_left, int32_t seam_right, int32_t rho_num, int32_t rho_den,
                         uint8_t* row_flags, int32_t* k_per_seq) {
  REQUIRE(n_seqs > 0, "n_seqs must be positive");
  REQUIRE_PTR(cu_seqlens);
  REQUIRE_PTR(row_flags);
  REQUIRE_PTR(k_per_seq);
  REQUIRE(n_chunks >= 0 && (n_chunks == 0 || chunks != nullptr), "bad chunk list");
  REQUIRE(chunk_len > 0 && n_sinks >= 0 && seam_left >= 0 && seam_right >= 0,
          "chunk_len must be positive; sinks and seam widths non-negative");
  REQUIRE(rho_den > 0 && rho_num >= 0, "rho must be rho_num / rho_den with rho_den > 0");
  REQUIRE(cu_seqlens[0] == 0, "cu_seqlens[0] must be 0");
  for (int32_t b = 0; b < n_seqs; ++b)
    REQUIRE(cu_seqlens[b + 1] >= cu_seqlens[b], "cu_seqlens must be non-decreasing");
  const int64_t T = cu_seqlens[n_seqs];
  memset(row_flags, 0, (size_t)T);
  for (int32_t c = 0; c < n_chunks; ++c) {
    const int64_t r0 = chunks[c].dst_row;
    REQUIRE(r0 >= 0 && r0 + chunk_len <= T, "chunk %d rows [%lld, %lld) outside [0, %lld)", c,
            (long long)r0, (long long)(r0 + chunk_len), (long long)T);
    for (int64_t r = r0; r < r0 + chunk_len; ++r) row_flags[r] = KVB_ROW_CANDIDATE;
  }
  for (int32_t b = 0; b < n_seqs; ++b) {
    const int64_t lo = cu_seqlens[b], hi = cu_seqlens[b + 1], Tb = hi - lo;
    int64_t n_cand = 0;
    for (int64_t r = lo; r < hi; ++r) {
      if (!(row_flags[r] & KVB_ROW_CANDIDATE)) row_flags[r] |= KVB_ROW_FORCED;  // live row
      else ++n_cand;
    }
    for (int64_t p = n_sinks; p < Tb; p += chunk_len) {
      if (p <= 0) continue;
      const int64_t a = p - seam_left > 0 ? p - seam_left : 0;
      const int64_t e = p + seam_right < Tb ? p + seam_right : Tb;
      for (int64_t r = lo + a; r < lo + e; ++r)
        if (row_flags[r] & KVB_ROW_CANDIDATE) row_flags[r] |= KVB_ROW_FORCED;
    }
    k_per_seq[b] = (int32_t)(((int64_t)rho_num * n_cand) / rho_den);
  }
  return ok();
}

kvb_status kvb_probe_gate(int32_t n_seqs, const int32_t* cu_seqlens, const uint8_t* row_flags,
                          int32_t min_num, int32_t min_den, int32_t* k_per_seq,
                          int32_t* n_probed) {
  REQUIRE(n_seqs > 0, "n_seqs must be positive");
  REQUIRE_PTR(cu_seqlens);
  REQUIRE_PTR(row_flags);
  REQUIRE_PTR(k_per_seq);
  REQUIRE(min_den > 0 && min_num >= 0, "the minimum hit ratio is min_num / min_den, min_den > 0");
  REQUIRE(cu_seqlens[0] == 0, "cu_seqlens[0] must be 0");
  for (int32_t b = 0; b < n_seqs; ++b)
    REQUIRE(cu_seqlens[b + 1] >= cu_seqlens[b], "cu_seqlens must be non-decreasing");
  int32_t probed = 0;
  for (int32_t b = 0; b < n_seqs; ++b) {
    const int64_t lo = cu_seqlens[b], hi = cu_seqlens[b + 1];
    int64_t n_cand = 0;
    for (int64_t r = lo; r < hi; ++r) n_cand += (row_flags[r] & KVB_ROW_CANDIDATE) ? 1 : 0;
    if (n_cand > 0 && n_cand * min_den >= (int64_t)min_num * (hi - lo))
      ++probed;
    else
      k_per_seq[b] = 0;
  }
  if (n_probed) *n_probed = probed;
  return ok();
}

kvb_status kvb_rope_rows(int32_t head_dim, int64_t n_outer, int64_t n_rows, int64_t n_inner,
                         const float* x, const int32_t* row_pos, const int32_t* outer_pos,
                         const float* table_cos, const float* table_sin, int32_t table_len,
                         kvb_dtype out_dtype, void* out, void* stream) {
  if (kvb_status s = check_head_dim(head_dim)) return s;
  REQUIRE(n_outer > 0 && n_rows > 0 && n_inner > 0, "sizes must be positive");
  REQUIRE_PTR(x);
  REQUIRE_PTR(out);
  REQUIRE_ALIGNED(x);
  REQUIRE_ALIGNED(out);
  REQUIRE((table_cos == nullptr) == (table_sin == nullptr), "give both tables or neither");
  if (table_cos) {
    REQUIRE_PTR(row_pos);
    REQUIRE(table_len > 0, "table_len must be positive");
    REQUIRE_ALIGNED(table_cos);
    REQUIRE_ALIGNED(table_sin);
  }
  REQUIRE(out_dtype == KVB_BF16 || out_dtype == KVB_F32 || out_dtype == KVB_F64,
          "unknown out_dtype %d", (int)out_dtype);
  return hip_status(kvb::launch_rope_rows(head_dim, n_outer, n_rows, n_inner, x, row_pos,
                                          outer_pos, table_cos, table_sin, table_len, out_dtype,
                                          out, (hipStream_t)stream),
                    "kvb_rope_rows");
}

kvb_status kvb_kivi_quantize(const kvb_pool_layout* pool, int32_t n_pool, int32_t first_layer,
                             int32_t n_in, kvb_dtype in_dtype, const void* k_in, const void* v_in,
                             uint8_t* k_codes, float* k_scale, float* k_zero, uint8_t* v_codes,
                             float* v_scale, float* v_zero, void* stream) {
  if (kvb_status s = check_pool(pool)) return s;
  REQUIRE(n_pool > 0 && n_in > 0, "n_pool and n_in must be positive");
  REQUIRE(first_layer >= 0 && first_layer + n_in <= pool->n_layers, "layers out of range");
  REQUIRE(in_dtype == KVB_F32 || in_dtype == KVB_F64, "in_dtype must be F32 or F64");
  const void* ptrs[] = {k_in, v_in, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero};
  for (const void* p : ptrs) REQUIRE(p != nullptr && aligned16(p), "null or misaligned tensor");
  return hip_status(kvb::launch_kivi_quantize(*pool, n_pool, first_layer, n_in, in_dtype, k_in,
                                              v_in, k_codes, k_scale, k_zero, v_codes, v_scale,
                                              v_zero, (hipStream_t)stream),
                    "kvb_kivi_quantize");
}

kvb_status kvb_chunk_importance(const kvb_pool_layout* pool, int32_t n_pool, int32_t n_in,
                                kvb_dtype in_dtype, const void* k_in, double* importance,
                                void* stream) {
  if (kvb_status s = check_pool(pool)) return s;
  REQUIRE(n_pool > 0 && n_pool <= INT32_MAX / 2, "n_pool must be positive");
  REQUIRE(n_in > 0 && n_in <= pool->n_layers, "n_in must be in [1, n_layers]");
  REQUIRE(in_dtype == KVB_F32 || in_dtype == KVB_F64, "in_dtype must be F32 or F64");
  REQUIRE((int64_t)n_in * pool->n_kv_heads * pool->chunk_len <= INT32_MAX,
          "too many key vectors per chunk");
  REQUIRE(k_in != nullptr && aligned16(k_in), "null or misaligned key tensor");
  REQUIRE(importance != nullptr && aligned16(importance), "null or misaligned importance");
  return hip_status(kvb::launch_chunk_importance(*pool, n_pool, n_in, in_dtype, k_in, importance,
                                                 (hipStream_t)stream),
                    "kvb_chunk_importance");
}

kvb_status kvb_stitch(const kvb_pool_layout* pool, int32_t n_pool, const uint8_t* k_codes,
                      const float* k_scale, const float* k_zero, const uint8_t* v_codes,
                      const float* v_scale, const float* v_zero, const kvb_chunk* chunks,
                      int32_t n_chunks, const float* rope_cos, const float* rope_sin,
                      int64_t t_total, kvb_dtype out_dtype, void* k_cache, void* v_cache,
                      void* stream) {
  if (kvb_status s = check_pool(pool)) return s;
  REQUIRE(n_pool >= 0 && n_chunks >= 0, "n_pool and n_chunks must be non-negative");
  REQUIRE(n_pool > 0 || n_chunks == 0, "chunks listed with an empty pool");
  REQUIRE(t_total > 0 && t_total <= INT32_MAX, "t_total must be in (0, 2^31)");
  REQUIRE(out_dtype == KVB_BF16 || out_dtype == KVB_F32, "out_dtype must be BF16 or F32");
  REQUIRE((int64_t)pool->n_layers * pool->n_kv_heads <= 65535, "n_layers * n_kv_heads > 65535");
  const void* ptrs[] = {k_cache, v_cache, k_codes, k_scale, k_zero, v_codes, v_scale, v_zero};
  // an empty pool (nothing cached) may come with NULL pool arrays
  for (size_t i = 0; i < (n_pool > 0 ? 8u : 2u); ++i)
    REQUIRE(ptrs[i] != nullptr && aligned16(ptrs[i]), "null or misaligned tensor");
  if (n_chunks == 0) return ok();
  REQUIRE(chunks != nullptr && rope_cos != nullptr && rope_sin != nullptr,
          "chunks and rotation tables are required");
  REQUIRE(aligned16(rope_cos) && aligned16(rope_sin), "rotation tables must be 16-byte aligned");
  return hip_status(kvb::launch_stitch(*pool, n_pool, k_codes, k_scale, k_zero, v_codes, v_scale,
                                       v_zero, chunks, n_chunks, rope_cos, rope_sin, t_total,
                                       out_dtype, k_cache, v_cache, (hipStream_t)stream),
                    "kvb_stitch");
}

kvb_status kvb_stitch_deviation(const kvb_pool_layout* pool, int32_t n_pool,
                                const uint8_t* k_codes, const float* k_scale, const float* k_zero,
                                const uint8_t* v_codes, const float* v_scale, const float* v_zero,
                                const kvb_chunk* chunks, int32_t n_chunks, const float* rope_cos,
                                const float* rope_sin, int64_t t_total, uint16_t* k_cache,
                                uint16_t* v_cache, const uint16_t* k_fresh, float* delta,
                                void* stream) {
  if (kvb_status s = check_pool(pool)) return s;
  REQUIRE(n_pool >= 0 && n_chunks >= 0, "n_pool and n_chunks must be non-negative");
  REQUIRE(n_pool > 0 || n_chunks == 0, "chunks listed with an empty pool");
  REQUIRE(t_total > 0 && t_total <= INT32_MAX, "t_total must be in (0, 2^31)");
  REQUIRE(pool->n_layers <= 65535, "n_layers > 65535");
  const void* ptrs[] = {k_cache, v_cache, k_fresh, delta, k_codes,
                        k_scale, k_zero,  v_codes, v_scale, v_zero};
  // an empty pool (nothing cached) may come with NULL pool arrays
  for (size_t i = 0; i < (n_pool > 0 ? 10u : 4u); ++i)
    REQUIRE(ptrs[i] != nullptr && aligned16(ptrs[i]), "null or misaligned tensor");
  if (n_chunks == 0) return ok();
  REQUIRE(chunks != nullptr && rope_cos != nullptr && rope_sin != nullptr,
          "chunks and rotation tables are required");
  REQUIRE(aligned16(rope_cos) && aligned16(rope_sin), "rotation tables must be 16-byte aligned");
  return hip_status(kvb::launch_stitch_deviation(*pool, n_pool, k_codes, k_scale, k_zero, v_codes,
                                                 v_scale, v_zero, chunks, n_chunks, rope_cos,
                                                 rope_sin, t_total, k_cache, v_cache, k_fresh,
                                                 delta, (hipStream_t)stream),
                    "kvb_stitch_deviation");
}

static kvb_status check_deviation(int32_t n_layers, int32_t n_kv_heads, int32_t head_dim,
                                  int64_t t_total, const uint16_t* k_cache,
                                  const uint16_t* k_fresh, const uint16_t* v_cache,
                                  const uint16_t* v_fresh, float* delta) {
  if (kvb_status s = check_head_dim(head_dim)) return s;
  REQUIRE(n_layers > 0 && n_kv_heads > 0, "n_layers and n_kv_heads must be positive");
  if (n_kv_heads > 16 || (n_kv_heads & (n_kv_heads - 1)))
    return fail(KVB_EUNSUPPORTED, "n_kv_heads %d: must be a power of two up to 16", n_kv_heads);
  REQUIRE(t_total > 0 && t_total <= INT32_MAX, "t_total must be in (0, 2^31)");
  REQUIRE((v_cache == nullptr) == (v_fresh == nullptr), "give both value tensors or neither");
  const void* ptrs[] = {k_cache, k_fresh, delta};
  for (const void* p : ptrs) REQUIRE(p != nullptr && aligned16(p), "null or misaligned tensor");
  if (v_cache) REQUIRE(aligned16(v_cache) && aligned16(v_fresh), "misaligned value tensor");
  return KVB_OK;
}

kvb_status kvb_deviation(int32_t n_layers, int32_t n_kv_heads, int32_t head_dim, int64_t t_total,
                         const uint16_t* k_cache, const uint16_t* k_fresh,
                         const uint16_t* v_cache, const uint16_t* v_fresh, int32_t per_layer,
                         float* delta, void* stream) {
  if (kvb_status s = check_deviation(n_layers, n_kv_heads, head_dim, t_total, k_cache, k_fresh,
                                     v_cache, v_fresh, delta))
    return s;
  return hip_status(kvb::launch_deviation(n_layers, n_kv_heads, head_dim, t_total, k_cache,
                                          k_fresh, v_cache, v_fresh, per_layer, delta,
                                          (hipStream_t)stream),
                    "kvb_deviation");
}

size_t kvb_select_workspace_bytes(int32_t n_sets, int64_t t_total, int32_t n_seqs) {
  if (n_sets <= 0 || t_total <= 0 || n_seqs <= 0) return 0;
  return kvb::select_workspace_bytes(n_sets, t_total, n_seqs);
}

static kvb_status check_select(int32_t n_sets, int64_t t_total, const int32_t* cu_seqlens,
                               int32_t n_seqs, const float* delta, const uint8_t* row_flags,
                               const int32_t* k_per_seq, int32_t* rows, int32_t* cu_rows,
                               void* workspace, size_t workspace_bytes,
                               bool has_workspace = true) {
  REQUIRE(n_sets > 0 && n_sets <= 65535, "n_sets must be in [1, 65535]");
  REQUIRE(n_seqs > 0 && n_seqs <= 65535, "n_seqs must be in [1, 65535]");
  REQUIRE(t_total > 0 && t_total <= INT32_MAX, "t_total must be in (0, 2^31)");
  const void* ptrs[] = {cu_seqlens, delta, row_flags, k_per_seq, rows, cu_rows};
  for (const void* p : ptrs) REQUIRE(p != nullptr, "a required pointer is NULL");
  if (!has_workspace) return KVB_OK;
  const size_t need = kvb::select_workspace_bytes(n_sets, t_total, n_seqs);
  REQUIRE(workspace_bytes >= need, "workspace %zu bytes, need %zu", workspace_bytes, need);
  if (need) REQUIRE(workspace != nullptr && aligned16(workspace), "workspace NULL or misaligned");
  return KVB_OK;
}

kvb_status kvb_select(int32_t n_sets, int64_t t_total, const int32_t* cu_seqlens, int32_t n_seqs,
                      const float* delta, const uint8_t* row_flags, const int32_t* k_per_seq,
                      int32_t* rows, int32_t* cu_rows, void* workspace, size_t workspace_bytes,
                      void* stream) {
  if (kvb_status s = check_select(n_sets, t_total, cu_seqlens, n_seqs, delta, row_flags, k_per_seq,
                                  rows, cu_rows, workspace, workspace_bytes))
    return s;
  return hip_status(kvb::launch_select(n_sets, t_total, cu_seqlens, n_seqs, delta, row_flags,
                                       k_per_seq, rows, cu_rows, workspace, (hipStream_t)stream),
                    "kvb_select");
}

kvb_status kvb_select_noalloc(int32_t n_sets, int64_t t_total, const int32_t* cu_seqlens,
                              int32_t n_seqs, const float* delta, const uint8_t* row_flags,
                              const int32_t* k_per_seq, int32_t* rows, int32_t* cu_rows,
                              void* stream) {
  REQUIRE(n_sets > 0 && n_sets <= 65535, "n_sets must be in [1, 65535]");
  REQUIRE(n_seqs > 0 && n_seqs <= 65535, "n_seqs must be in [1, 65535]");
  REQUIRE(t_total > 0 && t_total <= INT32_MAX, "t_total must be in (0, 2^31)");
  const size_t need = kvb::select_workspace_bytes(n_sets, t_total, n_seqs);
  REQUIRE(need <= kvb::kSelectScratchBytes,
          "kvb_select_noalloc: %d sets x %lld rows need %zu bytes of scratch, more than its "
          "%zu (use kvb_select with a workspace)",
          n_sets, (long long)t_total, need, kvb::kSelectScratchBytes);
  if (kvb_status s = check_select(n_sets, t_total, cu_seqlens, n_seqs, delta, row_flags,
                                  k_per_seq, rows, cu_rows, nullptr, 0, /*has_workspace=*/false))
    return s;
  return hip_status(kvb::launch_select_noalloc(n_sets, t_total, cu_seqlens, n_seqs, delta,
                                               row_flags, k_per_seq, rows, cu_rows,
                                               (hipStream_t)stream),
                    "kvb_select_noalloc");
}

size_t kvb_select_noalloc_max_bytes(void) { return kvb::kSelectScratchBytes; }

kvb_status kvb_deviation_topk(int32_t n_layers, int32_t n_kv_heads, int32_t head_dim,
                              int64_t t_total, const int32_t* cu_seqlens, int32_t n_seqs,
                              const uint16_t* k_cache, const uint16_t* k_fresh,
                              const uint16_t* v_cache, const uint16_t* v_fresh, int32_t per_layer,
                              const uint8_t* row_flags, const int32_t* k_per_seq, float* delta,
                              int32_t* rows, int32_t* cu_rows, void* workspace,
                              size_t workspace_bytes, void* stream) {
  if (kvb_status s = check_deviation(n_layers, n_kv_heads, head_dim, t_total, k_cache, k_fresh,
                                     v_cache, v_fresh, delta))
    return s;
  const int32_t n_sets = per_layer ? n_layers : 1;
  if (kvb_status s = check_select(n_sets, t_total, cu_seqlens, n_seqs, delta, row_flags, k_per_seq,
                                  rows, cu_rows, workspace, workspace_bytes))
    return s;
  hipStream_t s = (hipStream_t)stream;
  if (kvb_status st = hip_status(kvb::launch_deviation(n_layers, n_kv_heads, head_dim, t_total,
                                                       k_cache, k_fresh, v_cache, v_fresh,
                                                       per_layer, delta, s),
                                 "kvb_deviation_topk (deviation)"))
    return st;
  return hip_status(kvb::launch_select(n_sets, t_total, cu_seqlens, n_seqs, delta, row_flags,
                                       k_per_seq, rows, cu_rows, workspace, s),
                    "kvb_deviation_topk (select)");
}

size_t kvb_sparse_attn_workspace_bytes(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads,
                                       int32_t head_dim, int64_t t_total, int32_t n_seqs,
                                       int32_t max_seq_len, int32_t max_rows,
                                       int32_t v_f16_given) {
  if (n_layers <= 0 || n_q_heads <= 0 || n_kv_heads <= 0 || n_q_heads % n_kv_heads ||
      head_dim <= 0 || t_total <= 0 || n_seqs <= 0 || max_seq_len <= 0 || max_rows < 0)
    return 0;
  kvb::AttnPlan plan;
  if (!kvb::attn_plan(n_layers, n_q_heads, n_kv_heads, head_dim, t_total, n_seqs, max_seq_len,
                      max_rows, v_f16_given != 0, &plan))
    return 0;
  return plan.workspace;
}

}  // extern "C"

namespace {

// Size checks shared by the attention entry points.
kvb_status check_attn_sizes(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads,
                            int32_t head_dim, int64_t t_total, int32_t n_seqs,
                            int32_t max_seq_len, int32_t max_rows) {
  if (kvb_status s = check_head_dim(head_dim)) return s;
  REQUIRE(n_layers > 0 && n_q_heads > 0 && n_kv_heads > 0, "head counts and layers must be positive");
  REQUIRE(n_q_heads % n_kv_heads == 0, "n_q_heads %d not a multiple of n_kv_heads %d", n_q_heads,
          n_kv_heads);
  const int G = n_q_heads / n_kv_heads;
  if (G > 32 || (32 % G) != 0)
    return fail(KVB_EUNSUPPORTED, "n_q_heads / n_kv_heads = %d must divide 32", G);
  REQUIRE(t_total > 0 && t_total <= INT32_MAX, "t_total must be in (0, 2^31)");
  REQUIRE(n_seqs > 0, "n_seqs must be positive");
  REQUIRE(max_seq_len > 0 && max_seq_len <= t_total, "max_seq_len must be in (0, t_total]");
  REQUIRE(max_rows >= 0 && max_rows <= t_total, "max_rows must be in [0, t_total]");
  REQUIRE((int64_t)n_layers * n_kv_heads <= 65535, "n_layers * n_kv_heads > 65535");
  return ok();
}

// Plan of one layer's attention launch (the fp16 shadow of V given).
kvb_status layer_plan(int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int64_t t_total,
                      int32_t n_seqs, int32_t max_seq_len, int32_t max_rows, kvb::AttnPlan* plan) {
  if (!kvb::attn_plan(1, n_q_heads, n_kv_heads, head_dim, t_total, n_seqs, max_seq_len, max_rows,
                      true, plan))
    return fail(KVB_EUNSUPPORTED, "too many attention work units (kv heads x row tiles x key blocks)");
  return ok();
}

}  // namespace

extern "C" {

size_t kvb_attn_plans_bytes(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads,
                            int32_t head_dim, int64_t t_total, int32_t n_seqs, int32_t max_seq_len,
                            int32_t max_rows) {
  if (n_layers <= 0 || n_q_heads <= 0 || n_kv_heads <= 0 || n_q_heads % n_kv_heads ||
      head_dim <= 0 || t_total <= 0 || n_seqs <= 0 || max_seq_len <= 0 || max_rows < 0)
    return 0;
  kvb::AttnPlan plan;
  if (!kvb::attn_plan(1, n_q_heads, n_kv_heads, head_dim, t_total, n_seqs, max_seq_len, max_rows,
                      true, &plan))
    return 0;
  return (size_t)n_layers * kvb::layer_plan_stride(plan);
}

kvb_status kvb_patch(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                     int64_t t_total, const int32_t* cu_seqlens, int32_t n_seqs,
                     int32_t max_seq_len, const int32_t* rows, const int32_t* cu_rows,
                     int32_t rows_per_layer, int32_t max_rows, const uint16_t* k_fresh,
                     const uint16_t* v_fresh, uint16_t* k_cache, uint16_t* v_cache,
                     uint16_t* v_cache_f16, uint32_t* v_status, void* plans, size_t plans_bytes,
                     void* stream) {
  if (kvb_status s = check_attn_sizes(n_layers, n_q_heads, n_kv_heads, head_dim, t_total, n_seqs,
                                      max_seq_len, max_rows))
    return s;
  const void* ptrs[] = {cu_seqlens, rows, cu_rows};
  for (const void* p : ptrs) REQUIRE(p != nullptr, "a required index pointer is NULL");
  const void* tens[] = {k_fresh, v_fresh, k_cache, v_cache};
  for (const void* p : tens) REQUIRE(p != nullptr && aligned16(p), "null or misaligned tensor");
  if (v_cache_f16) REQUIRE(aligned16(v_cache_f16), "misaligned fp16 copy of V");
  REQUIRE(v_status == nullptr || v_cache_f16 != nullptr, "v_status without an fp16 copy of V");
  REQUIRE((reinterpret_cast<uintptr_t>(v_status) & 3u) == 0, "misaligned v_status");
  kvb::AttnPlan plan;
  if (kvb_status s = layer_plan(n_q_heads, n_kv_heads, head_dim, t_total, n_seqs, max_seq_len,
                                max_rows, &plan))
    return s;
  if (plans) {
    const size_t need = (size_t)n_layers * kvb::layer_plan_stride(plan);
    REQUIRE(plans_bytes >= need, "plans %zu bytes, need %zu", plans_bytes, need);
    REQUIRE(aligned16(plans), "misaligned plans");
  }
  if (max_rows == 0 && v_cache_f16 == nullptr) return ok();
  return hip_status(kvb::launch_patch_layers(plan, n_layers, n_kv_heads, head_dim, t_total,
                                             cu_seqlens, n_seqs, rows, cu_rows, rows_per_layer,
                                             max_rows, k_fresh, v_fresh, k_cache, v_cache,
                                             v_cache_f16, v_status, plans, (hipStream_t)stream),
                    "kvb_patch");
}

kvb_status kvb_sparse_attn_layer(int32_t layer, int32_t n_layers, int32_t n_q_heads,
                                 int32_t n_kv_heads, int32_t head_dim, int64_t t_total,
                                 const int32_t* cu_seqlens, int32_t n_seqs, int32_t max_seq_len,
                                 const int32_t* rows, const int32_t* cu_rows,
                                 int32_t rows_per_layer, int32_t max_rows, const uint16_t* q,
                                 const uint16_t* k_cache, const uint16_t* v_cache_f16,
                                 const void* plans, size_t plans_bytes, float softmax_scale,
                                 kvb_dtype out_dtype, void* out, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  if (kvb_status s = check_attn_sizes(n_layers, n_q_heads, n_kv_heads, head_dim, t_total, n_seqs,
                                      max_seq_len, max_rows))
    return s;
  REQUIRE(layer >= 0 && layer < n_layers, "layer %d outside [0, %d)", layer, n_layers);
  REQUIRE(out_dtype == KVB_BF16 || out_dtype == KVB_F32, "out_dtype must be BF16 or F32");
  REQUIRE(softmax_scale > 0.0f && isfinite(softmax_scale), "softmax_scale must be positive");
  const void* ptrs[] = {cu_seqlens, rows, cu_rows};
  for (const void* p : ptrs) REQUIRE(p != nullptr, "a required index pointer is NULL");
  const void* tens[] = {q, k_cache, v_cache_f16, out, plans};
  for (const void* p : tens)
    REQUIRE(p != nullptr && aligned16(p), "null or misaligned tensor, shadow of V or plans");
  kvb::AttnPlan plan;
  if (kvb_status s = layer_plan(n_q_heads, n_kv_heads, head_dim, t_total, n_seqs, max_seq_len,
                                max_rows, &plan))
    return s;
  const size_t need = (size_t)n_layers * kvb::layer_plan_stride(plan);
  REQUIRE(plans_bytes >= need, "plans %zu bytes, need %zu", plans_bytes, need);
  REQUIRE(workspace_bytes >= plan.workspace, "workspace %zu bytes, need %zu", workspace_bytes,
          plan.workspace);
  REQUIRE(workspace != nullptr && aligned16(workspace), "workspace NULL or misaligned");
  if (max_rows == 0) return ok();
  return hip_status(kvb::launch_sparse_attn_layer(plan, layer, n_q_heads, n_kv_heads, head_dim,
                                                  t_total, cu_seqlens, n_seqs, rows, cu_rows,
                                                  rows_per_layer, q, k_cache, v_cache_f16, plans,
                                                  softmax_scale, out_dtype, out, workspace,
                                                  (hipStream_t)stream),
                    "kvb_sparse_attn_layer");
}

kvb_status kvb_sparse_attn(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads,
                           int32_t head_dim, int64_t t_total, const int32_t* cu_seqlens,
                           int32_t n_seqs, int32_t max_seq_len, const int32_t* rows,
                           const int32_t* cu_rows, int32_t rows_per_layer, int32_t max_rows,
                           const uint16_t* q, const uint16_t* k_fresh, const uint16_t* v_fresh,
                           uint16_t* k_cache, uint16_t* v_cache, uint16_t* v_cache_f16,
                           uint32_t* v_status, float softmax_scale, kvb_dtype out_dtype, void* out,
                           void* workspace, size_t workspace_bytes, void* stream) {
  if (kvb_status s = check_attn_sizes(n_layers, n_q_heads, n_kv_heads, head_dim, t_total, n_seqs,
                                      max_seq_len, max_rows))
    return s;
  REQUIRE(out_dtype == KVB_BF16 || out_dtype == KVB_F32, "out_dtype must be BF16 or F32");
  REQUIRE(softmax_scale > 0.0f && isfinite(softmax_scale), "softmax_scale must be positive");
  const void* ptrs[] = {cu_seqlens, rows, cu_rows};
  for (const void* p : ptrs) REQUIRE(p != nullptr, "a required index pointer is NULL");
  const void* tens[] = {q, k_fresh, v_fresh, k_cache, v_cache, out};
  for (const void* p : tens) REQUIRE(p != nullptr && aligned16(p), "null or misaligned tensor");
  if (v_cache_f16) REQUIRE(aligned16(v_cache_f16), "misaligned fp16 copy of V");
  REQUIRE((reinterpret_cast<uintptr_t>(v_status) & 3u) == 0, "misaligned v_status");
  kvb::AttnPlan plan;
  if (!kvb::attn_plan(n_layers, n_q_heads, n_kv_heads, head_dim, t_total, n_seqs, max_seq_len,
                      max_rows, v_cache_f16 != nullptr, &plan))
    return fail(KVB_EUNSUPPORTED, "too many attention work units (layers x kv heads x row tiles x key blocks)");
  REQUIRE(workspace_bytes >= plan.workspace, "workspace %zu bytes, need %zu", workspace_bytes,
          plan.workspace);
  if (plan.workspace) REQUIRE(workspace != nullptr && aligned16(workspace), "workspace NULL or misaligned");
  if (max_rows == 0) {
    // nothing to patch or attend; a caller-kept fp16 copy of V still follows the cache
    if (v_cache_f16 == nullptr) return ok();
    return hip_status(kvb::launch_fp16_copy(n_layers, n_kv_heads, head_dim, t_total, v_cache,
                                            v_cache_f16, v_status, (hipStream_t)stream),
                      "kvb_sparse_attn");
  }
  return hip_status(kvb::launch_sparse_attn(plan, n_layers, n_q_heads, n_kv_heads, head_dim,
                                            t_total, cu_seqlens, n_seqs, rows, cu_rows,
                                            rows_per_layer, max_rows, q, k_fresh, v_fresh, k_cache,
                                            v_cache, v_cache_f16, v_status, softmax_scale,
                                            out_dtype, out, workspace, (hipStream_t)stream),
                    "kvb_sparse_attn");
}

}  // extern "C"
