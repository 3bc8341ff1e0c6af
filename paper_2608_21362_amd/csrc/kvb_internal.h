// Internal declarations shared by the HIP translation units of libkvb.
// Launchers validate nothing: the C entry points in kvb_api.cpp have already
// checked every host-visible argument.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvb.h"

namespace kvb {

// ---- population ---------------------------------------------------------
hipError_t launch_rope_rows(int head_dim, int64_t n_outer, int64_t n_rows, int64_t n_inner,
                            const float* x, const int32_t* row_pos, const int32_t* outer_pos,
                            const float* tcos, const float* tsin, int32_t table_len,
                            kvb_dtype out_dtype, void* out, hipStream_t s);

hipError_t launch_kivi_quantize(const kvb_pool_layout& p, int32_t n_pool, int32_t first_layer,
                                int32_t n_in, kvb_dtype in_dtype, const void* k_in,
                                const void* v_in, uint8_t* k_codes, float* k_scale, float* k_zero,
                                uint8_t* v_codes, float* v_scale, float* v_zero, hipStream_t s);
hipError_t launch_chunk_importance(const kvb_pool_layout& p, int32_t n_pool, int32_t n_in,
                                   kvb_dtype in_dtype, const void* k_in, double* importance,
                                   hipStream_t s);

// ---- hot path -------------------------------------------------------------
hipError_t launch_stitch(const kvb_pool_layout& p, int32_t n_pool, const uint8_t* k_codes,
                         const float* k_scale, const float* k_zero, const uint8_t* v_codes,
                         const float* v_scale, const float* v_zero, const kvb_chunk* chunks,
                         int32_t n_chunks, const float* rope_cos, const float* rope_sin,
                         int64_t t_total, kvb_dtype out_dtype, void* k_cache, void* v_cache,
                         hipStream_t s);

// Stitch plus the per-layer K deviation of the stitched rows (bf16 cache).
hipError_t launch_stitch_deviation(const kvb_pool_layout& p, int32_t n_pool,
                                   const uint8_t* k_codes, const float* k_scale,
                                   const float* k_zero, const uint8_t* v_codes,
                                   const float* v_scale, const float* v_zero,
                                   const kvb_chunk* chunks, int32_t n_chunks,
                                   const float* rope_cos, const float* rope_sin, int64_t t_total,
                                   void* k_cache, void* v_cache, const uint16_t* k_fresh,
                                   float* delta, hipStream_t s);

hipError_t launch_deviation(int n_layers, int n_kv_heads, int head_dim, int64_t t_total,
                            const uint16_t* k_cache, const uint16_t* k_fresh,
                            const uint16_t* v_cache, const uint16_t* v_fresh, int per_layer,
                            float* delta, hipStream_t s);

size_t select_workspace_bytes(int32_t n_sets, int64_t t_total, int32_t n_seqs);
hipError_t launch_select(int32_t n_sets, int64_t t_total, const int32_t* cu_seqlens,
                         int32_t n_seqs, const float* delta, const uint8_t* row_flags,
                         const int32_t* k_per_seq, int32_t* rows, int32_t* cu_rows,
                         void* workspace, hipStream_t s);

// Allocation-free selection: the staging of kvb_select in a static device
// array of kSelectScratchBytes bytes per device (no workspace argument).
constexpr size_t kSelectScratchBytes = size_t(16) << 20;
constexpr int kMaxDevices = 64;
hipError_t launch_select_noalloc(int32_t n_sets, int64_t t_total, const int32_t* cu_seqlens,
                                 int32_t n_seqs, const float* delta, const uint8_t* row_flags,
                                 const int32_t* k_per_seq, int32_t* rows, int32_t* cu_rows,
                                 hipStream_t s);

struct AttnPlan {
  int rows_per_tile;   // selected rows per workgroup tile
  int tile_slots;      // tile slots per (layer, kv head)
  int n_tiles;         // layers x kv heads x tile slots
  int n_wg_max;        // most attention workgroups a launch uses
  int n_rec;           // partial records (two per workgroup)
  int max_seq_len;     // longest prompt (bounds the key blocks of any tile)
  bool v16_in_ws;      // the fp16 copy of V lives in the workspace (no shadow given)
  size_t v16_offset;   // workspace offset of the fp16 copy of V
  size_t plan_offset;  // workspace offset of the work decomposition (int32)
  size_t parts_offset; // workspace offset of the partial records
  size_t workspace;    // total workspace bytes
};
bool attn_plan(int n_layers, int n_q_heads, int n_kv_heads, int head_dim, int64_t t_total,
               int n_seqs, int max_seq_len, int max_rows, bool v16_given, AttnPlan* plan);
hipError_t launch_sparse_attn(const AttnPlan& plan, int n_layers, int n_q_heads, int n_kv_heads,
                              int head_dim, int64_t t_total, const int32_t* cu_seqlens,
                              int n_seqs, const int32_t* rows, const int32_t* cu_rows,
                              int rows_per_layer, int max_rows, const uint16_t* q,
                              const uint16_t* k_fresh, const uint16_t* v_fresh,
                              uint16_t* k_cache, uint16_t* v_cache, uint16_t* v_cache_f16,
                              uint32_t* v_status, float softmax_scale, kvb_dtype out_dtype,
                              void* out, void* workspace, hipStream_t s);

// Bytes of one layer's plan in a buffer of per-layer plans (a multiple of 256).
size_t layer_plan_stride(const AttnPlan& layer_plan);
// Patch of n_layers layers; with plans != NULL also the per-layer plans
// (layer_plan is the one-layer plan, the fp16 copy of V given), and with
// v_cache_f16 != NULL the fp16 copy of the patched V cache.
hipError_t launch_patch_layers(const AttnPlan& layer_plan, int n_layers, int n_kv_heads,
                               int head_dim, int64_t t_total, const int32_t* cu_seqlens,
                               int n_seqs, const int32_t* rows, const int32_t* cu_rows,
                               int rows_per_layer, int max_rows, const uint16_t* k_fresh,
                               const uint16_t* v_fresh, uint16_t* k_cache, uint16_t* v_cache,
                               uint16_t* v_cache_f16, uint32_t* v_status, void* plans,
                               hipStream_t s);
// fp16 copy of the V cache of n_layers layers; with status != NULL, 1 is
// stored there when a value fp16 cannot hold is met.
hipError_t launch_fp16_copy(int n_layers, int n_kv_heads, int head_dim, int64_t t_total,
                            const uint16_t* v, uint16_t* v16, uint32_t* status, hipStream_t s);
// Attention of layer `layer` over the patched cache with its prebuilt plan.
hipError_t launch_sparse_attn_layer(const AttnPlan& layer_plan, int layer, int n_q_heads,
                                    int n_kv_heads, int head_dim, int64_t t_total,
                                    const int32_t* cu_seqlens, int n_seqs, const int32_t* rows,
                                    const int32_t* cu_rows, int rows_per_layer, const uint16_t* q,
                                    const uint16_t* k_cache, const uint16_t* v_cache_f16,
                                    const void* plans, float softmax_scale, kvb_dtype out_dtype,
                                    void* out, void* workspace, hipStream_t s);

}  // namespace kvb
