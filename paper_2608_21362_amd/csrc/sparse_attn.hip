// Patch and sparse-query causal GQA attention (Alg. 2 step 4; Eq. 2).
//
// patch_kernel: cache[l][h][t] <- fresh[l][h][t] for every selected row t,
// both tensors, every kv head (one wave per row).
//
// attn_kernel: one workgroup = one (layer, kv head g, tile of selected rows,
// KV split).  The tile packs rows x the G = Hq/Hkv query heads that share kv
// head g into the MFMA N dimension: each of the 4 waves owns 32 query vectors
// (32/G rows x G heads).  Keys stream through LDS in blocks of 64:
//
//   S^T (64 keys x 32 queries) = K Q^T      bf16 MFMA 32x32x16 (K from LDS as
//                                            the A operand, Q^T held in VGPRs)
//   online softmax over keys                fp32, base-2 exponent; each lane
//                                            holds 32 scores of one query, the
//                                            other 32 sit in lane ^ 32
//   O^T (d x 32 queries) += V^T P^T         fp16 MFMA 32x32x16 (V^T from LDS,
//                                            P^T straight from the S^T
//                                            accumulators)
//
// V is stored in LDS transposed ([d][key], fp16) with the keys of every
// 16-key group permuted so that the 8 keys a lane contributes to one P^T
// operand (the accumulator layout gives lane half h the keys
// {4h..4h+3, 8+4h..8+4h+3}) are 16 contiguous bytes.  The contraction
// dimension of both products is only ever indexed consistently on the two
// operands, so its lane order inside the MFMA does not matter.
//
// The next key block is loaded from HBM into registers while the current one
// is consumed from LDS.  A tile whose key range is longer than the split
// length is cut into splits whose (max, sum, O) partials go to the workspace
// and are merged in split order by combine_kernel (deterministic).
#include <math.h>

#include "kvb_device.h"
#include "kvb_internal.h"

namespace kvb {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
typedef __attribute__((ext_vector_type(2))) _Float16 f16x2;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kQW = 32;                 // query vectors per wave
constexpr int kQT = kQW * kWaves;       // query vectors per workgroup
constexpr int kKB = 64;                 // keys per block
constexpr int kVtStride = kKB + 8;      // fp16 elements per transposed-V row

// ---------------------------------------------------------------- patch ----
__global__ void __launch_bounds__(256)
patch_kernel(int32_t L, int32_t Hkv, int32_t D, int64_t t_total, int32_t n_seqs,
             const int32_t* __restrict__ rows, const int32_t* __restrict__ cu_rows,
             int32_t rows_per_layer, int32_t max_rows, const uint16_t* __restrict__ kf,
             const uint16_t* __restrict__ vf, uint16_t* __restrict__ kc,
             uint16_t* __restrict__ vc) {
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t l = wave / max_rows;
  const int64_t i = wave % max_rows;
  if (l >= L) return;
  const int64_t set = rows_per_layer ? l : 0;
  const int32_t n = cu_rows[set * (n_seqs + 1) + n_seqs];
  if (i >= n) return;
  const int64_t t = rows[set * t_total + i];
  if (t < 0 || t >= t_total) return;
  const int chunks = D / 8;  // 16-byte pieces per head row
  for (int e = lane; e < 2 * Hkv * chunks; e += 64) {
    const int tensor = e / (Hkv * chunks);
    const int h = (e / chunks) % Hkv;
    const int c = e % chunks;
    const int64_t off = (((l * Hkv + h) * t_total) + t) * D + c * 8;
    if (tensor == 0)
      *reinterpret_cast<uint4*>(kc + off) = *reinterpret_cast<const uint4*>(kf + off);
    else
      *reinterpret_cast<uint4*>(vc + off) = *reinterpret_cast<const uint4*>(vf + off);
  }
}

// ------------------------------------------------------------ tile lookup --
struct Tile {
  int b;          // prompt
  int r_begin;    // first entry of the tile in the set's row list
  int r_end;
};

__device__ __forceinline__ bool find_tile(const int32_t* cur, int n_seqs, int rows_per_tile,
                                          int slot, Tile* t) {
  int acc = 0;
  for (int b = 0; b < n_seqs; ++b) {
    const int nb = cur[b + 1] - cur[b];
    const int nt = (nb + rows_per_tile - 1) / rows_per_tile;
    if (slot < acc + nt) {
      t->b = b;
      t->r_begin = cur[b] + (slot - acc) * rows_per_tile;
      t->r_end = min(t->r_begin + rows_per_tile, cur[b + 1]);
      return true;
    }
    acc += nt;
  }
  return false;
}

__device__ __forceinline__ uint32_t bf16pair_to_f16pair(uint32_t w) {
  f32x2 f = {bf16_lo(w), bf16_hi(w)};
  f16x2 h = __builtin_convertvector(f, f16x2);
  return __builtin_bit_cast(uint32_t, h);
}

// ---------------------------------------------------------------- attention
template <int D>
__global__ void __launch_bounds__(kThreads, 2)
attn_kernel(int32_t Hq, int32_t Hkv, int32_t log2g, int64_t t_total,
            const int32_t* __restrict__ cu_seqlens, int32_t n_seqs,
            const int32_t* __restrict__ rows, const int32_t* __restrict__ cu_rows,
            int32_t rows_per_layer, int32_t rows_per_tile, int32_t tile_slots, int32_t split_len,
            int32_t n_split_max, const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
            const uint16_t* __restrict__ vc, float scale_log2, int32_t out_f32,
            void* __restrict__ out, float* __restrict__ ws) {
  constexpr int NS = D / 16;        // bf16 MFMA steps over d
  constexpr int ND = D / 32;        // 32-row tiles of d in O^T
  constexpr int KS = D + 8;         // bf16 elements per K row in LDS
  constexpr int KCH = D / 8;        // 16-byte chunks per K row
  constexpr int KLD = kKB * KCH / kThreads;  // K chunks per thread per block
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kKB * KS];
  __shared__ __attribute__((aligned(16))) uint16_t vt_lds[D * kVtStride];

  const int G = 1 << log2g;
  const int lg = blockIdx.z;
  const int l = lg / Hkv, g = lg % Hkv;
  const int slot = blockIdx.x, split = blockIdx.y;
  const int64_t set = rows_per_layer ? l : 0;
  const int32_t* cur = cu_rows + set * (n_seqs + 1);
  const int32_t* rws = rows + set * t_total;
  Tile tile;
  if (!find_tile(cur, n_seqs, rows_per_tile, slot, &tile)) return;
  const int64_t kstart = cu_seqlens[tile.b];
  const int64_t kend = min((int64_t)rws[tile.r_end - 1] + 1, t_total);
  if (kend <= kstart) return;
  const int n_split = (int)((kend - kstart + split_len - 1) / split_len);
  if (split >= n_split || n_split > n_split_max) return;
  const int64_t k_lo = kstart + (int64_t)split * split_len;
  const int64_t k_hi = min(k_lo + (int64_t)split_len, kend);
  const int64_t t_min = rws[tile.r_begin];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, n = lane & 31;
  const int rows_per_wave = kQW >> log2g;
  const int row_idx = tile.r_begin + wave * rows_per_wave + (n >> log2g);
  const int head = g * G + (n & (G - 1));
  int64_t t_q = row_idx < tile.r_end ? (int64_t)rws[row_idx] : -1;
  const bool qvalid = t_q >= kstart && t_q < kend;  // rows outside the prompt are skipped
  if (!qvalid) t_q = -1;

  // Q^T operand: query n, d = (D/2)*half + 8s + v
  bf16x8 qop[NS];
  {
    const uint16_t* qp = q + (((int64_t)l * t_total + (qvalid ? t_q : 0)) * Hq + head) * D +
                         (D / 2) * half;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      uint4 w = qvalid ? *reinterpret_cast<const uint4*>(qp + 8 * s) : make_uint4(0, 0, 0, 0);
      qop[s] = __builtin_bit_cast(bf16x8, w);
    }
  }

  const int64_t kv_base = ((int64_t)l * Hkv + g) * t_total;
  const uint16_t* kb_ptr = kc + kv_base * D;
  const uint16_t* vb_ptr = vc + kv_base * D;

  // register stage of one key block
  uint4 kreg[KLD];
  uint4 vreg[4];
  const bool v_job = tid < 16 * KCH;  // (key quad, 8-channel group) jobs
  const int kq = tid & 15, dg = tid >> 4;
  auto load_block = [&](int64_t kb) {
#pragma unroll
    for (int i = 0; i < KLD; ++i) {
      const int ci = tid + kThreads * i;
      int64_t key = kb + ci / KCH;
      key = key < t_total ? key : t_total - 1;
      kreg[i] = *reinterpret_cast<const uint4*>(kb_ptr + key * D + (ci % KCH) * 8);
    }
    if (v_job) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        int64_t key = kb + 4 * kq + r;
        key = key < t_total ? key : t_total - 1;
        vreg[r] = *reinterpret_cast<const uint4*>(vb_ptr + key * D + dg * 8);
      }
    }
  };
  auto store_block = [&]() {
#pragma unroll
    for (int i = 0; i < KLD; ++i) {
      const int ci = tid + kThreads * i;
      *reinterpret_cast<uint4*>(&k_lds[(ci / KCH) * KS + (ci % KCH) * 8]) = kreg[i];
    }
    if (v_job) {
      // key quad kq -> position base inside its 16-key group
      const int run = kq & 3;
      const int pos = (kq >> 2) * 16 + ((run == 1) ? 8 : (run == 2) ? 4 : (run == 3) ? 12 : 0);
      const uint32_t w[4][4] = {{vreg[0].x, vreg[0].y, vreg[0].z, vreg[0].w},
                                {vreg[1].x, vreg[1].y, vreg[1].z, vreg[1].w},
                                {vreg[2].x, vreg[2].y, vreg[2].z, vreg[2].w},
                                {vreg[3].x, vreg[3].y, vreg[3].z, vreg[3].w}};
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        // channel dg*8 + j of keys 4kq .. 4kq+3
        uint32_t e[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) e[r] = (j & 1) ? (w[r][j >> 1] >> 16) : (w[r][j >> 1] & 0xFFFFu);
        const uint32_t p01 = bf16pair_to_f16pair(e[0] | (e[1] << 16));
        const uint32_t p23 = bf16pair_to_f16pair(e[2] | (e[3] << 16));
        *reinterpret_cast<uint2*>(&vt_lds[(dg * 8 + j) * kVtStride + pos]) = make_uint2(p01, p23);
      }
    }
  };

  f32x16 o[ND];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) o[dt] = f32x16{};
  float m_run = -INFINITY, l_run = 0.0f;

  int64_t kb = k_lo;
  load_block(kb);
  for (; kb < k_hi; kb += kKB) {
    __syncthreads();
    store_block();
    __syncthreads();
    if (kb + kKB < k_hi) load_block(kb + kKB);

    // S^T = K Q^T for keys kb .. kb+63
    f32x16 sacc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      sacc[kt] = f32x16{};
      const uint16_t* krow = &k_lds[(kt * 32 + n) * KS + (D / 2) * half];
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(krow + 8 * s);
        sacc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qop[s], sacc[kt], 0, 0, 0);
      }
    }

    // mask, scale to log2 units, block max
    const bool full = (kb + kKB - 1 <= t_min) && (kb + kKB <= k_hi);
    float bmax = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v = sacc[kt][r] * scale_log2;
        if (!full) {
          const int64_t key = kb + kt * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          if (key > t_q || key >= k_hi) v = -INFINITY;
        }
        sacc[kt][r] = v;
        bmax = fmaxf(bmax, v);
      }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
    const float m_new = fmaxf(m_run, bmax);
    const float m_use = (m_new == -INFINITY) ? 0.0f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    float bsum = 0.0f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(sacc[kt][r] - m_use);
        sacc[kt][r] = p;
        bsum += p;
      }
    bsum += __shfl_xor(bsum, 32, 64);
    l_run = l_run * alpha + bsum;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;

    // O^T += V^T P^T, four 16-key steps
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int kt = ks >> 1, r0 = 8 * (ks & 1);
      f16x8 pb;
#pragma unroll
      for (int v = 0; v < 8; v += 2) {
        f32x2 f = {sacc[kt][r0 + v], sacc[kt][r0 + v + 1]};
        f16x2 h = __builtin_convertvector(f, f16x2);
        pb[v] = h[0];
        pb[v + 1] = h[1];
      }
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) {
        const f16x8 a = *reinterpret_cast<const f16x8*>(
            &vt_lds[(dt * 32 + n) * kVtStride + ks * 16 + 8 * half]);
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, pb, o[dt], 0, 0, 0);
      }
    }
  }

  if (!qvalid) return;
  if (n_split == 1) {
    const float inv = (l_run > 0.0f) ? 1.0f / l_run : 0.0f;
    const int64_t ob = (((int64_t)l * t_total + t_q) * Hq + head) * D;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int d0 = dt * 32 + 8 * j + 4 * half;
        const float a0 = o[dt][4 * j] * inv, a1 = o[dt][4 * j + 1] * inv;
        const float a2 = o[dt][4 * j + 2] * inv, a3 = o[dt][4 * j + 3] * inv;
        if (out_f32) {
          *reinterpret_cast<float4*>(reinterpret_cast<float*>(out) + ob + d0) =
              make_float4(a0, a1, a2, a3);
        } else {
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(out) + ob + d0) =
              make_uint2(pack_bf16x2(a0, a1), pack_bf16x2(a2, a3));
        }
      }
  } else {
    const int64_t item = ((int64_t)lg * tile_slots + slot) * n_split_max + split;
    float* wp = ws + (item * kQT + wave * kQW + n) * (D + 2);
#pragma unroll
    for (int dt = 0; dt < ND; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int d0 = dt * 32 + 8 * j + 4 * half;
        // D + 2 floats per query: 8-byte aligned, so store in pairs
        *reinterpret_cast<float2*>(wp + d0) = make_float2(o[dt][4 * j], o[dt][4 * j + 1]);
        *reinterpret_cast<float2*>(wp + d0 + 2) = make_float2(o[dt][4 * j + 2], o[dt][4 * j + 3]);
      }
    if (half == 0) {
      wp[D] = m_run;
      wp[D + 1] = l_run;
    }
  }
}

// Merge the split partials of every multi-split tile, in split order.
template <int D>
__global__ void __launch_bounds__(256)
combine_kernel(int32_t Hq, int32_t Hkv, int32_t log2g, int64_t t_total,
               const int32_t* __restrict__ cu_seqlens, int32_t n_seqs,
               const int32_t* __restrict__ rows, const int32_t* __restrict__ cu_rows,
               int32_t rows_per_layer, int32_t rows_per_tile, int32_t tile_slots,
               int32_t split_len, int32_t n_split_max, int32_t out_f32, void* __restrict__ out,
               const float* __restrict__ ws) {
  const int G = 1 << log2g;
  const int lg = blockIdx.y;
  const int l = lg / Hkv, g = lg % Hkv;
  const int slot = blockIdx.x;
  const int64_t set = rows_per_layer ? l : 0;
  const int32_t* cur = cu_rows + set * (n_seqs + 1);
  const int32_t* rws = rows + set * t_total;
  Tile tile;
  if (!find_tile(cur, n_seqs, rows_per_tile, slot, &tile)) return;
  const int64_t kstart = cu_seqlens[tile.b];
  const int64_t kend = min((int64_t)rws[tile.r_end - 1] + 1, t_total);
  if (kend <= kstart) return;
  const int n_split = (int)((kend - kstart + split_len - 1) / split_len);
  if (n_split <= 1 || n_split > n_split_max) return;
  const int qi = threadIdx.x >> 1;        // query vector within the tile
  const int dh = (threadIdx.x & 1) * (D / 2);
  const int wave = qi / kQW, nq = qi % kQW;
  const int row_idx = tile.r_begin + wave * (kQW >> log2g) + (nq >> log2g);
  if (row_idx >= tile.r_end) return;
  const int64_t t = rws[row_idx];
  if (t < kstart || t >= kend) return;
  const int head = g * G + (nq & (G - 1));
  const int64_t item0 = ((int64_t)lg * tile_slots + slot) * n_split_max;
  float M = -INFINITY;
  for (int s = 0; s < n_split; ++s) M = fmaxf(M, ws[((item0 + s) * kQT + qi) * (D + 2) + D]);
  float Lsum = 0.0f;
  float acc[D / 2];
#pragma unroll
  for (int d = 0; d < D / 2; ++d) acc[d] = 0.0f;
  for (int s = 0; s < n_split; ++s) {
    const float* wp = ws + ((item0 + s) * kQT + qi) * (D + 2);
    const float m = wp[D];
    const float w = (m == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m - M);
    Lsum += w * wp[D + 1];
#pragma unroll
    for (int d = 0; d < D / 2; ++d) acc[d] += w * wp[dh + d];
  }
  const float inv = Lsum > 0.0f ? 1.0f / Lsum : 0.0f;
  const int64_t ob = (((int64_t)l * t_total + t) * Hq + head) * D + dh;
  if (out_f32) {
    float* op = reinterpret_cast<float*>(out) + ob;
#pragma unroll
    for (int d = 0; d < D / 2; d += 4)
      *reinterpret_cast<float4*>(op + d) =
          make_float4(acc[d] * inv, acc[d + 1] * inv, acc[d + 2] * inv, acc[d + 3] * inv);
  } else {
    uint16_t* op = reinterpret_cast<uint16_t*>(out) + ob;
#pragma unroll
    for (int d = 0; d < D / 2; d += 8)
      *reinterpret_cast<uint4*>(op + d) =
          make_uint4(pack_bf16x2(acc[d] * inv, acc[d + 1] * inv),
                     pack_bf16x2(acc[d + 2] * inv, acc[d + 3] * inv),
                     pack_bf16x2(acc[d + 4] * inv, acc[d + 5] * inv),
                     pack_bf16x2(acc[d + 6] * inv, acc[d + 7] * inv));
  }
}

int ilog2(int x) {
  int r = 0;
  while ((1 << r) < x) ++r;
  return r;
}

}  // namespace

bool attn_plan(int n_layers, int n_q_heads, int n_kv_heads, int head_dim, int64_t t_total,
               int n_seqs, int max_seq_len, int max_rows, AttnPlan* plan) {
  const int G = n_q_heads / n_kv_heads;
  const int rows_per_tile = kQT / G;
  const int full_tiles = (max_rows + rows_per_tile - 1) / rows_per_tile;
  plan->rows_per_tile = rows_per_tile;
  plan->tile_slots = full_tiles + n_seqs;
  // enough workgroups to fill 256 CUs a few times over; never split below 1024 keys
  const int64_t est = (int64_t)n_layers * n_kv_heads * (full_tiles > 0 ? full_tiles : 1);
  int want = (int)((1024 + est - 1) / est);
  int split_len = max_seq_len;
  if (want > 1) {
    split_len = (max_seq_len + want - 1) / want;
    if (split_len < 1024) split_len = 1024;
  }
  split_len = ((split_len + kKB - 1) / kKB) * kKB;
  if (split_len < kKB) split_len = kKB;
  plan->split_len = split_len;
  plan->n_split_max = (max_seq_len + split_len - 1) / split_len;
  if (plan->n_split_max < 1) plan->n_split_max = 1;
  plan->workspace = plan->n_split_max > 1
                        ? (size_t)n_layers * n_kv_heads * plan->tile_slots * plan->n_split_max *
                              kQT * (head_dim + 2) * sizeof(float)
                        : 0;
  (void)t_total;
  return true;
}

hipError_t launch_sparse_attn(const AttnPlan& plan, int n_layers, int n_q_heads, int n_kv_heads,
                              int head_dim, int64_t t_total, const int32_t* cu_seqlens,
                              int n_seqs, const int32_t* rows, const int32_t* cu_rows,
                              int rows_per_layer, int max_rows, const uint16_t* q,
                              const uint16_t* k_fresh, const uint16_t* v_fresh,
                              uint16_t* k_cache, uint16_t* v_cache, float softmax_scale,
                              kvb_dtype out_dtype, void* out, void* workspace, hipStream_t s) {
  {
    const int64_t waves = (int64_t)n_layers * max_rows;
    const int64_t blocks = (waves * 64 + 255) / 256;
    if (blocks > 0)
      hipLaunchKernelGGL(patch_kernel, dim3((unsigned)blocks), dim3(256), 0, s, n_layers,
                         n_kv_heads, head_dim, t_total, n_seqs, rows, cu_rows, rows_per_layer,
                         max_rows, k_fresh, v_fresh, k_cache, v_cache);
  }
  const int log2g = ilog2(n_q_heads / n_kv_heads);
  const float scale_log2 = softmax_scale * 1.4426950408889634f;
  const int out_f32 = out_dtype == KVB_F32;
  const dim3 grid(plan.tile_slots, plan.n_split_max, n_layers * n_kv_heads);
  float* ws = reinterpret_cast<float*>(workspace);
#define KVB_ATTN(D)                                                                              \
  hipLaunchKernelGGL(attn_kernel<D>, grid, dim3(kThreads), 0, s, n_q_heads, n_kv_heads, log2g,   \
                     t_total, cu_seqlens, n_seqs, rows, cu_rows, rows_per_layer,                 \
                     plan.rows_per_tile, plan.tile_slots, plan.split_len, plan.n_split_max, q,    \
                     k_cache, v_cache, scale_log2, out_f32, out, ws)
#define KVB_COMBINE(D)                                                                           \
  hipLaunchKernelGGL(combine_kernel<D>, dim3(plan.tile_slots, n_layers * n_kv_heads), dim3(256), \
                     0, s, n_q_heads, n_kv_heads, log2g, t_total, cu_seqlens, n_seqs, rows,      \
                     cu_rows, rows_per_layer, plan.rows_per_tile, plan.tile_slots,               \
                     plan.split_len, plan.n_split_max, out_f32, out, ws)
  if (head_dim == 128) {
    KVB_ATTN(128);
    if (plan.n_split_max > 1) KVB_COMBINE(128);
  } else {
    KVB_ATTN(64);
    if (plan.n_split_max > 1) KVB_COMBINE(64);
  }
#undef KVB_ATTN
#undef KVB_COMBINE
  (void)max_rows;
  return hipGetLastError();
}

}  // namespace kvb
