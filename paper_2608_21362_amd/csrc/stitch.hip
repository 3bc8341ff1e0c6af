// Stitch: dequantise cached KIVI chunks and rotate their keys from the cached
// position to the new one (Sec. 4.3 assembly, Sec. 3.2 R^Delta, Sec. 4.5).
//
// One workgroup per (chunk, layer, kv head): 128 tokens x d channels of K and
// of V.  HBM-bound: per workgroup it reads the K and V code blocks (C*d*b/8
// bytes each) and their float statistics, and writes 2*C*d output elements.
//
// Key jobs: one thread takes 4 consecutive tokens (one statistic group,
// Gk % 4 == 0) and 8 channel pairs (j, j + d/2); statistics and the chunk's
// rotation row are loaded once per job and widened to double at each use.
// Value pieces: one thread takes one token and 8 consecutive channels (one statistic group,
// Gv % 8 == 0; the API asks Gv % 16), so 16 (d = 128) or 8 (d = 64) lanes
// store a whole row and a wave's stores are contiguous.  Every value input of
// the thread is loaded before the key work starts, so those loads overlap it.
// The fused kernel (below) instead stages each head's key statistics and the
// rotation row in LDS and reads them for every token, and loads its value
// inputs after the key work: neither is then held in registers while a key
// job's loads are in flight (158 instead of 231 registers, three waves per
// SIMD instead of two).
//
// Arithmetic is double with contraction off: x = fma(code, scale, zero) is
// exact in the product (8-bit code times 24-bit scale), so it equals the
// product-then-sum form; the rotation is mul, mul, sub / add.  The double is
// rounded to float, and for bfloat16 output the float is rounded again.
//
// Fused deviation (DEV): one workgroup per (chunk, layer) walks the kv heads;
// every key job also reads the fresh key pieces of its tokens and accumulates
// dot and both squared norms in double over the bf16 values it stores (Alg. 2
// step 2 on the stitched rows, K only, per layer).  The eight (d = 128) or four
// (d = 64) lanes of a token quad combine their sums with xor-shuffles, every
// lane forms the head's cosine and adds it to the token's running sum, and after
// the last head one lane per quad writes delta for its four tokens.  Summing
// dot and both norms in one order keeps identical rows at delta = 0 exactly.
#include <math.h>

#include "kvb_device.h"
#include "kvb_internal.h"

namespace kvb {
namespace {

constexpr int kC = 128;

// sum of x over the TPT adjacent lanes of a token quad (TPT a power of two)
template <int TPT>
__device__ __forceinline__ double quad_lanes_sum(double x) {
#pragma unroll
  for (int m = 1; m < TPT; m <<= 1) x += __shfl_xor(x, m, 64);
  return x;
}

template <int BITS, int D, bool BF16, bool DEV>
__global__ void __launch_bounds__(256)
stitch_kernel(int32_t L, int32_t Hkv, int32_t Gk, int32_t Gv, int32_t n_pool,
              const uint8_t* __restrict__ k_codes, const float* __restrict__ k_scale,
              const float* __restrict__ k_zero, const uint8_t* __restrict__ v_codes,
              const float* __restrict__ v_scale, const float* __restrict__ v_zero,
              const kvb_chunk* __restrict__ chunks, const float* __restrict__ rope_cos,
              const float* __restrict__ rope_sin, int64_t t_total, void* __restrict__ k_out,
              void* __restrict__ v_out, const uint16_t* __restrict__ k_fresh,
              float* __restrict__ delta) {
  constexpr int H = D / 2;
  constexpr int CB = D * BITS / 8;       // code bytes per token row
  constexpr int TPT = H / 8;             // key threads per token quad
  constexpr int KJOBS = (kC / 4) * TPT;  // 256 (d=128) or 128 (d=64)
  static_assert(!DEV || BF16, "the fused deviation reads the bf16 cache values");
  static_assert(KJOBS <= 256, "one key job per thread");
  const int c = blockIdx.x;
  const kvb_chunk ch = chunks[c];
  if (ch.pool_idx < 0 || ch.pool_idx >= n_pool || ch.dst_row < 0 ||
      (int64_t)ch.dst_row + kC > t_total)
    return;
  const int ngk = kC / Gk, ngv = D / Gv;
  // fused deviation: running cosine sum over heads of this thread's four tokens
  double cos_sum[4] = {0.0, 0.0, 0.0, 0.0};
  // fused: the head's key statistics (scale, then zero; at most C/4 groups)
  // and the chunk's rotation row (cos, then sin) staged in LDS, read per token
  __shared__ float4 st_k4[DEV ? 2 * (kC / 4) * D / 4 : 1];
  __shared__ float4 st_r4[DEV ? D / 4 : 1];
  const int n_heads = DEV ? Hkv : 1;
  for (int hh = 0; hh < n_heads; ++hh) {
    const int l = DEV ? (int)blockIdx.y : (int)blockIdx.y / Hkv;
    const int h = DEV ? hh : (int)blockIdx.y % Hkv;
    const int64_t slab = ((int64_t)ch.pool_idx * L + l) * Hkv + h;  // (p, l, h)
    const int64_t out_row0 = ((int64_t)l * Hkv + h) * t_total + ch.dst_row;
    if constexpr (DEV) {
      // the previous head's key jobs are done with the staged statistics
      __syncthreads();
      const int n4 = ngk * D / 4;
      const float4* ks4 = reinterpret_cast<const float4*>(k_scale + slab * ngk * D);
      const float4* kz4 = reinterpret_cast<const float4*>(k_zero + slab * ngk * D);
      for (int i = threadIdx.x; i < n4; i += blockDim.x) {
        st_k4[i] = ks4[i];
        st_k4[n4 + i] = kz4[i];
      }
      if (threadIdx.x < H / 4) {
        st_r4[threadIdx.x] = reinterpret_cast<const float4*>(rope_cos + (int64_t)c * H)[threadIdx.x];
        st_r4[H / 4 + threadIdx.x] =
            reinterpret_cast<const float4*>(rope_sin + (int64_t)c * H)[threadIdx.x];
      }
      __syncthreads();
    }

    // value inputs of this thread's pieces (token u, channels [j0, j0 + 8));
    // the plain stitch requests them before its key work (they are in flight
    // while the keys are computed), the fused one after it (fewer live
    // registers during the key jobs)
    constexpr int VP = D / 8;              // pieces per token row
    constexpr int VPT = kC * VP / 256;     // pieces per thread
    uint32_t vw[VPT][2];
    float vsc[VPT], vzr[VPT];
    auto load_values = [&]() {
#pragma unroll
      for (int k = 0; k < VPT; ++k) {
        const int vj = threadIdx.x + 256 * k;
        const int u = vj / VP, j0 = (vj % VP) * 8;
        const int64_t srow = slab * kC + u;
        vsc[k] = v_scale[srow * ngv + j0 / Gv];
        vzr[k] = v_zero[srow * ngv + j0 / Gv];
        const uint8_t* row = v_codes + srow * CB;
        if constexpr (BITS == 8) {
          const uint2 a = *reinterpret_cast<const uint2*>(row + j0);
          vw[k][0] = a.x;
          vw[k][1] = a.y;
        } else {
          vw[k][0] = *reinterpret_cast<const uint32_t*>(row + j0 / 2);
          vw[k][1] = 0;
        }
      }
    };
    if constexpr (!DEV) load_values();

    for (int job = threadIdx.x; job < KJOBS; job += blockDim.x) {
      {
        // ---- keys: tokens 4q..4q+3, channel pairs [8cg, 8cg + 8)
        const int q = job / TPT, cg = job % TPT;
        const int u0 = 4 * q, j0 = 8 * cg;
        const int g = u0 / Gk;
        // statistics and rotation row of the job's channels, kept as float
        // (half the registers of double) and widened exactly at use: loaded
        // once per job for the plain stitch, read from LDS for every token in
        // the fused kernel (so they are not live while its loads are in flight)
        float s_lo[8], s_hi[8], z_lo[8], z_hi[8], cs[8], sn[8];
        auto load_stats = [&]() {
          const float* sc = DEV ? reinterpret_cast<const float*>(st_k4) + g * D
                                : k_scale + (slab * ngk + g) * D;
          const float* zr = DEV ? reinterpret_cast<const float*>(st_k4) + (ngk + g) * D
                                : k_zero + (slab * ngk + g) * D;
          const float* rc = DEV ? reinterpret_cast<const float*>(st_r4) : rope_cos + (int64_t)c * H;
          const float* rs = DEV ? reinterpret_cast<const float*>(st_r4) + H : rope_sin + (int64_t)c * H;
#pragma unroll
          for (int k = 0; k < 8; k += 4) {
            const float4 a = *reinterpret_cast<const float4*>(sc + j0 + k);
            const float4 b = *reinterpret_cast<const float4*>(sc + H + j0 + k);
            const float4 e = *reinterpret_cast<const float4*>(zr + j0 + k);
            const float4 f = *reinterpret_cast<const float4*>(zr + H + j0 + k);
            const float4 cc = *reinterpret_cast<const float4*>(rc + j0 + k);
            const float4 ss = *reinterpret_cast<const float4*>(rs + j0 + k);
            s_lo[k] = a.x; s_lo[k + 1] = a.y; s_lo[k + 2] = a.z; s_lo[k + 3] = a.w;
            s_hi[k] = b.x; s_hi[k + 1] = b.y; s_hi[k + 2] = b.z; s_hi[k + 3] = b.w;
            z_lo[k] = e.x; z_lo[k + 1] = e.y; z_lo[k + 2] = e.z; z_lo[k + 3] = e.w;
            z_hi[k] = f.x; z_hi[k + 1] = f.y; z_hi[k + 2] = f.z; z_hi[k + 3] = f.w;
            cs[k] = cc.x; cs[k + 1] = cc.y; cs[k + 2] = cc.z; cs[k + 3] = cc.w;
            sn[k] = ss.x; sn[k + 1] = ss.y; sn[k + 2] = ss.z; sn[k + 3] = ss.w;
          }
        };
        if constexpr (!DEV) load_stats();
        // the codes of the four tokens (and, fused, their fresh key pieces)
        // are all requested before any is used: one memory round trip per job
        uint32_t cwl[4][2], cwh[4][2];
        uint4 fra[4], frb[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint8_t* row = k_codes + (slab * kC + u0 + i) * CB;
          if constexpr (BITS == 8) {
            const uint2 a = *reinterpret_cast<const uint2*>(row + j0);
            const uint2 b = *reinterpret_cast<const uint2*>(row + H + j0);
            cwl[i][0] = a.x; cwl[i][1] = a.y; cwh[i][0] = b.x; cwh[i][1] = b.y;
          } else {
            cwl[i][0] = *reinterpret_cast<const uint32_t*>(row + j0 / 2);
            cwh[i][0] = *reinterpret_cast<const uint32_t*>(row + (H + j0) / 2);
            cwl[i][1] = cwh[i][1] = 0;
          }
          if constexpr (DEV) {
            const uint16_t* fr = k_fresh + (out_row0 + u0 + i) * D;
            fra[i] = *reinterpret_cast<const uint4*>(fr + j0);
            frb[i] = *reinterpret_cast<const uint4*>(fr + H + j0);
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int u = u0 + i;
          if constexpr (DEV) {
            asm volatile("" ::: "memory");  // re-read the staged values for every token
            load_stats();
          }
          const uint32_t wl[2] = {cwl[i][0], cwl[i][1]}, wh[2] = {cwh[i][0], cwh[i][1]};
          float ylo[8], yhi[8];
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            const double xl = __builtin_fma((double)code_at<BITS>(wl, k), (double)s_lo[k], (double)z_lo[k]);
            const double xh = __builtin_fma((double)code_at<BITS>(wh, k), (double)s_hi[k], (double)z_hi[k]);
            const double a = xl * (double)cs[k];
            const double b = xh * (double)sn[k];
            const double e = xh * (double)cs[k];
            const double f = xl * (double)sn[k];
            ylo[k] = (float)(a - b);
            yhi[k] = (float)(e + f);
          }
          const int64_t o = (out_row0 + u) * D;
          if constexpr (BF16) {
            uint16_t* ko = reinterpret_cast<uint16_t*>(k_out) + o;
            uint4 A, B;
            A.x = pack_bf16x2(ylo[0], ylo[1]); A.y = pack_bf16x2(ylo[2], ylo[3]);
            A.z = pack_bf16x2(ylo[4], ylo[5]); A.w = pack_bf16x2(ylo[6], ylo[7]);
            B.x = pack_bf16x2(yhi[0], yhi[1]); B.y = pack_bf16x2(yhi[2], yhi[3]);
            B.z = pack_bf16x2(yhi[4], yhi[5]); B.w = pack_bf16x2(yhi[6], yhi[7]);
            *reinterpret_cast<uint4*>(ko + j0) = A;
            *reinterpret_cast<uint4*>(ko + H + j0) = B;
            if constexpr (DEV) {
              const uint4 FA = fra[i], FB = frb[i];
              const uint32_t cw[8] = {A.x, A.y, A.z, A.w, B.x, B.y, B.z, B.w};
              const uint32_t fw[8] = {FA.x, FA.y, FA.z, FA.w, FB.x, FB.y, FB.z, FB.w};
              double dot = 0.0, na = 0.0, nb = 0.0;
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const double a0 = bf16_lo(cw[e]), a1 = bf16_hi(cw[e]);
                const double b0 = bf16_lo(fw[e]), b1 = bf16_hi(fw[e]);
                dot = __builtin_fma(a0, b0, dot);
                dot = __builtin_fma(a1, b1, dot);
                na = __builtin_fma(a0, a0, na);
                na = __builtin_fma(a1, a1, na);
                nb = __builtin_fma(b0, b0, nb);
                nb = __builtin_fma(b1, b1, nb);
              }
              dot = quad_lanes_sum<TPT>(dot);
              na = quad_lanes_sum<TPT>(na);
              nb = quad_lanes_sum<TPT>(nb);
              const double den = na * nb;
              cos_sum[i] +=
                  (den == 0.0) ? ((na == 0.0 && nb == 0.0) ? 1.0 : 0.0) : dot / sqrt(den);
            }
          } else {
            float* ko = reinterpret_cast<float*>(k_out) + o;
            *reinterpret_cast<float4*>(ko + j0) = make_float4(ylo[0], ylo[1], ylo[2], ylo[3]);
            *reinterpret_cast<float4*>(ko + j0 + 4) = make_float4(ylo[4], ylo[5], ylo[6], ylo[7]);
            *reinterpret_cast<float4*>(ko + H + j0) = make_float4(yhi[0], yhi[1], yhi[2], yhi[3]);
            *reinterpret_cast<float4*>(ko + H + j0 + 4) = make_float4(yhi[4], yhi[5], yhi[6], yhi[7]);
          }
        }
      }
    }

    // ---- values
    if constexpr (DEV) load_values();
#pragma unroll
    for (int k = 0; k < VPT; ++k) {
      const int vj = threadIdx.x + 256 * k;
      const int u = vj / VP, j0 = (vj % VP) * 8;
      const double sc = vsc[k], zr = vzr[k];
      float y[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = (float)__builtin_fma((double)code_at<BITS>(vw[k], e), sc, zr);
      const int64_t o = (out_row0 + u) * D + j0;
      if constexpr (BF16) {
        const uint4 A = make_uint4(pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]),
                                   pack_bf16x2(y[4], y[5]), pack_bf16x2(y[6], y[7]));
        *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(v_out) + o) = A;
      } else {
        float* vo = reinterpret_cast<float*>(v_out) + o;
        *reinterpret_cast<float4*>(vo) = make_float4(y[0], y[1], y[2], y[3]);
        *reinterpret_cast<float4*>(vo + 4) = make_float4(y[4], y[5], y[6], y[7]);
      }
    }
  }  // heads
  if constexpr (DEV) {
    // one lane per token quad: delta[l][dst_row + 4q .. + 3], one 16-byte
    // store when the quad is 16-byte aligned (dst_row and t_total multiples
    // of 4), else four 4-byte stores (e.g. after one to three sink rows)
    const int job = threadIdx.x;
    if (job < KJOBS && job % TPT == 0) {
      const int q = job / TPT;
      const double n = (double)Hkv;
      const int64_t first = (int64_t)blockIdx.y * t_total + ch.dst_row;
      float* dp = delta + first + 4 * q;
      const float4 dv = make_float4((float)(1.0 - cos_sum[0] / n), (float)(1.0 - cos_sum[1] / n),
                                    (float)(1.0 - cos_sum[2] / n), (float)(1.0 - cos_sum[3] / n));
      if ((first & 3) == 0) {
        *reinterpret_cast<float4*>(dp) = dv;
      } else {
        dp[0] = dv.x;
        dp[1] = dv.y;
        dp[2] = dv.z;
        dp[3] = dv.w;
      }
    }
  }
}

}  // namespace

hipError_t launch_stitch(const kvb_pool_layout& p, int32_t n_pool, const uint8_t* k_codes,
                         const float* k_scale, const float* k_zero, const uint8_t* v_codes,
                         const float* v_scale, const float* v_zero, const kvb_chunk* chunks,
                         int32_t n_chunks, const float* rope_cos, const float* rope_sin,
                         int64_t t_total, kvb_dtype out_dtype, void* k_cache, void* v_cache,
                         hipStream_t s) {
  const dim3 grid(n_chunks, p.n_layers * p.n_kv_heads), block(256);
  const bool bf = out_dtype == KVB_BF16;
#define KVB_STITCH(B, D, F)                                                                       \
  hipLaunchKernelGGL((stitch_kernel<B, D, F, false>), grid, block, 0, s, p.n_layers,             \
                     p.n_kv_heads, p.k_group, p.v_group, n_pool, k_codes, k_scale, k_zero,       \
                     v_codes, v_scale, v_zero, chunks, rope_cos, rope_sin, t_total, k_cache,     \
                     v_cache, nullptr, nullptr)
  if (p.bits == 8) {
    if (p.head_dim == 128) { if (bf) KVB_STITCH(8, 128, true); else KVB_STITCH(8, 128, false); }
    else { if (bf) KVB_STITCH(8, 64, true); else KVB_STITCH(8, 64, false); }
  } else {
    if (p.head_dim == 128) { if (bf) KVB_STITCH(4, 128, true); else KVB_STITCH(4, 128, false); }
    else { if (bf) KVB_STITCH(4, 64, true); else KVB_STITCH(4, 64, false); }
  }
#undef KVB_STITCH
  return hipGetLastError();
}

hipError_t launch_stitch_deviation(const kvb_pool_layout& p, int32_t n_pool,
                                   const uint8_t* k_codes, const float* k_scale,
                                   const float* k_zero, const uint8_t* v_codes,
                                   const float* v_scale, const float* v_zero,
                                   const kvb_chunk* chunks, int32_t n_chunks,
                                   const float* rope_cos, const float* rope_sin, int64_t t_total,
                                   void* k_cache, void* v_cache, const uint16_t* k_fresh,
                                   float* delta, hipStream_t s) {
  const dim3 grid(n_chunks, p.n_layers), block(256);
#define KVB_STITCH_DEV(B, D)                                                                      \
  hipLaunchKernelGGL((stitch_kernel<B, D, true, true>), grid, block, 0, s, p.n_layers,           \
                     p.n_kv_heads, p.k_group, p.v_group, n_pool, k_codes, k_scale, k_zero,       \
                     v_codes, v_scale, v_zero, chunks, rope_cos, rope_sin, t_total, k_cache,     \
                     v_cache, k_fresh, delta)
  if (p.bits == 8) {
    if (p.head_dim == 128) KVB_STITCH_DEV(8, 128); else KVB_STITCH_DEV(8, 64);
  } else {
    if (p.head_dim == 128) KVB_STITCH_DEV(4, 128); else KVB_STITCH_DEV(4, 64);
  }
#undef KVB_STITCH_DEV
  return hipGetLastError();
}

}  // namespace kvb
