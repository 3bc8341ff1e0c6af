// Per-token deviation, CacheBlendRecompute step 2 (Alg. 2):
//   delta_t = 1 - mean over (layers, kv heads, tensors) of cos(cache_t, fresh_t).
//
// HBM-bound streaming reduction.  A 32-lane half-wave owns one row: each lane
// loads 16 bytes (8 bf16) of the cached and the fresh vector, so d/8 lanes
// cover one head and 32/(d/8) heads are in flight per pass.  Partial dot and
// squared norms are accumulated in double and reduced with xor-shuffles inside
// the head's lane group; the per-head cosines are then summed over the
// half-wave.  With `per_layer` every layer is its own set; otherwise one
// half-wave walks all layers of its row.
#include <math.h>

#include "kvb_device.h"
#include "kvb_internal.h"

namespace kvb {
namespace {

__device__ __forceinline__ double shfl_xor_d(double v, int m) {
  return __shfl_xor(v, m, 64);
}

template <int D>
__global__ void __launch_bounds__(256)
deviation_kernel(int32_t L, int32_t Hkv, int64_t t_total, const uint16_t* __restrict__ kc,
                 const uint16_t* __restrict__ kf, const uint16_t* __restrict__ vc,
                 const uint16_t* __restrict__ vf, int32_t per_layer, float* __restrict__ delta) {
  constexpr int LPH = D / 8;       // lanes per head
  constexpr int HPP = 32 / LPH;    // heads per pass
  const int lane = threadIdx.x & 63;
  const int half = lane >> 5, hl = lane & 31;
  const int64_t item = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 5;  // half-wave id
  const int64_t n_sets = per_layer ? L : 1;
  if (item >= n_sets * t_total) return;  // both halves of a wave exit together or run alike
  const int64_t set = item / t_total;
  const int64_t t = item % t_total;
  const int l_begin = per_layer ? (int)set : 0;
  const int l_end = per_layer ? (int)set + 1 : L;
  const int n_tensors = vc ? 2 : 1;
  double total = 0.0;
  for (int l = l_begin; l < l_end; ++l) {
    for (int tensor = 0; tensor < n_tensors; ++tensor) {
      const uint16_t* A = tensor ? vc : kc;
      const uint16_t* B = tensor ? vf : kf;
      for (int h0 = 0; h0 < Hkv; h0 += HPP) {
        const int h = h0 + hl / LPH;
        double dot = 0.0, na = 0.0, nb = 0.0;
        if (h < Hkv) {
          const int64_t off = (((int64_t)l * Hkv + h) * t_total + t) * D + (hl % LPH) * 8;
          const uint4 a = *reinterpret_cast<const uint4*>(A + off);
          const uint4 b = *reinterpret_cast<const uint4*>(B + off);
          const uint32_t aw[4] = {a.x, a.y, a.z, a.w};
          const uint32_t bw[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const double a0 = bf16_lo(aw[k]), a1 = bf16_hi(aw[k]);
            const double b0 = bf16_lo(bw[k]), b1 = bf16_hi(bw[k]);
            dot = __builtin_fma(a0, b0, dot);
            dot = __builtin_fma(a1, b1, dot);
            na = __builtin_fma(a0, a0, na);
            na = __builtin_fma(a1, a1, na);
            nb = __builtin_fma(b0, b0, nb);
            nb = __builtin_fma(b1, b1, nb);
          }
        }
#pragma unroll
        for (int m = 1; m < LPH; m <<= 1) {
          dot += shfl_xor_d(dot, m);
          na += shfl_xor_d(na, m);
          nb += shfl_xor_d(nb, m);
        }
        double cosv = 0.0;
        if (h < Hkv && (hl % LPH) == 0) {
          const double den = na * nb;
          if (den == 0.0) cosv = (na == 0.0 && nb == 0.0) ? 1.0 : 0.0;
          else cosv = dot / sqrt(den);
        }
#pragma unroll
        for (int m = LPH; m < 32; m <<= 1) cosv += shfl_xor_d(cosv, m);
        total += cosv;
      }
    }
  }
  if (hl == 0) {
    const double count = (double)(l_end - l_begin) * Hkv * n_tensors;
    delta[set * t_total + t] = (float)(1.0 - total / count);
  }
  (void)half;
}

}  // namespace

hipError_t launch_deviation(int n_layers, int n_kv_heads, int head_dim, int64_t t_total,
                            const uint16_t* k_cache, const uint16_t* k_fresh,
                            const uint16_t* v_cache, const uint16_t* v_fresh, int per_layer,
                            float* delta, hipStream_t s) {
  const int64_t items = (per_layer ? (int64_t)n_layers : 1) * t_total;
  const int64_t blocks = (items * 32 + 255) / 256;
  if (head_dim == 128)
    hipLaunchKernelGGL(deviation_kernel<128>, dim3((unsigned)blocks), dim3(256), 0, s, n_layers,
                       n_kv_heads, t_total, k_cache, k_fresh, v_cache, v_fresh, per_layer, delta);
  else
    hipLaunchKernelGGL(deviation_kernel<64>, dim3((unsigned)blocks), dim3(256), 0, s, n_layers,
                       n_kv_heads, t_total, k_cache, k_fresh, v_cache, v_fresh, per_layer, delta);
  return hipGetLastError();
}

}  // namespace kvb
