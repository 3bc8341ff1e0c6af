// Per-token deviation, CacheBlendRecompute step 2 (Alg. 2):
//   delta_t = 1 - mean over (layers, kv heads, tensors) of cos(cache_t, fresh_t).
//
// HBM-bound streaming reduction.  Four lanes own one (row, kv head) vector:
// lane q of the four takes the 16-byte pieces q, q + 4, ... of the head's
// cached and fresh row (so a load instruction covers 64 contiguous bytes of
// every vector it touches) and accumulates dot and both squared norms in
// double over the exact bf16 values; two DPP quad permutations give all four
// lanes the totals, every lane forms the cosine, and the Hkv quads of a row
// (adjacent lanes) are summed with xor-shuffles.  A wave covers 16 / Hkv rows
// (Hkv a power of two up to 16).  With `per_layer` every layer is its own set;
// otherwise the wave walks all layers of its rows.
#include <math.h>

#include "kvb_device.h"
#include "kvb_internal.h"

namespace kvb {
namespace {

// x from the lane chosen by DPP control CTRL (a permutation within each quad),
// for a double split into its two 32-bit halves
template <int CTRL>
__device__ __forceinline__ double dpp_d(double x) {
  const uint64_t u = __builtin_bit_cast(uint64_t, x);
  const int lo = __builtin_amdgcn_mov_dpp((int)(uint32_t)u, CTRL, 0xF, 0xF, true);
  const int hi = __builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), CTRL, 0xF, 0xF, true);
  return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// sum over each quad of lanes; all four lanes end with the total
__device__ __forceinline__ double quad_sum(double x) {
  x += dpp_d<0xB1>(x);  // quad_perm [1,0,3,2]
  x += dpp_d<0x4E>(x);  // quad_perm [2,3,0,1]
  return x;
}

template <int D>
__global__ void __launch_bounds__(256)
deviation_kernel(int32_t L, int32_t Hkv, int32_t log2hkv, int64_t t_total,
                 const uint16_t* __restrict__ kc, const uint16_t* __restrict__ kf,
                 const uint16_t* __restrict__ vc, const uint16_t* __restrict__ vf,
                 int32_t per_layer, float* __restrict__ delta) {
  constexpr int CPL = D / 32;  // 16-byte pieces per lane per head vector
  const int lane = threadIdx.x & 63, grp = lane >> 2, q = lane & 3;
  const int rows_per_wave = 16 >> log2hkv;
  const int h = grp & (Hkv - 1), rsub = grp >> log2hkv;
  const int64_t wave = __builtin_amdgcn_readfirstlane(
      (int)(((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6));
  const int64_t n_sets = per_layer ? L : 1;
  const int64_t n_items = n_sets * t_total;
  // the wave's first item, split once (scalar); its rows then step by one
  const int64_t base = wave * rows_per_wave;
  int64_t set = base / t_total, t = base % t_total + rsub;
  while (t >= t_total) {  // only when t_total < 16
    t -= t_total;
    ++set;
  }
  const bool ok = base + rsub < n_items;
  if (!ok) set = t = 0;
  const int n_tensors = vc ? 2 : 1;
  const int n_l = per_layer ? 1 : L;
  double total = 0.0;
  for (int li = 0; li < n_l; ++li) {
    const int64_t l = per_layer ? set : li;
    for (int tensor = 0; tensor < n_tensors; ++tensor) {
      const uint16_t* A = tensor ? vc : kc;
      const uint16_t* B = tensor ? vf : kf;
      const int64_t row = ((l * Hkv + h) * t_total + t) * D;
      uint4 a[CPL], b[CPL];
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        const int64_t off = row + (q + 4 * k) * 8;
        a[k] = ok ? *reinterpret_cast<const uint4*>(A + off) : make_uint4(0, 0, 0, 0);
        b[k] = ok ? *reinterpret_cast<const uint4*>(B + off) : make_uint4(0, 0, 0, 0);
      }
      double dot = 0.0, na = 0.0, nb = 0.0;
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        const uint32_t aw[4] = {a[k].x, a[k].y, a[k].z, a[k].w};
        const uint32_t bw[4] = {b[k].x, b[k].y, b[k].z, b[k].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const double a0 = bf16_lo(aw[e]), a1 = bf16_hi(aw[e]);
          const double b0 = bf16_lo(bw[e]), b1 = bf16_hi(bw[e]);
          dot = __builtin_fma(a0, b0, dot);
          dot = __builtin_fma(a1, b1, dot);
          na = __builtin_fma(a0, a0, na);
          na = __builtin_fma(a1, a1, na);
          nb = __builtin_fma(b0, b0, nb);
          nb = __builtin_fma(b1, b1, nb);
        }
      }
      dot = quad_sum(dot);
      na = quad_sum(na);
      nb = quad_sum(nb);
      const double den = na * nb;
      double cosv = (den == 0.0) ? ((na == 0.0 && nb == 0.0) ? 1.0 : 0.0) : dot / sqrt(den);
      for (int m = 4; m < 4 * Hkv; m <<= 1) cosv += __shfl_xor(cosv, m, 64);
      total += cosv;
    }
  }
  if (ok && q == 0 && h == 0) {
    const double count = (double)n_l * Hkv * n_tensors;
    delta[set * t_total + t] = (float)(1.0 - total / count);
  }
}

}  // namespace

hipError_t launch_deviation(int n_layers, int n_kv_heads, int head_dim, int64_t t_total,
                            const uint16_t* k_cache, const uint16_t* k_fresh,
                            const uint16_t* v_cache, const uint16_t* v_fresh, int per_layer,
                            float* delta, hipStream_t s) {
  int log2hkv = 0;
  while ((1 << log2hkv) < n_kv_heads) ++log2hkv;
  const int64_t items = (per_layer ? (int64_t)n_layers : 1) * t_total;
  const int64_t rows_per_wave = 16 >> log2hkv;
  const int64_t waves = (items + rows_per_wave - 1) / rows_per_wave;
  const int64_t blocks = (waves * 64 + 255) / 256;
  if (head_dim == 128)
    hipLaunchKernelGGL(deviation_kernel<128>, dim3((unsigned)blocks), dim3(256), 0, s, n_layers,
                       n_kv_heads, log2hkv, t_total, k_cache, k_fresh, v_cache, v_fresh,
                       per_layer, delta);
  else
    hipLaunchKernelGGL(deviation_kernel<64>, dim3((unsigned)blocks), dim3(256), 0, s, n_layers,
                       n_kv_heads, log2hkv, t_total, k_cache, k_fresh, v_cache, v_fresh,
                       per_layer, delta);
  return hipGetLastError();
}

}  // namespace kvb
