// Cache population kernels: RoPE at absolute positions (Eq. 3), KIVI
// quantisation of cached chunks (Sec. 4.5, Eq. 7) and the chunks' importance
// for the eviction order (Sec. 4.4).  These prepare the chunk pool and the
// probe-pass tensors; they are not timed as part of the path.
#include <math.h>

#include "kvb_device.h"
#include "kvb_internal.h"

namespace kvb {
namespace {

// One thread per (vector, group of 4 channel pairs).  Double arithmetic:
// y_lo = x_lo*c - x_hi*s, y_hi = x_hi*c + x_lo*s (contraction is off for this
// file, so each product and sum rounds once).
template <int D, int OUT>
__global__ void __launch_bounds__(256)
rope_rows_kernel(int64_t n_outer, int64_t n_rows, int64_t n_inner, const float* __restrict__ x,
                 const int32_t* __restrict__ row_pos, const int32_t* __restrict__ outer_pos,
                 const float* __restrict__ tcos, const float* __restrict__ tsin, int32_t table_len,
                 void* __restrict__ out) {
  constexpr int H = D / 2;
  constexpr int G = H / 4;  // threads per vector
  const int64_t n_vec = n_outer * n_rows * n_inner;
  for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < n_vec * G;
       w += (int64_t)gridDim.x * blockDim.x) {
    const int64_t v = w / G;
    const int i0 = (int)(w % G) * 4;
    const int64_t r = (v / n_inner) % n_rows;
    const int64_t o = v / (n_inner * n_rows);
    const float4 lo = *reinterpret_cast<const float4*>(x + v * D + i0);
    const float4 hi = *reinterpret_cast<const float4*>(x + v * D + H + i0);
    double xl[4] = {lo.x, lo.y, lo.z, lo.w};
    double xh[4] = {hi.x, hi.y, hi.z, hi.w};
    double yl[4], yh[4];
    if (tcos != nullptr) {
      const int64_t p = (int64_t)row_pos[r] + (outer_pos ? (int64_t)outer_pos[o] : 0);
      if (p < 0 || p >= table_len) {
        for (int k = 0; k < 4; ++k) yl[k] = yh[k] = __builtin_nan("");
      } else {
        const float4 c4 = *reinterpret_cast<const float4*>(tcos + p * H + i0);
        const float4 s4 = *reinterpret_cast<const float4*>(tsin + p * H + i0);
        const double c[4] = {c4.x, c4.y, c4.z, c4.w};
        const double s[4] = {s4.x, s4.y, s4.z, s4.w};
        for (int k = 0; k < 4; ++k) {
          yl[k] = xl[k] * c[k] - xh[k] * s[k];
          yh[k] = xh[k] * c[k] + xl[k] * s[k];
        }
      }
    } else {
      for (int k = 0; k < 4; ++k) { yl[k] = xl[k]; yh[k] = xh[k]; }
    }
    if constexpr (OUT == KVB_F64) {
      double* o64 = reinterpret_cast<double*>(out) + v * D;
      *reinterpret_cast<double2*>(o64 + i0) = make_double2(yl[0], yl[1]);
      *reinterpret_cast<double2*>(o64 + i0 + 2) = make_double2(yl[2], yl[3]);
      *reinterpret_cast<double2*>(o64 + H + i0) = make_double2(yh[0], yh[1]);
      *reinterpret_cast<double2*>(o64 + H + i0 + 2) = make_double2(yh[2], yh[3]);
    } else if constexpr (OUT == KVB_F32) {
      float* o32 = reinterpret_cast<float*>(out) + v * D;
      *reinterpret_cast<float4*>(o32 + i0) =
          make_float4((float)yl[0], (float)yl[1], (float)yl[2], (float)yl[3]);
      *reinterpret_cast<float4*>(o32 + H + i0) =
          make_float4((float)yh[0], (float)yh[1], (float)yh[2], (float)yh[3]);
    } else {
      uint16_t* o16 = reinterpret_cast<uint16_t*>(out) + v * D;
      uint2 a, b;
      a.x = pack_bf16x2((float)yl[0], (float)yl[1]);
      a.y = pack_bf16x2((float)yl[2], (float)yl[3]);
      b.x = pack_bf16x2((float)yh[0], (float)yh[1]);
      b.y = pack_bf16x2((float)yh[2], (float)yh[3]);
      *reinterpret_cast<uint2*>(o16 + i0) = a;
      *reinterpret_cast<uint2*>(o16 + H + i0) = b;
    }
  }
}

template <typename T>
__device__ __forceinline__ double load_d(const void* p, int64_t i) {
  return (double)reinterpret_cast<const T*>(p)[i];
}

// Keys: one thread per (slot, layer, head, token group, channel pair).
template <typename T>
__global__ void __launch_bounds__(256)
quant_keys_kernel(int32_t n_pool, int32_t L, int32_t first_layer, int32_t n_in, int32_t Hkv,
                  int32_t C, int32_t D, int32_t bits, int32_t Gk, const void* __restrict__ in,
                  uint8_t* __restrict__ codes, float* __restrict__ scale,
                  float* __restrict__ zero) {
  const int64_t pairs = D / 2;
  const int64_t n_groups = C / Gk;
  const int64_t total = (int64_t)n_pool * n_in * Hkv * n_groups * pairs;
  const double levels = (double)((1 << bits) - 1);
  const int cb = D * bits / 8;
  for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < total;
       w += (int64_t)gridDim.x * blockDim.x) {
    const int j0 = (int)(w % pairs) * 2;
    int64_t rest = w / pairs;
    const int g = (int)(rest % n_groups);
    rest /= n_groups;
    const int h = (int)(rest % Hkv);
    rest /= Hkv;
    const int li = (int)(rest % n_in);
    const int64_t p = rest / n_in;
    const int l = first_layer + li;
    const int64_t in_base = (((p * n_in + li) * Hkv + h) * C) * (int64_t)D;
    const int64_t out_row = ((p * L + l) * Hkv + h) * (int64_t)C;
    double mn[2], mx[2];
    for (int e = 0; e < 2; ++e) {
      mn[e] = INFINITY;
      mx[e] = -INFINITY;
    }
    for (int u = g * Gk; u < (g + 1) * Gk; ++u)
      for (int e = 0; e < 2; ++e) {
        const double x = load_d<T>(in, in_base + (int64_t)u * D + j0 + e);
        mn[e] = fmin(mn[e], x);
        mx[e] = fmax(mx[e], x);
      }
    uint32_t cd[2];
    for (int u = g * Gk; u < (g + 1) * Gk; ++u) {
      for (int e = 0; e < 2; ++e) {
        const double x = load_d<T>(in, in_base + (int64_t)u * D + j0 + e);
        const double r = mx[e] - mn[e];
        double c = 0.0;
        if (r != 0.0) {
          c = rint(((x - mn[e]) / r) * levels);
          c = fmin(fmax(c, 0.0), levels);
        }
        cd[e] = (uint32_t)c;
      }
      uint8_t* row = codes + (out_row + u) * cb;
      if (bits == 8) {
        row[j0] = (uint8_t)cd[0];
        row[j0 + 1] = (uint8_t)cd[1];
      } else {
        row[j0 / 2] = (uint8_t)(cd[0] | (cd[1] << 4));
      }
    }
    const int64_t st = (((p * L + l) * Hkv + h) * n_groups + g) * (int64_t)D + j0;
    for (int e = 0; e < 2; ++e) {
      const double r = mx[e] - mn[e];
      scale[st + e] = r == 0.0 ? 0.0f : (float)(r / levels);
      zero[st + e] = (float)mn[e];
    }
  }
}

// Values: one thread per (slot, layer, head, token, channel group).
template <typename T>
__global__ void __launch_bounds__(256)
quant_values_kernel(int32_t n_pool, int32_t L, int32_t first_layer, int32_t n_in, int32_t Hkv,
                    int32_t C, int32_t D, int32_t bits, int32_t Gv, const void* __restrict__ in,
                    uint8_t* __restrict__ codes, float* __restrict__ scale,
                    float* __restrict__ zero) {
  const int64_t n_groups = D / Gv;
  const int64_t total = (int64_t)n_pool * n_in * Hkv * C * n_groups;
  const double levels = (double)((1 << bits) - 1);
  const int cb = D * bits / 8;
  for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < total;
       w += (int64_t)gridDim.x * blockDim.x) {
    const int g = (int)(w % n_groups);
    int64_t rest = w / n_groups;
    const int u = (int)(rest % C);
    rest /= C;
    const int h = (int)(rest % Hkv);
    rest /= Hkv;
    const int li = (int)(rest % n_in);
    const int64_t p = rest / n_in;
    const int l = first_layer + li;
    const int64_t in_base = ((((p * n_in + li) * Hkv + h) * C) + u) * (int64_t)D + g * Gv;
    double mn = INFINITY, mx = -INFINITY;
    for (int j = 0; j < Gv; ++j) {
      const double x = load_d<T>(in, in_base + j);
      mn = fmin(mn, x);
      mx = fmax(mx, x);
    }
    const double r = mx - mn;
    uint8_t* row = codes + ((((p * L + l) * Hkv + h) * C) + u) * (int64_t)cb;
    for (int j = 0; j < Gv; j += 2) {
      uint32_t cd[2];
      for (int e = 0; e < 2; ++e) {
        const double x = load_d<T>(in, in_base + j + e);
        double c = 0.0;
        if (r != 0.0) {
          c = rint(((x - mn) / r) * levels);
          c = fmin(fmax(c, 0.0), levels);
        }
        cd[e] = (uint32_t)c;
      }
      const int ch = g * Gv + j;
      if (bits == 8) {
        row[ch] = (uint8_t)cd[0];
        row[ch + 1] = (uint8_t)cd[1];
      } else {
        row[ch / 2] = (uint8_t)(cd[0] | (cd[1] << 4));
      }
    }
    const int64_t st = ((((p * L + l) * Hkv + h) * C) + u) * n_groups + g;
    scale[st] = r == 0.0 ? 0.0f : (float)(r / levels);
    zero[st] = (float)mn;
  }
}

int grid_for(int64_t work) {
  int64_t b = (work + 255) / 256;
  if (b > 65536) b = 65536;
  return (int)(b < 1 ? 1 : b);
}

}  // namespace

hipError_t launch_rope_rows(int head_dim, int64_t n_outer, int64_t n_rows, int64_t n_inner,
                            const float* x, const int32_t* row_pos, const int32_t* outer_pos,
                            const float* tcos, const float* tsin, int32_t table_len,
                            kvb_dtype out_dtype, void* out, hipStream_t s) {
  const int64_t work = n_outer * n_rows * n_inner * (head_dim / 8);
  const dim3 grid(grid_for(work)), block(256);
#define KVB_ROPE(D, O)                                                                     \
  hipLaunchKernelGGL((rope_rows_kernel<D, O>), grid, block, 0, s, n_outer, n_rows, n_inner, \
                     x, row_pos, outer_pos, tcos, tsin, table_len, out)
  if (head_dim == 64) {
    if (out_dtype == KVB_F64) KVB_ROPE(64, KVB_F64);
    else if (out_dtype == KVB_F32) KVB_ROPE(64, KVB_F32);
    else KVB_ROPE(64, KVB_BF16);
  } else {
    if (out_dtype == KVB_F64) KVB_ROPE(128, KVB_F64);
    else if (out_dtype == KVB_F32) KVB_ROPE(128, KVB_F32);
    else KVB_ROPE(128, KVB_BF16);
  }
#undef KVB_ROPE
  return hipGetLastError();
}

// Chunk importance (Sec. 4.4): one workgroup of 1024 lanes per chunk.  Each key
// vector is read by 8 adjacent lanes: 16-byte piece i of the vector goes to
// lane i % 8, so every load instruction of a wave reads 8 whole 128-byte
// segments (8 vectors).  All of a lane's pieces are requested before any is
// summed; a lane sums its squares in piece order (double), the 8 lanes combine
// theirs with a fixed xor tree (every level adds two values, so all 8 end with
// the same bits), and the vector's first lane adds the norm to its running
// sum.  The lanes' sums are combined with a fixed xor-shuffle tree, the 16 wave
// sums in wave order, and the chunk's share is added to importance[p].  Fixed
// assignment and order: deterministic.
constexpr int kImpLanes = 8;  // lanes per key vector

template <typename T>
__device__ __forceinline__ double sum_sq_piece(const T* p) {  // one 16-byte piece
  if constexpr (sizeof(T) == 8) {
    const double2 a = *reinterpret_cast<const double2*>(p);
    return __builtin_fma(a.y, a.y, a.x * a.x);
  } else {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const double x0 = a.x, x1 = a.y, x2 = a.z, x3 = a.w;
    return __builtin_fma(x3, x3, __builtin_fma(x2, x2, __builtin_fma(x1, x1, x0 * x0)));
  }
}

template <typename T, int D>
__global__ void __launch_bounds__(1024)
importance_kernel(int32_t n_vectors, double inv_count, const void* __restrict__ in,
                  double* __restrict__ importance) {
  constexpr int PER = 16 / (int)sizeof(T);    // elements per piece
  constexpr int NP = D / PER;                 // pieces per vector
  constexpr int LP = NP / kImpLanes;          // pieces per lane
  static_assert(LP >= 1 && NP % kImpLanes == 0, "a vector spans whole pieces of every lane");
  __shared__ double wave_sum[16];
  const int p = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = threadIdx.x % kImpLanes;
  const T* base = reinterpret_cast<const T*>(in) + (int64_t)p * n_vectors * D;
  double acc = 0.0;
  for (int v = threadIdx.x / kImpLanes; v < n_vectors; v += 1024 / kImpLanes) {
    const T* row = base + (int64_t)v * D + sub * PER;
    double part[LP];
#pragma unroll
    for (int j = 0; j < LP; ++j) part[j] = sum_sq_piece<T>(row + j * kImpLanes * PER);
    double ss = 0.0;
#pragma unroll
    for (int j = 0; j < LP; ++j) ss += part[j];
#pragma unroll
    for (int m = 1; m < kImpLanes; m <<= 1) ss += __shfl_xor(ss, m, 64);
    if (sub == 0) acc += sqrt(ss);
  }
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) acc += __shfl_xor(acc, m, 64);
  if (lane == 0) wave_sum[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double total = 0.0;
    for (int w = 0; w < 16; ++w) total += wave_sum[w];
    importance[p] += total * inv_count;
  }
}

hipError_t launch_kivi_quantize(const kvb_pool_layout& p, int32_t n_pool, int32_t first_layer,
                                int32_t n_in, kvb_dtype in_dtype, const void* k_in,
                                const void* v_in, uint8_t* k_codes, float* k_scale, float* k_zero,
                                uint8_t* v_codes, float* v_scale, float* v_zero, hipStream_t s) {
  const int64_t kw = (int64_t)n_pool * n_in * p.n_kv_heads * (p.chunk_len / p.k_group) * (p.head_dim / 2);
  const int64_t vw = (int64_t)n_pool * n_in * p.n_kv_heads * p.chunk_len * (p.head_dim / p.v_group);
  if (in_dtype == KVB_F64) {
    hipLaunchKernelGGL(quant_keys_kernel<double>, dim3(grid_for(kw)), dim3(256), 0, s, n_pool,
                       p.n_layers, first_layer, n_in, p.n_kv_heads, p.chunk_len, p.head_dim,
                       p.bits, p.k_group, k_in, k_codes, k_scale, k_zero);
    hipLaunchKernelGGL(quant_values_kernel<double>, dim3(grid_for(vw)), dim3(256), 0, s, n_pool,
                       p.n_layers, first_layer, n_in, p.n_kv_heads, p.chunk_len, p.head_dim,
                       p.bits, p.v_group, v_in, v_codes, v_scale, v_zero);
  } else {
    hipLaunchKernelGGL(quant_keys_kernel<float>, dim3(grid_for(kw)), dim3(256), 0, s, n_pool,
                       p.n_layers, first_layer, n_in, p.n_kv_heads, p.chunk_len, p.head_dim,
                       p.bits, p.k_group, k_in, k_codes, k_scale, k_zero);
    hipLaunchKernelGGL(quant_values_kernel<float>, dim3(grid_for(vw)), dim3(256), 0, s, n_pool,
                       p.n_layers, first_layer, n_in, p.n_kv_heads, p.chunk_len, p.head_dim,
                       p.bits, p.v_group, v_in, v_codes, v_scale, v_zero);
  }
  return hipGetLastError();
}

hipError_t launch_chunk_importance(const kvb_pool_layout& p, int32_t n_pool, int32_t n_in,
                                   kvb_dtype in_dtype, const void* k_in, double* importance,
                                   hipStream_t s) {
  const int32_t n_vectors = n_in * p.n_kv_heads * p.chunk_len;
  const double inv_count = 1.0 / ((double)p.n_layers * p.n_kv_heads * p.chunk_len);
#define KVB_IMPORTANCE(T, D)                                                                    \
  hipLaunchKernelGGL((importance_kernel<T, D>), dim3(n_pool), dim3(1024), 0, s, n_vectors,      \
                     inv_count, k_in, importance)
  if (in_dtype == KVB_F64) {
    if (p.head_dim == 128) KVB_IMPORTANCE(double, 128); else KVB_IMPORTANCE(double, 64);
  } else {
    if (p.head_dim == 128) KVB_IMPORTANCE(float, 128); else KVB_IMPORTANCE(float, 64);
  }
#undef KVB_IMPORTANCE
  return hipGetLastError();
}

}  // namespace kvb
