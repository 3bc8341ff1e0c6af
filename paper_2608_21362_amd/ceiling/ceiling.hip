// Practical ceilings of the chip, measured next to the path's kernels so that
// their roofline fractions can be read against what the device sustains as
// well as against its published peaks.  Not part of the path: built into a
// library of its own that only the benchmark loads.
//
//   kvb_ceiling_mfma  every workgroup runs back-to-back bf16 32x32x16 matrix
//                     products on eight independent accumulators per wave (no
//                     memory traffic), with the attention kernel's launch shape
//                     (256 threads, two workgroups per CU)
//   kvb_ceiling_read  a streaming read of a buffer (16-byte loads, grid-stride)
//   kvb_ceiling_copy  a streaming copy (16-byte loads and stores)

// Results are never used; a store guarded by a test that cannot pass keeps the
// compiler from removing the work.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

__global__ void __launch_bounds__(256, 2) mfma_loop(int32_t iters, float* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)((lane + i) & 7));
    b[i] = (__bf16)(0.002f * (float)((lane * 3 + i) & 7));
  }
  f32x16 acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = f32x16{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[k], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < 8; ++k) s += acc[k][0] + acc[k][15];
  if (s == -1.0f) sink[blockIdx.x * blockDim.x + threadIdx.x] = s;  // never taken
}

// Both streaming kernels walk the buffer in chunks of kUnroll x 256 16-byte
// pieces, one chunk per workgroup at a time (grid-stride over chunks): thread
// t takes pieces t, t + 256, ... of the chunk, so every load instruction of a
// wave covers 1 KiB and a workgroup's kUnroll loads in flight cover 16 KiB of
// contiguous memory.
constexpr int kUnroll = 4;

__global__ void __launch_bounds__(256) read_loop(const uint4* __restrict__ in, int64_t n16,
                                                 uint32_t* __restrict__ sink) {
  uint32_t x = 0;
  constexpr int64_t CH = kUnroll * 256;
  for (int64_t c = (int64_t)blockIdx.x * CH; c < n16; c += (int64_t)gridDim.x * CH) {
    uint4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = c + u * 256 + threadIdx.x;
      v[u] = i < n16 ? in[i] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (x == 0x9E3779B9u) sink[blockIdx.x * blockDim.x + threadIdx.x] = x;  // never taken in practice
}

__global__ void __launch_bounds__(256) copy_loop(const uint4* __restrict__ in,
                                                 uint4* __restrict__ out, int64_t n16) {
  constexpr int64_t CH = kUnroll * 256;
  for (int64_t c = (int64_t)blockIdx.x * CH; c < n16; c += (int64_t)gridDim.x * CH) {
    uint4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = c + u * 256 + threadIdx.x;
      if (i < n16) v[u] = in[i];
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = c + u * 256 + threadIdx.x;
      if (i < n16) out[i] = v[u];
    }
  }
}

int fail(hipError_t e) { return e == hipSuccess ? 0 : (int)e; }

}  // namespace

extern "C" {

// Launches n_wg workgroups of 256 threads, each wave doing iters x 8 products
// of 32x32x16 (32,768 flops each).  sink: device float[n_wg * 256] (never
// written in practice).  Returns 0 or the HIP error code.
int kvb_ceiling_mfma(int32_t n_wg, int32_t iters, float* sink, void* stream) {
  if (n_wg <= 0 || iters <= 0 || !sink) return -1;
  hipLaunchKernelGGL(mfma_loop, dim3(n_wg), dim3(256), 0, (hipStream_t)stream, iters, sink);
  return fail(hipGetLastError());
}

// Reads bytes (a multiple of 16) from device buffer in.  sink: device
// uint32[n_wg * 256].
int kvb_ceiling_read(const void* in, int64_t bytes, int32_t n_wg, uint32_t* sink, void* stream) {
  if (!in || !sink || bytes <= 0 || bytes % 16 || n_wg <= 0) return -1;
  hipLaunchKernelGGL(read_loop, dim3(n_wg), dim3(256), 0, (hipStream_t)stream,
                     reinterpret_cast<const uint4*>(in), bytes / 16, sink);
  return fail(hipGetLastError());
}

// Copies bytes (a multiple of 16) between device buffers.
int kvb_ceiling_copy(const void* in, void* out, int64_t bytes, int32_t n_wg, void* stream) {
  if (!in || !out || bytes <= 0 || bytes % 16 || n_wg <= 0) return -1;
  hipLaunchKernelGGL(copy_loop, dim3(n_wg), dim3(256), 0, (hipStream_t)stream,
                     reinterpret_cast<const uint4*>(in), reinterpret_cast<uint4*>(out), bytes / 16);
  return fail(hipGetLastError());
}

}  // extern "C"
