// Row selection (Alg. 2 step 3, Alg. 1 seam windows, live rows).
//
// One 1024-thread workgroup per (set, prompt) segment.  Deviations are mapped
// to order-preserving uint32 keys (NaN lowest, -0 equal to +0); a 4-pass
// 8-bit radix select over the segment's candidate rows finds the k-th largest
// key tau and how many rows equal to tau are still needed.  One ordered pass
// over the rows then takes: forced rows, candidates with key > tau, and the
// first `need_eq` candidates with key == tau in row order (the lower row wins
// a tie).  Positions come from wave ballots and a block-wide prefix, so the
// output is ascending without a sort and no atomic decides an order.  LDS
// atomics only count histogram bins.
//
// Segments of up to 48K rows use select_reg_kernel: every thread keeps the keys
// and flags of its KPT rows (rows lo + j * 1024 + tid) in registers, so the
// four histogram passes touch no memory but LDS, and the compaction takes one
// ballot per register slot with a single block-wide prefix over all of them.
// Longer segments use select_kernel, which re-reads the keys on every pass.
//
// Several prompts per set: rows go to a staging area at the prompt's own row
// offset and a second small kernel packs them and writes cu_rows.
#include "kvb_device.h"
#include "kvb_internal.h"

#include <mutex>

namespace kvb {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;

__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0u;  // NaN: below everything
  if (u == 0x80000000u) u = 0u;                     // -0 -> +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

struct ScanLds {
  uint32_t wave_tot[kWaves];
};

// Block-wide exclusive prefix of a 0/1 flag (every thread must call).
__device__ __forceinline__ uint32_t block_excl(bool bit, ScanLds& s, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t m = __ballot(bit);
  const uint32_t below = (uint32_t)__popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) s.wave_tot[wave] = (uint32_t)__popcll(m);
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t c = s.wave_tot[w];
    before += (w < wave) ? c : 0u;
    tot += c;
  }
  __syncthreads();
  *total = tot;
  return before + below;
}

__global__ void __launch_bounds__(kThreads)
select_kernel(int64_t t_total, const int32_t* __restrict__ cu_seqlens, int32_t n_seqs,
              const float* __restrict__ delta, const uint8_t* __restrict__ flags,
              const int32_t* __restrict__ k_per_seq, int32_t* __restrict__ rows_out,
              int32_t* __restrict__ cu_rows, int32_t* __restrict__ staging,
              int32_t* __restrict__ counts) {
  __shared__ uint32_t hist[256];
  __shared__ ScanLds scan;
  __shared__ uint32_t sh_prefix, sh_remaining;
  const int b = blockIdx.x;
  const int64_t set = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t lo = cu_seqlens[b], hi = cu_seqlens[b + 1];
  const float* dl = delta + set * t_total;

  // candidates in the segment
  uint32_t n_cand = 0;
  for (int64_t base = lo; base < hi; base += kThreads) {
    const int64_t r = base + tid;
    const bool c = r < hi && (flags[r] & KVB_ROW_CANDIDATE);
    uint32_t tot;
    block_excl(c, scan, &tot);
    n_cand += tot;
  }
  int64_t k = k_per_seq[set * n_seqs + b];
  if (k < 0) k = 0;
  const bool take_all = k >= (int64_t)n_cand;
  const bool take_none = k == 0;

  uint32_t tau = 0, need_eq = 0;
  if (!take_all && !take_none) {
    uint32_t prefix = 0, remaining = (uint32_t)k;
    for (int digit = 3; digit >= 0; --digit) {
      for (int i = tid; i < 256; i += kThreads) hist[i] = 0;
      __syncthreads();
      const uint32_t hi_mask = digit == 3 ? 0u : (0xFFFFFFFFu << (8 * (digit + 1)));
      int run_bin = -1;
      uint32_t run_n = 0;
      for (int64_t r = lo + tid; r < hi; r += kThreads) {
        if (!(flags[r] & KVB_ROW_CANDIDATE)) continue;
        const uint32_t key = order_key(dl[r]);
        if ((key & hi_mask) != (prefix & hi_mask)) continue;
        const int bin = (key >> (8 * digit)) & 0xFF;
        if (bin == run_bin) {
          ++run_n;
        } else {
          if (run_n) atomicAdd(&hist[run_bin], run_n);
          run_bin = bin;
          run_n = 1;
        }
      }
      if (run_n) atomicAdd(&hist[run_bin], run_n);
      __syncthreads();
      if (wave == 0) {
        // lane i owns bins 255-4i .. 252-4i (walking from the top)
        uint32_t hb[4], s = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          hb[j] = hist[255 - 4 * lane - j];
          s += hb[j];
        }
        uint32_t incl = s;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const uint32_t v = __shfl_up(incl, off, 64);
          if (lane >= off) incl += v;
        }
        const uint64_t hit = __ballot(incl >= remaining);
        const int first = __ffsll((unsigned long long)hit) - 1;
        if (lane == first) {
          uint32_t cum = incl - s;
          for (int j = 0; j < 4; ++j) {
            if (cum + hb[j] >= remaining) {
              sh_prefix = prefix | ((uint32_t)(255 - 4 * lane - j) << (8 * digit));
              sh_remaining = remaining - cum;
              break;
            }
            cum += hb[j];
          }
        }
      }
      __syncthreads();
      prefix = sh_prefix;
      remaining = sh_remaining;
    }
    tau = prefix;
    need_eq = remaining;
  }

  // ordered compaction
  uint32_t run_sel = 0, run_eq = 0;
  int32_t* dst = (n_seqs == 1) ? rows_out + set * t_total : staging + set * t_total + lo;
  for (int64_t base = lo; base < hi; base += kThreads) {
    const int64_t r = base + tid;
    const bool valid = r < hi;
    const uint32_t f = valid ? flags[r] : 0u;
    const bool cand = f & KVB_ROW_CANDIDATE;
    const bool forced = f & KVB_ROW_FORCED;
    bool gt = false, eq = false;
    if (cand) {
      if (take_all) {
        gt = true;
      } else if (!take_none) {
        const uint32_t key = order_key(dl[r]);
        gt = key > tau;
        eq = key == tau;
      }
    }
    uint32_t eq_tot;
    const uint32_t eq_rank = run_eq + block_excl(eq, scan, &eq_tot);
    const bool sel = forced || gt || (eq && eq_rank < need_eq);
    uint32_t sel_tot;
    const uint32_t idx = run_sel + block_excl(sel, scan, &sel_tot);
    if (sel) dst[idx] = (int32_t)r;
    run_sel += sel_tot;
    run_eq += eq_tot;
  }
  if (tid == 0) {
    if (n_seqs == 1) {
      cu_rows[set * 2] = 0;
      cu_rows[set * 2 + 1] = (int32_t)run_sel;
    } else {
      counts[set * n_seqs + b] = (int32_t)run_sel;
    }
  }
  (void)lane;
}


// Radix select of the k-th largest key among the candidate keys of this
// thread's register slots; every thread must call.  Returns tau and how many
// candidates equal to tau are still needed.
template <int KPT>
__device__ __forceinline__ void radix_select_reg(const uint32_t (&key)[KPT], uint64_t candm,
                                                 uint32_t k, uint32_t* hist, uint32_t* sh_prefix,
                                                 uint32_t* sh_remaining, uint32_t* tau,
                                                 uint32_t* need_eq) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint32_t prefix = 0, remaining = k;
  for (int digit = 3; digit >= 0; --digit) {
    for (int i = tid; i < 256; i += kThreads) hist[i] = 0;
    __syncthreads();
    const uint32_t hi_mask = digit == 3 ? 0u : (0xFFFFFFFFu << (8 * (digit + 1)));
    int run_bin = -1;
    uint32_t run_n = 0;
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      if (!((candm >> j) & 1ull)) continue;
      if ((key[j] & hi_mask) != (prefix & hi_mask)) continue;
      const int bin = (key[j] >> (8 * digit)) & 0xFF;
      if (bin == run_bin) {
        ++run_n;
      } else {
        if (run_n) atomicAdd(&hist[run_bin], run_n);
        run_bin = bin;
        run_n = 1;
      }
    }
    if (run_n) atomicAdd(&hist[run_bin], run_n);
    __syncthreads();
    if (wave == 0) {
      // lane i owns bins 255-4i .. 252-4i (walking from the top)
      uint32_t hb[4], sum = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        hb[j] = hist[255 - 4 * lane - j];
        sum += hb[j];
      }
      uint32_t incl = sum;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t v = __shfl_up(incl, off, 64);
        if (lane >= off) incl += v;
      }
      const uint64_t hit = __ballot(incl >= remaining);
      const int first = __ffsll((unsigned long long)hit) - 1;
      if (lane == first) {
        uint32_t cum = incl - sum;
        for (int j = 0; j < 4; ++j) {
          if (cum + hb[j] >= remaining) {
            *sh_prefix = prefix | ((uint32_t)(255 - 4 * lane - j) << (8 * digit));
            *sh_remaining = remaining - cum;
            break;
          }
          cum += hb[j];
        }
      }
    }
    __syncthreads();
    prefix = *sh_prefix;
    remaining = *sh_remaining;
  }
  *tau = prefix;
  *need_eq = remaining;
}

// Per-slot, per-wave counts of a bit (slot-major, then thread order) into
// wcnt; returns the block-wide total.  Every thread must call; wcnt is valid
// until the next call.
template <int KPT>
__device__ __forceinline__ uint32_t slot_counts(uint64_t bits, uint32_t (*wcnt)[kWaves],
                                                int nslots) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();  // the previous user of wcnt is done
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    if (j < nslots) {
      const uint64_t ball = __ballot((bits >> j) & 1ull);
      if (lane == 0) wcnt[j][wave] = (uint32_t)__popcll(ball);
    }
  }
  __syncthreads();
  uint32_t tot = 0;
  for (int j = 0; j < nslots; ++j)
#pragma unroll
    for (int w = 0; w < kWaves; ++w) tot += wcnt[j][w];
  return tot;
}

// Exclusive rank of slot j's bit among all set bits (slot-major, then thread),
// from the counts of slot_counts and the running total of slots before j.
__device__ __forceinline__ uint32_t slot_rank(uint64_t bits, int j, const uint32_t (*wcnt)[kWaves],
                                              uint32_t run_before, uint32_t* slot_total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t ball = __ballot((bits >> j) & 1ull);
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t c = wcnt[j][w];
    before += (w < wave) ? c : 0u;
    tot += c;
  }
  *slot_total = tot;
  return run_before + before + (uint32_t)__popcll(ball & ((1ull << lane) - 1ull));
}

template <int KPT>
__global__ void __launch_bounds__(kThreads)
select_reg_kernel(int64_t t_total, const int32_t* __restrict__ cu_seqlens, int32_t n_seqs,
                  const float* __restrict__ delta, const uint8_t* __restrict__ flags,
                  const int32_t* __restrict__ k_per_seq, int32_t* __restrict__ rows_out,
                  int32_t* __restrict__ cu_rows, int32_t* __restrict__ staging,
                  int32_t* __restrict__ counts) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t wcnt[KPT][kWaves];
  __shared__ uint32_t sh_prefix, sh_remaining;
  const int b = blockIdx.x;
  const int64_t set = blockIdx.y;
  const int tid = threadIdx.x;
  const int64_t lo = cu_seqlens[b], hi = cu_seqlens[b + 1];
  const int nslots = (int)((hi - lo + kThreads - 1) / kThreads);  // <= KPT by the launch
  const float* dl = delta + set * t_total;

  // this thread's rows lo + j * kThreads + tid: keys and flags, loaded once
  uint32_t key[KPT];
  uint64_t candm = 0, forcedm = 0;
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    key[j] = 0;
    const int64_t r = lo + (int64_t)j * kThreads + tid;
    if (j < nslots && r < hi) {
      const uint32_t f = flags[r];
      if (f & KVB_ROW_CANDIDATE) {
        candm |= 1ull << j;
        key[j] = order_key(dl[r]);
      }
      if (f & KVB_ROW_FORCED) forcedm |= 1ull << j;
    }
  }
  const uint32_t n_cand = slot_counts<KPT>(candm, wcnt, nslots);
  int64_t k = k_per_seq[set * n_seqs + b];
  if (k < 0) k = 0;
  const bool take_all = k >= (int64_t)n_cand;
  const bool take_none = k == 0;

  uint64_t gtm = 0, eqm = 0;
  if (take_all) {
    gtm = candm;
  } else if (!take_none) {
    uint32_t tau, need_eq;
    radix_select_reg<KPT>(key, candm, (uint32_t)k, hist, &sh_prefix, &sh_remaining, &tau,
                          &need_eq);
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      if ((candm >> j) & 1ull) {
        if (key[j] > tau) gtm |= 1ull << j;
        if (key[j] == tau) eqm |= 1ull << j;
      }
    }
    // the first need_eq keys equal to tau, in row order (the lower row wins a tie)
    const uint32_t n_eq = slot_counts<KPT>(eqm, wcnt, nslots);
    if (need_eq < n_eq) {
      uint32_t run = 0;
      uint64_t keep = 0;
#pragma unroll
      for (int j = 0; j < KPT; ++j) {
        if (j < nslots) {
          uint32_t tot;
          const uint32_t rk = slot_rank(eqm, j, wcnt, run, &tot);
          if (((eqm >> j) & 1ull) && rk < need_eq) keep |= 1ull << j;
          run += tot;
        }
      }
      eqm = keep;
    }
  }
  const uint64_t selm = forcedm | gtm | eqm;
  const uint32_t n_sel = slot_counts<KPT>(selm, wcnt, nslots);
  int32_t* dst = (n_seqs == 1) ? rows_out + set * t_total : staging + set * t_total + lo;
  uint32_t run = 0;
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    if (j < nslots) {
      uint32_t tot;
      const uint32_t rk = slot_rank(selm, j, wcnt, run, &tot);
      if ((selm >> j) & 1ull) dst[rk] = (int32_t)(lo + (int64_t)j * kThreads + tid);
      run += tot;
    }
  }
  if (tid == 0) {
    if (n_seqs == 1) {
      cu_rows[set * 2] = 0;
      cu_rows[set * 2 + 1] = (int32_t)n_sel;
    } else {
      counts[set * n_seqs + b] = (int32_t)n_sel;
    }
  }
}

__global__ void __launch_bounds__(256)
pack_kernel(int64_t t_total, const int32_t* __restrict__ cu_seqlens, int32_t n_seqs,
            const int32_t* __restrict__ staging, const int32_t* __restrict__ counts,
            int32_t* __restrict__ rows_out, int32_t* __restrict__ cu_rows) {
  const int b = blockIdx.x;
  const int64_t set = blockIdx.y;
  const int32_t* cnt = counts + set * n_seqs;
  int64_t off = 0;
  for (int i = 0; i < b; ++i) off += cnt[i];
  const int64_t lo = cu_seqlens[b];
  const int32_t n = cnt[b];
  const int32_t* src = staging + set * t_total + lo;
  int32_t* dst = rows_out + set * t_total + off;
  for (int i = threadIdx.x; i < n; i += blockDim.x) dst[i] = src[i];
  if (b == 0 && threadIdx.x == 0) {
    int32_t* cu = cu_rows + set * (n_seqs + 1);
    int32_t acc = 0;
    cu[0] = 0;
    for (int i = 0; i < n_seqs; ++i) {
      acc += cnt[i];
      cu[i + 1] = acc;
    }
  }
}

}  // namespace

size_t select_workspace_bytes(int32_t n_sets, int64_t t_total, int32_t n_seqs) {
  if (n_seqs <= 1) return 0;
  const size_t staging = (size_t)n_sets * (size_t)t_total * sizeof(int32_t);
  const size_t counts = (size_t)n_sets * (size_t)n_seqs * sizeof(int32_t);
  return ((staging + 255) / 256) * 256 + counts;
}

hipError_t launch_select(int32_t n_sets, int64_t t_total, const int32_t* cu_seqlens,
                         int32_t n_seqs, const float* delta, const uint8_t* row_flags,
                         const int32_t* k_per_seq, int32_t* rows, int32_t* cu_rows,
                         void* workspace, hipStream_t s) {
  int32_t* staging = nullptr;
  int32_t* counts = nullptr;
  if (n_seqs > 1) {
    staging = reinterpret_cast<int32_t*>(workspace);
    const size_t st = (size_t)n_sets * (size_t)t_total * sizeof(int32_t);
    counts = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(workspace) + ((st + 255) / 256) * 256);
  }
  // the longest prompt is at most t_total rows: pick the register-slot count from it
  const dim3 grid(n_seqs, n_sets);
#define KVB_SELECT_REG(K)                                                                       \
  hipLaunchKernelGGL(select_reg_kernel<K>, grid, dim3(kThreads), 0, s, t_total, cu_seqlens,     \
                     n_seqs, delta, row_flags, k_per_seq, rows, cu_rows, staging, counts)
  if (t_total <= 8 * kThreads)
    KVB_SELECT_REG(8);
  else if (t_total <= 16 * kThreads)
    KVB_SELECT_REG(16);
  else if (t_total <= 32 * kThreads)
    KVB_SELECT_REG(32);
  else if (t_total <= 48 * kThreads)
    KVB_SELECT_REG(48);
  else
    hipLaunchKernelGGL(select_kernel, grid, dim3(kThreads), 0, s, t_total, cu_seqlens, n_seqs,
                       delta, row_flags, k_per_seq, rows, cu_rows, staging, counts);
#undef KVB_SELECT_REG
  if (n_seqs > 1)
    hipLaunchKernelGGL(pack_kernel, dim3(n_seqs, n_sets), dim3(256), 0, s, t_total, cu_seqlens,
                       n_seqs, staging, counts, rows, cu_rows);
  return hipGetLastError();
}

// Scratch of the allocation-free selection (kvb_select_noalloc): the staging
// rows and per-prompt counts that kvb_select keeps in the caller's workspace.
// Every device the library runs on holds one copy for the life of the process.
// In host code `scratch` names a host-side stand-in, not device memory: host
// code reaches the array only through the address select_scratch returns.
static __device__ __align__(256) unsigned char scratch[kSelectScratchBytes];

// Device address of this device's copy of `scratch`, looked up once per device
// (with that device current) and kept.
hipError_t select_scratch(void** ptr) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

hipError_t launch_select_noalloc(int32_t n_sets, int64_t t_total, const int32_t* cu_seqlens,
                                 int32_t n_seqs, const float* delta, const uint8_t* row_flags,
                                 const int32_t* k_per_seq, int32_t* rows, int32_t* cu_rows,
                                 hipStream_t s) {
  void* ws = nullptr;
  if (n_seqs > 1) {
    hipError_t e = select_scratch(&ws);
    if (e != hipSuccess) return e;
  }
  return launch_select(n_sets, t_total, cu_seqlens, n_seqs, delta, row_flags, k_per_seq, rows,
                       cu_rows, ws, s);
}

}  // namespace kvb
