// Patch and sparse-query causal GQA attention (Alg. 2 step 4; Eq. 2).
//
// Per call, on one stream:
//
//   patch_kernel     cache[l][h][t] <- fresh[l][h][t] for every selected row t
//                    (both tensors, every kv head); its first workgroups build
//                    the work decomposition when the launch uses balanced
//                    ranges (below)
//   v16_kernel       the fp16 copy of the patched V cache that the P.V product
//                    takes as its operand (exact for |v| < 65536: a bf16
//                    significand fits an fp16 one; values fp16 cannot hold are
//                    reported in a status word)
//   attn_kernel      the attention itself (below)
//   combine_kernel   merges the partial records of tiles that were cut between
//                    workgroups (balanced ranges only)
//
// attn_kernel: a tile is up to 128 / G selected rows of one prompt for one
// (layer, kv head g): rows x the G = Hq/Hkv query heads that share kv head g
// fill the MFMA N dimension, each of the 4 waves owning 32 query vectors
// (32/G rows x G heads).  A workgroup runs one whole tile, or a range of key
// blocks that may span tiles (see attn_kernel).  Keys stream in blocks of 32
// through a five-stage LDS ring filled by asynchronous global->LDS loads (no
// VGPR staging), XOR-swizzled on 16-byte chunks so the operand reads below are
// free of bank conflicts:
//
//   S^T (32 keys x 32 queries) = K Q^T     bf16 MFMA 32x32x16: K rows from LDS
//                                           (A operand), Q^T kept in VGPRs
//   online softmax over keys               fp32, base-2 exponent.  Each lane
//                                           holds 16 scores of one query, the
//                                           other 16 sit in lane ^ 32.  The
//                                           running maximum is refreshed only
//                                           when a block raises it by more
//                                           than 15 (log2 units), so partial
//                                           probabilities stay below 2^15
//   O^T (d x 32 queries) += V^T P^T        fp16 MFMA 32x32x16: V^T read from
//                                           the row-major fp16 V block with the
//                                           LDS transpose read, P^T converted
//                                           from the S^T accumulators
//
// The loop is software-pipelined: the scores of block j+1 are computed while
// block j's probabilities are formed, and the LDS operands of the next step
// are read at the end of the current one; one barrier per block.
//
// The accumulator layout of a 32x32 MFMA gives lane half h the keys
// {4h..4h+3, 8+4h..8+4h+3} of every 16-key step; the transpose reads fetch V
// for exactly those keys, so no permutation is needed anywhere.  The
// contraction index of each product is laid out identically on its two
// operands, so its order inside the MFMA does not matter.
#include <math.h>

#include <type_traits>

#include "kvb_device.h"
#include "kvb_internal.h"

namespace kvb {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((ext_vector_type(2))) unsigned u32x2;
typedef __attribute__((ext_vector_type(4))) unsigned u32x4;
typedef __attribute__((ext_vector_type(2))) _Float16 f16x2;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(16))) float f32x16;

#ifndef KVB_ATTN_WAVES
#define KVB_ATTN_WAVES 4
#endif
constexpr int kWaves = KVB_ATTN_WAVES;  // waves per workgroup (each owns 32 query vectors)
constexpr int kThreads = 64 * kWaves;
constexpr int kQW = 32;                 // query vectors per wave
constexpr int kQT = kQW * kWaves;       // query vectors per workgroup
// Workgroups per CU the register allocator targets (compile-time tunable).
#ifndef KVB_ATTN_WG_PER_CU
#define KVB_ATTN_WG_PER_CU 2
#endif
constexpr int kKB = 32;                 // keys per block = one 32-row MFMA tile
constexpr int kStages = 5;              // LDS ring depth (80 KiB per workgroup at d = 128)
constexpr int kAttnMaxWorkgroups = 1024;  // attention workgroups (sizes the partial records)
// Balanced ranges charge every tile a fixed cost, in 32-key block units, for a
// segment's start (tile rows, queries and the first blocks fetched) and end
// (output or partial record written), so that workgroups covering many short
// tiles get fewer blocks.  Measured on MI355X at 8K keys per prompt: a
// segment's start and end take as long as five to eight blocks; with a CU's
// two workgroups on adjacent ranges, 11 gave the shortest per-layer launches
// of the values tried (7, 9, 11, 13).
constexpr int kSegCost = 11;
// With two workgroups per CU the dispatcher gives workgroups 0 .. CUs-1 the
// first slot of every CU and the rest the second; the hardware issues the
// older (first) workgroup's waves first, so it progresses faster while both
// run (per unit of the plan about 1.5 times as fast in a timestamped per-layer
// launch at 8K keys per prompt).  Balanced ranges give first-slot workgroups
// 3/2 of the units of second-slot ones so that the two finish together
// (measured on MI355X: 3/2 gave the shortest per-layer launches, 8/5 and 7/5
// 0.3 to 0.9 % longer; a different placement only costs balance, never
// correctness).
constexpr int kFirstShareNum = 3, kFirstShareDen = 2;
// Lazy rescaling: the running maximum (the reference of the probabilities)
// moves only when a block's maximum exceeds it by more than kLazy log2 units,
// so probabilities stay below 2^15 (fp16 holds up to 65504).  The reference
// is never above the true maximum: a reference above it would push the
// largest probabilities toward fp16's subnormal range.
constexpr float kLazy = 15.0f;
// Reference of a lane that has seen no visible key: finite and far below any
// scaled score, so that the first visible block always moves the reference
// (with factor exp2(kNoKey - m) = 0 for the still empty sums), a masked score
// (-inf) gives probability 0 against it, and no special case is needed for
// infinities in the block loop.
constexpr float kNoKey = -1.0e30f;

#define LDS_PTR(T, p) ((__attribute__((address_space(3))) T*)(p))

// wait until at most n vector-memory operations of this wave are outstanding
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// wait until this wave's LDS operations have completed
__device__ __forceinline__ void wait_lgkmcnt0() {
  __builtin_amdgcn_s_waitcnt((0xF) | (0x3 << 14) | (0x7 << 4) | (0x0 << 8));
}

// Keep the compiler from moving memory accesses across this point (the raw
// s_barrier builtin is not a memory barrier for it); emits no instruction.
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

// ------------------------------------------------------------ V to fp16 ----
// fp16 holds a bf16 value exactly unless its magnitude is 65536 or more (bf16
// magnitude bits 0x4780 and up, infinities and NaN included).
__device__ __forceinline__ bool f16_out_of_range(uint32_t w) {
  return (w & 0x7FFFu) >= 0x4780u || ((w >> 16) & 0x7FFFu) >= 0x4780u;
}

// v16 <- fp16(v), n8 pieces of 8 values.  With status != NULL, a value fp16
// cannot hold stores 1 there (plain stores of the same value by any thread
// that found one; the caller clears the word).
__global__ void __launch_bounds__(256)
v16_kernel(int64_t n8, const uint16_t* __restrict__ v, uint16_t* __restrict__ v16,
           uint32_t* __restrict__ status) {
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n8;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint4 a = reinterpret_cast<const uint4*>(v)[i];
    bad |= f16_out_of_range(a.x) || f16_out_of_range(a.y) || f16_out_of_range(a.z) ||
           f16_out_of_range(a.w);
    reinterpret_cast<uint4*>(v16)[i] =
        make_uint4(bf16x2_to_f16x2(a.x), bf16x2_to_f16x2(a.y),
                   bf16x2_to_f16x2(a.z), bf16x2_to_f16x2(a.w));
  }
  if (status != nullptr && bad) *status = 1u;
}

// ------------------------------------------------------------ tile lookup --
struct Tile {
  int b;          // prompt
  int r_begin;    // first entry of the tile in the set's row list
  int r_end;
};

// What a segment needs to know about its tile.
struct SegTile {
  int lg;               // layer * Hkv + kv head
  int r_begin, r_end;   // entries of the tile in the set's row list
  int kstart;           // first key (row) of the tile's prompt
  int kend;             // one past the tile's last query row
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

// ---------------------------------------------------------------- attention
template <int D>
struct AttnCfg {
  static constexpr int ROWB = D * 2;                 // bytes per K / V16 row
  static constexpr int CPR = ROWB / 16;              // 16-byte chunks per row
  static constexpr int BLK = kKB * ROWB;             // bytes of one K (or V) block
  static constexpr int RPI = 1024 / ROWB;            // rows per wave-wide 1 KiB load
  static constexpr int LOADS = BLK / (kThreads * 16);  // per-thread loads per tensor per block
  static constexpr int NS = D / 16;                  // 16-deep MFMA steps over d
  static constexpr int ND = D / 32;                  // 32-row d tiles of O^T
  // 16-byte-chunk swizzles (slot = chunk ^ f(row))
  static __device__ __forceinline__ int swz_k(int r) { return r % CPR; }
  static __device__ __forceinline__ int swz_v(int r) { return (CPR / 4) * (r & 3); }
};

// Per-lane byte offsets (inside a block) of this thread's asynchronous loads:
// piece i of the block is the 1 KiB a wave writes with one instruction; lane L
// writes LDS bytes 16 L of it, i.e. row piece*RPI + L/CPR, slot L % CPR, and
// fetches the global chunk that the swizzle maps to that slot.
template <int D>
struct LoadOffsets {
  int k[AttnCfg<D>::LOADS];
  int v[AttnCfg<D>::LOADS];
};

template <int D>
__device__ __forceinline__ LoadOffsets<D> load_offsets(int wave, int lane) {
  using C = AttnCfg<D>;
  LoadOffsets<D> o;
#pragma unroll
  for (int i = 0; i < C::LOADS; ++i) {
    const int r = (wave * C::LOADS + i) * C::RPI + lane / C::CPR;
    const int slot = lane % C::CPR;
    o.k[i] = r * C::ROWB + 16 * (slot ^ C::swz_k(r));
    o.v[i] = r * C::ROWB + 16 * (slot ^ C::swz_v(r));
  }
  return o;
}

// Raw buffer resource (128-bit, stride 0) over `bytes` bytes at `base`; loads
// at offsets >= bytes return zero.
typedef __attribute__((ext_vector_type(4))) int i32x4;
__device__ __forceinline__ i32x4 buffer_rsrc(const void* base, int bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xFFFFu));
  r[2] = __builtin_amdgcn_readfirstlane(bytes);
  r[3] = 0x00020000;
  return r;
}

// One asynchronous 16-byte-per-lane load from a buffer straight into LDS: lane
// L's data lands at lds_addr + 16 L.  Issued as inline assembly so the compiler
// does not order LDS reads of the *other* ring stage behind it; completion is
// awaited explicitly with wait_vmcnt before the stage is read.
__device__ __forceinline__ void lds_dma16(i32x4 rsrc, uint32_t lds_addr, int voff, int soff) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %1, %2, %3 offen lds"
      :
      : "s"(lds_addr), "v"(voff), "s"(rsrc), "s"(soff)
      : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)LDS_PTR(const char, p);
}

// Issue the asynchronous loads of one 32-key block of K (bf16) and V (fp16)
// into one LDS stage.  Each load takes a buffer resource that starts at the
// block's first row and covers the cache rows of this (layer, kv head) from
// there on (built on the scalar unit: the lanes add no block offset); rows
// past the end read as zero (their scores are masked).
template <int D>
__device__ __forceinline__ void issue_block(const uint16_t* kbase, const uint16_t* vbase, int T,
                                            int kb, const LoadOffsets<D>& lo, char* k_st,
                                            char* v_st, int wave) {
  using C = AttnCfg<D>;
  const int bytes = max(T - kb, 0) * C::ROWB;
  const i32x4 krs = buffer_rsrc(kbase + (int64_t)kb * D, bytes);
  const i32x4 vrs = buffer_rsrc(vbase + (int64_t)kb * D, bytes);
  const uint32_t kl = __builtin_amdgcn_readfirstlane(lds_addr(k_st) + wave * C::LOADS * 1024);
  const uint32_t vl = __builtin_amdgcn_readfirstlane(lds_addr(v_st) + wave * C::LOADS * 1024);
#pragma unroll
  for (int i = 0; i < C::LOADS; ++i) {
    lds_dma16(krs, kl + i * 1024, lo.k[i], 0);
    lds_dma16(vrs, vl + i * 1024, lo.v[i], 0);
  }
}

template <int D>
struct AttnState {
  f32x16 o[AttnCfg<D>::ND];
  float mc;      // reference of the probabilities in log2 units (the running
                 // maximum of the scaled scores, stale by at most kLazy), or
                 // kNoKey while this lane has seen no visible key
  float l_part;  // this lane's share of the running sum
};

// max / sum of x over lanes l and l ^ 32.  v_permlane32_swap exchanges the
// upper half of its first operand with the lower half of its second, so with
// both holding x, lane l ends with x[l] and x[l ^ 32] in its two registers.  It
// is written as inline assembly: the compiler builtin, given the same value
// twice, has been lowered to read both results from one register.
__device__ __forceinline__ void swap_halves(float& a, float& b) {
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ float max_halves(float x) {
  float a = x, b = x;
  swap_halves(a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float sum_halves(float x) {
  float a = x, b = x;
  swap_halves(a, b);
  return a + b;
}

// K operand of one 32-key block: lane (row n, half h) holds d = (D/2) h + 8 s + v
template <int D>
__device__ __forceinline__ void read_k(const char* k_st, int lane,
                                       bf16x8 (&kr)[AttnCfg<D>::NS]) {
  using C = AttnCfg<D>;
  const int half = lane >> 5, n = lane & 31;
  const char* krow = k_st + n * C::ROWB;
#pragma unroll
  for (int s = 0; s < C::NS; ++s) {
    const int chunk = (D / 16) * half + s;
    kr[s] = *reinterpret_cast<const bf16x8*>(krow + 16 * (chunk ^ C::swz_k(n)));
  }
}

// V^T operands of one 32-key block, for 16-key step ks and 32-row d tile dt.
// Transpose-read lane address: row 16 ks + 8 hh + 4 half + j/4, d = dbase + 4 (j % 4);
// the two reads are joined as whole registers (keys 4h..4h+3, then 8+4h..8+4h+3:
// element-wise 16-bit extraction here has been miscompiled into a broadcast).
template <int D>
__device__ __forceinline__ void read_v(const char* v_st, int lane,
                                       f16x8 (&vr)[2][AttnCfg<D>::ND]) {
  using C = AttnCfg<D>;
  const int half = lane >> 5, j = lane & 15, grp = (lane >> 4) & 1;
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int dt = 0; dt < C::ND; ++dt) {
      const int elem = dt * 32 + 16 * grp + 4 * (j & 3);
      const int chunk = elem >> 3;
      u32x2 part[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int row = ks * 16 + 8 * hh + 4 * half + (j >> 2);
        const char* addr = v_st + row * C::ROWB + 16 * (chunk ^ C::swz_v(row)) + 2 * (elem & 7);
        part[hh] = __builtin_bit_cast(
            u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, addr)));
      }
      const u32x4 w = {part[0][0], part[0][1], part[1][0], part[1][1]};
      vr[ks][dt] = __builtin_bit_cast(f16x8, w);
    }
}

// S^T (32 keys x 32 queries) = K Q^T
template <int D>
__device__ __forceinline__ f32x16 scores(const bf16x8 (&kr)[AttnCfg<D>::NS],
                                         const bf16x8 (&qop)[AttnCfg<D>::NS]) {
  f32x16 acc = {};
#pragma unroll
  for (int s = 0; s < AttnCfg<D>::NS; ++s)
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kr[s], qop[s], acc, 0, 0, 0);
  return acc;
}

// Online-softmax update for one block of scores: masks keys past the query
// (or past the split), refreshes the running maximum when it grew by more than
// kLazy, and returns the probabilities as the fp16 P^T operands of the two
// 16-key steps (accumulator registers 0..7 and 8..15).
template <int D>
__device__ __forceinline__ void softmax_block(f32x16 sacc, AttnState<D>& st, float c_log2,
                                              bool full, int kb, int t_q, int k_hi, int lane,
                                              f16x8 (&pb)[2]) {
  using C = AttnCfg<D>;
  const int half = lane >> 5;
  if (__builtin_expect(!full, 0)) {
    // key kb + off is allowed iff off <= lim (off = 8(r/4) + 4 half + r%4)
    const int lim = min(t_q, k_hi - 1) - kb - 4 * half;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (8 * (r >> 2) + (r & 3) > lim) sacc[r] = -INFINITY;
  }
  float bmax = sacc[0];
#pragma unroll
  for (int r = 1; r < 16; ++r) bmax = fmaxf(bmax, sacc[r]);
  // the block's maximum in log2 units (-inf for a lane with no visible key in
  // it: such a lane never forces a rescale)
  const float bm = max_halves(bmax) * c_log2;
  if (__builtin_expect(__builtin_amdgcn_ballot_w64(bm - st.mc > kLazy) != 0, 0)) {
    const float mc_new = fmaxf(st.mc, bm);
    const float alpha = __builtin_amdgcn_exp2f(st.mc - mc_new);
    st.l_part *= alpha;
#pragma unroll
    for (int dt = 0; dt < C::ND; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) st.o[dt][r] *= alpha;
    st.mc = mc_new;
  }
  const float mc = st.mc;
  const f16x2 ones = {(_Float16)1.0f, (_Float16)1.0f};
  float psum = st.l_part;
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int v = 0; v < 8; v += 2) {
      const f32x2 e = {__builtin_amdgcn_exp2f(__builtin_fmaf(sacc[8 * ks + v], c_log2, -mc)),
                       __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[8 * ks + v + 1], c_log2, -mc))};
      const f16x2 h = __builtin_convertvector(e, f16x2);
      // the running sum adds the same fp16 values the P.V product uses
      psum = __builtin_amdgcn_fdot2(h, ones, psum, false);
      pb[ks][v] = h[0];
      pb[ks][v + 1] = h[1];
    }
  st.l_part = psum;
}

// Partial records: n_rec x kQT x D fp16 normalised outputs, then n_rec x kQT
// (max, sum) float pairs at this byte offset.
template <int D>
__host__ __device__ constexpr int64_t rec_ml_offset(int64_t n_rec) {
  return ((n_rec * kQT * D * 2 + 255) / 256) * 256;
}

// One segment: key blocks [blk_lo, blk_hi) (32 keys each, counted from the
// tile's prompt start) of one tile of selected rows of (layer, kv head).  With
// rec < 0 the segment covers the whole tile and writes the normalised output;
// otherwise it writes partial record `rec` (O normalised by this segment's
// sum, running maximum in log2 units, running sum) for the combine pass.
template <int D>
__device__ __forceinline__ void attend_segment(
    const SegTile& tl, int blk_lo, int blk_hi, int rec, int n_rec, char* k_ring, char* v_ring,
    int32_t Hq, int32_t Hkv, int32_t log2g, int64_t t_total, const int32_t* __restrict__ rows,
    int32_t rows_per_layer, const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
    const uint16_t* __restrict__ v16, float c_log2, int32_t out_f32, void* __restrict__ out,
    float* __restrict__ parts) {
  using C = AttnCfg<D>;
  const int G = 1 << log2g;
  const int l = tl.lg / Hkv, g = tl.lg % Hkv;
  const int32_t* rws = rows + (rows_per_layer ? (int64_t)l : 0) * t_total;
  const int T = (int)t_total;
  const int k_lo = tl.kstart + blk_lo * kKB;
  const int k_hi = min(tl.kstart + blk_hi * kKB, tl.kend);
  if (k_hi <= k_lo) return;

  // the previous segment of this workgroup is done with the LDS ring
  wait_lgkmcnt0();
  __builtin_amdgcn_s_barrier();
  compiler_fence();

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, n = lane & 31;
  const int rows_per_wave = kQW >> log2g;
  const int row_idx = tl.r_begin + wave * rows_per_wave + (n >> log2g);
  const int head = g * G + (n & (G - 1));
  // this lane's query row, and the smallest query row of this wave (rows are
  // ascending within a tile): blocks wholly at or below it need no mask
  int t_q = row_idx < tl.r_end ? rws[row_idx] : -1;
  const int t_min = rws[min(tl.r_begin + wave * rows_per_wave, tl.r_end - 1)];

  const int64_t kv_base = ((int64_t)l * Hkv + g) * t_total * D;
  const uint16_t* const kbase = kc + kv_base;
  const uint16_t* const vbase = v16 + kv_base;
  const LoadOffsets<D> lo = load_offsets<D>(wave, lane);
  const int nblk = (k_hi - k_lo + kKB - 1) / kKB;
  static_assert(kStages == 5, "stage index arithmetic assumes a 5-deep ring");

  // The first four blocks depend only on the tile: they are requested while
  // the query rows are on their way.
  issue_block<D>(kbase, vbase, T, k_lo, lo, k_ring, v_ring, wave);
  if (nblk > 1) issue_block<D>(kbase, vbase, T, k_lo + kKB, lo, k_ring + C::BLK, v_ring + C::BLK, wave);
  if (nblk > 2)
    issue_block<D>(kbase, vbase, T, k_lo + 2 * kKB, lo, k_ring + 2 * C::BLK, v_ring + 2 * C::BLK, wave);
  if (nblk > 3)
    issue_block<D>(kbase, vbase, T, k_lo + 3 * kKB, lo, k_ring + 3 * C::BLK, v_ring + 3 * C::BLK, wave);

  const bool qvalid = t_q >= tl.kstart && t_q < tl.kend;  // rows outside the prompt are skipped
  if (!qvalid) t_q = -1;
  // Q^T operand: query n, d = (D/2) h + 8 s + v
  bf16x8 qop[C::NS];
  {
    const uint16_t* qrow = q + (((int64_t)l * t_total + (qvalid ? t_q : 0)) * Hq + head) * D +
                           (D / 2) * half;
#pragma unroll
    for (int s = 0; s < C::NS; ++s) {
      const uint4 w = qvalid ? *reinterpret_cast<const uint4*>(qrow + 8 * s) : make_uint4(0, 0, 0, 0);
      qop[s] = __builtin_bit_cast(bf16x8, w);
    }
  }
  // Queries and the first blocks land before the loop: the compiler then never
  // waits on the queries -- and so on the in-flight prefetch -- later on.
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  compiler_fence();

  AttnState<D> st;
#pragma unroll
  for (int dt = 0; dt < C::ND; ++dt) st.o[dt] = f32x16{};
  st.mc = kNoKey;
  st.l_part = 0.0f;

  // Software pipeline over blocks: step j turns the scores of block j into
  // probabilities on the vector units while the matrix cores compute the
  // scores of block j + 1, then accumulates P V for block j, and last reads
  // the LDS operands of the next step (K of block j + 2, V of block j + 1), so
  // no step starts by waiting on LDS.  The ring holds blocks j .. j + 4: a step
  // waits for block j + 2 to land (block j + 3 may be in flight) and, after
  // the barrier that every wave reaches once done with block j - 1, requests
  // block j + 4 into that block's stage.  The waves raise their issue priority
  // while they send P V to the matrix cores.  The loop is unrolled over the
  // five ring stages so every LDS address is a per-lane base plus a constant.
  bf16x8 kr[C::NS];
  read_k<D>(k_ring, lane, kr);
  f32x16 sacc = scores<D>(kr, qop);
  f16x8 vr[2][C::ND];
  read_k<D>(k_ring + C::BLK, lane, kr);  // stale when nblk == 1: never used
  read_v<D>(v_ring, lane, vr);
  auto step = [&](auto stage, int j) {
    constexpr int S = decltype(stage)::value;  // ring stage of block j
    const int kb = k_lo + j * kKB;
    if (j + 3 < nblk)
      wait_vmcnt<2 * C::LOADS>();  // block j + 2 landed, block j + 3 may be in flight
    else
      wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    if (j + 4 < nblk)
      issue_block<D>(kbase, vbase, T, kb + 4 * kKB, lo, k_ring + ((S + 4) % 5) * C::BLK,
                     v_ring + ((S + 4) % 5) * C::BLK, wave);
    const bool full = (kb + kKB - 1 <= t_min) && (kb + kKB <= k_hi);
    f16x8 pb[2];
    softmax_block<D>(sacc, st, c_log2, full, kb, t_q, k_hi, lane, pb);
    sacc = scores<D>(kr, qop);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int dt = 0; dt < C::ND; ++dt)
        st.o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vr[ks][dt], pb[ks], st.o[dt], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(0);
    // operands of the next step (landed and visible since this step's
    // barrier; stale past the end of the segment, never used).  K first: LDS
    // reads return in order and the next step starts with the score products.
    read_k<D>(k_ring + ((S + 2) % 5) * C::BLK, lane, kr);
    compiler_fence();
    read_v<D>(v_ring + ((S + 1) % 5) * C::BLK, lane, vr);
  };
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;
  using S3 = std::integral_constant<int, 3>;
  using S4 = std::integral_constant<int, 4>;
  int j = 0;
  for (; j + 5 <= nblk; j += 5) {
    step(S0{}, j);
    step(S1{}, j + 1);
    step(S2{}, j + 2);
    step(S3{}, j + 3);
    step(S4{}, j + 4);
  }
  if (j < nblk) step(S0{}, j);
  if (j + 1 < nblk) step(S1{}, j + 1);
  if (j + 2 < nblk) step(S2{}, j + 2);
  if (j + 3 < nblk) step(S3{}, j + 3);

  if (!qvalid) return;
  const float l_run = sum_halves(st.l_part);
  if (rec < 0) {
    const float inv = (l_run > 0.0f) ? 1.0f / l_run : 0.0f;
    const int64_t ob = (((int64_t)l * t_total + t_q) * Hq + head) * D;
#pragma unroll
    for (int dt = 0; dt < C::ND; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int d0 = dt * 32 + 8 * j + 4 * half;
        const float a0 = st.o[dt][4 * j] * inv, a1 = st.o[dt][4 * j + 1] * inv;
        const float a2 = st.o[dt][4 * j + 2] * inv, a3 = st.o[dt][4 * j + 3] * inv;
        if (out_f32) {
          *reinterpret_cast<float4*>(reinterpret_cast<float*>(out) + ob + d0) =
              make_float4(a0, a1, a2, a3);
        } else {
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(out) + ob + d0) =
              make_uint2(pack_bf16x2(a0, a1), pack_bf16x2(a2, a3));
        }
      }
  } else {
    // partial record: O normalised by this segment's own sum, in fp16 (|O| is
    // bounded by max |V|, which fits fp16), plus (running max in log2 units, sum)
    const int qi = wave * kQW + n;
    const float inv = (l_run > 0.0f) ? 1.0f / l_run : 0.0f;
    uint16_t* wo = reinterpret_cast<uint16_t*>(parts) + ((int64_t)rec * kQT + qi) * D;
#pragma unroll
    for (int dt = 0; dt < C::ND; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x2 lo2 = {st.o[dt][4 * j] * inv, st.o[dt][4 * j + 1] * inv};
        const f32x2 hi2 = {st.o[dt][4 * j + 2] * inv, st.o[dt][4 * j + 3] * inv};
        const u32x2 h = {__builtin_bit_cast(unsigned, __builtin_convertvector(lo2, f16x2)),
                         __builtin_bit_cast(unsigned, __builtin_convertvector(hi2, f16x2))};
        *reinterpret_cast<u32x2*>(wo + dt * 32 + 8 * j + 4 * half) = h;
      }
    if (half == 0) {
      float* ml = reinterpret_cast<float*>(reinterpret_cast<char*>(parts) + rec_ml_offset<D>(n_rec)) +
                  ((int64_t)rec * kQT + qi) * 2;
      *reinterpret_cast<float2*>(ml) =
          make_float2(st.mc == kNoKey ? -INFINITY : st.mc, l_run);
    }
  }
}

// Plan area (int32): [0] c1, [1] c2, [2] n_first, [3] total, [4 .. 4+n_tiles]
// prefix, then the per-tile metadata (int4) at tile_meta_offset, then one
// 32-byte first-segment descriptor per workgroup at range_seg_offset.
__host__ __device__ constexpr int64_t tile_meta_offset(int64_t n_tiles) {
  return ((5 + n_tiles + 3) / 4) * 4;
}
__host__ __device__ constexpr int64_t range_seg_offset(int64_t n_tiles) {
  return tile_meta_offset(n_tiles) + 4 * n_tiles;
}
__host__ __device__ constexpr int64_t plan_ints(int64_t n_tiles, int64_t n_wg_max) {
  return range_seg_offset(n_tiles) + 8 * n_wg_max;
}

// Ranges are numbered by a range index v in unit order.  With two workgroups
// per CU (n_first > 0: workgroups 0 .. n_first-1 take the first slot of every
// CU, the other n_first the second), range 2p belongs to the second-slot
// workgroup of CU position p and range 2p + 1 to its first-slot partner, so a
// CU's two workgroups cover adjacent units (the same tiles, and so the same key
// blocks); second-slot ranges hold c2 units, first-slot ones c1.  With one
// workgroup per CU (n_first == 0) range v holds c2 units.  CU positions are
// grouped by XCD: workgroup offset o of a group of g (XCD o % 8 under
// round-robin dispatch) takes position (o % 8) g/8 + o / 8 when g is a multiple
// of 8 (else the identity), so consecutive ranges share an XCD and its L2.
__device__ __forceinline__ int unit_start(int v, int c1, int c2, int n_first) {
  return n_first > 0 ? (v / 2) * (c1 + c2) + (v % 2) * c2 : v * c2;
}

// Range index whose units hold unit u.
__device__ __forceinline__ int unit_owner(int u, int c1, int c2, int n_first) {
  if (n_first == 0) return u / c2;
  const int j = u / (c1 + c2);
  return 2 * j + (u - j * (c1 + c2) >= c2 ? 1 : 0);
}

__device__ __forceinline__ int xcd_pos(int o, int g) {
  return (g % 8 == 0) ? (o % 8) * (g / 8) + o / 8 : o;
}
__device__ __forceinline__ int xcd_off(int i, int g) {
  return (g % 8 == 0) ? 8 * (i % (g / 8)) + i / (g / 8) : i;
}

// Range index of workgroup w of n_wg (n_wg = 2 n_first when n_first > 0).
__device__ __forceinline__ int range_of(int w, int n_first, int n_wg) {
  if (n_first == 0) return xcd_pos(w, n_wg);
  return w >= n_first ? 2 * xcd_pos(w - n_first, n_first) : 2 * xcd_pos(w, n_first) + 1;
}

// Workgroup of range index v (inverse of range_of).
__device__ __forceinline__ int wg_of_range(int v, int n_first, int n_wg) {
  if (n_first == 0) return xcd_off(v, n_wg);
  return (v % 2 == 0) ? n_first + xcd_off(v / 2, n_first) : xcd_off(v / 2, n_first);
}

// Work decomposition.  Work unit = one 32-key block of one tile, and a tile
// with blocks also counts kSegCost units for its fixed cost (they come first
// and hold no blocks); units are numbered tile by tile, tiles ordered by
// (layer x kv head) and within it by row slot (tile index = layer x kv head *
// tile_slots + slot: a (layer, kv head)'s tiles, which share their key blocks,
// are adjacent, and its first row tiles, which attend to the fewest keys, come
// first; launches of whole tiles order them slot-major instead).  One workgroup
// builds the exclusive prefix sum of the tiles' unit counts, then the
// attention workgroup with range index v takes the contiguous units
// [unit_start(v), unit_start(v + 1)): c2 units for second-slot workgroups,
// c1 for first-slot ones (above), sized to cover every unit.
//   plan[0] = c1, plan[1] = c2, plan[2] = n_first, plan[3] = total,
//   plan[4 .. 4+n_tiles] = prefix,
//   per tile an int4 {first row entry, end row entry, key start, key end} at
//   the 16-byte aligned offset tile_meta_offset(n_tiles),
//   per attention workgroup w (indexed by w, not by range index, so that a
//   workgroup fetches it together with the plan's head) two int4 at
//   range_seg_offset(n_tiles): {t, prefix[t], prefix[t + 1], 0} and the
//   metadata of t, where t is the tile holding the first unit of w's range
//   (t = n_tiles for a range past the last unit).
__device__ __forceinline__ void build_plan(
    int32_t n_tiles, int32_t tile_slots, int32_t Hkv, int64_t t_total,
    const int32_t* __restrict__ cu_seqlens, int32_t n_seqs, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ cu_rows, int32_t rows_per_layer, int32_t rows_per_tile,
    int32_t n_wg, int32_t n_first, int32_t n_wg_max, int32_t* __restrict__ plan) {
  __shared__ int warp_sums[16];
  __shared__ int carry_sh;
  __shared__ int prefix_sh[2 * kAttnMaxWorkgroups + 1];  // balanced ranges: n_tiles < 2 n_wg
  int32_t* prefix = plan + 4;
  int4* meta = reinterpret_cast<int4*>(plan + tile_meta_offset(n_tiles));
  int4* seg = reinterpret_cast<int4*>(plan + range_seg_offset(n_tiles));
  const int nt = blockDim.x;  // a multiple of 64, at most 1024
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (tid == 0) carry_sh = 0;
  __syncthreads();
  for (int base = 0; base < n_tiles; base += nt) {
    const int t = base + tid;
    int nb = 0;
    if (t < n_tiles) {
      const int lg = t / tile_slots, slot = t % tile_slots;
      const int64_t set = rows_per_layer ? lg / Hkv : 0;
      const int32_t* cur = cu_rows + set * (n_seqs + 1);
      Tile tile;
      int4 mt = make_int4(0, 0, 0, 0);
      if (find_tile(cur, n_seqs, rows_per_tile, slot, &tile)) {
        const int64_t kstart = cu_seqlens[tile.b];
        const int64_t kend = min((int64_t)rows[set * t_total + tile.r_end - 1] + 1, t_total);
        if (kend > kstart) nb = (int)((kend - kstart + kKB - 1) / kKB) + kSegCost;
        mt = make_int4(tile.r_begin, tile.r_end, (int)kstart, (int)kend);
      }
      meta[t] = mt;
    }
    // inclusive scan over the block: within each wave, then over waves
    int x = nb;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    if (lane == 63) warp_sums[wv] = x;
    __syncthreads();
    int before = carry_sh;
    for (int i = 0; i < wv; ++i) before += warp_sums[i];
    if (t < n_tiles) {
      prefix[t] = before + x - nb;
      prefix_sh[t] = before + x - nb;
    }
    __syncthreads();
    if (tid == nt - 1) carry_sh = before + x;
    __syncthreads();
  }
  const int total = carry_sh;
  // n_first c1 + (n_wg - n_first) c2 >= total with c1 / c2 >= kFirstShareNum / kFirstShareDen
  const int64_t weight = (int64_t)kFirstShareNum * n_first + (int64_t)kFirstShareDen * (n_wg - n_first);
  const int c2 = (int)max((int64_t)1, ((int64_t)kFirstShareDen * total + weight - 1) / weight);
  const int c1 = (int)(((int64_t)kFirstShareNum * c2 + kFirstShareDen - 1) / kFirstShareDen);
  if (tid == 0) {
    plan[0] = c1;
    plan[1] = c2;
    plan[2] = n_first;
    plan[3] = total;
    prefix[n_tiles] = total;
    prefix_sh[n_tiles] = total;
  }
  __syncthreads();
  // first-segment descriptors: every non-empty tile [p0, p1) writes those of
  // the ranges whose first unit lies in it (one pass, no search); ranges that
  // start past the last unit get tile n_tiles (they have no work).  meta[t]
  // was stored by this same thread in the first pass.
  for (int t = tid; t < n_tiles; t += nt) {
    const int p0 = prefix_sh[t], p1 = prefix_sh[t + 1];
    if (p1 <= p0) continue;
    const int4 mt = meta[t];
    for (int v = unit_owner(p0, c1, c2, n_first); v < n_wg; ++v) {
      const int u = unit_start(v, c1, c2, n_first);
      if (u >= p1) break;
      if (u >= p0) {
        const int w = wg_of_range(v, n_first, n_wg);
        seg[2 * w] = make_int4(t, p0, p1, 0);
        seg[2 * w + 1] = mt;
      }
    }
  }
  for (int v = tid; v < n_wg; v += nt)
    if (unit_start(v, c1, c2, n_first) >= total) {
      const int w = wg_of_range(v, n_first, n_wg);
      seg[2 * w] = make_int4(n_tiles, total, total, 0);
      seg[2 * w + 1] = make_int4(0, 0, 0, 0);
    }
}

constexpr int kPatchRows = 4;  // row-list entries per patch wave

// Patch: cache[l][h][t] <- fresh[l][h][t] for every selected row t (both
// tensors, every kv head; one wave per kPatchRows rows).  With plan != NULL the first
// n_plans workgroups build work decompositions instead: one plan over all L
// layers (n_plans = 1), or one plan per layer (n_plans = L, plan p at
// plan + p * plan_stride, over layer p's row set alone).  n_tiles counts the
// tiles of one plan.
__global__ void __launch_bounds__(256)
patch_kernel(int32_t L, int32_t Hkv, int32_t D, int64_t t_total, int32_t n_seqs,
             const int32_t* __restrict__ rows, const int32_t* __restrict__ cu_rows,
             int32_t rows_per_layer, int32_t max_rows, const uint16_t* __restrict__ kf,
             const uint16_t* __restrict__ vf, uint16_t* __restrict__ kc,
             uint16_t* __restrict__ vc,
             const int32_t* __restrict__ cu_seqlens, int32_t n_tiles, int32_t tile_slots,
             int32_t rows_per_tile, int32_t n_wg, int32_t n_first, int32_t n_wg_max,
             int32_t* __restrict__ plan, int32_t n_plans, int64_t plan_stride) {
  // the plan builders come first: dispatched first, they start their chains of
  // dependent loads while the copying workgroups are still being dispatched
  if (plan != nullptr && (int)blockIdx.x < n_plans) {
    const int p = blockIdx.x;
    if (n_plans == 1) {
      build_plan(n_tiles, tile_slots, Hkv, t_total, cu_seqlens, n_seqs, rows, cu_rows,
                 rows_per_layer, rows_per_tile, n_wg, n_first, n_wg_max, plan);
    } else {
      const int64_t set = rows_per_layer ? p : 0;
      build_plan(n_tiles, tile_slots, Hkv, t_total, cu_seqlens, n_seqs, rows + set * t_total,
                 cu_rows + set * (n_seqs + 1), 0, rows_per_tile, n_wg, n_first, n_wg_max,
                 plan + p * plan_stride);
    }
    return;
  }
  const int64_t copy_block = (int64_t)blockIdx.x - (plan != nullptr ? n_plans : 0);
  const int64_t wave = (copy_block * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  // each wave copies kPatchRows consecutive entries of the row list, with all
  // their loads in flight together
  const int64_t groups = (max_rows + kPatchRows - 1) / kPatchRows;
  const int64_t l = wave / groups;
  const int64_t i0 = (wave % groups) * kPatchRows;
  if (l >= L) return;
  const int64_t set = rows_per_layer ? l : 0;
  const int32_t n = cu_rows[set * (n_seqs + 1) + n_seqs];
  if (i0 >= n) return;
  int64_t t[kPatchRows];
  bool ok[kPatchRows];
#pragma unroll
  for (int r = 0; r < kPatchRows; ++r) {
    t[r] = rows[set * t_total + min(i0 + r, (int64_t)n - 1)];
    ok[r] = i0 + r < n && t[r] >= 0 && t[r] < t_total;
  }
  // an entry that is not copied reads a valid row (loads stay unconditional)
  int64_t t_any = -1;
#pragma unroll
  for (int r = kPatchRows - 1; r >= 0; --r)
    if (ok[r]) t_any = t[r];
  if (t_any < 0) return;
  const int chunks = D / 8;  // 16-byte pieces per head row
  for (int e = lane; e < 2 * Hkv * chunks; e += 64) {
    const int tensor = e / (Hkv * chunks);
    const int h = (e / chunks) % Hkv;
    const int c = e % chunks;
    const int64_t base = (l * Hkv + h) * t_total;
    const uint16_t* src = tensor == 0 ? kf : vf;
    uint4 a[kPatchRows];
#pragma unroll
    for (int r = 0; r < kPatchRows; ++r)
      a[r] = *reinterpret_cast<const uint4*>(src + (base + (ok[r] ? t[r] : t_any)) * D + c * 8);
#pragma unroll
    for (int r = 0; r < kPatchRows; ++r) {
      if (!ok[r]) continue;
      const int64_t off = (base + t[r]) * D + c * 8;
      *reinterpret_cast<uint4*>((tensor == 0 ? kc : vc) + off) = a[r];
    }
  }
}

// Two launch shapes:
//  * whole tiles (many tiles): workgroup t finishes tile t;
//  * balanced ranges (few tiles): workgroup w walks the tiles that overlap its
//    units [unit_start(w), unit_start(w + 1)); a tile whose blocks it covers
//    whole is finished here, the cut ones (at most its first and its last)
//    leave partial records 2w and 2w + 1.
template <int D>
__global__ void __launch_bounds__(kThreads, KVB_ATTN_WG_PER_CU)
attn_kernel(int32_t balanced, int32_t n_tiles, int32_t Hq, int32_t Hkv, int32_t log2g,
            int64_t t_total, const int32_t* __restrict__ cu_seqlens, int32_t n_seqs,
            const int32_t* __restrict__ rows, const int32_t* __restrict__ cu_rows,
            int32_t rows_per_layer, int32_t rows_per_tile, int32_t tile_slots,
            const int32_t* __restrict__ plan, int32_t n_wg_max, int32_t n_rec,
            const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
            const uint16_t* __restrict__ v16, float c_log2, int32_t out_f32,
            void* __restrict__ out, float* __restrict__ parts) {
  using C = AttnCfg<D>;
  __shared__ __attribute__((aligned(1024))) char k_ring[kStages * C::BLK];
  __shared__ __attribute__((aligned(1024))) char v_ring[kStages * C::BLK];
  if (!balanced) {
    // tiles in reverse order: the last row tiles of a prompt, which attend to
    // the most keys, are dispatched first and the launch ends on short ones
    const int t = n_tiles - 1 - (int)blockIdx.x;
    const int n_lg = n_tiles / tile_slots;
    const int lg = t % n_lg;
    const int64_t set = rows_per_layer ? lg / Hkv : 0;
    Tile tile;
    if (!find_tile(cu_rows + set * (n_seqs + 1), n_seqs, rows_per_tile, t / n_lg, &tile))
      return;
    SegTile tl;
    tl.lg = lg;
    tl.r_begin = tile.r_begin;
    tl.r_end = tile.r_end;
    tl.kstart = cu_seqlens[tile.b];
    tl.kend = min(rows[set * t_total + tile.r_end - 1] + 1, (int)t_total);
    const int whole = (int)((t_total + kKB - 1) / kKB) + 1;
    attend_segment<D>(tl, 0, whole, -1, n_rec, k_ring, v_ring, Hq, Hkv, log2g, t_total, rows,
                      rows_per_layer, q, kc, v16, c_log2, out_f32, out, parts);
    return;
  }
  // the plan's head and this workgroup's first-segment descriptor are
  // independent loads: the first tile's blocks can be requested right after
  const int c1 = plan[0], c2 = plan[1], n_first = plan[2], total = plan[3];
  const int4* sd = reinterpret_cast<const int4*>(plan + range_seg_offset(n_tiles)) + 2 * blockIdx.x;
  const int4 s0 = sd[0];
  int4 mt = sd[1];
  const int v = range_of(blockIdx.x, n_first, (int)gridDim.x);  // range index
  const int32_t* prefix = plan + 4;
  const int4* meta = reinterpret_cast<const int4*>(plan + tile_meta_offset(n_tiles));
  int u = unit_start(v, c1, c2, n_first);
  const int u_end = min(unit_start(v + 1, c1, c2, n_first), total);
  int t = s0.x, p0 = s0.y, p1 = s0.z;
  for (int seg = 0; u < u_end && t < n_tiles;) {
    if (p1 > u) {  // else an empty tile
      const int e = min(u_end, p1);
      // units [p0, p0 + kSegCost) of a tile stand for its fixed cost and hold no block
      const int b_lo = max(u - p0 - kSegCost, 0), b_hi = max(e - p0 - kSegCost, 0);
      if (b_hi > b_lo) {
        const int rec = (u <= p0 + kSegCost && p1 <= u_end) ? -1 : 2 * v + (seg == 0 ? 0 : 1);
        SegTile tl;
        tl.lg = t / tile_slots;
        tl.r_begin = mt.x;
        tl.r_end = mt.y;
        tl.kstart = mt.z;
        tl.kend = mt.w;
        attend_segment<D>(tl, b_lo, b_hi, rec, n_rec, k_ring, v_ring, Hq, Hkv, log2g, t_total,
                          rows, rows_per_layer, q, kc, v16, c_log2, out_f32, out, parts);
        ++seg;
      }
      u = e;
    }
    // later tiles of the range: their prefix end and metadata from the plan
    if (++t < n_tiles && u < u_end) {
      p0 = p1;
      p1 = prefix[t + 1];
      mt = meta[t];
    }
  }
}

// Merge the partial records of every tile that was cut between workgroups, in
// key order.  One thread per (query vector, 8 channels).  Every load a thread
// needs depends only on the plan: the records are requested together with the
// query's row.
template <int D>
__global__ void __launch_bounds__(256)
combine_kernel(int32_t n_tiles, int32_t n_wg_max, int32_t Hq, int32_t Hkv, int32_t log2g,
               int64_t t_total, const int32_t* __restrict__ rows, int32_t rows_per_layer,
               int32_t tile_slots, const int32_t* __restrict__ plan, int32_t n_rec,
               int32_t out_f32, void* __restrict__ out, const float* __restrict__ parts) {
  const int t = blockIdx.x;
  const int c1 = plan[0], c2 = plan[1], n_first = plan[2];
  const int p0 = plan[4 + t], p1 = plan[5 + t];
  const int4 mt = reinterpret_cast<const int4*>(plan + tile_meta_offset(n_tiles))[t];
  if (p1 <= p0) return;
  // the tile's blocks are units [p0 + kSegCost, p1), held by ranges w_a .. w_b
  const int w_a = unit_owner(p0 + kSegCost, c1, c2, n_first),
            w_b = unit_owner(p1 - 1, c1, c2, n_first);
  if (w_a == w_b) return;  // finished by one workgroup
  constexpr int Q8 = D / 8;  // 8-channel pieces per query vector
  const int e = blockIdx.y * blockDim.x + threadIdx.x;
  if (e >= kQT * Q8) return;
  const int qi = e / Q8, c8 = (e % Q8) * 8;
  const int lg = t / tile_slots;
  const int l = lg / Hkv, g = lg % Hkv;
  const int wave = qi / kQW, nq = qi % kQW;
  const int row_idx = mt.x + wave * (kQW >> log2g) + (nq >> log2g);
  if (row_idx >= mt.y) return;
  const int64_t set = rows_per_layer ? l : 0;
  const int tq = rows[set * t_total + row_idx];
  // the tile is the first segment of every range after w_a, and of w_a only
  // if w_a's range starts inside the tile (a range that starts before it ends
  // with blocks of an earlier tile)
  const int rec_a = 2 * w_a + (unit_start(w_a, c1, c2, n_first) < p0 ? 1 : 0);
  const int n_parts = w_b - w_a + 1;
  const uint16_t* o16 = reinterpret_cast<const uint16_t*>(parts);
  const float* ml = reinterpret_cast<const float*>(reinterpret_cast<const char*>(parts) +
                                                   rec_ml_offset<D>(n_rec));
  // records are taken 8 at a time, all loads of a group issued before any is
  // used (indices past the last record repeat it with weight zero); groups are
  // merged with the usual running-maximum rescale
  constexpr int U = 8;
  float M = -INFINITY, Lsum = 0.0f;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < n_parts; s0 += U) {
    float m[U], ls[U];
    u32x4 o[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = min(s0 + u, n_parts - 1);
      const int rec = (i == 0) ? rec_a : 2 * (w_a + i);
      const int64_t it = (int64_t)rec * kQT + qi;
      const float2 v = *reinterpret_cast<const float2*>(ml + it * 2);
      m[u] = (s0 + u < n_parts) ? v.x : -INFINITY;
      ls[u] = v.y;
      o[u] = *reinterpret_cast<const u32x4*>(o16 + it * D + c8);
    }
    float Mn = M;
#pragma unroll
    for (int u = 0; u < U; ++u) Mn = fmaxf(Mn, m[u]);
    if (Mn == -INFINITY) continue;
    const float a = (M == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(M - Mn);
    Lsum *= a;
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] *= a;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      // weight of a record = its sum rescaled to the common maximum (its O is
      // already divided by its own sum)
      const float wgt = (m[u] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m[u] - Mn) * ls[u];
      Lsum += wgt;
      const f16x8 h = __builtin_bit_cast(f16x8, o[u]);
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[c] += wgt * (float)h[c];
    }
    M = Mn;
  }
  if (tq < mt.z || tq >= mt.w) return;  // not a query of this prompt
  const int head = g * (1 << log2g) + (nq & ((1 << log2g) - 1));
  const float inv = Lsum > 0.0f ? 1.0f / Lsum : 0.0f;
  const int64_t ob = (((int64_t)l * t_total + tq) * Hq + head) * D + c8;
  if (out_f32) {
    float* op = reinterpret_cast<float*>(out) + ob;
    *reinterpret_cast<float4*>(op) = make_float4(acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
    *reinterpret_cast<float4*>(op + 4) = make_float4(acc[4] * inv, acc[5] * inv, acc[6] * inv, acc[7] * inv);
  } else {
    *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(out) + ob) =
        make_uint4(pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv),
                   pack_bf16x2(acc[4] * inv, acc[5] * inv), pack_bf16x2(acc[6] * inv, acc[7] * inv));
  }
}

// Workgroups of the attention kernel the current device holds at once.
int resident_workgroups() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
    cached[dev] = cus * KVB_ATTN_WG_PER_CU;
  }
  return cached[dev];
}

int ilog2(int x) {
  int r = 0;
  while ((1 << r) < x) ++r;
  return r;
}

}  // namespace

bool attn_plan(int n_layers, int n_q_heads, int n_kv_heads, int head_dim, int64_t t_total,
               int n_seqs, int max_seq_len, int max_rows, bool v16_given, AttnPlan* plan) {
  const int G = n_q_heads / n_kv_heads;
  const int rows_per_tile = kQT / G;
  const int64_t full_tiles = ((int64_t)max_rows + rows_per_tile - 1) / rows_per_tile;
  const int64_t tile_slots = full_tiles + n_seqs;
  const int64_t n_tiles = (int64_t)n_layers * n_kv_heads * tile_slots;
  // work units must fit int32: at most n_tiles * (ceil(max_seq_len / 32) + kSegCost)
  if (n_tiles * ((max_seq_len + kKB - 1) / kKB + kSegCost) > INT32_MAX / 2) return false;
  plan->rows_per_tile = rows_per_tile;
  plan->tile_slots = (int)tile_slots;
  plan->n_tiles = (int)n_tiles;
  plan->n_wg_max = kAttnMaxWorkgroups;
  plan->n_rec = 2 * kAttnMaxWorkgroups;
  plan->v16_in_ws = !v16_given;
  const size_t v16 =
      v16_given ? 0 : (size_t)n_layers * n_kv_heads * (size_t)t_total * head_dim * 2;
  const size_t n_plan_ints = (size_t)plan_ints(n_tiles, plan->n_wg_max);
  const size_t parts = (size_t)(head_dim == 128 ? rec_ml_offset<128>(plan->n_rec)
                                                 : rec_ml_offset<64>(plan->n_rec)) +
                       (size_t)plan->n_rec * kQT * 2 * sizeof(float);
  auto up = [](size_t x) { return ((x + 255) / 256) * 256; };
  plan->v16_offset = 0;
  plan->plan_offset = up(v16);
  plan->parts_offset = up(plan->plan_offset + n_plan_ints * sizeof(int32_t));
  plan->workspace = plan->parts_offset + parts;
  plan->max_seq_len = max_seq_len;
  return true;
}

namespace {

// Attention workgroups and first-slot workgroups of a launch on this device.
void launch_shape(const AttnPlan& plan, int* n_wg, int* n_first) {
  int w = resident_workgroups();
  if (w > plan.n_wg_max) w = plan.n_wg_max;
  // first-slot workgroups (see kFirstShareNum) exist only with two per CU
  *n_first = (KVB_ATTN_WG_PER_CU == 2 && w == resident_workgroups()) ? w / 2 : 0;
  *n_wg = w;
}

// One tile per workgroup (no partial records, no combine launch) when there
// are enough tiles to keep every resident workgroup busy twice over, or when
// no prompt is longer than kWholeTileMaxSeq rows: no tile then has more than
// 16 key blocks, and a launch of short whole tiles ends sooner than balanced
// ranges followed by the merge of their cut tiles.  Otherwise balanced ranges.
constexpr int kWholeTileMaxSeq = 512;
bool is_balanced(const AttnPlan& plan, int n_wg) {
  return plan.n_tiles < 2 * n_wg && plan.max_seq_len > kWholeTileMaxSeq;
}

// Patch launch: copies the selected rows of n_layers layers; with plans != NULL
// its first n_plans workgroups build the plans (see patch_kernel).
void launch_patch(int n_layers, int n_kv_heads, int head_dim, int64_t t_total,
                  const int32_t* cu_seqlens, int n_seqs, const int32_t* rows,
                  const int32_t* cu_rows, int rows_per_layer, int max_rows,
                  const uint16_t* k_fresh, const uint16_t* v_fresh, uint16_t* k_cache,
                  uint16_t* v_cache, const AttnPlan& plan, int n_wg, int n_first,
                  int32_t* plans, int n_plans, int64_t plan_stride, hipStream_t s) {
  const int64_t waves = (int64_t)n_layers * ((max_rows + kPatchRows - 1) / kPatchRows);
  const int64_t blocks = (waves * 64 + 255) / 256 + (plans ? n_plans : 0);
  if (blocks > 0)
    hipLaunchKernelGGL(patch_kernel, dim3((unsigned)blocks), dim3(256), 0, s, n_layers, n_kv_heads,
                       head_dim, t_total, n_seqs, rows, cu_rows, rows_per_layer, max_rows, k_fresh,
                       v_fresh, k_cache, v_cache, cu_seqlens, plan.n_tiles, plan.tile_slots,
                       plan.rows_per_tile, n_wg, n_first, plan.n_wg_max, plans, n_plans,
                       plan_stride);
}

// fp16 copy of the V cache of n_layers layers (status as for v16_kernel).
void launch_v16(int n_layers, int n_kv_heads, int head_dim, int64_t t_total, const uint16_t* v,
                uint16_t* v16, uint32_t* status, hipStream_t s) {
  const int64_t n8 = (int64_t)n_layers * n_kv_heads * t_total * head_dim / 8;
  int64_t blocks = (n8 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks > 0)
    hipLaunchKernelGGL(v16_kernel, dim3((unsigned)blocks), dim3(256), 0, s, n8, v, v16, status);
}

// Attention (and, for balanced ranges, the merge of cut tiles) over an already
// patched cache; wplan is the plan of exactly these layers.
void launch_attend(const AttnPlan& plan, int n_wg, bool balanced, int n_q_heads, int n_kv_heads,
                   int head_dim, int64_t t_total, const int32_t* cu_seqlens, int n_seqs,
                   const int32_t* rows, const int32_t* cu_rows, int rows_per_layer,
                   const uint16_t* q, const uint16_t* k_cache, const uint16_t* v16,
                   float softmax_scale, kvb_dtype out_dtype, void* out, const int32_t* wplan,
                   float* parts, hipStream_t s) {
  const int log2g = ilog2(n_q_heads / n_kv_heads);
  const float c_log2 = softmax_scale * 1.4426950408889634f;
  const int out_f32 = out_dtype == KVB_F32;
  const dim3 grid(balanced ? n_wg : plan.n_tiles);
#define KVB_ATTN(D)                                                                              \
  hipLaunchKernelGGL(attn_kernel<D>, grid, dim3(kThreads), 0, s, (int)balanced, plan.n_tiles,     \
                     n_q_heads, n_kv_heads, log2g, t_total, cu_seqlens, n_seqs, rows, cu_rows,    \
                     rows_per_layer, plan.rows_per_tile, plan.tile_slots, wplan, plan.n_wg_max,   \
                     plan.n_rec, q, k_cache, v16, c_log2, out_f32, out, parts)
#define KVB_COMBINE(D)                                                                           \
  hipLaunchKernelGGL(combine_kernel<D>, dim3(plan.n_tiles, kQT * (D / 8) / 256), dim3(256), 0, s, \
                     plan.n_tiles, plan.n_wg_max, n_q_heads, n_kv_heads, log2g, t_total, rows,    \
                     rows_per_layer, plan.tile_slots, wplan, plan.n_rec, out_f32, out, parts)
  if (head_dim == 128) {
    KVB_ATTN(128);
    if (balanced) KVB_COMBINE(128);
  } else {
    KVB_ATTN(64);
    if (balanced) KVB_COMBINE(64);
  }
#undef KVB_ATTN
#undef KVB_COMBINE
}

}  // namespace

hipError_t launch_sparse_attn(const AttnPlan& plan, int n_layers, int n_q_heads, int n_kv_heads,
                              int head_dim, int64_t t_total, const int32_t* cu_seqlens,
                              int n_seqs, const int32_t* rows, const int32_t* cu_rows,
                              int rows_per_layer, int max_rows, const uint16_t* q,
                              const uint16_t* k_fresh, const uint16_t* v_fresh,
                              uint16_t* k_cache, uint16_t* v_cache, uint16_t* v_cache_f16,
                              uint32_t* v_status, float softmax_scale, kvb_dtype out_dtype,
                              void* out, void* workspace, hipStream_t s) {
  char* wsb = reinterpret_cast<char*>(workspace);
  uint16_t* v16 = plan.v16_in_ws ? reinterpret_cast<uint16_t*>(wsb + plan.v16_offset) : v_cache_f16;
  int32_t* wplan = reinterpret_cast<int32_t*>(wsb + plan.plan_offset);
  float* parts = reinterpret_cast<float*>(wsb + plan.parts_offset);
  int n_wg = 0, n_first = 0;
  launch_shape(plan, &n_wg, &n_first);
  const bool balanced = is_balanced(plan, n_wg);
  launch_patch(n_layers, n_kv_heads, head_dim, t_total, cu_seqlens, n_seqs, rows, cu_rows,
               rows_per_layer, max_rows, k_fresh, v_fresh, k_cache, v_cache, plan, n_wg, n_first,
               balanced ? wplan : nullptr, 1, 0, s);
  launch_v16(n_layers, n_kv_heads, head_dim, t_total, v_cache, v16, v_status, s);
  launch_attend(plan, n_wg, balanced, n_q_heads, n_kv_heads, head_dim, t_total, cu_seqlens, n_seqs,
                rows, cu_rows, rows_per_layer, q, k_cache, v16, softmax_scale, out_dtype, out,
                wplan, parts, s);
  return hipGetLastError();
}

hipError_t launch_fp16_copy(int n_layers, int n_kv_heads, int head_dim, int64_t t_total,
                            const uint16_t* v, uint16_t* v16, uint32_t* status, hipStream_t s) {
  launch_v16(n_layers, n_kv_heads, head_dim, t_total, v, v16, status, s);
  return hipGetLastError();
}

size_t layer_plan_stride(const AttnPlan& layer_plan) {
  const size_t ints = (size_t)plan_ints(layer_plan.n_tiles, layer_plan.n_wg_max);
  return ((ints * sizeof(int32_t) + 255) / 256) * 256;
}

hipError_t launch_patch_layers(const AttnPlan& layer_plan, int n_layers, int n_kv_heads,
                               int head_dim, int64_t t_total, const int32_t* cu_seqlens,
                               int n_seqs, const int32_t* rows, const int32_t* cu_rows,
                               int rows_per_layer, int max_rows, const uint16_t* k_fresh,
                               const uint16_t* v_fresh, uint16_t* k_cache, uint16_t* v_cache,
                               uint16_t* v_cache_f16, uint32_t* v_status, void* plans,
                               hipStream_t s) {
  int n_wg = 0, n_first = 0;
  launch_shape(layer_plan, &n_wg, &n_first);
  // plans are needed (and built) only for balanced ranges
  int32_t* p = (plans && is_balanced(layer_plan, n_wg)) ? reinterpret_cast<int32_t*>(plans) : nullptr;
  if (max_rows > 0 || p != nullptr)
    launch_patch(n_layers, n_kv_heads, head_dim, t_total, cu_seqlens, n_seqs, rows, cu_rows,
                 rows_per_layer, max_rows, k_fresh, v_fresh, k_cache, v_cache, layer_plan, n_wg,
                 n_first, p, n_layers,
                 (int64_t)(layer_plan_stride(layer_plan) / sizeof(int32_t)), s);
  if (v_cache_f16 != nullptr)
    launch_v16(n_layers, n_kv_heads, head_dim, t_total, v_cache, v_cache_f16, v_status, s);
  return hipGetLastError();
}

hipError_t launch_sparse_attn_layer(const AttnPlan& layer_plan, int layer, int n_q_heads,
                                    int n_kv_heads, int head_dim, int64_t t_total,
                                    const int32_t* cu_seqlens, int n_seqs, const int32_t* rows,
                                    const int32_t* cu_rows, int rows_per_layer, const uint16_t* q,
                                    const uint16_t* k_cache, const uint16_t* v_cache_f16,
                                    const void* plans, float softmax_scale, kvb_dtype out_dtype,
                                    void* out, void* workspace, hipStream_t s) {
  int n_wg = 0, n_first = 0;
  launch_shape(layer_plan, &n_wg, &n_first);
  const bool balanced = is_balanced(layer_plan, n_wg);
  const int64_t set = rows_per_layer ? layer : 0;
  const int64_t kv = (int64_t)layer * n_kv_heads * t_total * head_dim;
  const int64_t qo = (int64_t)layer * t_total * n_q_heads * head_dim;
  const int32_t* wplan = reinterpret_cast<const int32_t*>(
      reinterpret_cast<const char*>(plans) + (size_t)layer * layer_plan_stride(layer_plan));
  float* parts = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) + layer_plan.parts_offset);
  void* out_l = out_dtype == KVB_F32 ? (void*)(reinterpret_cast<float*>(out) + qo)
                                     : (void*)(reinterpret_cast<uint16_t*>(out) + qo);
  launch_attend(layer_plan, n_wg, balanced, n_q_heads, n_kv_heads, head_dim, t_total, cu_seqlens,
                n_seqs, rows + set * t_total, cu_rows + set * (n_seqs + 1), 0, q + qo,
                k_cache + kv, v_cache_f16 + kv, softmax_scale, out_dtype, out_l,
                balanced ? wplan : nullptr, parts, s);
  return hipGetLastError();
}

}  // namespace kvb
