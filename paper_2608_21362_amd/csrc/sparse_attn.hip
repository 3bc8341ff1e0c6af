// Patch and sparse-query causal GQA attention (Alg. 2 step 4; Eq. 2).
//
// Per layer the call runs four kernels on one stream:
//
//   patch_kernel     cache[l][h][t] <- fresh[l][h][t] for every selected row t
//                    (both tensors, every kv head; one wave per row)
//   v16_kernel       the patched V of the layer converted to fp16 in the
//                    workspace (exact for |v| <= 65504: a bf16 significand fits
//                    an fp16 one), so the P.V product can take fp16 operands
//                    straight from LDS
//   attn_kernel      the attention itself (below)
//   combine_kernel   merges KV-split partials in split order (only when a
//                    tile's key range was split)
//
// attn_kernel: one workgroup = one (layer, kv head g, tile of selected rows,
// KV split).  The tile packs rows x the G = Hq/Hkv query heads that share kv
// head g into the MFMA N dimension: each of the 4 waves owns 32 query vectors
// (32/G rows x G heads).  Keys stream in blocks of 64 through a two-stage LDS
// ring filled by asynchronous global->LDS loads (no VGPR staging), XOR-swizzled
// on 16-byte chunks so the operand reads below are free of bank conflicts:
//
//   S^T (64 keys x 32 queries) = K Q^T     bf16 MFMA 32x32x16: K rows from LDS
//                                           (A operand), Q^T kept in VGPRs
//   online softmax over keys               fp32, base-2 exponent.  Each lane
//                                           holds 32 scores of one query, the
//                                           other 32 sit in lane ^ 32.  The
//                                           running maximum is refreshed only
//                                           when a block raises it by more
//                                           than 8 (log2 units), so partial
//                                           probabilities stay below 2^8
//   O^T (d x 32 queries) += V^T P^T        fp16 MFMA 32x32x16: V^T read from
//                                           the row-major fp16 V block with the
//                                           LDS transpose read, P^T converted
//                                           from the S^T accumulators
//
// The accumulator layout of a 32x32 MFMA gives lane half h the keys
// {4h..4h+3, 8+4h..8+4h+3} of every 16-key step; the transpose reads fetch V
// for exactly those keys, so no permutation is needed anywhere.  The
// contraction index of each product is laid out identically on its two
// operands, so its order inside the MFMA does not matter.
#include <math.h>

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
constexpr int kStages = 4;              // LDS ring depth (blocks in flight: 2 ahead)
constexpr float kLazy = 8.0f;           // max growth (log2 units) tolerated before a rescale

#define LDS_PTR(T, p) ((__attribute__((address_space(3))) T*)(p))

// wait until at most n vector-memory operations of this wave are outstanding
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Keep the compiler from moving memory accesses across this point (the raw
// s_barrier builtin is not a memory barrier for it); emits no instruction.
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

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

// ------------------------------------------------------------ V to fp16 ----
__device__ __forceinline__ uint32_t bf16pair_to_f16pair(uint32_t w) {
  f32x2 f = {bf16_lo(w), bf16_hi(w)};
  f16x2 h = __builtin_convertvector(f, f16x2);
  return __builtin_bit_cast(uint32_t, h);
}

__global__ void __launch_bounds__(256)
v16_kernel(int64_t n8, const uint16_t* __restrict__ v, uint16_t* __restrict__ v16) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n8;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint4 a = reinterpret_cast<const uint4*>(v)[i];
    reinterpret_cast<uint4*>(v16)[i] =
        make_uint4(bf16pair_to_f16pair(a.x), bf16pair_to_f16pair(a.y),
                   bf16pair_to_f16pair(a.z), bf16pair_to_f16pair(a.w));
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

// Issue the asynchronous loads of one 64-key block of K (bf16) and V (fp16)
// into one LDS stage.  The buffer resources cover exactly the cache rows of
// this (layer, kv head); rows past the end read as zero (their scores are
// masked).
template <int D>
__device__ __forceinline__ void issue_block(i32x4 krs, i32x4 vrs, int kb, const LoadOffsets<D>& lo,
                                            char* k_st, char* v_st, int wave) {
  using C = AttnCfg<D>;
  // the block offset goes into the lane offset: the buffer range check covers
  // the lane offset, not the scalar one
  const int boff = kb * C::ROWB;
  const uint32_t kbase = __builtin_amdgcn_readfirstlane(lds_addr(k_st) + wave * C::LOADS * 1024);
  const uint32_t vbase = __builtin_amdgcn_readfirstlane(lds_addr(v_st) + wave * C::LOADS * 1024);
#pragma unroll
  for (int i = 0; i < C::LOADS; ++i) {
    lds_dma16(krs, kbase + i * 1024, boff + lo.k[i], 0);
    lds_dma16(vrs, vbase + i * 1024, boff + lo.v[i], 0);
  }
}

template <int D>
struct AttnState {
  f32x16 o[AttnCfg<D>::ND];
  float m_raw;   // running maximum of raw scores (stale by at most kLazy / scale)
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
  bmax = max_halves(bmax);
  const float m_new = fmaxf(st.m_raw, bmax);
  const bool grow = (m_new - st.m_raw) * c_log2 > kLazy || st.m_raw == -INFINITY;
  if (__builtin_expect(__builtin_amdgcn_ballot_w64(grow) != 0, 0)) {
    const float alpha = (st.m_raw == -INFINITY || m_new == -INFINITY)
                            ? (m_new == -INFINITY ? 1.0f : 0.0f)
                            : __builtin_amdgcn_exp2f((st.m_raw - m_new) * c_log2);
    st.l_part *= alpha;
#pragma unroll
    for (int dt = 0; dt < C::ND; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) st.o[dt][r] *= alpha;
    st.m_raw = m_new;
  }
  const float mc = st.m_raw == -INFINITY ? 0.0f : st.m_raw * c_log2;
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

// One work item: (layer, kv head, tile slot, KV split).  Returns without work
// when the slot holds no tile or the tile has fewer splits.
template <int D>
__device__ __forceinline__ void attend_item(
    int lg, int slot, int split, int n_lg, char* k_ring, char* v_ring,
    int32_t Hq, int32_t Hkv, int32_t log2g, int64_t t_total, const int32_t* __restrict__ cu_seqlens,
    int32_t n_seqs, const int32_t* __restrict__ rows, const int32_t* __restrict__ cu_rows,
    int32_t rows_per_layer, int32_t rows_per_tile, int32_t tile_slots, int32_t split_len,
    int32_t n_split_max, const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
    const uint16_t* __restrict__ v16, float c_log2, int32_t out_f32, void* __restrict__ out,
    float* __restrict__ ws) {
  using C = AttnCfg<D>;
  const int G = 1 << log2g;
  const int l = lg / Hkv, g = lg % Hkv;
  const int64_t set = rows_per_layer ? l : 0;
  const int32_t* cur = cu_rows + set * (n_seqs + 1);
  const int32_t* rws = rows + set * t_total;
  Tile tile;
  if (!find_tile(cur, n_seqs, rows_per_tile, slot, &tile)) return;
  const int T = (int)t_total;
  const int kstart = cu_seqlens[tile.b];
  const int kend = min(rws[tile.r_end - 1] + 1, T);
  if (kend <= kstart) return;
  const int n_split = (kend - kstart + split_len - 1) / split_len;
  if (split >= n_split || n_split > n_split_max) return;
  const int k_lo = kstart + split * split_len;
  const int k_hi = min(k_lo + split_len, kend);
  const int t_min = rws[tile.r_begin];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, n = lane & 31;
  const int rows_per_wave = kQW >> log2g;
  const int row_idx = tile.r_begin + wave * rows_per_wave + (n >> log2g);
  const int head = g * G + (n & (G - 1));
  int t_q = row_idx < tile.r_end ? rws[row_idx] : -1;
  const bool qvalid = t_q >= kstart && t_q < kend;  // rows outside the prompt are skipped
  if (!qvalid) t_q = -1;

  const int64_t kv_base = ((int64_t)l * Hkv + g) * t_total * D;
  const i32x4 krs = buffer_rsrc(kc + kv_base, T * C::ROWB);
  const i32x4 vrs = buffer_rsrc(v16 + kv_base, T * C::ROWB);
  const LoadOffsets<D> lo = load_offsets<D>(wave, lane);
  const int nblk = (k_hi - k_lo + kKB - 1) / kKB;
  static_assert(kStages == 4, "stage index arithmetic assumes a 4-deep ring");
  auto kst = [&](int b) { return k_ring + (b & 3) * C::BLK; };  // ring stage of block b
  auto vst = [&](int b) { return v_ring + (b & 3) * C::BLK; };

  issue_block<D>(krs, vrs, k_lo, lo, kst(0), vst(0), wave);

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
  // Q and block 0 land before anything else is issued: the compiler then never
  // waits on the queries -- and so on the in-flight prefetch -- later on.
  wait_vmcnt<0>();
  if (nblk > 1) issue_block<D>(krs, vrs, k_lo + kKB, lo, kst(1), vst(1), wave);
  if (nblk > 2) issue_block<D>(krs, vrs, k_lo + 2 * kKB, lo, kst(2), vst(2), wave);
  __builtin_amdgcn_s_barrier();
  compiler_fence();

  AttnState<D> st;
#pragma unroll
  for (int dt = 0; dt < C::ND; ++dt) st.o[dt] = f32x16{};
  st.m_raw = -INFINITY;
  st.l_part = 0.0f;

  // Software pipeline over blocks: iteration j computes the scores of block
  // j + 1 on the matrix cores while the vector units turn the scores of block j
  // into probabilities, then accumulates P V for block j.  The ring holds
  // blocks j .. j + 3; block j + 3 is requested once every wave has finished
  // block j - 1 (the barrier), whose stage it reuses.
  bf16x8 kr[C::NS];
  read_k<D>(kst(0), lane, kr);
  f32x16 sacc = scores<D>(kr, qop);
  for (int j = 0; j < nblk; ++j) {
    const int kb = k_lo + j * kKB;
    if (j + 2 < nblk)
      wait_vmcnt<2 * C::LOADS>();  // block j + 1 landed, block j + 2 may be in flight
    else
      wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    if (j + 3 < nblk) issue_block<D>(krs, vrs, kb + 3 * kKB, lo, kst(j + 3), vst(j + 3), wave);
    // on the last iteration this reads a stale stage; those scores are never used
    read_k<D>(kst(j + 1), lane, kr);
    f16x8 vr[2][C::ND];
    read_v<D>(vst(j), lane, vr);
    const bool full = (kb + kKB - 1 <= t_min) && (kb + kKB <= k_hi);
    f16x8 pb[2];
    softmax_block<D>(sacc, st, c_log2, full, kb, t_q, k_hi, lane, pb);
    sacc = scores<D>(kr, qop);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int dt = 0; dt < C::ND; ++dt)
        st.o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vr[ks][dt], pb[ks], st.o[dt], 0, 0, 0);
  }

  if (!qvalid) return;
  const float l_run = sum_halves(st.l_part);
  if (n_split == 1) {
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
    // partial (unnormalised O, running max in log2 units, sum) of this split
    const int64_t item = ((int64_t)lg * tile_slots + slot) * n_split_max + split;
    const int qi = wave * kQW + n;
    float* wo = ws + (item * kQT + qi) * D;
#pragma unroll
    for (int dt = 0; dt < C::ND; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *reinterpret_cast<float4*>(wo + dt * 32 + 8 * j + 4 * half) =
            make_float4(st.o[dt][4 * j], st.o[dt][4 * j + 1], st.o[dt][4 * j + 2],
                        st.o[dt][4 * j + 3]);
    if (half == 0) {
      const int64_t n_items = (int64_t)n_lg * tile_slots * n_split_max;
      float* ml = ws + n_items * kQT * D;
      ml[(item * kQT + qi) * 2] = st.m_raw == -INFINITY ? -INFINITY : st.m_raw * c_log2;
      ml[(item * kQT + qi) * 2 + 1] = l_run;
    }
  }
}


// Grid (tile slot, KV split, layer x kv head).  Workgroups whose slot holds no
// tile, or whose tile has fewer splits, exit at once; the hardware dispatcher
// hands their place to the next workgroup, so the grid load-balances itself.
template <int D>
__global__ void __launch_bounds__(kThreads, KVB_ATTN_WG_PER_CU)
attn_kernel(int32_t Hq, int32_t Hkv, int32_t log2g, int64_t t_total,
            const int32_t* __restrict__ cu_seqlens, int32_t n_seqs,
            const int32_t* __restrict__ rows, const int32_t* __restrict__ cu_rows,
            int32_t rows_per_layer, int32_t rows_per_tile, int32_t tile_slots, int32_t split_len,
            int32_t n_split_max, const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
            const uint16_t* __restrict__ v16, float c_log2, int32_t out_f32,
            void* __restrict__ out, float* __restrict__ ws) {
  using C = AttnCfg<D>;
  __shared__ __attribute__((aligned(1024))) char k_ring[kStages * C::BLK];
  __shared__ __attribute__((aligned(1024))) char v_ring[kStages * C::BLK];
  attend_item<D>(blockIdx.z, blockIdx.x, blockIdx.y, gridDim.z, k_ring, v_ring, Hq,
                 Hkv, log2g, t_total, cu_seqlens, n_seqs, rows, cu_rows, rows_per_layer,
                 rows_per_tile, tile_slots, split_len, n_split_max, q, kc, v16, c_log2, out_f32,
                 out, ws);
}

// Merge the split partials of every multi-split tile, in split order.  One
// thread per (query vector, 4 channels); consecutive threads read consecutive
// 16-byte pieces of a partial.
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
  const int64_t n_items = (int64_t)gridDim.y * tile_slots * n_split_max;
  const float* ml = ws + n_items * kQT * D;
  const int64_t item0 = ((int64_t)lg * tile_slots + slot) * n_split_max;
  constexpr int Q4 = D / 4;  // 4-channel pieces per query vector
  for (int e = blockIdx.z * blockDim.x + threadIdx.x; e < kQT * Q4; e += gridDim.z * blockDim.x) {
    const int qi = e / Q4, c4 = (e % Q4) * 4;
    const int wave = qi / kQW, nq = qi % kQW;
    const int row_idx = tile.r_begin + wave * (kQW >> log2g) + (nq >> log2g);
    if (row_idx >= tile.r_end) continue;
    const int64_t t = rws[row_idx];
    if (t < kstart || t >= kend) continue;
    const int head = g * G + (nq & (G - 1));
    // splits are taken 8 at a time with every load of a group issued before
    // any is used; groups are merged with the usual running-maximum rescale
    constexpr int U = 8;
    float M = -INFINITY, Lsum = 0.0f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s0 = 0; s0 < n_split; s0 += U) {
      float m[U], ls[U];
      float4 o[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (s0 + u < n_split) {
          const int64_t it = (item0 + s0 + u) * kQT + qi;
          const float2 v = *reinterpret_cast<const float2*>(ml + it * 2);
          m[u] = v.x;
          ls[u] = v.y;
          o[u] = *reinterpret_cast<const float4*>(ws + it * D + c4);
        } else {
          m[u] = -INFINITY;
          ls[u] = 0.0f;
          o[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
      float Mn = M;
#pragma unroll
      for (int u = 0; u < U; ++u) Mn = fmaxf(Mn, m[u]);
      if (Mn == -INFINITY) continue;
      const float a = (M == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(M - Mn);
      Lsum *= a;
      acc.x *= a;
      acc.y *= a;
      acc.z *= a;
      acc.w *= a;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float w = (m[u] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m[u] - Mn);
        Lsum += w * ls[u];
        acc.x += w * o[u].x;
        acc.y += w * o[u].y;
        acc.z += w * o[u].z;
        acc.w += w * o[u].w;
      }
      M = Mn;
    }
    const float inv = Lsum > 0.0f ? 1.0f / Lsum : 0.0f;
    const int64_t ob = (((int64_t)l * t_total + t) * Hq + head) * D + c4;
    if (out_f32) {
      *reinterpret_cast<float4*>(reinterpret_cast<float*>(out) + ob) =
          make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
    } else {
      *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(out) + ob) =
          make_uint2(pack_bf16x2(acc.x * inv, acc.y * inv), pack_bf16x2(acc.z * inv, acc.w * inv));
    }
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
  const size_t v16 = (size_t)n_layers * n_kv_heads * (size_t)t_total * head_dim * 2;
  plan->v16_offset = 0;
  size_t parts = 0;
  if (plan->n_split_max > 1) {
    const size_t items = (size_t)n_layers * n_kv_heads * plan->tile_slots * plan->n_split_max;
    parts = items * kQT * (head_dim + 2) * sizeof(float);
  }
  const int64_t n_items = (int64_t)n_layers * n_kv_heads * plan->tile_slots * plan->n_split_max;
  if (n_items > INT32_MAX) return false;
  plan->parts_offset = ((v16 + 255) / 256) * 256;
  plan->workspace = plan->parts_offset + parts;
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
  uint16_t* v16 = reinterpret_cast<uint16_t*>(reinterpret_cast<char*>(workspace) + plan.v16_offset);
  float* parts = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) + plan.parts_offset);
  {
    const int64_t n8 = (int64_t)n_layers * n_kv_heads * t_total * head_dim / 8;
    int64_t blocks = (n8 + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(v16_kernel, dim3((unsigned)blocks), dim3(256), 0, s, n8, v_cache, v16);
  }
  const int log2g = ilog2(n_q_heads / n_kv_heads);
  const float c_log2 = softmax_scale * 1.4426950408889634f;
  const int out_f32 = out_dtype == KVB_F32;
  const dim3 grid(plan.tile_slots, plan.n_split_max, n_layers * n_kv_heads);
#define KVB_ATTN(D)                                                                              \
  hipLaunchKernelGGL(attn_kernel<D>, grid, dim3(kThreads), 0, s, n_q_heads, n_kv_heads, log2g,   \
                     t_total, cu_seqlens, n_seqs, rows, cu_rows, rows_per_layer,                 \
                     plan.rows_per_tile, plan.tile_slots, plan.split_len, plan.n_split_max, q,    \
                     k_cache, v16, c_log2, out_f32, out, parts)
#define KVB_COMBINE(D)                                                                           \
  hipLaunchKernelGGL(combine_kernel<D>, dim3(plan.tile_slots, n_layers * n_kv_heads, 4),         \
                     dim3(256), 0, s, n_q_heads, n_kv_heads, log2g, t_total, cu_seqlens, n_seqs,  \
                     rows, cu_rows, rows_per_layer, plan.rows_per_tile, plan.tile_slots,          \
                     plan.split_len, plan.n_split_max, out_f32, out, parts)
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
