/*
 * kvb.h -- C ABI of the stitched-prefill path of KVBoost (arXiv 2608.21362)
 * on one AMD Instinct MI355X (gfx950).
 *
 * The path turns independently cached, KIVI-quantised 128-token KV chunks into
 * a usable prompt cache and runs the repair forward's attention:
 *
 *   kvb_stitch          dequantise cached chunks, re-rotate keys to their new
 *                       position (Sec. 4.3, Sec. 3.2 Eq. 3, Sec. 4.5 Eq. 7)
 *   kvb_stitch_deviation  kvb_stitch plus the deviation of the stitched rows in
 *                       the same pass (Alg. 2 steps 1-2 fused)
 *   kvb_deviation       per-token cosine deviation (Alg. 2 step 2)
 *   kvb_select          top floor(rho n) rows + seam windows + live rows
 *                       (Alg. 2 step 3, Alg. 1, Sec. 4.1 sinks)
 *   kvb_deviation_topk  kvb_deviation followed by kvb_select
 *   kvb_sparse_attn     patch the selected rows (Alg. 2 step 4), then causal
 *                       GQA attention of the selected query rows (Eq. 2)
 *   kvb_patch           Alg. 2 step 4 alone, every layer at once, with the
 *                       attention's fp16 copy of V and work plans of every
 *                       layer
 *   kvb_sparse_attn_layer  the repair forward's attention of one layer over
 *                       the patched cache (Eq. 2), with its prebuilt plan
 *
 * plus the host helpers that prepare their inputs (rotation tables, row
 * flags, the threshold-activated probe of Sec. 7.4) and the cache-population
 * kernels (RoPE at absolute positions, KIVI quantisation, chunk importance;
 * Sec. 4.7 warm, Sec. 4.4).
 *
 * Conventions
 *   - Every pointer named as a tensor, descriptor, index or workspace is a
 *     DEVICE pointer owned by the caller, unless its comment says HOST.
 *     Tensor pointers must be 16-byte aligned.
 *   - The library never allocates, frees or synchronises.  Every GPU call only
 *     enqueues kernels on `stream` (a hipStream_t passed as void*; NULL is the
 *     default stream) and returns.  Asynchronous device faults surface at the
 *     caller's next synchronisation.
 *   - Return value: KVB_OK when every argument passed validation and every
 *     launch was enqueued; KVB_EINVAL for a bad argument (null pointer,
 *     non-positive size, misalignment, inconsistent sizes, workspace too
 *     small); KVB_EUNSUPPORTED for a shape outside the built kernels;
 *     KVB_EHIP for a HIP runtime failure (including "no device").  Validation
 *     runs on the host before any HIP call.  kvb_last_error() returns a
 *     thread-local message ("" after KVB_OK).
 *   - Contents of device arrays (descriptor ranges, row lists) are the
 *     caller's contract; kernels that index with them bound-check and skip
 *     (writing nothing) rather than read or write out of range.
 *   - Layouts (row-major, innermost last):
 *       cache K / V           bf16 [L][Hkv][T][d]      (T = t_total rows)
 *       fp16 copy of V        fp16 [L][Hkv][T][d]      (see kvb_patch)
 *       queries / outputs     bf16 [L][T][Hq][d]
 *       chunk-pool codes      u8   [P][L][Hkv][C][d*b/8]
 *       key statistics        f32  [P][L][Hkv][C/Gk][d]    (scale, zero)
 *       value statistics      f32  [P][L][Hkv][C][d/Gv]    (scale, zero)
 *     A row is an absolute index into the ragged batch; prompt b owns rows
 *     cu_seqlens[b] .. cu_seqlens[b+1]-1 and a row's position is its offset
 *     from cu_seqlens[b].
 *   - bfloat16 and fp16 are passed as their uint16 bit patterns.
 */
#ifndef KVB_H
#define KVB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { KVB_OK = 0, KVB_EINVAL = 1, KVB_EUNSUPPORTED = 2, KVB_EHIP = 3 } kvb_status;
typedef enum { KVB_BF16 = 0, KVB_F32 = 1, KVB_F64 = 2 } kvb_dtype;

/* row_flags bits used by kvb_select */
enum { KVB_ROW_CANDIDATE = 1u, KVB_ROW_FORCED = 2u };

/* Shape of the chunk pool (HOST struct). */
typedef struct {
  int32_t n_layers;    /* L */
  int32_t n_kv_heads;  /* Hkv */
  int32_t head_dim;    /* d: 64 or 128 */
  int32_t chunk_len;   /* C: 128 (fixed-size chunking, Sec. 4.1) */
  int32_t bits;        /* b: 8, or 4 (two codes per byte along d, even channel in the low nibble) */
  int32_t k_group;     /* Gk: tokens per key-statistic group; divides C */
  int32_t v_group;     /* Gv: channels per value-statistic group; divides d */
} kvb_pool_layout;

/* One cached chunk placed into the prompt (DEVICE array element).
 * pool_idx: slot in the chunk pool; src_pos: position the chunk was cached at;
 * dst_row: first cache row it fills; dst_pos: its position in the new prompt.
 * The rotation table row used for the chunk is its index in the array. */
typedef struct {
  int32_t pool_idx, src_pos, dst_row, dst_pos;
} kvb_chunk;

/* 7 for this header (version 2 added the optional fp16 shadow of V to
 * kvb_stitch, kvb_sparse_attn and kvb_sparse_attn_workspace_bytes; version 3
 * added kvb_stitch_deviation and kvb_chunk_importance; version 4 added
 * kvb_probe_gate; version 5 added kvb_attn_plans_bytes, kvb_patch and
 * kvb_sparse_attn_layer; version 6 added kvb_select_noalloc and
 * kvb_select_noalloc_max_bytes; version 7 moved the fp16 copy of V from the
 * stitch to the patch: kvb_patch / kvb_sparse_attn build it from the patched
 * cache, kvb_stitch and kvb_stitch_deviation no longer take it, and the
 * building calls report values fp16 cannot hold in a status word). */
int kvb_abi_version(void);

/* Thread-local message of the last failing call on this thread. */
const char* kvb_last_error(void);

/* ---- host helpers ------------------------------------------------------ */

/* Rotation table for position offsets (Sec. 3.2, Eq. 3; HOST only, no GPU).
 * For each offset delta[n] and i < head_dim/2:
 *   cos_out[n][i] = cos(delta[n] * omega_i), sin_out[n][i] = sin(delta[n] * omega_i),
 *   omega_i = theta^(-2i/head_dim)  (rotate-half pairing: channel i with i + d/2),
 * evaluated in double precision and rounded once to float.  With delta =
 * dst_pos - src_pos per chunk it is the stitch's R^Delta table; with
 * delta = 0..n-1 it is the absolute-position table of kvb_rope_rows.
 * All arrays HOST; cos_out / sin_out [n][head_dim/2].
 * Errors: KVB_EINVAL (null pointer, n < 0, head_dim not even and positive,
 * theta <= 0). */
kvb_status kvb_rope_delta_table(double theta, int32_t head_dim, const int32_t* delta, int32_t n,
                                float* cos_out, float* sin_out);

/* Row flags and top-k sizes from a fixed-size chunk map (HOST only, no GPU).
 * Candidates are the rows covered by `chunks` (cached chunks; Alg. 2 scores
 * the cached tokens).  Forced rows are live rows (not covered: miss chunks
 * and the n_sinks sink rows at the start of every prompt, Sec. 4.1) plus, for
 * every chunk boundary p > 0 of a prompt (p = n_sinks + chunk_len * c), the
 * candidate rows at positions [max(0, p - seam_left), min(T_b, p + seam_right))
 * (Alg. 1 re-encodes [p - R, p): seam_left = R, seam_right = 0).
 * k_per_seq[b] = floor(rho_num * n_b / rho_den), n_b = candidates of prompt b.
 * cu_seqlens [n_seqs+1], chunks [n_chunks], row_flags [t_total], k_per_seq
 * [n_seqs]: all HOST.  Errors: KVB_EINVAL (null pointer, bad sizes, a chunk
 * outside the rows, rho_den <= 0). */
kvb_status kvb_row_flags(int32_t n_seqs, const int32_t* cu_seqlens, int32_t n_sinks,
                         int32_t chunk_len, const kvb_chunk* chunks, int32_t n_chunks,
                         int32_t seam_left, int32_t seam_right, int32_t rho_num, int32_t rho_den,
                         uint8_t* row_flags, int32_t* k_per_seq);

/* Threshold-activated probe (Sec. 7.4: the probe pass costs time in
 * proportion to the cached tokens and can be skipped when the hit ratio is
 * below a minimum; HOST only, no GPU).  For prompt b with n_b candidate rows
 * (row_flags bit KVB_ROW_CANDIDATE) out of T_b rows, the probe runs iff
 * n_b > 0 and n_b * min_den >= min_num * T_b (64-bit integers, exact).  A
 * prompt without the probe has no deviation to rank: k_per_seq[b] is set to 0,
 * so kvb_select keeps only its forced rows (live rows and seam windows,
 * SelectiveRecompute alone); the other entries are left as they are.
 * *n_probed (optional, NULL for none) receives the number of probed prompts;
 * with 0 the caller can skip the deviation pass altogether (kvb_stitch
 * instead of kvb_stitch_deviation, then kvb_select: the deviations of
 * prompts with k = 0 are never read).  min_num = 0 keeps every prompt that
 * has a candidate.  cu_seqlens [n_seqs+1], row_flags [t_total], k_per_seq
 * [n_seqs] (in/out): all HOST.  Errors: KVB_EINVAL (null pointer, n_seqs <= 0,
 * min_den <= 0, min_num < 0, cu_seqlens not starting at 0 or decreasing). */
kvb_status kvb_probe_gate(int32_t n_seqs, const int32_t* cu_seqlens, const uint8_t* row_flags,
                          int32_t min_num, int32_t min_den, int32_t* k_per_seq,
                          int32_t* n_probed);

/* ---- cache population (Sec. 4.7 warm, Sec. 4.5, Eq. 3) ----------------- */

/* RoPE at absolute positions (Eq. 3) and storage conversion.
 * x: f32 [n_outer][n_rows][n_inner][head_dim]; vector (o, r, i) is rotated by
 * the table row row_pos[r] + (outer_pos ? outer_pos[o] : 0), which must lie in
 * [0, table_len) (a vector with an out-of-range position is written as NaN).
 * table_cos / table_sin: f32 [table_len][head_dim/2] (kvb_rope_delta_table
 * with delta = 0..table_len-1); both NULL = no rotation (conversion only).
 * Arithmetic is double: y_i = x_i c - x_{i+d/2} s, y_{i+d/2} = x_{i+d/2} c + x_i s,
 * each product and sum rounded once.  out: same shape, dtype out_dtype
 * (F64; F32 = RNE of the double; BF16 = RNE to float then RNE to bfloat16).
 * row_pos [n_rows], outer_pos [n_outer] int32.
 * Errors: KVB_EINVAL, KVB_EUNSUPPORTED (head_dim not 64 or 128). */
kvb_status kvb_rope_rows(int32_t head_dim, int64_t n_outer, int64_t n_rows, int64_t n_inner,
                         const float* x, const int32_t* row_pos, const int32_t* outer_pos,
                         const float* table_cos, const float* table_sin, int32_t table_len,
                         kvb_dtype out_dtype, void* out, void* stream);

/* KIVI asymmetric quantisation of cached chunks (Sec. 4.5, Eq. 7).
 * k_in / v_in: in_dtype (F32 or F64) [n_pool][n_in][Hkv][C][d], written into
 * pool layers first_layer .. first_layer + n_in - 1.  Keys: per channel over
 * groups of Gk tokens; values: per token over groups of Gv channels.
 * code = clamp(rint((x - min) / (max - min) * (2^b - 1)), 0, 2^b - 1) in double
 * (ties to even); scale = float((max - min) / (2^b - 1)), zero = float(min);
 * a constant group gets scale 0 and codes 0.  Outputs in the pool layout.
 * Errors: KVB_EINVAL, KVB_EUNSUPPORTED (bits, head_dim, chunk_len). */
kvb_status kvb_kivi_quantize(const kvb_pool_layout* pool, int32_t n_pool, int32_t first_layer,
                             int32_t n_in, kvb_dtype in_dtype, const void* k_in, const void* v_in,
                             uint8_t* k_codes, float* k_scale, float* k_zero,
                             uint8_t* v_codes, float* v_scale, float* v_zero, void* stream);

/* Chunk importance for the cache manager's eviction order (Sec. 4.4, the
 * importance equation): importance(C) = 1/(L Hkv C) sum over layers, kv heads
 * and tokens of the chunk of ||k||_2, the mean Euclidean norm of its cached key
 * vectors.  k_in: in_dtype (F32 or F64) [n_pool][n_in][Hkv][C][d], n_in of the
 * pool's L layers (the keys as cached, e.g. the same input kvb_kivi_quantize
 * takes); importance: f64 [n_pool], ACCUMULATED: every call adds its layers'
 * share (sum of their norms / (L Hkv C)), so calls over disjoint layer sets
 * starting from zero leave the mean over all layers.  Double arithmetic; the
 * order of the sums is fixed (deterministic), so it can differ from a plain
 * left-to-right sum in the last bits.  For callers that rank chunks for
 * eviction; not part of the timed path.
 * Errors: KVB_EINVAL, KVB_EUNSUPPORTED (head_dim, bits, chunk_len as in
 * kvb_pool_layout). */
kvb_status kvb_chunk_importance(const kvb_pool_layout* pool, int32_t n_pool, int32_t n_in,
                                kvb_dtype in_dtype, const void* k_in, double* importance,
                                void* stream);

/* ---- the hot path ------------------------------------------------------- */

/* Stitch (Sec. 4.3 CHUNK_REUSE assembly; Sec. 3.2 position correction R^Delta;
 * Sec. 4.5 dequantisation).  For every chunk c of `chunks`, layer l, kv head h,
 * token u < C and channel j:
 *   K[l][h][dst_row + u] = R^(dst_pos - src_pos) (code * scale + zero)   (key stats of token group u/Gk)
 *   V[l][h][dst_row + u] =                        code * scale + zero    (value stats of channel group j/Gv)
 * with the rotation from table row c of rope_cos / rope_sin (f32 [n_chunks][d/2]).
 * Arithmetic is double, no fused multiply-add; the result is stored as f32
 * (RNE) or bf16 (RNE to float, then RNE to bfloat16) per out_dtype.
 * k_cache / v_cache: [L][Hkv][t_total][d] of out_dtype (KVB_BF16 or KVB_F32);
 * only rows of the listed chunks are written -- live rows (misses, sinks) are
 * the caller's.  Chunks must not overlap.  A chunk whose pool_idx or rows fall
 * outside the arrays is skipped.  n_pool bounds pool_idx; n_pool = 0 (nothing
 * cached: a cold prompt) is allowed with n_chunks = 0 and then the pool arrays
 * may be NULL (the call returns KVB_OK and writes nothing).
 * Errors: KVB_EINVAL, KVB_EUNSUPPORTED (bits not 4/8, d not 64/128, C != 128). */
kvb_status kvb_stitch(const kvb_pool_layout* pool, int32_t n_pool,
                      const uint8_t* k_codes, const float* k_scale, const float* k_zero,
                      const uint8_t* v_codes, const float* v_scale, const float* v_zero,
                      const kvb_chunk* chunks, int32_t n_chunks,
                      const float* rope_cos, const float* rope_sin,
                      int64_t t_total, kvb_dtype out_dtype, void* k_cache, void* v_cache,
                      void* stream);

/* kvb_stitch with a bf16 cache, fused with the per-layer deviation of the rows
 * it stitches (Alg. 2 steps 1-2 in one pass: the stitched keys are compared
 * with k_fresh while they are in registers instead of being read back).
 * Stitch outputs (k_cache, v_cache) are bit-identical to kvb_stitch(...,
 * KVB_BF16, ...).  For every row t of a chunk in the list
 * and every layer l, delta[l][t] = 1 - (1/Hkv) sum_h cos(k_cache[l][h][t],
 * k_fresh[l][h][t]) with cos as in kvb_deviation (double sums over the bf16
 * values, the same zero-norm rule; the summation order differs, so values can
 * differ from kvb_deviation's in the last float bit; identical rows still give
 * 0 exactly).  K only, every layer its own set.  Rows outside the listed
 * chunks (live rows, whose cache already holds the fresh values) are not
 * written: kvb_select reads delta only at candidate rows, which are the
 * stitched rows.  k_cache, v_cache, k_fresh bf16 [L][Hkv][t_total][d]; delta
 * f32 [L][t_total].
 * Errors: as kvb_stitch (also the empty-pool rule); k_fresh and delta must be
 * non-NULL and aligned. */
kvb_status kvb_stitch_deviation(const kvb_pool_layout* pool, int32_t n_pool,
                                const uint8_t* k_codes, const float* k_scale, const float* k_zero,
                                const uint8_t* v_codes, const float* v_scale, const float* v_zero,
                                const kvb_chunk* chunks, int32_t n_chunks,
                                const float* rope_cos, const float* rope_sin, int64_t t_total,
                                uint16_t* k_cache, uint16_t* v_cache, const uint16_t* k_fresh,
                                float* delta, void* stream);

/* Per-token deviation (Alg. 2 step 2):
 *   delta[s][t] = 1 - (1/N) * sum cos(cache[l][h][t], fresh[l][h][t])
 * over kv heads h, tensors {K} (or {K, V} when v_cache and v_fresh are both
 * non-NULL) and layers l (each layer its own set s = l when per_layer, else one
 * set over every layer).  cos = dot / sqrt(|a|^2 |b|^2), evaluated in double
 * over the bf16 inputs; when |a|^2 |b|^2 == 0 it is 1 if both vectors are zero
 * and 0 otherwise.  delta: f32 [per_layer ? L : 1][t_total] (the double rounded
 * once).  Inputs bf16 [L][Hkv][t_total][d].
 * Errors: KVB_EINVAL (incl. exactly one V pointer NULL), KVB_EUNSUPPORTED (d not
 * 64/128, Hkv not a power of two up to 16). */
kvb_status kvb_deviation(int32_t n_layers, int32_t n_kv_heads, int32_t head_dim, int64_t t_total,
                         const uint16_t* k_cache, const uint16_t* k_fresh,
                         const uint16_t* v_cache, const uint16_t* v_fresh,
                         int32_t per_layer, float* delta, void* stream);

/* Workspace bytes kvb_select needs (pure function). */
size_t kvb_select_workspace_bytes(int32_t n_sets, int64_t t_total, int32_t n_seqs);

/* Row selection (Alg. 2 step 3 with Alg. 1 windows and live rows).
 * For every set s and prompt b: TopK = the first k_per_seq[s][b] candidate rows
 * (row_flags bit KVB_ROW_CANDIDATE) of the prompt ordered by delta[s][row]
 * descending, then row ascending (the lower row wins a tie; -0 equals +0; NaN
 * ranks below every number); S = TopK united with the rows flagged
 * KVB_ROW_FORCED, ascending.  rows[s][...] holds the sets' prompts one after
 * another; cu_rows[s][b] is where prompt b starts in rows[s], cu_rows[s][n_seqs]
 * the set's total.  A k larger than the prompt's candidates takes them all.
 * delta f32 [n_sets][t_total]; row_flags u8 [t_total]; k_per_seq i32
 * [n_sets][n_seqs]; rows i32 [n_sets][t_total]; cu_rows i32 [n_sets][n_seqs+1];
 * cu_seqlens i32 [n_seqs+1].  Deterministic (no atomics decide an order).
 * Errors: KVB_EINVAL (incl. workspace smaller than kvb_select_workspace_bytes). */
kvb_status kvb_select(int32_t n_sets, int64_t t_total, const int32_t* cu_seqlens, int32_t n_seqs,
                      const float* delta, const uint8_t* row_flags,
                      const int32_t* k_per_seq, int32_t* rows, int32_t* cu_rows,
                      void* workspace, size_t workspace_bytes, void* stream);

/* kvb_select for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same selection, bit-identical outputs, with no workspace argument.  Its
 * staging lives in a static device array of the library, one copy per device,
 * held until the process ends; kvb_select_noalloc_max_bytes() returns its size
 * (16 MiB).  The call allocates nothing.  Every call on a device shares that
 * device's array (each call overwrites what it needs before reading it), so
 * calls that overlap on one device race: order them on one stream.  Arguments
 * as kvb_select without workspace / workspace_bytes.
 * Errors: as kvb_select; KVB_EINVAL also when kvb_select_workspace_bytes(n_sets,
 * t_total, n_seqs) exceeds kvb_select_noalloc_max_bytes(). */
kvb_status kvb_select_noalloc(int32_t n_sets, int64_t t_total, const int32_t* cu_seqlens,
                              int32_t n_seqs, const float* delta, const uint8_t* row_flags,
                              const int32_t* k_per_seq, int32_t* rows, int32_t* cu_rows,
                              void* stream);

/* Bytes of the static scratch behind kvb_select_noalloc (pure function). */
size_t kvb_select_noalloc_max_bytes(void);

/* kvb_deviation then kvb_select on the same stream (Alg. 2 steps 2-3).
 * Arguments as in those two calls; delta is written as well. */
kvb_status kvb_deviation_topk(int32_t n_layers, int32_t n_kv_heads, int32_t head_dim,
                              int64_t t_total, const int32_t* cu_seqlens, int32_t n_seqs,
                              const uint16_t* k_cache, const uint16_t* k_fresh,
                              const uint16_t* v_cache, const uint16_t* v_fresh, int32_t per_layer,
                              const uint8_t* row_flags, const int32_t* k_per_seq, float* delta,
                              int32_t* rows, int32_t* cu_rows, void* workspace,
                              size_t workspace_bytes, void* stream);

/* The fp16 copy of V (the attention's P.V operand): fp16 [L][Hkv][T][d], each
 * value the fp16 image of the bf16 V cache value at the same index (exact
 * while |v| < 65536: a bf16 significand fits an fp16 one; bf16 values below
 * 2^-14 become fp16 subnormals).  Built from the patched cache by kvb_patch
 * (or inside kvb_sparse_attn).  Optional status word (v_status,
 * DEVICE uint32, 4-byte aligned, NULL for none): the building call stores 1
 * there when a V value fp16 cannot hold (|v| >= 65536, infinite or NaN) --
 * the attention's P.V product would then see an infinity -- and never writes
 * it otherwise, so the caller clears it before the call and reads it after
 * (when it is 1 the outputs of those rows' prompts are not to be trusted:
 * no fp16 variant of the product can hold such values). */

/* Workspace bytes kvb_sparse_attn needs (pure function); v_f16_given is
 * non-zero when the call passes an fp16 copy of V (the workspace then holds none
 * of its own).  0 for invalid sizes. */
size_t kvb_sparse_attn_workspace_bytes(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads,
                                       int32_t head_dim, int64_t t_total, int32_t n_seqs,
                                       int32_t max_seq_len, int32_t max_rows,
                                       int32_t v_f16_given);

/* Patch then sparse-query causal attention (Alg. 2 step 4; Eq. 2).
 * For each layer l and its row set S_l (rows[l] / cu_rows[l] when
 * rows_per_layer, else rows[0] / cu_rows[0] for every layer):
 *   1. k_cache[l][h][t] = k_fresh[l][h][t] and v_cache[l][h][t] = v_fresh[l][h][t]
 *      for every t in S_l and kv head h;
 *   2. the fp16 copy of the patched V cache of these layers, into
 *      v_cache_f16 when given (n_layers x the layout above), else into the
 *      workspace; v_status as described above;
 *   3. for every t in S_l and query head h, with g = floor(h * Hkv / Hq) and
 *      b the prompt of t:
 *        out[l][t][h] = sum_{u = cu_seqlens[b]}^{t} softmax_u(scale * q[l][t][h] . K[l][g][u]) V[l][g][u]
 *      over the patched cache.  q is already rotated at the row's position.
 * QK^T runs as bf16 MFMA, the softmax in float (online, base-2 exponent), PV
 * as fp16 MFMA (probabilities and the copy of V in fp16), accumulation in
 * float.  Only rows of S_l are written in out (bf16 or f32 per out_dtype,
 * [L][t_total][Hq][d]).  max_rows bounds |S_l| and max_seq_len bounds T_b (host
 * values used to size the grid).  Deterministic: a tile's key ranges split
 * between workgroups are combined in key order.  Rows of S_l must be ascending
 * within each prompt and belong to it.
 * Errors: KVB_EINVAL (incl. workspace too small, Hq % Hkv != 0),
 * KVB_EUNSUPPORTED (d not 64/128, Hq/Hkv not dividing 32). */
kvb_status kvb_sparse_attn(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads,
                           int32_t head_dim, int64_t t_total, const int32_t* cu_seqlens,
                           int32_t n_seqs, int32_t max_seq_len, const int32_t* rows,
                           const int32_t* cu_rows, int32_t rows_per_layer, int32_t max_rows,
                           const uint16_t* q, const uint16_t* k_fresh, const uint16_t* v_fresh,
                           uint16_t* k_cache, uint16_t* v_cache, uint16_t* v_cache_f16,
                           uint32_t* v_status, float softmax_scale, kvb_dtype out_dtype, void* out,
                           void* workspace, size_t workspace_bytes, void* stream);

/* ---- patch once, then attention layer by layer -------------------------
 * Alg. 2 takes the rows it patches (K~, V~) from the probe pass, which covers
 * every layer before the selection (step 1), and step 4 completes before the
 * repair forward runs.  A caller that runs the repair forward layer by layer
 * can therefore patch every layer with one kvb_patch call right after the
 * selection, then make one kvb_sparse_attn_layer call per layer.  Results
 * (cache, fp16 copy of V, out) are bit-identical to kvb_sparse_attn over the
 * same rows. */

/* Bytes of the plan buffer kvb_patch fills for n_layers layers (pure
 * function; 0 for invalid sizes).  The plans depend on the sizes given here and
 * on the device's compute-unit count: build and use them on one device. */
size_t kvb_attn_plans_bytes(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads,
                            int32_t head_dim, int64_t t_total, int32_t n_seqs,
                            int32_t max_seq_len, int32_t max_rows);

/* Patch (Alg. 2 step 4) of every layer: for each layer l and t in S_l (rows[l]
 * / cu_rows[l] when rows_per_layer, else rows[0] / cu_rows[0]) and kv head h,
 * k_cache[l][h][t] = k_fresh[l][h][t] and v_cache[l][h][t] = v_fresh[l][h][t];
 * then, when v_cache_f16 is given, the fp16 copy of every layer of the
 * patched V cache (every row, whatever wrote it: the stitch, the caller's
 * live rows, this patch), with the optional range status v_status (both as
 * described above kvb_sparse_attn_workspace_bytes).  Layouts and sizes as
 * kvb_sparse_attn.  When plans is not NULL the same launch also writes the
 * attention work plan of every layer into it (at least kvb_attn_plans_bytes
 * bytes, 16-byte aligned; the contents are opaque), for the
 * kvb_sparse_attn_layer calls that follow on the same rows.  Rows of S_l must
 * be ascending within each prompt and belong to it (as kvb_sparse_attn).
 * Errors: KVB_EINVAL (incl. plans smaller than kvb_attn_plans_bytes, v_status
 * without v_cache_f16), KVB_EUNSUPPORTED (as kvb_sparse_attn). */
kvb_status kvb_patch(int32_t n_layers, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                     int64_t t_total, const int32_t* cu_seqlens, int32_t n_seqs,
                     int32_t max_seq_len, const int32_t* rows, const int32_t* cu_rows,
                     int32_t rows_per_layer, int32_t max_rows, const uint16_t* k_fresh,
                     const uint16_t* v_fresh, uint16_t* k_cache, uint16_t* v_cache,
                     uint16_t* v_cache_f16, uint32_t* v_status, void* plans, size_t plans_bytes,
                     void* stream);

/* Attention (Eq. 2) of layer `layer` of n_layers for the rows of S_layer, over
 * the already patched cache: for every t in S_layer and query head h,
 *   out[layer][t][h] = sum_{u = cu_seqlens[b]}^{t}
 *                      softmax_u(scale * q[layer][t][h] . K[layer][g][u]) V[layer][g][u]
 * with the arithmetic of kvb_sparse_attn.  Every pointer is the whole tensor
 * as kvb_sparse_attn takes it (the call offsets to the layer).  v_cache_f16 is
 * required: the fp16 copy of the patched V cache (as kvb_patch builds
 * them); plans as filled by kvb_patch with the same sizes on this device;
 * workspace of at least kvb_sparse_attn_workspace_bytes(1, ..., v_f16_given =
 * 1) bytes (partial records; calls that share it must be ordered on one
 * stream).  Reads q, k_cache, v_cache_f16, rows, plans; writes out (rows of
 * S_layer only) and the workspace.
 * Errors: KVB_EINVAL (incl. layer outside [0, n_layers), plans or workspace
 * too small, v_cache_f16 NULL), KVB_EUNSUPPORTED (as kvb_sparse_attn). */
kvb_status kvb_sparse_attn_layer(int32_t layer, int32_t n_layers, int32_t n_q_heads,
                                 int32_t n_kv_heads, int32_t head_dim, int64_t t_total,
                                 const int32_t* cu_seqlens, int32_t n_seqs, int32_t max_seq_len,
                                 const int32_t* rows, const int32_t* cu_rows,
                                 int32_t rows_per_layer, int32_t max_rows, const uint16_t* q,
                                 const uint16_t* k_cache, const uint16_t* v_cache_f16,
                                 const void* plans, size_t plans_bytes, float softmax_scale,
                                 kvb_dtype out_dtype, void* out, void* workspace,
                                 size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KVB_H */
