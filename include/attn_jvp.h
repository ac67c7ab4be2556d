/*
 * attn_jvp.h -- C ABI of the MI355X (gfx950) masked-attention forward + JVP library.
 *
 * Operation (paper App. B, "FlashAttention-2 JVP kernel with custom masks"):
 *   O   = softmax(s * Q K^T + M) V                      (masked-attention equation)
 *   dS  = s * (dQ K^T + Q dK^T), dS = 0 where M = -inf  (score-tangent equation;
 *                                                        the mask has no tangent)
 *   dO  = P dV + (P o (dS - rowsum(P o dS))) V          (tangent-output equation)
 *   LSE = rowmax + ln(rowsum exp(S - rowmax))            (Algorithm 1, normalisation)
 * computed in one fused online-softmax pass (Algorithm 1; epilogue equation
 * dO = diag(l)^-1 (A + B - diag(r) O)).  M is the teacher-forcing chunk mask of
 * autoregressive video diffusion (paper Sec. 3.1.1, packed [clean | noisy]
 * forward): a clean query in chunk j sees clean chunks <= j; a noisy query in
 * chunk i sees clean chunks < i and noisy chunk i.  Block-causal and full masks
 * are the other two layouts of the same range-list representation (App. B,
 * "Sparse custom-mask representation").
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Tensors are contiguous row-major [B, H, L, D] (batch, head, token, head_dim),
 *   all with the same dtype (ATTN_DTYPE_*); LSE is fp32 [B, H, L].
 * - Tensor pointers are DEVICE pointers; the mask layout is a HOST struct whose
 *   arrays are HOST memory, read during the call only.
 * - softmax_scale <= 0 selects s = 1/sqrt(D).
 * - Work is enqueued on `stream` (a hipStream_t passed as void*, NULL = default
 *   stream) and the call returns without synchronising: outputs are valid once
 *   the stream has been synchronised.
 * - The caller owns every buffer.  The library allocates no device memory and
 *   keeps no per-call state, so calls are reentrant and may be captured in a
 *   HIP graph.  Inputs are never written.  Outputs must not overlap inputs or
 *   each other (checked by address range; overlap is ATTN_ERR_INVALID).
 * - Alignment: every [B, H, L, D] tensor pointer (inputs, tangents, O, dO, gO, gQ, gK,
 *   gV) must be 16-byte aligned, LSE and Delta 4-byte aligned; otherwise
 *   ATTN_ERR_INVALID.
 * - Sizes: B, H, L >= 1, B * H <= 2^20, ceil(L / 128) * B * H <= 2^31 - 1 (work-groups
 *   of one launch); the kernels address a head with 32-bit byte offsets, so bf16 inputs
 *   need L * D <= 2^31 and fp32 inputs L * D <= 2^30.  Larger sizes are
 *   ATTN_ERR_INVALID.
 * - Return codes: ATTN_OK, or ATTN_ERR_INVALID (bad pointer, size or layout),
 *   ATTN_ERR_UNSUPPORTED (dtype / head_dim not built), ATTN_ERR_HIP (a HIP
 *   launch error).  All argument and layout validation happens before any HIP
 *   call.  attn_last_error() returns a thread-local message for the last
 *   nonzero return of this thread.  Nothing aborts or throws across the ABI.
 * - Rows with no admissible key (impossible for the three built-in layouts)
 *   produce O = 0, dO = 0, LSE = -inf.
 */
#ifndef ATTN_JVP_H
#define ATTN_JVP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* element types of Q, K, V, dQ, dK, dV, O, dO */
enum {
  ATTN_DTYPE_F32 = 0,  /* fp32 in, fp32 math (fp32 matrix cores), fp32 out; D in {64, 128} */
  ATTN_DTYPE_BF16 = 1  /* bf16 in, bf16 MFMA with fp32 accumulation, bf16 out; D in {64, 128} */
};

/* attention mask kinds (paper Sec. 3.1.1 and the background on TF / DF training) */
enum {
  ATTN_MASK_FULL = 0,             /* every query sees every key; num_chunks/offsets ignored */
  ATTN_MASK_BLOCK_CAUSAL = 1,     /* query in chunk i sees chunks <= i; requires L == o_N */
  ATTN_MASK_TEACHER_FORCING = 2,  /* [clean c_1..c_N | noisy c_1..c_N]; requires L == 2 o_N */
  ATTN_MASK_RANGES = 3            /* explicit query groups with key ranges (see attn_chunk_layout) */
};

enum {
  ATTN_OK = 0,
  ATTN_ERR_INVALID = 1,
  ATTN_ERR_UNSUPPORTED = 2,
  ATTN_ERR_HIP = 3
};

/* largest number of chunks a layout may have (the derived query-group table
 * travels in the kernel arguments, so its size is bounded) */
#define ATTN_MAX_CHUNKS 64
/* largest number of query groups of an ATTN_MASK_RANGES layout */
#define ATTN_MAX_GROUPS 128
/* largest number of key ranges, over all groups, after a layout's ranges are
 * normalised (empty ranges dropped, touching ranges of a group merged) */
#define ATTN_MAX_RANGES 256

/* Mask layout.
 *
 * Block-causal and teacher-forcing: chunk_offsets (HOST memory) holds num_chunks + 1
 * strictly increasing prefix offsets 0 = o_0 < o_1 < ... < o_N of the chunk
 * boundaries within ONE half of the TF sequence (teacher forcing) or within the
 * sequence (block-causal).  Uniform chunks of C tokens use o_i = i * C.
 *
 * ATTN_MASK_RANGES gives the query-group / key-range representation directly (paper
 * App. B, "Sparse custom-mask representation": query group g owns the query interval
 * Q_g = [q_g, q_{g+1}) and admits the keys of its list K_g of R_g >= 0 key intervals).
 * All arrays are HOST memory, read during the call only:
 *   num_chunks     = G query groups (1 .. ATTN_MAX_GROUPS)
 *   chunk_offsets  = G + 1 query-group bounds 0 = q_0 < q_1 < ... < q_G = L (the groups
 *                    tile the sequence; a row that should see no key belongs to a group
 *                    with no key range)
 *   range_offsets  = G + 1 non-decreasing ints, range_offsets[0] = 0: the key ranges of
 *                    group g are entries range_offsets[g] .. range_offsets[g + 1] - 1
 *   ranges         = 2 * range_offsets[G] ints, k0 k1 per key range [k0, k1), with
 *                    0 <= k0 <= k1 <= L; the ranges of one group may come in any order,
 *                    may be empty (k0 == k1) or touch, but must not overlap (a key in two
 *                    ranges of a group would enter the softmax twice)
 * Rows of a group with no (non-empty) key range are fully masked: O = 0, dO = 0,
 * LSE = -inf.  After empty ranges are dropped and touching ones merged, at most
 * ATTN_MAX_RANGES ranges may remain; beyond that the layout is ATTN_ERR_INVALID. */
typedef struct attn_chunk_layout {
  int32_t kind;                  /* ATTN_MASK_* */
  int32_t num_chunks;            /* N (chunks) or G (groups, ATTN_MASK_RANGES); ignored for FULL */
  const int32_t* chunk_offsets;  /* N + 1 chunk offsets, or G + 1 query-group bounds (RANGES) */
  const int32_t* range_offsets;  /* G + 1 range offsets (ATTN_MASK_RANGES only; else may be NULL) */
  const int32_t* ranges;         /* 2 * range_offsets[G] ints (ATTN_MASK_RANGES only; else may be NULL) */
} attn_chunk_layout;

/* Fused masked attention forward + JVP (paper App. B, Algorithm 1).
 *   in : Q, K, V, dQ, dK, dV  device [B, H, L, D], dtype `dtype`
 *   out: O, dO                device [B, H, L, D], dtype `dtype`
 *        LSE                  device fp32 [B, H, L], natural log, scaled-score domain
 * B, H, L >= 1; D in {64, 128}. */
int attn_jvp_fwd(int dtype, int B, int H, int L, int D,
                 const void* Q, const void* K, const void* V,
                 const void* dQ, const void* dK, const void* dV,
                 const attn_chunk_layout* layout, float softmax_scale,
                 void* O, void* dO, float* LSE, void* stream);

/* Fused forward + JVP for the teacher-forcing sCM tangent (paper Sec. 3.1.2, the
 * TF-sCM tangent equation: the packed input tangent is [0^clean, t^noisy], i.e. the
 * clean context carries zero tangent).  `layout` must be ATTN_MASK_TEACHER_FORCING;
 * with half = L / 2 the tangents of the clean rows [0, half) are zero and are not
 * passed:
 *   in : Q, K, V              device [B, H, L, D]
 *        dQn, dKn, dVn        device [B, H, L - half, D]: tangents of the noisy rows
 *                             [half, L) (row x of the sequence is row x - half here)
 *   out: O                    device [B, H, L, D]
 *        dOn                  device [B, H, L - half, D]: dO of the noisy rows
 *        LSE                  device fp32 [B, H, L]
 * The result equals attn_jvp_fwd on the zero-padded tangents [0, dQn] etc.; the dO
 * of the clean rows is exactly zero (a clean query sees clean keys only, whose K and
 * V tangents vanish, and its own dQ vanishes), so it is not written.  The kernels
 * skip the work the zeros make vanish: clean query tiles run the forward only, and
 * noisy queries drop the dK and dV terms over clean keys.  Same conventions, dtypes
 * and error behaviour as attn_jvp_fwd; a layout of another kind is
 * ATTN_ERR_INVALID. */
int attn_jvp_fwd_zero_clean(int dtype, int B, int H, int L, int D,
                            const void* Q, const void* K, const void* V,
                            const void* dQn, const void* dKn, const void* dVn,
                            const attn_chunk_layout* layout, float softmax_scale,
                            void* O, void* dOn, float* LSE, void* stream);

/* Masked attention forward only (the primal part of Algorithm 1): O and LSE
 * exactly as attn_jvp_fwd would produce them from the same Q, K, V. */
int attn_fwd(int dtype, int B, int H, int L, int D,
             const void* Q, const void* K, const void* V,
             const attn_chunk_layout* layout, float softmax_scale,
             void* O, float* LSE, void* stream);

/* Gradient of masked attention (reverse mode): the vector-Jacobian product of the
 * masked-attention equation (paper App. B) for a cotangent gO of O, as the student's
 * packed teacher-forcing forward needs for training (Sec. 3.1.2, TF-sCM objective).
 * With P = exp(s Q K^T - LSE) on admissible pairs and 0 elsewhere:
 *   Delta = rowsum(gO o O),  gS = P o (gO V^T - Delta),
 *   gQ = s gS K,  gK = s gS^T Q,  gV = P^T gO.
 *   in : Q, K, V, O, gO        device [B, H, L, D], dtype `dtype` (O as returned by
 *                              attn_fwd / attn_jvp_fwd for the same inputs)
 *        LSE                   device fp32 [B, H, L] from the same call
 *   out: gQ, gK, gV            device [B, H, L, D], dtype `dtype`
 *        Delta                 device fp32 [B, H, L]: rowsum(gO o O) (written by the
 *                              first of the two kernels, read by the second)
 * Same conventions and error behaviour as attn_jvp_fwd; every layout the forward
 * accepts is accepted.  Deterministic (no atomics): two launches on `stream`. */
int attn_bwd(int dtype, int B, int H, int L, int D,
             const void* Q, const void* K, const void* V, const void* O, const void* gO,
             const float* LSE, const attn_chunk_layout* layout, float softmax_scale,
             void* gQ, void* gK, void* gV, float* Delta, void* stream);

/* Host only.  Query-block plan of key tile `ktile` of the backward's key-tile pass
 * (keys [ktile*K, ktile*K + K) with K = 128, query blocks of 64 rows) as the bf16
 * kernel executes it: the visited query-block indices in visiting order go to
 * blocks[], and full[i] = 1 if every query of block i admits every key of the tile
 * (no per-element mask applied), else 0.  Returns the number of visited blocks, or
 * -1 on an invalid layout, tile index or a too-small buffer (capacity `cap`). */
int attn_key_tile_plan(const attn_chunk_layout* layout, int L, int ktile, int32_t* blocks, int32_t* full, int cap);

/* Host only.  Number of admissible (query, key) pairs of the layout over a
 * sequence of L tokens: the pairs whose work the throughput figures count (the
 * entries of the mask M of the masked-attention equation, paper App. B, that are 0
 * rather than -inf).  Returns -1 (and sets the error message) for an invalid layout. */
int64_t attn_count_unmasked_pairs(const attn_chunk_layout* layout, int L);

/* Host only.  Number of (query, key) pairs the bf16 kernel actually evaluates
 * for this layout, for one (batch, head): whole key blocks of the tile plans,
 * including the masked lanes of partial blocks (the key/value tiles streamed by
 * Algorithm 1's inner loop, paper App. B, under this library's tiling).  Returns -1
 * on an invalid layout or head_dim. */
int64_t attn_count_computed_pairs(const attn_chunk_layout* layout, int L, int D);

/* Host only.  The query-group / key-range table derived from the layout (paper
 * App. B, "Sparse custom-mask representation": query interval [q_g, q_{g+1}) with a
 * list of admissible key intervals), normalised: the ranges of each group sorted,
 * without empty ones, touching ones merged.  Writes G + 1 bounds, G + 1 range offsets
 * and 2 R ints k0 k1 (R = range_offsets[G]) in the form of an ATTN_MASK_RANGES layout;
 * capacities max_groups groups and max_ranges ranges.  Returns G, or -1 on an
 * invalid layout or a too-small buffer. */
int attn_query_groups(const attn_chunk_layout* layout, int L, int32_t* bounds, int32_t* range_offsets,
                      int32_t* ranges, int max_groups, int max_ranges);

/* Host only.  Shape of the work decomposition of the bf16 JVP kernels: query rows
 * per work-group tile and keys per streamed key block (the forward-only kernel takes
 * tiles of half as many rows). */
void attn_tile_shape(int* rows_per_tile, int* keys_per_block);

/* Host only.  Key-block plan of query tile `qtile` (rows [qtile*R, qtile*R + R)
 * with R from attn_tile_shape) as the bf16 kernels execute it: the visited key
 * block indices in visiting order go to blocks[], and full[i] = 1 if block i is
 * admissible for every row of the tile (no per-row mask applied), else 0.
 * Returns the number of visited blocks, or -1 on an invalid layout, tile index
 * or a too-small buffer (capacity `cap`). */
int attn_tile_plan(const attn_chunk_layout* layout, int L, int qtile,
                   int32_t* blocks, int32_t* full, int cap);

/* Host only.  Order in which the bf16 kernels' work-groups of one (batch, head)
 * take query tiles: order[t] = query tile of the t-th work-group (a permutation
 * of 0 .. ceil(L / R) - 1, heaviest tiles first where the layout makes the
 * per-tile work predictable).  zero_clean != 0 gives the order of
 * attn_jvp_fwd_zero_clean, else that of attn_jvp_fwd / attn_fwd.  Returns the
 * number of tiles, or -1 on an invalid layout or a too-small buffer. */
int attn_tile_order(const attn_chunk_layout* layout, int L, int zero_clean, int32_t* order, int cap);

/* Thread-local description of the last nonzero return on this thread ("" if none). */
const char* attn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_JVP_H */
