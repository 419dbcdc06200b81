/*
 * cobs.h - C ABI of the COBS decode-step library for AMD Instinct MI355X (gfx950).
 *
 * COBS (Cumulant Order Block Sparse Attention) selects, per KV head and per
 * decode step, the KV-cache blocks with the largest estimated attention mass
 * and attends only to them plus a sliding window.  Notation of the paper:
 * a query q in R^d attends over keys/values k_t, v_t of T cached tokens,
 * split into contiguous blocks of L tokens (Sec. 2); G query heads share
 * one KV head (GQA); c is the attention scale (the paper absorbs it into q).
 *
 * Stages (one decode step of one layer, for every batch row and KV head):
 *   1. block statistics: count n_b, mean kbar_b, top-r scaled eigenvectors
 *      xi_i of the population covariance (Sec. 5.3 eq. lowrank, Gram trick of
 *      Sec. 5.6), stored as fp32, bf16 or FP4 E2M1 (Sec. 5.5);
 *   2. second-order log-mass estimate per block and query head
 *        l_b^g = ln n_b + c q_g.kbar_b + (c^2/2) sum_i (xi_i . q_g)^2
 *      (eq. trunc with eq. gram), GQA group score
 *        sigma_b = ln sum_g exp(l_b^g - ln sum_b' exp(l_b'^g))
 *      (log of eq. gqa-secondorder);
 *   3. top-s candidate blocks by sigma (ties to the lower block index);
 *   4. softmax attention over the union of the selected blocks and the last w
 *      tokens, each token once (eq. oracle-true), split over workgroups and
 *      merged through log-sum-exp.
 *
 * Conventions
 *   - Every tensor pointer is a DEVICE pointer unless stated otherwise; the
 *     caller owns every buffer, the workspace included.  The library allocates
 *     no device memory, keeps no state between calls and never synchronises.
 *   - Every call validates its arguments on the host before any launch and
 *     returns COBS_ERR_INVALID_ARG / COBS_ERR_UNSUPPORTED without touching the
 *     GPU; otherwise it enqueues its kernels on `stream` (a hipStream_t; NULL
 *     is the default stream) and returns COBS_OK, or COBS_ERR_HIP if a launch
 *     failed.  It never aborts.
 *   - seq_lens[b] (device int32) is the number of valid tokens T of batch row
 *     b.  Values are clamped to [0, max_seq_len] on the device; a row with
 *     T = 0 selects nothing and yields out = 0, lse = -inf.
 *   - Blocks: NB(T) = ceil(T/L); block b holds n_b = min(L, T - bL) tokens.
 *     A block is a selection candidate iff bL < T - w (it has a token before
 *     the window).
 *   - Query head j belongs to KV head j / G (contiguous groups), G = Hq / Hkv.
 *   - Workspace: `ws` must hold cobs_workspace_bytes(cfg, op) bytes, be 256-byte
 *     aligned and be zero-filled before its first use; every call leaves its
 *     arrival counters zero again on completion, so the same workspace can be
 *     reused by later calls on the same stream.  Calls that share a workspace
 *     must not overlap in time (different streams race).
 *   - Results are deterministic: identical inputs give bitwise identical
 *     outputs (no floating-point atomics; work is split statically and
 *     reduced in a fixed order).
 */
#ifndef COBS_H
#define COBS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  COBS_OK = 0,
  COBS_ERR_INVALID_ARG = 1, /* null pointer, inconsistent shape, bad stride ...   */
  COBS_ERR_UNSUPPORTED = 2, /* valid but outside what the kernels implement       */
  COBS_ERR_WORKSPACE = 3,   /* ws too small or misaligned                          */
  COBS_ERR_HIP = 4          /* a HIP launch or runtime call failed                 */
} cobs_status_t;

typedef enum { COBS_F32 = 0, COBS_BF16 = 1, COBS_E2M1 = 2 } cobs_dtype_t;

typedef enum {
  COBS_OP_BUILD = 0,  /* cobs_build_block_stats */
  COBS_OP_SELECT = 1, /* cobs_select            */
  COBS_OP_DECODE = 2, /* cobs_sparse_decode     */
  COBS_OP_STEP = 3,   /* cobs_decode_step       */
  COBS_OP_SELECT_EXACT = 4 /* cobs_select_exact, cobs_select_quest */
} cobs_op_t;

/* Optional record parts (cobs_config_t.options).
 *   COBS_OPT_SKEW: the diagonal third-cumulant term of Sec. 7.7.  Per factor the
 *     record stores gamma_i = g_i / lambda_i^(3/2), where lambda_i = |xi_i|^2,
 *     u_i = xi_i / |xi_i| and g_i = (1/n) sum_t (u_i . (k_t - kbar))^3 (the
 *     paper's scalar), computed from the fp32 factors before storage rounding;
 *     the selector adds (c^3/6) sum_i gamma_i (xi_i . q)^3, the paper's
 *     (1/6) sum_i (u_i . q)^3 g_i, to l_b^g.  A diagnostic selector variant.
 *   COBS_OPT_VALUE_MEAN: the record also stores the block's mean value (in the
 *     mean dtype), the pooled value of the mean-pool compression branch
 *     (Sec. 2 branch (i), kept by Sec. 5.2); needed by cobs_compression_branch. */
typedef enum { COBS_OPT_SKEW = 1, COBS_OPT_VALUE_MEAN = 2 } cobs_option_t;

/* Problem description shared by every call (host struct, passed by pointer). */
typedef struct {
  int32_t batch;         /* B >= 1                                                  */
  int32_t num_q_heads;   /* Hq, a multiple of num_kv_heads; G = Hq/Hkv in {1,2,4,8,16} */
  int32_t num_kv_heads;  /* Hkv >= 1                                                */
  int32_t head_dim;      /* d in {64, 128}                                          */
  int32_t max_seq_len;   /* T_max, cache capacity in tokens, a multiple of block_size */
  int32_t block_size;    /* L in {32, 64, 128}                                      */
  int32_t rank;          /* r in [0, 16]; 0 gives the first-order (mean-pool) score */
  int32_t budget;        /* s >= 0 selected blocks per (batch row, KV head)         */
  int32_t window;        /* w >= 0 most recent tokens always attended               */
  cobs_dtype_t kv_dtype;     /* K/V cache element type: COBS_F32 or COBS_BF16          */
  cobs_dtype_t mean_dtype;   /* stored block mean: F32, BF16 or E2M1                  */
  cobs_dtype_t factor_dtype; /* stored scaled eigenvectors: F32, BF16 or E2M1         */
  float softmax_scale;   /* c; 0 selects 1/sqrt(d)                                  */
  int32_t options;       /* bitwise OR of cobs_option_t; 0 for the plain method    */
  /* Subspace factors (Sec. 5.4): with subspace_dim = s' > 0 every block stores
   * the top-r scaled eigenvectors xi^ss of B_b = U_Q^T Sigma_b U_Q (s'
   * elements each) instead of those of Sigma_b, and the curvature term is
   * sum_i (xi^ss_i . U_Q^T q)^2; the mean term keeps the full q.
   * subspace_dim: 0 (full-space factors) or s' in {32, 64, 96} below d
   *   (COBS_ERR_UNSUPPORTED otherwise); needs rank in [1, 4] (INVALID_ARG
   *   for rank 0, UNSUPPORTED above 4).  cobs_select and the decode steps score
   *   subspace factors with BF16 or E2M1 mean and factors only (UNSUPPORTED
   *   for F32); cobs_build_block_stats also writes F32 ones.
   * query_basis: device fp32 [Hkv, d, s'], 16-byte aligned, U_Q of each KV
   *   head (orthonormal columns spanning its query heads' subspace, e.g. the
   *   top-s' eigenvectors of their E[q q^T]); read by the build, select and
   *   step calls, owned by the caller; NULL exactly when subspace_dim = 0
   *   (COBS_ERR_INVALID_ARG otherwise).                                       */
  int32_t subspace_dim;
  const float* query_basis;
} cobs_config_t;

/* KV cache of one layer.
 * Contiguous mode (block_table == NULL): element (b, h, t, i) of K lives at
 *   k + b*stride_b + h*stride_h + t*stride_t + i   (strides in elements, i < d
 *   contiguous), likewise V with the same strides.  d <= stride_t <= 2^22, and
 *   every stride a multiple of 16 bytes' worth of elements (COBS_ERR_INVALID_ARG
 *   otherwise; a larger stride_t gives COBS_ERR_UNSUPPORTED).
 * Paged mode (block_table != NULL): block_table is a device int32 array
 *   [B, T_max/L] of page ids; page p of the K pool holds [Hkv, L, d] contiguous
 *   elements, so (b, h, t, i) lives at
 *   k + ((block_table[b*(T_max/L) + t/L]*Hkv + h)*L + t%L)*d + i.
 *   Strides are ignored; page ids must lie in [0, num_pages) (an id outside it is
 *   never dereferenced: the decode leaves that page's tokens out, the
 *   statistics build reads them as zero keys, and the exact-mass and Quest
 *   selectors score such a block -inf for every head).
 * k, v: 16-byte aligned.                                                          */
typedef struct {
  const void* k;
  const void* v;
  int64_t stride_b, stride_h, stride_t;
  const int32_t* block_table;
  int64_t num_pages;
} cobs_kv_t;

/* Descriptor record of one block (Sec. 5.3 / 5.5), little-endian, 16-byte aligned:
 *   0        int32   n_b
 *   4        float   scale of the E2M1 mean (0 for F32/BF16 means)
 *   8        float   scale of the E2M1 value mean (COBS_OPT_VALUE_MEAN, else 0)
 *   12       4 zero bytes
 *   16       float   scale of factor i, i < r (E2M1 factors only), zero padded to 16 B
 *   S        float   skew coefficient gamma_i, i < r (COBS_OPT_SKEW only), zero padded to 16 B
 *   M        mean: d elements of mean_dtype
 *   M+|mean| factors: r vectors of d (subspace: s') elements of factor_dtype,
 *            vector-major
 *   V        value mean: d elements of mean_dtype (COBS_OPT_VALUE_MEAN only)
 *   size     rounded up to 16 B
 * Element sizes: F32 4 B, BF16 2 B, E2M1 one nibble (element 2j in the low nibble
 * of byte j).  E2M1 vectors use scale = fp32(max|x|)/6, y = x/scale in fp32,
 * round to nearest of {0,.5,1,1.5,2,3,4,6} with ties to the even code, |y| <= 6,
 * no negative zero, scale 0 for an all-zero vector.  A block with n_b < L stores
 * zero factors (and zero skew coefficients).  Summaries of one layer:
 * [B, Hkv, T_max/L] records.
 * Returns 0 if cfg is invalid.                                                     */
size_t cobs_record_bytes(const cobs_config_t* cfg);

/* Workspace bytes needed by `op` for this configuration (0 if none or invalid). */
size_t cobs_workspace_bytes(const cobs_config_t* cfg, cobs_op_t op);

/* Block statistics (Sec. 5.3, Gram trick of Sec. 5.6, storage of Sec. 5.5).
 * For every batch row b and KV head h, (re)build the records of blocks
 * first_block <= j < first_block + num_blocks that exist at T = seq_lens[b]
 * (j < ceil(T/L)); other records are left untouched.  A full block gets
 * its count, mean and top-r factors (fixed-count block power iteration on the
 * L x L Gram matrix of the centred keys, Rayleigh-Ritz, xi = Kc^T w / sqrt(n),
 * sign fixed so the largest-magnitude entry is positive); a partial block gets
 * its count, mean and zero factors.
 *   summaries: device [B, Hkv, T_max/L, cobs_record_bytes(cfg)] bytes, written. */
cobs_status_t cobs_build_block_stats(const cobs_config_t* cfg, const cobs_kv_t* kv,
                                     const int32_t* seq_lens, int32_t first_block,
                                     int32_t num_blocks, void* summaries, void* ws,
                                     size_t ws_bytes, void* stream);

/* Block selection (eq. trunc, eq. gram, eq. gqa-secondorder, top-s).
 *   q:         device fp32 [B, Hq, d], unscaled queries.
 *   summaries: device records as built above (read only).
 *   sel:       device int32 [B, Hkv, budget], written: the min(s, #candidates)
 *              best candidate blocks in ascending order, then -1.
 *   scores:    optional device fp32 [B, Hkv, T_max/L], written: sigma_b for
 *              candidates, -inf for every other index.
 * With subspace factors a first small launch writes U_Q^T q of every query
 * head into the workspace (its size includes that region).                     */
cobs_status_t cobs_select(const cobs_config_t* cfg, const float* q, const void* summaries,
                          const int32_t* seq_lens, int32_t* sel, float* scores, void* ws,
                          size_t ws_bytes, void* stream);

/* Exact-mass block selection: the Oracle Sparse Attention ranking of Sec. 3.5.
 * For every block b and query head g of a KV head, the exact log-mass
 * l_b^g = ln sum_{t in b} exp(c q_g . k_t) over the block's T-clamped tokens
 * (eq. bg-defs) replaces the descriptor estimate; normaliser, group score
 * (eq. prop-gqa in log form), candidates, top-s and outputs are those of
 * cobs_select.  Reads every key of the cache once (a recall ceiling for the
 * summary-based selectors, not a decode-time path).
 *   kv:   bf16 keys only (COBS_ERR_UNSUPPORTED for fp32); V is not read.
 *   ws:   cobs_workspace_bytes(cfg, COBS_OP_SELECT_EXACT), zero-filled before
 *         its first use and left zeroed by every call.
 *   q, seq_lens, sel, scores: as for cobs_select.                              */
cobs_status_t cobs_select_exact(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                                const int32_t* seq_lens, int32_t* sel, float* scores, void* ws,
                                size_t ws_bytes, void* stream);

/* Block-sparse decode attention (eq. oracle-true over the kept-token union).
 *   sel:  device int32 [B, Hkv, budget] block ids.  The longest prefix that is
 *         strictly ascending with every entry in [0, #candidates) is used; the
 *         entries after it (e.g. -1 padding) are ignored.
 *   out:  device fp32 [B, Hq, d], written.
 *   lse:  optional device fp32 [B, Hq], written: ln sum_{t in U} exp(c q.k_t).  */
cobs_status_t cobs_sparse_decode(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                                 const int32_t* seq_lens, const int32_t* sel, float* out,
                                 float* lse, void* ws, size_t ws_bytes, void* stream);

/* Quest block selection, an alternate selector for diagnostics (Sec. 6.4):
 * per block the element-wise minimum and maximum of its keys (eq.
 * rw-quest-box), per query head the box's largest inner product with the query
 * (eq. rw-quest-score), and c times that bound in place of l_b^g in the group
 * score; candidates, top-s and outputs as for cobs_select.  Reads every key
 * once.  Arguments and workspace (COBS_OP_SELECT_EXACT) as for
 * cobs_select_exact; bf16 keys only.                                           */
cobs_status_t cobs_select_quest(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                                const int32_t* seq_lens, int32_t* sel, float* scores, void* ws,
                                size_t ws_bytes, void* stream);

/* The decode attention split into the two branches a caller-side gate
 * combines (the selection and sliding-window branches of the NSA layout the
 * paper builds on, Sec. 2): out_sel / lse_sel over the selected blocks' tokens
 * before the window start, out_win / lse_win over the last w tokens.  The two
 * token sets are disjoint and their union is cobs_sparse_decode's, so merging
 * the pairs by log-sum-exp gives its out and lse.  An empty branch gives 0 and
 * -inf.  Arguments as for cobs_sparse_decode (same workspace size); bf16 K/V
 * only (COBS_ERR_UNSUPPORTED for fp32).  lse_sel, lse_win optional.           */
cobs_status_t cobs_sparse_decode_branches(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                                          const int32_t* seq_lens, const int32_t* sel, float* out_sel,
                                          float* lse_sel, float* out_win, float* lse_win, void* ws,
                                          size_t ws_bytes, void* stream);

/* One decode step: refresh the record of the block holding token T-1 (the
 * caller has already written the new token's K/V at position T-1 and counted
 * it in seq_lens), then select and attend.  Equivalent to
 * cobs_build_block_stats on block (T-1)/L, cobs_select and cobs_sparse_decode.
 * With bf16 K/V, rank <= 4, L = 64 and full-space factors it is two launches
 * (the selector's workgroup that scores the newest block recomputes its record
 * first), else three (with subspace factors the newest block's build launch also
 * writes U_Q^T q).
 *   summaries: in/out.   sel: optional device int32 [B, Hkv, budget] output.    */
cobs_status_t cobs_decode_step(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                               const int32_t* seq_lens, void* summaries, int32_t* sel,
                               float* out, float* lse, void* ws, size_t ws_bytes, void* stream);

/* Size of the library's own workspace for cobs_decode_step_noalloc, per GPU. */
#define COBS_NOALLOC_SCRATCH_BYTES (32u << 20)

/* cobs_decode_step without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The workspace is a static device array
 * of the library, COBS_NOALLOC_SCRATCH_BYTES on every GPU the library runs on,
 * held until the process ends; the call itself allocates nothing.
 *   Arguments and results: as for cobs_decode_step.
 *   Errors: COBS_ERR_WORKSPACE if cobs_workspace_bytes(cfg, COBS_OP_STEP)
 *   exceeds COBS_NOALLOC_SCRATCH_BYTES (32 MiB holds e.g. B = 32, Hq = 32,
 *   Hkv = 8, T_max = 32768, budget 85; B = 8, Hq = 64, Hkv = 8, T_max = 131072);
 *   COBS_ERR_HIP if the array's address cannot be obtained.
 *   Each call first clears its arrival counters in the array (one extra small
 *   launch), so a call needs no state from the previous one.  Every call on one
 *   GPU uses the same array: calls that overlap in time on one GPU (different
 *   streams, or host threads) race and must be serialised by the caller.      */
cobs_status_t cobs_decode_step_noalloc(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                                       const int32_t* seq_lens, void* summaries, int32_t* sel,
                                       float* out, float* lse, void* stream);

/* The mean-pool compression branch (Sec. 2 branch (i), kept by COBS beside its
 * covariance selector, Sec. 5.2), for a caller-side gate with the selection and
 * window branches: per query head, softmax attention over the pooled blocks,
 * block b entering as one key (its stored mean key) with one value (its stored
 * mean value), for every block b < ceil(T/L):
 *   out_g = sum_b exp(c q_g . kbar_b) vbar_b / sum_b exp(c q_g . kbar_b),
 *   lse_g = ln sum_b exp(c q_g . kbar_b).
 * Needs records built with COBS_OPT_VALUE_MEAN (COBS_ERR_INVALID_ARG otherwise).
 *   q:    device fp32 [B, Hq, d].   summaries: records (read only).
 *   out:  device fp32 [B, Hq, d], written; a row with T = 0 gives 0.
 *   lse:  optional device fp32 [B, Hq], written (-inf for T = 0).
 * One workgroup per (batch row, KV head); no workspace.                         */
cobs_status_t cobs_compression_branch(const cobs_config_t* cfg, const float* q, const void* summaries,
                                      const int32_t* seq_lens, float* out, float* lse, void* stream);

/* FP4 E2M1 encoder used for descriptor storage (Sec. 5.5), exposed so the
 * rounding rule can be checked on its own.
 *   x:      device fp32 [num_vectors, dim], dim even, 2 <= dim <= 4096.
 *   codes:  device uint8 [num_vectors, dim/2], written (element 2j low nibble).
 *   scales: device fp32 [num_vectors], written.                                 */
cobs_status_t cobs_pack_e2m1(const float* x, int64_t num_vectors, int32_t dim, uint8_t* codes,
                             float* scales, void* stream);

/* Static string for a status code. */
const char* cobs_status_string(cobs_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* COBS_H */
