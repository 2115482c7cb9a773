/*
 * losa.h -- C ABI of liblosa.so, the MI355X (gfx950) hot path of LoSA
 * ("Near-Lossless Sparse Attention for Training-Free Video Diffusion
 * Acceleration"): exact block masses at the construction step, the
 * shortest-prefix block selection, and block-sparse attention over the frozen
 * support.
 *
 * Conventions shared by every call
 * --------------------------------
 * - All tensor pointers are caller-owned HIP DEVICE memory (16-byte aligned)
 *   unless stated otherwise.  The library never allocates device memory and
 *   keeps no state between calls except a thread-local error string, and for
 *   losa_sparse_attn_fwd_noalloc a scratch array per GPU (reserved when the
 *   library's code is loaded on that GPU) with a table of its addresses.
 * - Q, K, V, O are contiguous [B][H][N_pad][d] in the element type `dtype`,
 *   N_pad = N rounded up to max(block_q, block_k).  Token positions n >= N
 *   are padding: as keys they never enter a softmax; as queries they are left
 *   out of every block mass and their output rows are written as 0 (lse as
 *   -inf).  Padding rows of Q/K/V may hold any finite values.
 * - n_q = N_pad / block_q query blocks and n_k = N_pad / block_k key/value
 *   blocks per head (the partition of Sec. 3.1); row r = (b*H + h)*n_q + i
 *   addresses query block i of head h in batch b (a classifier-free-guidance
 *   branch is simply another b).
 * - `scale` (> 0) multiplies Q K^T before the softmax; the method uses 1/sqrt(d).
 * - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued
 *   asynchronously; outputs are valid once the stream has reached that point.
 *   No call allocates, synchronizes or enqueues a memset, and each launches
 *   only on `stream`, so calls can be captured into a HIP graph and replayed
 *   (tested for losa_construct, losa_select_blocks, losa_select_blocks_topk,
 *   losa_sparse_attn_fwd and both losa_calibrate_mass schemes, which also set
 *   their kernel's dynamic LDS size on the host).
 * - Validation is synchronous and happens before any HIP call: on an error
 *   nothing is launched, outputs are untouched, and losa_last_error() holds a
 *   description.  Launch failures return LOSA_ERR_HIP.
 * - Supported: dtype BF16 or F32, d in {64, 128}, block_q in {64, 128} and
 *   block_k either equal to block_q or 32 (the paper's rectangular setting,
 *   Sec. 5.1: 128-row query blocks, 32-key key blocks).  Other valid
 *   combinations return LOSA_ERR_UNSUPPORTED.
 * - Calls are deterministic: the same inputs give bitwise identical outputs.
 */
#ifndef LOSA_H
#define LOSA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LOSA_OK = 0,
  LOSA_ERR_NULL_POINTER = 1,  /* a required pointer is NULL                              */
  LOSA_ERR_INVALID_SHAPE = 2, /* B, H, N, d <= 0; block not a power of two in [16, 256];
                                 sizes overflow the 32-bit index ranges of the kernels    */
  LOSA_ERR_INVALID_TAU = 3,   /* tau is NaN or not in (0, 1]                              */
  LOSA_ERR_ALIGNMENT = 4,     /* a tensor pointer is not 16-byte aligned                  */
  LOSA_ERR_UNSUPPORTED = 5,   /* valid, but not implemented (see "Supported" above)       */
  LOSA_ERR_CAPACITY = 6,      /* col_idx capacity or workspace too small                  */
  LOSA_ERR_HIP = 7            /* a HIP runtime / launch error; see losa_last_error()      */
} losa_status;

typedef enum {
  LOSA_DTYPE_F32 = 0,
  LOSA_DTYPE_BF16 = 1,
  /* not element types: they give losa_dtype the range of int, so that any int
     a caller passes is a value of the type and is rejected with
     LOSA_ERR_UNSUPPORTED instead of being out of the enumeration's range */
  LOSA_DTYPE_RANGE_MIN_ = -2147483647 - 1,
  LOSA_DTYPE_RANGE_MAX_ = 2147483647
} losa_dtype;

/*
 * Exact block attention masses of one dense step (Sec. 3.1, Eq. (1); used at
 * the construction step t0 of Sec. 4.1).
 *
 * For every (b, h, i) with R_i >= 1 valid query rows:
 *   mass[b][h][i][j] = (1/R_i) * sum_{q in B^Q_i, q < N} sum_{k in B^K_j, k < N} A(q, k),
 *   A(q, .) = softmax over the N valid keys of scale * Q[q] . K[k],
 * i.e. Eq. (1)'s M(i, j) divided by R_i, so each row of `mass` sums to 1 (the
 * paper's threshold theta*R then reads mass >= theta).  Rows of query blocks
 * with no valid query are all zero; key blocks with no valid key get 0.
 *
 * q, k       [B][H][N_pad][d] of `dtype` (read only).
 * mass       out, fp32 [B][H][n_q][n_k].
 * lse        out, nullable, fp32 [B][H][N_pad]: natural-log logsumexp of the
 *            scaled scores of each query over all valid keys; -inf on padding.
 * workspace  bf16, optional.  NULL: two sweeps over the keys per query block,
 *            the first for lse, the second for the masses; no extra memory.
 *            Non-NULL: one sweep that also stores, for every query q and key
 *            block j, log2 of q's unnormalised probability sum over block j
 *            (4 bytes each); a reduction with lse then gives the masses.  It
 *            must hold at least one head's share, which is
 *            losa_workspace_bytes(0, dtype, 1, 1, N, d, block_q, block_k);
 *            heads are processed as many at a time as it holds, and
 *            losa_workspace_bytes(0, ...) suggests room for all of them, up to
 *            16 GiB.  Contents on entry are ignored and overwritten.  f32:
 *            ignored (two sweeps).
 * Arithmetic: bf16 inputs use bf16 matrix-core products with fp32
 * accumulation; f32 inputs use fp32 arithmetic, with each query's softmax
 * normaliser carried across 32-key chunks in fp64.  Both bf16 schemes compute
 * the same scores; their masses differ only by fp32 rounding.
 */
losa_status losa_calibrate_mass(const void* q, const void* k, losa_dtype dtype, int B, int H,
                                int N, int d, int block_q, int block_k, float scale, float* mass,
                                float* lse, void* workspace, size_t workspace_bytes,
                                void* stream);

/*
 * Shortest-prefix selection of retained key blocks and its CSR storage
 * (Sec. 4.1, Eq. (3)).
 *
 * For each row r: order the row's key blocks by decreasing mass, ties by the
 * smaller block index (the paper leaves ties arbitrary); keep the shortest
 * prefix whose cumulative mass (summed in fp64) reaches tau (the exact fp32
 * value passed).  tau >= 1 keeps every key block that holds a valid key, so
 * the sparse forward then equals dense attention.  A row whose masses never
 * reach tau also keeps every such block.  Rows of query blocks with no valid
 * query are empty.  Masses that are negative or NaN count as 0.
 *
 * mass              fp32 [B][H][n_q][n_k] (e.g. from losa_calibrate_mass).
 * row_ptr           out, int32 [B*H*n_q + 1]: row_ptr[0] = 0, row_ptr[end] = nnz.
 * col_idx           out, int32: row r's kept block ids, strictly ascending, at
 *                   col_idx[row_ptr[r] .. row_ptr[r+1]).
 * col_idx_capacity  elements available at col_idx; must be >= B*H*n_q*n_k
 *                   (the worst case), checked before launching.
 * workspace         >= losa_workspace_bytes(1, ...) bytes of device memory.
 * nnz is produced on the device (row_ptr[B*H*n_q]); read it after a sync.
 */
losa_status losa_select_blocks(const float* mass, int B, int H, int N, int block_q, int block_k,
                               float tau, int32_t* row_ptr, int32_t* col_idx,
                               int64_t col_idx_capacity, void* workspace, size_t workspace_bytes,
                               void* stream);

/*
 * Fixed-ratio top-k selection: the rule the paper's selection ablation
 * compares against (Sec. 5, Table 2), a uniform budget of k key blocks per
 * query block instead of a retained-mass threshold.
 *
 * For each row r: the same order as losa_select_blocks (decreasing mass, ties
 * by the smaller block index); keep its first min(k, n_kv) blocks, n_kv the
 * key blocks holding a valid key.  Rows of query blocks with no valid query
 * are empty.  Arguments, CSR output, capacity and workspace exactly as for
 * losa_select_blocks (workspace: losa_workspace_bytes(1, ...)).  k < 1
 * returns LOSA_ERR_INVALID_SHAPE.  To match the coverage of a threshold
 * selection (as Table 2 does), pass k = round(nnz / (B*H*n_q)).
 */
losa_status losa_select_blocks_topk(const float* mass, int B, int H, int N, int block_q,
                                    int block_k, int k, int32_t* row_ptr, int32_t* col_idx,
                                    int64_t col_idx_capacity, void* workspace,
                                    size_t workspace_bytes, void* stream);

/*
 * Recall of a frozen support on the block masses of another step (Sec. 3.1,
 * Eq. (2)): how much attention mass the support fixed at the construction
 * step still captures later (the paper's frozen-pattern analysis, Sec. 3.3).
 *
 * mass          fp32 [B][H][n_q][n_k], e.g. losa_calibrate_mass of step t.
 * row_ptr, col_idx, col_idx_len   the support, with the conventions of
 *               losa_sparse_attn_fwd (ids in any order, a repeated id counts
 *               once, ids outside [0, n_k) ignored, row bounds clamped to
 *               [0, col_idx_len]).  n_k <= 4096.
 * recall_rows   out, nullable, fp32 [B*H*n_q]: per row the sum of its distinct
 *               retained masses (masses of a query block sum to one, so this is
 *               Eq. (2) restricted to that block); 0 for empty rows.
 * recall_heads  out, nullable, fp32 [B*H]: Eq. (2) per head,
 *               sum_i R_i * kept_i / sum_i R_i * total_i, R_i = valid rows of
 *               query block i, total_i = the row's mass sum.
 * workspace     >= losa_workspace_bytes(3, ...) bytes (per-row fp64 sums).
 * Sums are taken in fp64 in a fixed order: results are bitwise repeatable.
 */
losa_status losa_block_recall(const float* mass, int B, int H, int N, int block_q, int block_k,
                              const int32_t* row_ptr, const int32_t* col_idx, int64_t col_idx_len,
                              float* recall_rows, float* recall_heads, void* workspace,
                              size_t workspace_bytes, void* stream);

/*
 * Frozen-support block-sparse attention (Sec. 4.2, Eq. (4)).
 *
 * For every valid query q of query block i in head (b, h):
 *   O[q] = sum_{k in K(q)} softmax_{K(q)}(scale * Q[q] . K[k]) V[k],
 *   K(q) = union over j in col_idx[row_ptr[r] .. row_ptr[r+1]) of the valid
 *          keys of key block j,
 * i.e. the softmax is renormalised over the retained keys only.  Reused
 * unchanged across the later steps (Sec. 4.2): only Q, K, V change.
 *
 * q, k, v     [B][H][N_pad][d] of `dtype`.
 * row_ptr     int32 [B*H*n_q + 1]; col_idx int32 [col_idx_len].  A row's ids
 *             may come in any order; a repeated id counts once (K(q) is a set);
 *             ids outside [0, n_k) are ignored; row bounds are clamped to
 *             [0, col_idx_len], so a malformed CSR cannot make the kernel read
 *             outside col_idx.  n_k <= 4096, else LOSA_ERR_UNSUPPORTED.
 * o           out, [B][H][N_pad][d] of `dtype`.  Rows with an empty key set and
 *             padding rows are 0.
 * lse         out, nullable, fp32 [B][H][N_pad]: natural-log logsumexp over
 *             K(q) of the scaled scores; -inf for empty or padding rows.
 * workspace   >= losa_workspace_bytes(2, ...) bytes, rewritten by every call
 *             (bf16: a transposed copy of V in the kernel's tile layout,
 *             B*H*N_pad*d*2 bytes rounded up to 256, then the rows' dispatch
 *             order, 4*B*H*n_q bytes; f32: none).
 * Arithmetic (bf16): Q K^T and P V on bf16 matrix cores with fp32
 * accumulation, softmax in fp32, P rounded to bf16 for the P V product, O
 * rounded to bf16 once at the end.  f32: fp32 arithmetic, the softmax
 * normaliser carried across 32-key chunks in fp64.
 */
losa_status losa_sparse_attn_fwd(const void* q, const void* k, const void* v, losa_dtype dtype,
                                 int B, int H, int N, int d, int block_q, int block_k,
                                 float scale, const int32_t* row_ptr, const int32_t* col_idx,
                                 int64_t col_idx_len, void* o, float* lse, void* workspace,
                                 size_t workspace_bytes, void* stream);

/*
 * losa_sparse_attn_fwd for callers that cannot allocate device memory: code
 * running under HIP graph capture that may not call hipMalloc, tight serving
 * loops, harnesses that forbid allocation.  Same arguments, results and
 * kernels as losa_sparse_attn_fwd (bitwise the same output), without the
 * workspace: the bf16 forward's scratch (the transposed copy of V and the
 * rows' dispatch order, B*H*N_pad*d*2 bytes rounded up to 256 plus 4*B*H*n_q
 * bytes) lives in a device array the library holds, LOSA_NOALLOC_SCRATCH_BYTES
 * per GPU, reserved on each GPU the library runs on until the process ends.
 * Neither this call nor anything it calls allocates or frees memory.
 *
 * - A shape whose scratch exceeds LOSA_NOALLOC_SCRATCH_BYTES returns
 *   LOSA_ERR_CAPACITY before anything is launched (128 MiB holds, e.g., the
 *   Wan2.1-1.3B shape: 12 heads of 32,768 x 128; use losa_sparse_attn_fwd
 *   with a workspace for larger ones).
 * - The scratch of the current device is used; `stream` (if not NULL) must
 *   belong to that device, else LOSA_ERR_HIP.  The first call on a device
 *   looks up that device's copy of the array (a host-side table, no device
 *   memory); later calls reuse it.
 * - Every call on one GPU shares that GPU's scratch.  Calls that overlap in
 *   time on one GPU (other streams, or other host threads without ordering)
 *   race on it and give undefined results; order them on one stream.
 * - fp32 needs no scratch and runs exactly as losa_sparse_attn_fwd.
 */
#define LOSA_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
losa_status losa_sparse_attn_fwd_noalloc(const void* q, const void* k, const void* v,
                                         losa_dtype dtype, int B, int H, int N, int d,
                                         int block_q, int block_k, float scale,
                                         const int32_t* row_ptr, const int32_t* col_idx,
                                         int64_t col_idx_len, void* o, float* lse, void* stream);

/*
 * The construction step (Sec. 4.1; Sec. 5.1: one dense attention step that also
 * yields the exact block masses).  Step t0 is a dense step, so the sampler
 * needs its dense attention output anyway; this call returns it together with
 * the masses that losa_select_blocks turns into the frozen support.
 *
 * o     out, [B][H][N_pad][d] of `dtype`: dense attention over all N valid
 *       keys (Sec. 3.1), padding rows 0.
 * mass  out, fp32 [B][H][n_q][n_k]: as losa_calibrate_mass.
 * lse   out, nullable, fp32 [B][H][N_pad]: natural-log logsumexp of the scaled
 *       scores over all valid keys, -inf on padding.
 * workspace  bf16: required, at least one head's share, which is
 *       losa_workspace_bytes(4, dtype, 1, 1, N, d, block_q, block_k); heads
 *       are processed as many at a time as it holds, and
 *       losa_workspace_bytes(4, ...) suggests room for all of them, up to
 *       16 GiB.  f32: unused.
 * bf16 runs the sparse forward's kernel over every valid key block.  Besides
 * O and lse it stores, for every query and key block, log2 of the query's
 * unnormalised probability sum over the block (in the workspace); one
 * reduction with lse turns these into the masses.  The whole step costs one
 * dense attention plus a pass over 4 bytes per (query, key block), where the
 * separate calls would cost a dense attention plus the calibration's sweeps
 * over Q K^T.  o equals losa_sparse_attn_fwd over a full support bitwise;
 * mass and lse agree with losa_calibrate_mass to fp32 rounding.
 * f32 runs losa_calibrate_mass and a dense fp32 forward.
 */
losa_status losa_construct(const void* q, const void* k, const void* v, losa_dtype dtype, int B,
                           int H, int N, int d, int block_q, int block_k, float scale, void* o,
                           float* mass, float* lse, void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * Workspace bytes needed by: which = 0 losa_calibrate_mass (bf16: the suggested
 * size of its optional workspace), 1 losa_select_blocks and
 * losa_select_blocks_topk, 2 losa_sparse_attn_fwd, 3 losa_block_recall,
 * 4 losa_construct (the suggested size; the least it accepts is the value
 * for B = H = 1).  Returns 0 for invalid arguments (then the call itself
 * reports the error).
 */
size_t losa_workspace_bytes(int which, losa_dtype dtype, int B, int H, int N, int d, int block_q,
                            int block_k);

/* Static text for a status code ("LOSA_OK", ...). */
const char* losa_status_string(losa_status s);

/* Thread-local description of the last non-OK status returned on this thread. */
const char* losa_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int losa_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LOSA_H */
