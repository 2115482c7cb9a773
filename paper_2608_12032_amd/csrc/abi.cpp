// C ABI of liblosa.so: argument validation, workspace sizing, dispatch to the
// HIP launchers, and status reporting.  See include/losa.h for the contract.
#include "losa.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>

#include "launch.hpp"

static_assert(LOSA_NOALLOC_SCRATCH_BYTES == losa::kNoAllocScratchBytes,
              "the header and the library agree on the no-alloc scratch size");

namespace {

thread_local char g_err[512] = "";

losa_status fail(losa_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

bool pow2_in(int x, int lo, int hi) { return x >= lo && x <= hi && (x & (x - 1)) == 0; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Shape {
  int B, H, N, d, bq, bk;
  int n_pad, n_q, n_k;
  int64_t rows;
};

// Checks shared by every entry point.  Fills `s` on success.
losa_status check_shape(int B, int H, int N, int d, int bq, int bk, Shape* s) {
  if (B <= 0 || H <= 0 || N <= 0 || d <= 0)
    return fail(LOSA_ERR_INVALID_SHAPE, "B=%d H=%d N=%d d=%d must all be > 0", B, H, N, d);
  if (!pow2_in(bq, 16, 256) || !pow2_in(bk, 16, 256))
    return fail(LOSA_ERR_INVALID_SHAPE, "block_q=%d block_k=%d must be powers of two in [16,256]",
                bq, bk);
  const int64_t L = bq > bk ? bq : bk;
  const int64_t n_pad = (N + L - 1) / L * L;
  // kernels index one head with 32-bit byte offsets (fp32 elements at most)
  if (n_pad * (int64_t)d * 4 >= ((int64_t)1 << 31))
    return fail(LOSA_ERR_INVALID_SHAPE, "N_pad*d = %lld exceeds the per-head index range",
                (long long)(n_pad * d));
  const int64_t rows = (int64_t)B * H * (n_pad / bq);
  if (rows >= ((int64_t)1 << 31) || (int64_t)B * H >= 65536)
    return fail(LOSA_ERR_INVALID_SHAPE, "B*H*n_q = %lld rows is too many", (long long)rows);
  s->B = B;
  s->H = H;
  s->N = N;
  s->d = d;
  s->bq = bq;
  s->bk = bk;
  s->n_pad = (int)n_pad;
  s->n_q = (int)(n_pad / bq);
  s->n_k = (int)(n_pad / bk);
  s->rows = rows;
  return LOSA_OK;
}

losa_status check_supported(losa_dtype dtype, const Shape& s) {
  if (dtype != LOSA_DTYPE_F32 && dtype != LOSA_DTYPE_BF16)
    return fail(LOSA_ERR_UNSUPPORTED, "unknown dtype %d", (int)dtype);
  if (s.d != 64 && s.d != 128)
    return fail(LOSA_ERR_UNSUPPORTED, "head dim d=%d not supported (64 or 128)", s.d);
  if (s.bq != 64 && s.bq != 128)
    return fail(LOSA_ERR_UNSUPPORTED, "block_q=%d not supported (64 or 128)", s.bq);
  if (s.bk != s.bq && s.bk != 32)
    return fail(LOSA_ERR_UNSUPPORTED, "block_k=%d not supported (block_q=%d, or 32)", s.bk, s.bq);
  return LOSA_OK;
}

losa_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return LOSA_OK;
  return fail(LOSA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

size_t elem_bytes(losa_dtype dt) { return dt == LOSA_DTYPE_BF16 ? 2 : 4; }

constexpr size_t kMaxLds = 160 * 1024;

// Workspace of the one-sweep bf16 calibration and of the bf16 construction
// step for a group of G heads: the block statistics, the heads' lse, then
// (construction only) the dense forward's V^T.  Heads are processed G at a
// time; G follows from the bytes the caller gives.
constexpr size_t kStatGroupCap = (size_t)16 << 30;  // suggested size: up to 16 GiB of groups

size_t up256(size_t x) { return (x + 255) / 256 * 256; }

struct StatLayout {
  size_t lse, fwd, total;  // byte offsets of lse and V^T (statistics at 0), total size
};

StatLayout stat_layout(const Shape& s, int G, bool with_fwd) {
  StatLayout L;
  L.lse = up256((size_t)G * losa::stat_bytes_per_head(s.n_pad, s.bk));
  L.fwd = L.lse + up256((size_t)G * s.n_pad * sizeof(float));
  L.total = L.fwd + (with_fwd ? up256(losa::sparse_fwd_bf16_workspace(1, G, s.n_pad, s.d, s.n_q))
                              : 0);
  return L;
}

// bytes for one head; a workspace of x bytes holds min(B*H, x / this) heads
size_t stat_bytes_one_head(const Shape& s, bool with_fwd) {
  return stat_layout(s, 1, with_fwd).total;
}

size_t stat_bytes_suggested(const Shape& s, bool with_fwd) {
  const size_t one = stat_bytes_one_head(s, with_fwd);
  const int64_t BH = (int64_t)s.B * s.H;
  int64_t G = (int64_t)(kStatGroupCap / one);
  G = G < 1 ? 1 : (G > BH ? BH : G);
  return (size_t)G * one;
}

}  // namespace

extern "C" {

losa_status losa_calibrate_mass(const void* q, const void* k, losa_dtype dtype, int B, int H,
                                int N, int d, int block_q, int block_k, float scale, float* mass,
                                float* lse, void* workspace, size_t workspace_bytes,
                                void* stream) {
  if (!q || !k || !mass) return fail(LOSA_ERR_NULL_POINTER, "q, k and mass must be non-NULL");
  Shape s;
  losa_status st = check_shape(B, H, N, d, block_q, block_k, &s);
  if (st != LOSA_OK) return st;
  if (!std::isfinite(scale) || !(scale > 0.f))
    return fail(LOSA_ERR_INVALID_SHAPE, "scale must be finite and > 0");
  if (!aligned16(q) || !aligned16(k) || !aligned16(mass) || (lse && !aligned16(lse)))
    return fail(LOSA_ERR_ALIGNMENT, "tensor pointers must be 16-byte aligned");
  st = check_supported(dtype, s);
  if (st != LOSA_OK) return st;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (dtype == LOSA_DTYPE_BF16 && workspace != nullptr) {
    // one sweep over the keys writing block statistics, a group of heads at a time
    if (!aligned16(workspace)) return fail(LOSA_ERR_ALIGNMENT, "workspace must be 16-byte aligned");
    const size_t one = stat_bytes_one_head(s, false);
    if (workspace_bytes < one)
      return fail(LOSA_ERR_CAPACITY, "workspace_bytes=%zu < %zu (one head; NULL for no workspace)",
                  workspace_bytes, one);
    const int BH = B * H;
    const int G = (int)((size_t)BH < workspace_bytes / one ? (size_t)BH : workspace_bytes / one);
    const StatLayout L = stat_layout(s, G, false);
    char* ws = static_cast<char*>(workspace);
    const size_t head_bytes = (size_t)s.n_pad * d * 2;
    for (int bh0 = 0; bh0 < BH; bh0 += G) {
      const int g = BH - bh0 < G ? BH - bh0 : G;
      float* l = lse ? lse + (size_t)bh0 * s.n_pad : reinterpret_cast<float*>(ws + L.lse);
      st = hip_status(losa::launch_calibrate_bf16(
                          d, block_q, block_k, static_cast<const char*>(q) + bh0 * head_bytes,
                          static_cast<const char*>(k) + bh0 * head_bytes, 1, g, N, s.n_pad, scale,
                          mass + (size_t)bh0 * s.n_q * s.n_k, l, reinterpret_cast<float*>(ws), hs),
                      "losa_calibrate_mass");
      if (st != LOSA_OK) return st;
    }
    return LOSA_OK;
  }
  if (dtype == LOSA_DTYPE_BF16) {
    // no workspace: two sweeps over the keys
    if (losa::calib_bf16_lds_bytes(d, block_q, s.n_k) > kMaxLds)
      return fail(LOSA_ERR_UNSUPPORTED, "n_k=%d key blocks exceed the calibration LDS budget",
                  s.n_k);
    return hip_status(
        losa::launch_calibrate_bf16(d, block_q, block_k, q, k, B, H, N, s.n_pad, scale, mass, lse,
                                    nullptr, hs),
        "losa_calibrate_mass");
  }
  return hip_status(
      losa::launch_calibrate_f32(d, block_q, block_k, q, k, B, H, N, s.n_pad, scale, mass, lse, hs),
      "losa_calibrate_mass");
}

}  // extern "C"

namespace {

// Checks and launch shared by the threshold rule (topk = 0) and the
// fixed-ratio top-k rule (topk > 0).
losa_status select_common(const char* where, const float* mass, int B, int H, int N, int block_q,
                          int block_k, float tau, int topk, int32_t* row_ptr, int32_t* col_idx,
                          int64_t col_idx_capacity, void* workspace, size_t workspace_bytes,
                          void* stream) {
  if (!mass || !row_ptr || !col_idx || !workspace)
    return fail(LOSA_ERR_NULL_POINTER, "mass, row_ptr, col_idx and workspace must be non-NULL");
  Shape s;
  losa_status st = check_shape(B, H, N, 1, block_q, block_k, &s);
  if (st != LOSA_OK) return st;
  if (!aligned16(mass) || !aligned16(row_ptr) || !aligned16(col_idx) || !aligned16(workspace))
    return fail(LOSA_ERR_ALIGNMENT, "pointers must be 16-byte aligned");
  if (s.n_k > losa::select_max_nk())
    return fail(LOSA_ERR_UNSUPPORTED, "n_k=%d key blocks per row exceeds %d", s.n_k,
                losa::select_max_nk());
  const int64_t worst = s.rows * s.n_k;
  if (worst >= ((int64_t)1 << 31))
    return fail(LOSA_ERR_INVALID_SHAPE, "rows*n_k=%lld exceeds the int32 CSR range",
                (long long)worst);
  if (col_idx_capacity < worst)
    return fail(LOSA_ERR_CAPACITY, "col_idx_capacity=%lld < B*H*n_q*n_k=%lld",
                (long long)col_idx_capacity, (long long)worst);
  const size_t need = losa::select_workspace_bytes((int)s.rows, s.n_k);
  if (workspace_bytes < need)
    return fail(LOSA_ERR_CAPACITY, "workspace_bytes=%zu < %zu", workspace_bytes, need);
  return hip_status(losa::launch_select(mass, B, H, N, block_q, block_k, tau, topk, row_ptr,
                                        col_idx, workspace, static_cast<hipStream_t>(stream)),
                    where);
}

}  // namespace

extern "C" {

losa_status losa_select_blocks(const float* mass, int B, int H, int N, int block_q, int block_k,
                               float tau, int32_t* row_ptr, int32_t* col_idx,
                               int64_t col_idx_capacity, void* workspace, size_t workspace_bytes,
                               void* stream) {
  if (std::isnan(tau) || !(tau > 0.f) || tau > 1.f)
    return fail(LOSA_ERR_INVALID_TAU, "tau=%g must be in (0, 1]", (double)tau);
  return select_common("losa_select_blocks", mass, B, H, N, block_q, block_k, tau, 0, row_ptr,
                       col_idx, col_idx_capacity, workspace, workspace_bytes, stream);
}

losa_status losa_select_blocks_topk(const float* mass, int B, int H, int N, int block_q,
                                    int block_k, int k, int32_t* row_ptr, int32_t* col_idx,
                                    int64_t col_idx_capacity, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  if (k < 1) return fail(LOSA_ERR_INVALID_SHAPE, "k=%d must be >= 1", k);
  return select_common("losa_select_blocks_topk", mass, B, H, N, block_q, block_k, 1.0f, k,
                       row_ptr, col_idx, col_idx_capacity, workspace, workspace_bytes, stream);
}

losa_status losa_block_recall(const float* mass, int B, int H, int N, int block_q, int block_k,
                              const int32_t* row_ptr, const int32_t* col_idx, int64_t col_idx_len,
                              float* recall_rows, float* recall_heads, void* workspace,
                              size_t workspace_bytes, void* stream) {
  if (!mass || !row_ptr || !workspace)
    return fail(LOSA_ERR_NULL_POINTER, "mass, row_ptr and workspace must be non-NULL");
  if (col_idx_len < 0) return fail(LOSA_ERR_INVALID_SHAPE, "col_idx_len must be >= 0");
  if (col_idx_len > 0 && !col_idx)
    return fail(LOSA_ERR_NULL_POINTER, "col_idx is NULL but col_idx_len > 0");
  Shape s;
  losa_status st = check_shape(B, H, N, 1, block_q, block_k, &s);
  if (st != LOSA_OK) return st;
  if (!aligned16(mass) || !aligned16(row_ptr) || (col_idx && !aligned16(col_idx)) ||
      !aligned16(workspace) || (recall_rows && !aligned16(recall_rows)) ||
      (recall_heads && !aligned16(recall_heads)))
    return fail(LOSA_ERR_ALIGNMENT, "pointers must be 16-byte aligned");
  if (s.n_k > losa::kSparseFwdMaxNk)
    return fail(LOSA_ERR_UNSUPPORTED, "n_k=%d key blocks per row exceeds %d", s.n_k,
                losa::kSparseFwdMaxNk);
  const size_t need = losa::recall_workspace_bytes((int)s.rows);
  if (workspace_bytes < need)
    return fail(LOSA_ERR_CAPACITY, "workspace_bytes=%zu < %zu", workspace_bytes, need);
  return hip_status(losa::launch_recall(mass, B, H, N, block_q, s.n_q, s.n_k, row_ptr, col_idx,
                                        col_idx_len, recall_rows, recall_heads, workspace,
                                        static_cast<hipStream_t>(stream)),
                    "losa_block_recall");
}

}  // extern "C"

namespace {

// Argument checks of the sparse forward (both entry points).  Fills `s`.
losa_status fwd_checks(const void* q, const void* k, const void* v, losa_dtype dtype, int B, int H,
                       int N, int d, int block_q, int block_k, float scale,
                       const int32_t* row_ptr, const int32_t* col_idx, int64_t col_idx_len,
                       const void* o, const float* lse, Shape* s) {
  if (!q || !k || !v || !row_ptr || !o)
    return fail(LOSA_ERR_NULL_POINTER, "q, k, v, row_ptr and o must be non-NULL");
  if (col_idx_len < 0) return fail(LOSA_ERR_INVALID_SHAPE, "col_idx_len must be >= 0");
  if (col_idx_len > 0 && !col_idx)
    return fail(LOSA_ERR_NULL_POINTER, "col_idx is NULL but col_idx_len > 0");
  losa_status st = check_shape(B, H, N, d, block_q, block_k, s);
  if (st != LOSA_OK) return st;
  if (!std::isfinite(scale) || !(scale > 0.f))
    return fail(LOSA_ERR_INVALID_SHAPE, "scale must be finite and > 0");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) ||
      (lse && !aligned16(lse)) || !aligned16(row_ptr) || (col_idx && !aligned16(col_idx)))
    return fail(LOSA_ERR_ALIGNMENT, "pointers must be 16-byte aligned");
  st = check_supported(dtype, *s);
  if (st != LOSA_OK) return st;
  if (s->n_k > losa::kSparseFwdMaxNk)
    return fail(LOSA_ERR_UNSUPPORTED, "n_k=%d key blocks per head exceeds %d", s->n_k,
                losa::kSparseFwdMaxNk);
  return LOSA_OK;
}

}  // namespace

extern "C" {

losa_status losa_sparse_attn_fwd(const void* q, const void* k, const void* v, losa_dtype dtype,
                                 int B, int H, int N, int d, int block_q, int block_k,
                                 float scale, const int32_t* row_ptr, const int32_t* col_idx,
                                 int64_t col_idx_len, void* o, float* lse, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  Shape s;
  losa_status st = fwd_checks(q, k, v, dtype, B, H, N, d, block_q, block_k, scale, row_ptr,
                              col_idx, col_idx_len, o, lse, &s);
  if (st != LOSA_OK) return st;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (dtype == LOSA_DTYPE_BF16) {
    const size_t need = losa::sparse_fwd_bf16_workspace(B, H, s.n_pad, d, s.n_q);
    if (!workspace) return fail(LOSA_ERR_NULL_POINTER, "bf16 needs a workspace of %zu bytes", need);
    if (!aligned16(workspace)) return fail(LOSA_ERR_ALIGNMENT, "workspace must be 16-byte aligned");
    if (workspace_bytes < need)
      return fail(LOSA_ERR_CAPACITY, "workspace_bytes=%zu < %zu", workspace_bytes, need);
    return hip_status(losa::launch_sparse_fwd_bf16(d, block_q, block_k, q, k, v, B, H, N, s.n_pad, scale,
                                                   row_ptr, col_idx, col_idx_len, o, lse,
                                                   workspace, hs),
                      "losa_sparse_attn_fwd");
  }
  return hip_status(losa::launch_sparse_fwd_f32(d, block_q, block_k, q, k, v, B, H, N, s.n_pad, scale,
                                                row_ptr, col_idx, col_idx_len, o, lse, hs),
                    "losa_sparse_attn_fwd");
}

losa_status losa_sparse_attn_fwd_noalloc(const void* q, const void* k, const void* v,
                                         losa_dtype dtype, int B, int H, int N, int d, int block_q,
                                         int block_k, float scale, const int32_t* row_ptr,
                                         const int32_t* col_idx, int64_t col_idx_len, void* o,
                                         float* lse, void* stream) {
  Shape s;
  losa_status st = fwd_checks(q, k, v, dtype, B, H, N, d, block_q, block_k, scale, row_ptr,
                              col_idx, col_idx_len, o, lse, &s);
  if (st != LOSA_OK) return st;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (dtype == LOSA_DTYPE_BF16) {
    const size_t need = losa::sparse_fwd_bf16_workspace(B, H, s.n_pad, d, s.n_q);
    if (need > losa::kNoAllocScratchBytes)
      return fail(LOSA_ERR_CAPACITY,
                  "losa_sparse_attn_fwd_noalloc: this shape needs %zu bytes of scratch, more than "
                  "the %zu the library holds; use losa_sparse_attn_fwd with a workspace",
                  need, losa::kNoAllocScratchBytes);
    void* ws = nullptr;
    int dev = -1;
    const hipError_t e = losa::noalloc_scratch(hs, &ws, &dev);
    if (e == hipErrorInvalidResourceHandle)
      return fail(LOSA_ERR_HIP,
                  "losa_sparse_attn_fwd_noalloc: the stream belongs to another device than the "
                  "current device %d",
                  dev);
    st = hip_status(e, "losa_sparse_attn_fwd_noalloc (scratch lookup)");
    if (st != LOSA_OK) return st;
    return hip_status(losa::launch_sparse_fwd_bf16(d, block_q, block_k, q, k, v, B, H, N,
                                                   s.n_pad, scale, row_ptr, col_idx, col_idx_len,
                                                   o, lse, ws, hs),
                      "losa_sparse_attn_fwd_noalloc");
  }
  // fp32 needs no scratch: the same kernel as losa_sparse_attn_fwd
  return hip_status(losa::launch_sparse_fwd_f32(d, block_q, block_k, q, k, v, B, H, N, s.n_pad,
                                                scale, row_ptr, col_idx, col_idx_len, o, lse, hs),
                    "losa_sparse_attn_fwd_noalloc");
}

losa_status losa_construct(const void* q, const void* k, const void* v, losa_dtype dtype, int B,
                           int H, int N, int d, int block_q, int block_k, float scale, void* o,
                           float* mass, float* lse, void* workspace, size_t workspace_bytes,
                           void* stream) {
  if (!q || !k || !v || !o || !mass)
    return fail(LOSA_ERR_NULL_POINTER, "q, k, v, o and mass must be non-NULL");
  Shape s;
  losa_status st = check_shape(B, H, N, d, block_q, block_k, &s);
  if (st != LOSA_OK) return st;
  if (!std::isfinite(scale) || !(scale > 0.f))
    return fail(LOSA_ERR_INVALID_SHAPE, "scale must be finite and > 0");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(mass) ||
      (lse && !aligned16(lse)))
    return fail(LOSA_ERR_ALIGNMENT, "tensor pointers must be 16-byte aligned");
  st = check_supported(dtype, s);
  if (st != LOSA_OK) return st;
  if (s.n_k > losa::kSparseFwdMaxNk)
    return fail(LOSA_ERR_UNSUPPORTED, "n_k=%d key blocks per head exceeds %d", s.n_k,
                losa::kSparseFwdMaxNk);
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (dtype == LOSA_DTYPE_F32) {
    // fp32: the calibration kernel's own two sweeps, then the dense forward
    st = losa_calibrate_mass(q, k, dtype, B, H, N, d, block_q, block_k, scale, mass, lse,
                             nullptr, 0, stream);
    if (st != LOSA_OK) return st;
    return hip_status(losa::launch_sparse_fwd_f32(d, block_q, block_k, q, k, v, B, H, N, s.n_pad,
                                                  scale, nullptr, nullptr, 0, o, nullptr, hs),
                      "losa_construct");
  }
  // bf16: the dense forward writes O, lse and the block statistics; the masses
  // follow from one reduction.  A group of heads at a time.
  const size_t one = stat_bytes_one_head(s, true);
  if (!workspace) return fail(LOSA_ERR_NULL_POINTER, "bf16 needs a workspace of >= %zu bytes", one);
  if (!aligned16(workspace)) return fail(LOSA_ERR_ALIGNMENT, "workspace must be 16-byte aligned");
  if (workspace_bytes < one)
    return fail(LOSA_ERR_CAPACITY, "workspace_bytes=%zu < %zu (one head)", workspace_bytes, one);
  const int BH = B * H;
  const int G = (int)((size_t)BH < workspace_bytes / one ? (size_t)BH : workspace_bytes / one);
  const StatLayout L = stat_layout(s, G, true);
  char* ws = static_cast<char*>(workspace);
  float* stat = reinterpret_cast<float*>(ws);
  const size_t head_bytes = (size_t)s.n_pad * d * 2;
  for (int bh0 = 0; bh0 < BH; bh0 += G) {
    const int g = BH - bh0 < G ? BH - bh0 : G;
    const size_t off = bh0 * head_bytes;
    float* l = lse ? lse + (size_t)bh0 * s.n_pad : reinterpret_cast<float*>(ws + L.lse);
    st = hip_status(losa::launch_dense_bf16(d, block_q, block_k,
                                            static_cast<const char*>(q) + off,
                                            static_cast<const char*>(k) + off,
                                            static_cast<const char*>(v) + off, 1, g, N, s.n_pad,
                                            scale, static_cast<char*>(o) + off, l, stat,
                                            ws + L.fwd, hs),
                    "losa_construct (dense attention)");
    if (st != LOSA_OK) return st;
    st = hip_status(losa::launch_stat_mass(block_q, block_k, stat, l, g, N, s.n_pad,
                                           mass + (size_t)bh0 * s.n_q * s.n_k, hs),
                    "losa_construct (block masses)");
    if (st != LOSA_OK) return st;
  }
  return LOSA_OK;
}

size_t losa_workspace_bytes(int which, losa_dtype dtype, int B, int H, int N, int d, int block_q,
                            int block_k) {
  Shape s;
  if (check_shape(B, H, N, (which == 1 || which == 3) ? 1 : d, block_q, block_k, &s) != LOSA_OK)
    return 0;
  switch (which) {
    case 0:  // losa_calibrate_mass: optional for bf16 (NULL = two sweeps), unused for fp32
      return dtype == LOSA_DTYPE_BF16 ? stat_bytes_suggested(s, false) : 0;
    case 1:
      return losa::select_workspace_bytes((int)s.rows, s.n_k);
    case 2:
      return dtype == LOSA_DTYPE_BF16 ? losa::sparse_fwd_bf16_workspace(B, H, s.n_pad, d, s.n_q) : 0;
    case 3:
      return losa::recall_workspace_bytes((int)s.rows);
    case 4:  // losa_construct
      return dtype == LOSA_DTYPE_BF16 ? stat_bytes_suggested(s, true) : 0;
    default:
      return 0;
  }
}

const char* losa_status_string(losa_status s) {
  switch (s) {
    case LOSA_OK: return "LOSA_OK";
    case LOSA_ERR_NULL_POINTER: return "LOSA_ERR_NULL_POINTER";
    case LOSA_ERR_INVALID_SHAPE: return "LOSA_ERR_INVALID_SHAPE";
    case LOSA_ERR_INVALID_TAU: return "LOSA_ERR_INVALID_TAU";
    case LOSA_ERR_ALIGNMENT: return "LOSA_ERR_ALIGNMENT";
    case LOSA_ERR_UNSUPPORTED: return "LOSA_ERR_UNSUPPORTED";
    case LOSA_ERR_CAPACITY: return "LOSA_ERR_CAPACITY";
    case LOSA_ERR_HIP: return "LOSA_ERR_HIP";
  }
  return "LOSA_ERR_UNKNOWN";
}

const char* losa_last_error(void) { return g_err; }

int losa_version(void) { return 100; }

}  // extern "C"
