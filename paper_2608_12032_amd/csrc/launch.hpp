// Internal launchers behind the C ABI (include/losa.h).  Every launcher only
// enqueues work on `stream`; argument validation happens in abi.cpp before
// any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace losa {

// Padded sequence length: N rounded up to the larger block size.
__host__ __device__ inline int padded_len(int N, int block_q, int block_k) {
  const int L = block_q > block_k ? block_q : block_k;
  return (N + L - 1) / L * L;
}

// blk = query block rows, blk_k = key block keys (blk, or 32)
// stat == nullptr: two sweeps over the keys, lse optional.
// stat != nullptr: one sweep that writes the block statistics
//   [B*H][n_k][n_pad] fp32 and lse (then required), then launch_stat_mass.
hipError_t launch_calibrate_bf16(int d, int blk, int blk_k, const void* q, const void* k, int B,
                                 int H, int N, int n_pad, float scale, float* mass, float* lse,
                                 float* stat, hipStream_t stream);
// Block masses [BH][n_q][n_k] from block statistics and natural-log lse.
hipError_t launch_stat_mass(int blk, int blk_k, const float* stat, const float* lse, int BH, int N,
                            int n_pad, float* mass, hipStream_t stream);
inline size_t stat_bytes_per_head(int n_pad, int blk_k) {
  return (size_t)(n_pad / blk_k) * n_pad * sizeof(float);
}
hipError_t launch_calibrate_f32(int d, int blk, int blk_k, const void* q, const void* k, int B,
                                int H, int N, int n_pad, float scale, float* mass, float* lse,
                                hipStream_t stream);
size_t calib_bf16_lds_bytes(int d, int blk, int n_k);

// topk > 0: keep the topk heaviest blocks of each row instead of the prefix reaching tau
hipError_t launch_select(const float* mass, int B, int H, int N, int block_q, int block_k,
                         float tau, int topk, int32_t* row_ptr, int32_t* col_idx, void* workspace,
                         hipStream_t stream);
size_t select_workspace_bytes(int rows, int n_k);
int select_max_nk();

hipError_t launch_sparse_fwd_bf16(int d, int blk, int blk_k, const void* q, const void* k,
                                  const void* v, int B, int H, int N, int n_pad, float scale,
                                  const int32_t* row_ptr, const int32_t* col_idx,
                                  int64_t col_len, void* o, float* lse, void* workspace,
                                  hipStream_t stream);
// dense attention over every valid key (row_ptr == nullptr for the f32 path)
// stat != nullptr: also the block statistics [B*H][n_k][n_pad] (log2 units)
hipError_t launch_dense_bf16(int d, int blk, int blk_k, const void* q, const void* k,
                             const void* v, int B, int H, int N, int n_pad, float scale, void* o,
                             float* lse, float* stat, void* workspace, hipStream_t stream);
hipError_t launch_sparse_fwd_f32(int d, int blk, int blk_k, const void* q, const void* k,
                                 const void* v, int B, int H, int N, int n_pad, float scale,
                                 const int32_t* row_ptr, const int32_t* col_idx, int64_t col_len,
                                 void* o, float* lse, hipStream_t stream);
size_t sparse_fwd_bf16_workspace(int B, int H, int n_pad, int d, int n_q);

// Recall of a frozen support (Eq. (2)): per row the retained and the total
// mass (fp64, in the workspace), then per head the row-weighted ratio.
hipError_t launch_recall(const float* mass, int B, int H, int N, int block_q, int n_q, int n_k,
                         const int32_t* row_ptr, const int32_t* col_idx, int64_t col_len,
                         float* recall_rows, float* recall_heads, void* workspace,
                         hipStream_t stream);
size_t recall_workspace_bytes(int rows);

// Largest n_k (key blocks per head) the sparse forward kernels accept: each
// workgroup keeps one flag per key block of its row in LDS.
constexpr int kSparseFwdMaxNk = 4096;

// Scratch held by the library for losa_sparse_attn_fwd_noalloc (a device
// array per GPU, noalloc.hip).  Must equal LOSA_NOALLOC_SCRATCH_BYTES.
constexpr size_t kNoAllocScratchBytes = (size_t)128 << 20;
// Device address of the current device's copy of the scratch array, looked up
// once per device.  Fails with hipErrorInvalidResourceHandle if `stream`
// (non-null) belongs to another device than the current one; `device`
// receives the current device.
hipError_t noalloc_scratch(hipStream_t stream, void** ptr, int* device);

}  // namespace losa
