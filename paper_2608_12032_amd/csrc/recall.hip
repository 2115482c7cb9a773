// Recall of a frozen support (Sec. 3.1, Eq. (2)), measured on the block
// masses of a later step: how much attention mass the support fixed at the
// construction step still captures (the quantity behind the paper's
// frozen-pattern analysis, Sec. 3.3).
//
//   recall_rows   per row r = (b*H + h)*n_q + i: sum over the distinct ids j of
//                 Omega_r inside [0, n_k) of mass[r][j]; masses of a query
//                 block sum to one, so this is Eq. (2) restricted to block i.
//   recall_heads  per (b, h): sum_i R_i * kept_i / sum_i R_i * total_i, with
//                 R_i the valid rows of query block i and total_i the row's
//                 mass sum (Eq. (2)'s M(i, j) = R_i * mass(i, j)).
//
// Two launches.  recall_rows_kernel: one workgroup per row flags the row's
// ids in LDS (a repeated id counts once, stray ids are dropped, row bounds are
// clamped to the col_idx allocation) and sums the flagged and all masses in
// fp64 in a fixed order; the fp64 pair goes to the workspace.
// recall_heads_kernel: one wave per head reduces its rows in a fixed order.
// No atomics: results are bitwise repeatable.
#include "common.hpp"
#include "launch.hpp"

namespace losa {

namespace {

constexpr int RT = 256;  // threads of the per-row workgroup

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__global__ void __launch_bounds__(RT)
    recall_rows_kernel(const float* __restrict__ mass, int n_k, const int32_t* __restrict__ row_ptr,
                       const int32_t* __restrict__ col_idx, int64_t col_len,
                       double* __restrict__ kept_tot, float* __restrict__ recall_rows) {
  __shared__ uint8_t flag[kSparseFwdMaxNk];
  __shared__ double part[2][RT / 64];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int r = blockIdx.x;
  const float* mrow = mass + (size_t)r * n_k;
  for (int j = t; j < n_k; j += RT) flag[j] = 0;
  __syncthreads();
  int64_t e0 = row_ptr[r], e1 = row_ptr[r + 1];
  e0 = e0 < 0 ? 0 : (e0 > col_len ? col_len : e0);
  e1 = e1 < e0 ? e0 : (e1 > col_len ? col_len : e1);
  for (int64_t e = e0 + t; e < e1; e += RT) {
    const int j = col_idx[e];
    if (j >= 0 && j < n_k) flag[j] = 1;
  }
  __syncthreads();
  double kept = 0.0, tot = 0.0;
  for (int j = t; j < n_k; j += RT) {
    const double m = (double)mrow[j];
    tot += m;
    if (flag[j]) kept += m;
  }
  kept = wave_sum_f64(kept);
  tot = wave_sum_f64(tot);
  if (lane == 0) {
    part[0][w] = kept;
    part[1][w] = tot;
  }
  __syncthreads();
  if (t == 0) {
    double k2 = 0.0, t2 = 0.0;
#pragma unroll
    for (int x = 0; x < RT / 64; ++x) {
      k2 += part[0][x];
      t2 += part[1][x];
    }
    kept_tot[2 * (size_t)r] = k2;
    kept_tot[2 * (size_t)r + 1] = t2;
    if (recall_rows != nullptr) recall_rows[r] = (float)k2;
  }
}

__global__ void __launch_bounds__(64)
    recall_heads_kernel(const double* __restrict__ kept_tot, int n_q, int N, int block_q,
                        float* __restrict__ recall_heads) {
  const int bh = blockIdx.x;
  const int lane = threadIdx.x;
  double num = 0.0, den = 0.0;
  for (int i = lane; i < n_q; i += 64) {
    const int rows_valid = max(0, min(block_q, N - i * block_q));
    const size_t r = (size_t)bh * n_q + i;
    num += rows_valid * kept_tot[2 * r];
    den += rows_valid * kept_tot[2 * r + 1];
  }
  num = wave_sum_f64(num);
  den = wave_sum_f64(den);
  if (lane == 0) recall_heads[bh] = den > 0.0 ? (float)(num / den) : 0.f;
}

}  // namespace

size_t recall_workspace_bytes(int rows) { return (size_t)rows * 2 * sizeof(double); }

hipError_t launch_recall(const float* mass, int B, int H, int N, int block_q, int n_q, int n_k,
                         const int32_t* row_ptr, const int32_t* col_idx, int64_t col_len,
                         float* recall_rows, float* recall_heads, void* workspace,
                         hipStream_t stream) {
  const int BH = B * H;
  const int rows = BH * n_q;
  double* kept_tot = static_cast<double*>(workspace);
  hipLaunchKernelGGL(recall_rows_kernel, dim3(rows), dim3(RT), 0, stream, mass, n_k, row_ptr,
                     col_idx, col_len, kept_tot, recall_rows);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || recall_heads == nullptr) return err;
  hipLaunchKernelGGL(recall_heads_kernel, dim3(BH), dim3(64), 0, stream, kept_tot, n_q, N, block_q,
                     recall_heads);
  return hipGetLastError();
}

}  // namespace losa
