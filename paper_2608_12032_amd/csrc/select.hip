// Shortest-prefix block selection (Sec. 4.1, Eq. (3)) and CSR emission.
//
// Three launches:
//   select_rows  one workgroup per row r = (b*H + h)*n_q + i.  The row's n_k
//                masses become 64-bit keys  (~bits(m) << 32) | j : masses are
//                >= 0, so their float bits order like the values and the
//                complemented bits sort descending; the low word breaks ties
//                by the smaller block index.  A bitonic sort in LDS, then an
//                fp64 inclusive scan of the sorted masses; the prefix length
//                s is the first position whose cumulative mass reaches tau.
//                tau >= 1 keeps every key block that holds a real key.  In
//                the fixed-ratio top-k mode (topk > 0; the ablation of Sec. 5,
//                Table 2) the scan is skipped and s = min(topk, blocks holding
//                a real key).  The kept blocks are flagged in a per-row byte
//                mask and s is stored as the row's count.
//   scan_counts  one workgroup: exclusive scan of the counts -> row_ptr.
//   compact_rows one workgroup per row: the flagged block ids, ascending, at
//                col_idx[row_ptr[r] ...].
// Every step is per row or a fixed-order scan: results are deterministic.
#include "common.hpp"
#include "launch.hpp"

namespace losa {

namespace {

constexpr int SEL_T = 256;

__device__ __forceinline__ float clean_mass(float m) { return (m > 0.f) ? m : 0.f; }  // NaN -> 0

template <int NKP>
__global__ void __launch_bounds__(SEL_T)
    select_rows_kernel(const float* __restrict__ mass, int n_q, int n_k, int n_kv, int N,
                       int block_q, float tau, int topk, int32_t* __restrict__ counts,
                       uint8_t* __restrict__ flags) {
  constexpr int PER = NKP / SEL_T > 0 ? NKP / SEL_T : 1;  // sorted slots per thread
  __shared__ uint64_t key[NKP];
  __shared__ double tot[SEL_T];
  __shared__ int s_found;
  const int t = threadIdx.x;
  const int r = blockIdx.x;
  const int i = r % n_q;
  const float* mrow = mass + (size_t)r * n_k;
  uint8_t* frow = flags + (size_t)r * n_k;

  if (i * block_q >= N) {  // query block made only of padding: empty row
    for (int j = t; j < n_k; j += SEL_T) frow[j] = 0;
    if (t == 0) counts[r] = 0;
    return;
  }
  if (topk <= 0 && tau >= 1.0f) {
    for (int j = t; j < n_k; j += SEL_T) frow[j] = (j < n_kv) ? 1 : 0;
    if (t == 0) counts[r] = n_kv;
    return;
  }

  for (int p = t; p < NKP; p += SEL_T) {
    if (p < n_k) {
      const uint32_t bits = __float_as_uint(clean_mass(mrow[p]));
      key[p] = ((uint64_t)(~bits) << 32) | (uint32_t)p;
    } else {
      key[p] = ~0ull;  // sorts after every real block
    }
  }
  __syncthreads();

  // bitonic sort, ascending
  for (int size = 2; size <= NKP; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int c = t; c < NKP / 2; c += SEL_T) {
        const int lo = 2 * c - (c & (stride - 1));
        const int hi = lo + stride;
        const bool up = ((lo & size) == 0);
        const uint64_t a = key[lo], b = key[hi];
        if ((a > b) == up) {
          key[lo] = b;
          key[hi] = a;
        }
      }
      __syncthreads();
    }
  }

  if (topk > 0) {  // fixed-ratio top-k: the first min(topk, n_kv) of the order
    const int s = topk < n_kv ? topk : n_kv;
    for (int p = t; p < n_k; p += SEL_T) {
      const int j = (int)(uint32_t)key[p];
      frow[j] = (p < s) ? 1 : 0;
    }
    if (t == 0) counts[r] = s;
    return;
  }

  // fp64 inclusive scan: thread t owns sorted slots [t*PER, t*PER + PER)
  double loc[PER];
  double run = 0.0;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int p = t * PER + u;
    double m = 0.0;
    if (p < NKP && p < n_k) m = (double)__uint_as_float(~(uint32_t)(key[p] >> 32));
    run += m;
    loc[u] = run;
  }
  tot[t] = run;
  if (t == 0) s_found = 0x7fffffff;
  __syncthreads();
  for (int off = 1; off < SEL_T; off <<= 1) {  // Hillis-Steele over thread totals
    const double add = (t >= off) ? tot[t - off] : 0.0;
    __syncthreads();
    tot[t] += add;
    __syncthreads();
  }
  const double base = (t > 0) ? tot[t - 1] : 0.0;
  // s = 1 + the first sorted position whose cumulative mass reaches tau
  int first = 0x7fffffff;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int p = t * PER + u;
    if (p < n_k && base + loc[u] >= (double)tau && p + 1 < first) first = p + 1;
  }
  if (first != 0x7fffffff) atomicMin(&s_found, first);
  __syncthreads();
  const int s = s_found;
  if (s == 0x7fffffff) {  // threshold never reached (masses sum below tau): keep every real block
    for (int j = t; j < n_k; j += SEL_T) frow[j] = (j < n_kv) ? 1 : 0;
    if (t == 0) counts[r] = n_kv;
    return;
  }
  for (int p = t; p < n_k; p += SEL_T) {
    const int j = (int)(uint32_t)key[p];
    frow[j] = (p < s) ? 1 : 0;
  }
  if (t == 0) counts[r] = s;
}

constexpr int SCAN_T = 1024;

__global__ void __launch_bounds__(SCAN_T)
    scan_counts_kernel(const int32_t* __restrict__ counts, int rows, int32_t* __restrict__ row_ptr) {
  __shared__ int32_t tot[SCAN_T];
  const int t = threadIdx.x;
  const int per = (rows + SCAN_T - 1) / SCAN_T;
  const int lo = min(rows, t * per), hi = min(rows, lo + per);
  int32_t s = 0;
  for (int r = lo; r < hi; ++r) s += counts[r];
  tot[t] = s;
  __syncthreads();
  for (int off = 1; off < SCAN_T; off <<= 1) {
    const int32_t add = (t >= off) ? tot[t - off] : 0;
    __syncthreads();
    tot[t] += add;
    __syncthreads();
  }
  int32_t run = (t > 0) ? tot[t - 1] : 0;
  for (int r = lo; r < hi; ++r) {
    row_ptr[r] = run;
    run += counts[r];
  }
  if (t == SCAN_T - 1) row_ptr[rows] = tot[SCAN_T - 1];
}

__global__ void __launch_bounds__(SEL_T)
    compact_rows_kernel(const uint8_t* __restrict__ flags, const int32_t* __restrict__ row_ptr,
                        int n_k, int32_t* __restrict__ col_idx) {
  __shared__ int wtot[SEL_T / 64];
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int r = blockIdx.x;
  const uint8_t* frow = flags + (size_t)r * n_k;
  int out = row_ptr[r];
  for (int c0 = 0; c0 < n_k; c0 += SEL_T) {
    const int j = c0 + t;
    const bool f = (j < n_k) && frow[j];
    const uint64_t ball = __ballot(f);
    const int before = __popcll(ball & ((1ull << lane) - 1ull));
    if (lane == 0) wtot[w] = __popcll(ball);
    __syncthreads();
    int woff = 0, all = 0;
#pragma unroll
    for (int ww = 0; ww < SEL_T / 64; ++ww) {
      woff += (ww < w) ? wtot[ww] : 0;
      all += wtot[ww];
    }
    if (f) col_idx[out + woff + before] = j;
    out += all;
    __syncthreads();
  }
}

template <int NKP>
void launch_sel(const float* mass, int rows, int n_q, int n_k, int n_kv, int N, int block_q,
                float tau, int topk, int32_t* counts, uint8_t* flags, hipStream_t stream) {
  hipLaunchKernelGGL(select_rows_kernel<NKP>, dim3(rows), dim3(SEL_T), 0, stream, mass, n_q, n_k,
                     n_kv, N, block_q, tau, topk, counts, flags);
}

}  // namespace

size_t select_workspace_bytes(int rows, int n_k) {
  const size_t counts = ((size_t)rows * 4 + 255) & ~(size_t)255;
  return counts + (size_t)rows * n_k;
}

int select_max_nk() { return 4096; }

hipError_t launch_select(const float* mass, int B, int H, int N, int block_q, int block_k,
                         float tau, int topk, int32_t* row_ptr, int32_t* col_idx, void* workspace,
                         hipStream_t stream) {
  const int n_pad = padded_len(N, block_q, block_k);
  const int n_q = n_pad / block_q, n_k = n_pad / block_k;
  const int n_kv = (N + block_k - 1) / block_k;
  const int rows = B * H * n_q;
  int32_t* counts = static_cast<int32_t*>(workspace);
  uint8_t* flags =
      static_cast<uint8_t*>(workspace) + (((size_t)rows * 4 + 255) & ~(size_t)255);
  if (n_k <= 64) launch_sel<64>(mass, rows, n_q, n_k, n_kv, N, block_q, tau, topk, counts, flags, stream);
  else if (n_k <= 256) launch_sel<256>(mass, rows, n_q, n_k, n_kv, N, block_q, tau, topk, counts, flags, stream);
  else if (n_k <= 1024) launch_sel<1024>(mass, rows, n_q, n_k, n_kv, N, block_q, tau, topk, counts, flags, stream);
  else if (n_k <= 4096) launch_sel<4096>(mass, rows, n_q, n_k, n_kv, N, block_q, tau, topk, counts, flags, stream);
  else return hipErrorInvalidValue;
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(scan_counts_kernel, dim3(1), dim3(SCAN_T), 0, stream, counts, rows, row_ptr);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(compact_rows_kernel, dim3(rows), dim3(SEL_T), 0, stream, flags, row_ptr, n_k,
                     col_idx);
  return hipGetLastError();
}

}  // namespace losa
