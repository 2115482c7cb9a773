// fp32 inputs: block masses (Sec. 3.1, Eq. (1)) and frozen-support attention
// (Sec. 4.2, Eq. (4)) with fp32 vector arithmetic throughout.
//
// fp32 is the small-workload path (no bf16 rounding anywhere), so these
// kernels keep to a plain per-thread layout: one thread holds one query row
// (its scaled q and its running output in registers), one workgroup owns one
// query block of BLK rows, and key/value rows are staged through LDS in chunks
// of 32 keys that every thread reads as broadcasts.  The workgroup holds KS
// copies of the block's rows (512 threads at d = 64, 256 at d = 128): copy s
// takes the row's s-th, (s+KS)-th, ... key block, and the KS partial softmax
// states (running max, sum, output) are merged in a fixed order at the end, so
// a row's keys are worked through by KS threads instead of one.  Masking and
// padding follow the bf16 kernels: keys >= N never enter a softmax, query rows
// >= N read Q as 0 and get O = 0 and lse = -inf, and so do rows whose key set
// is empty; col_idx entries outside [0, n_k) are ignored, a repeated entry
// counts once (the row's ids are flagged in LDS and listed in ascending
// order), and row bounds are clamped to [0, col_idx_len].
//
// Row sums.  The softmax normaliser is summed per 32-key chunk in fp32 and the
// chunk sums are carried in an fp64 running sum (and merged in fp64).  Added
// one by one to an fp32 accumulator, the many small terms of far keys fall
// below half its ulp and are lost: over 131k keys that biases the sum low by
// ~2e-4.
#include "common.hpp"
#include "launch.hpp"

namespace losa {

namespace {

constexpr int CK = 32;  // keys per LDS chunk

template <int D, int BLK>
struct F32Cfg {
  static constexpr int NT = D == 64 ? 512 : 256;  // threads
  static constexpr int KS = NT / BLK;             // copies of the block's rows (key splits)
  static constexpr int BUF = 32768;               // floats of the staging / merge buffer
  static_assert(KS * 2 * CK * D <= BUF && NT * D <= BUF, "staging and partial outputs fit");
};

// CK consecutive rows of D floats starting at row key0 of src, copied by the
// nts threads ts = 0..nts-1 of one key split
template <int D>
__device__ __forceinline__ void stage_rows(float* dst, const float* src, int key0, int ts,
                                           int nts) {
  for (int idx = ts; idx < CK * D / 4; idx += nts) {
    const int row = idx / (D / 4);
    const int col = (idx % (D / 4)) * 4;
    *reinterpret_cast<f32x4_t*>(dst + row * D + col) =
        *reinterpret_cast<const f32x4_t*>(src + (size_t)(key0 + row) * D + col);
  }
}

// The row's distinct valid key blocks, ascending, into list (dense: every
// block holding a valid key); returns their count.  flag and wcount are LDS
// scratch.  All NT threads call it.
template <int NT>
__device__ int block_list(int dense, int n_kv, int n_k, const int32_t* __restrict__ row_ptr,
                          const int32_t* __restrict__ col_idx, int64_t col_len, int r,
                          uint8_t* flag, uint16_t* list, int* wcount) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (dense) {
    for (int j = tid; j < n_kv; j += NT) list[j] = (uint16_t)j;
    __syncthreads();
    return n_kv;
  }
  for (int j = tid; j < n_k; j += NT) flag[j] = 0;
  __syncthreads();
  int64_t e0 = row_ptr[r], e1 = row_ptr[r + 1];
  e0 = e0 < 0 ? 0 : (e0 > col_len ? col_len : e0);
  e1 = e1 < e0 ? e0 : (e1 > col_len ? col_len : e1);
  for (int64_t e = e0 + tid; e < e1; e += NT) {
    const int j = col_idx[e];
    if (j >= 0 && j < n_k) flag[j] = 1;
  }
  __syncthreads();
  int nb = 0;
  for (int c0 = 0; c0 < n_k; c0 += NT) {
    const int j = c0 + tid;
    const bool f = (j < n_k) && flag[j] != 0;
    const uint64_t bal = __ballot(f);
    const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                 __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
    if (lane == 0) wcount[w] = __popcll(bal);
    __syncthreads();
    int before = 0, total = 0;
    for (int x = 0; x < NT / 64; ++x) {
      before += (x < w) ? wcount[x] : 0;
      total += wcount[x];
    }
    if (f) list[nb + before + below] = (uint16_t)j;
    nb += total;
    __syncthreads();
  }
  return nb;
}

template <int D, int BLK, int BK>
__global__ void __launch_bounds__((F32Cfg<D, BLK>::NT))
    sparse_fwd_f32_kernel(const float* __restrict__ Q, const float* __restrict__ K,
                          const float* __restrict__ V, const int32_t* __restrict__ row_ptr,
                          const int32_t* __restrict__ col_idx, int64_t col_len,
                          float* __restrict__ O, float* __restrict__ lse, int n_q, int n_k, int N,
                          int n_pad, float scale_log2, int dense) {
  using C = F32Cfg<D, BLK>;
  __shared__ __attribute__((aligned(16))) float buf[C::BUF];
  __shared__ uint8_t flag[kSparseFwdMaxNk];
  __shared__ uint16_t list[kSparseFwdMaxNk];
  __shared__ int wcount[C::NT / 64];
  __shared__ float mpart[C::NT];
  __shared__ double lpart[C::NT];
  const int tid = threadIdx.x;
  const int sp = tid / BLK;  // key split
  const int t = tid % BLK;   // row of the block
  const int r = blockIdx.x;
  const int bh = r / n_q;
  const int i = r - bh * n_q;
  const size_t head = (size_t)bh * n_pad * D;
  const int qrow = i * BLK + t;

  // padding query rows take Q = 0: their scores stay finite whatever the
  // padding holds (their output is written as 0 at the end)
  const bool qvalid = qrow < N;
  float q[D], o[D];
#pragma unroll
  for (int dd = 0; dd < D; ++dd) {
    q[dd] = qvalid ? Q[head + (size_t)qrow * D + dd] * scale_log2 : 0.f;
    o[dd] = 0.f;
  }
  float m = kNegBig;
  double l = 0.0;

  const int nb = block_list<C::NT>(dense, (N + BK - 1) / BK, n_k, row_ptr, col_idx, col_len, r,
                                   flag, list, wcount);
  float* Kc = buf + sp * 2 * CK * D;
  float* Vc = Kc + CK * D;
  const int rounds = (nb + C::KS - 1) / C::KS;
  for (int rd = 0; rd < rounds; ++rd) {
    const int x = rd * C::KS + sp;
    const int j = x < nb ? (int)list[x] : 0;
    const int kvalid = x < nb ? min(BK, N - j * BK) : 0;
    for (int c0 = 0; c0 < BK; c0 += CK) {  // the same trip count in every split
      __syncthreads();
      const bool live = c0 < kvalid;
      if (live) {
        stage_rows<D>(Kc, K + head, j * BK + c0, t, BLK);
        stage_rows<D>(Vc, V + head, j * BK + c0, t, BLK);
      }
      __syncthreads();
      if (!live) continue;  // the same for every thread of the split
      const int nk = min(CK, kvalid - c0);
      float s[CK];
      float mx = m;
#pragma unroll
      for (int kk = 0; kk < CK; ++kk) {
        float acc = 0.f;
#pragma unroll
        for (int dd = 0; dd < D; ++dd) acc = fmaf(q[dd], Kc[kk * D + dd], acc);
        s[kk] = kk < nk ? acc : -INFINITY;
        mx = fmaxf(mx, s[kk]);
      }
      const float alpha = fast_exp2(m - mx);
      m = mx;
      l *= (double)alpha;
#pragma unroll
      for (int dd = 0; dd < D; ++dd) o[dd] *= alpha;
      float part = 0.f;
#pragma unroll
      for (int kk = 0; kk < CK; ++kk) {
        const float p = fast_exp2(s[kk] - m);
        part += p;
#pragma unroll
        for (int dd = 0; dd < D; ++dd) o[dd] = fmaf(p, Vc[kk * D + dd], o[dd]);
      }
      l += (double)part;
    }
  }

  // merge the KS partial states of each row in split order: the common max,
  // then the sums and outputs rescaled to it.  Partial outputs go to LDS
  // d-major, so consecutive threads write consecutive words.
  __syncthreads();  // every split is done with its staging buffers
  mpart[tid] = m;
  lpart[tid] = l;
#pragma unroll
  for (int dd = 0; dd < D; ++dd) buf[dd * C::NT + tid] = o[dd];
  __syncthreads();
  if (sp != 0) return;
  float M = kNegBig;
  for (int s2 = 0; s2 < C::KS; ++s2) M = fmaxf(M, mpart[s2 * BLK + t]);
  float wgt[C::KS];
  double lt = 0.0;
#pragma unroll
  for (int s2 = 0; s2 < C::KS; ++s2) {
    wgt[s2] = fast_exp2(mpart[s2 * BLK + t] - M);
    lt += lpart[s2 * BLK + t] * (double)wgt[s2];
  }
  const float lf = (float)lt;
  const bool ok = qvalid && (lf > 0.f);
  const float inv = ok ? 1.0f / lf : 0.f;
#pragma unroll
  for (int dd = 0; dd < D; ++dd) {
    float acc = 0.f;
#pragma unroll
    for (int s2 = 0; s2 < C::KS; ++s2) acc = fmaf(buf[dd * C::NT + s2 * BLK + t], wgt[s2], acc);
    O[head + (size_t)qrow * D + dd] = acc * inv;
  }
  if (lse != nullptr) lse[(size_t)bh * n_pad + qrow] = ok ? (M + __log2f(lf)) * kLn2 : -INFINITY;
}

template <int D, int BLK, int BK>
__global__ void __launch_bounds__((F32Cfg<D, BLK>::NT))
    calib_f32_kernel(const float* __restrict__ Q, const float* __restrict__ K,
                     float* __restrict__ mass, float* __restrict__ lse, int n_q, int n_k, int N,
                     int n_pad, float scale_log2) {
  using C = F32Cfg<D, BLK>;
  constexpr int WPS = BLK / 64;  // waves per key split
  __shared__ __attribute__((aligned(16))) float buf[C::KS * CK * D];
  __shared__ float mpart[C::NT];
  __shared__ double lpart[C::NT];
  __shared__ float red[C::NT / 64];
  const int tid = threadIdx.x;
  const int sp = tid / BLK;
  const int t = tid % BLK;
  const int lane = tid & 63;
  const int r = blockIdx.x;
  const int bh = r / n_q;
  const int i = r - bh * n_q;
  const size_t head = (size_t)bh * n_pad * D;
  const int qrow = i * BLK + t;
  const int rows_valid = min(BLK, N - i * BLK);
  float* mrow = mass + (size_t)r * n_k;
  if (rows_valid <= 0) {
    for (int j = tid; j < n_k; j += C::NT) mrow[j] = 0.f;
    if (lse != nullptr && sp == 0) lse[(size_t)bh * n_pad + qrow] = -INFINITY;
    return;
  }
  // padding query rows take Q = 0 (finite scores whatever the padding holds;
  // they are never read into a mass)
  const bool qvalid = qrow < N;
  float q[D];
#pragma unroll
  for (int dd = 0; dd < D; ++dd) q[dd] = qvalid ? Q[head + (size_t)qrow * D + dd] * scale_log2 : 0.f;
  const int n_kv = (N + BK - 1) / BK;  // key blocks holding a real key; split s takes s, s+KS, ...
  const int rounds = (n_kv + C::KS - 1) / C::KS;
  float* Kc = buf + sp * CK * D;

  // sweep 1: running max / sum over this split's keys, then merged over the
  // splits in split order (every thread merges its row, so all splits hold it)
  float m = kNegBig;
  double l = 0.0;
  for (int rd = 0; rd < rounds; ++rd) {
    const int j = rd * C::KS + sp;
    const int kvalid = j < n_kv ? min(BK, N - j * BK) : 0;
    for (int c0 = 0; c0 < BK; c0 += CK) {
      __syncthreads();
      const bool live = c0 < kvalid;
      if (live) stage_rows<D>(Kc, K + head, j * BK + c0, t, BLK);
      __syncthreads();
      if (!live) continue;
      const int nk = min(CK, kvalid - c0);
      float s[CK];
      float mx = m;
#pragma unroll
      for (int kk = 0; kk < CK; ++kk) {
        float acc = 0.f;
#pragma unroll
        for (int dd = 0; dd < D; ++dd) acc = fmaf(q[dd], Kc[kk * D + dd], acc);
        s[kk] = kk < nk ? acc : -INFINITY;
        mx = fmaxf(mx, s[kk]);
      }
      l *= (double)fast_exp2(m - mx);
      m = mx;
      float part = 0.f;
#pragma unroll
      for (int kk = 0; kk < CK; ++kk) part += fast_exp2(s[kk] - m);
      l += (double)part;
    }
  }
  mpart[tid] = m;
  lpart[tid] = l;
  __syncthreads();
  float M = kNegBig;
  for (int s2 = 0; s2 < C::KS; ++s2) M = fmaxf(M, mpart[s2 * BLK + t]);
  double lt = 0.0;
  for (int s2 = 0; s2 < C::KS; ++s2)
    lt += lpart[s2 * BLK + t] * (double)fast_exp2(mpart[s2 * BLK + t] - M);
  const float lse2 = M + __log2f((float)lt);
  if (lse != nullptr && sp == 0) lse[(size_t)bh * n_pad + qrow] = qvalid ? lse2 * kLn2 : -INFINITY;
  const float sub = qvalid ? lse2 : INFINITY;

  // sweep 2: per key block of this split, the normalised probabilities summed
  // over the block's keys and the query block's rows (waves of the split added
  // in order)
  const float inv_rows = 1.0f / (float)rows_valid;
  for (int rd = 0; rd < rounds; ++rd) {
    const int j = rd * C::KS + sp;
    const int kvalid = j < n_kv ? min(BK, N - j * BK) : 0;
    float acc = 0.f;
    for (int c0 = 0; c0 < BK; c0 += CK) {
      __syncthreads();
      const bool live = c0 < kvalid;
      if (live) stage_rows<D>(Kc, K + head, j * BK + c0, t, BLK);
      __syncthreads();
      if (!live) continue;
      const int nk = min(CK, kvalid - c0);
#pragma unroll
      for (int kk = 0; kk < CK; ++kk) {
        float s = 0.f;
#pragma unroll
        for (int dd = 0; dd < D; ++dd) s = fmaf(q[dd], Kc[kk * D + dd], s);
        acc += kk < nk ? fast_exp2(s - sub) : 0.f;
      }
    }
    acc = wave_sum(acc);
    if (lane == 0) red[tid >> 6] = acc;
    __syncthreads();
    if (t == 0 && j < n_kv) {
      float tot = 0.f;
      for (int ww = 0; ww < WPS; ++ww) tot += red[sp * WPS + ww];
      mrow[j] = tot * inv_rows;
    }
  }
  for (int j = n_kv + tid; j < n_k; j += C::NT) mrow[j] = 0.f;
}

template <int D, int BLK, int BK>
hipError_t launch_f32(const void* q, const void* k, const void* v, int B, int H, int N, int n_pad,
                      float scale, const int32_t* row_ptr, const int32_t* col_idx,
                      int64_t col_len, void* o, float* lse, int dense, hipStream_t stream) {
  const int n_q = n_pad / BLK, n_k = n_pad / BK;
  hipLaunchKernelGGL((sparse_fwd_f32_kernel<D, BLK, BK>), dim3(B * H * n_q),
                     dim3(F32Cfg<D, BLK>::NT), 0, stream,
                     static_cast<const float*>(q), static_cast<const float*>(k),
                     static_cast<const float*>(v), row_ptr, col_idx, col_len,
                     static_cast<float*>(o), lse, n_q, n_k, N, n_pad, scale * kLog2e, dense);
  return hipGetLastError();
}

template <int D, int BLK, int BK>
hipError_t launch_cal_f32(const void* q, const void* k, int B, int H, int N, int n_pad, float scale,
                          float* mass, float* lse, hipStream_t stream) {
  const int n_q = n_pad / BLK, n_k = n_pad / BK;
  hipLaunchKernelGGL((calib_f32_kernel<D, BLK, BK>), dim3(B * H * n_q), dim3(F32Cfg<D, BLK>::NT),
                     0, stream,
                     static_cast<const float*>(q), static_cast<const float*>(k), mass, lse, n_q,
                     n_k, N, n_pad, scale * kLog2e);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sparse_fwd_f32(int d, int blk, int blk_k, const void* q, const void* k,
                                 const void* v, int B, int H, int N, int n_pad, float scale,
                                 const int32_t* row_ptr, const int32_t* col_idx, int64_t col_len,
                                 void* o, float* lse, hipStream_t stream) {
  const int dense = row_ptr == nullptr;  // internal: the construction step's dense attention
#define LOSA_F32_FWD(DD, BB, KK)                                                               \
  if (d == DD && blk == BB && blk_k == KK)                                                     \
    return launch_f32<DD, BB, KK>(q, k, v, B, H, N, n_pad, scale, row_ptr, col_idx, col_len, o, \
                                  lse, dense, stream);
  LOSA_F32_FWD(64, 64, 64)
  LOSA_F32_FWD(64, 128, 128)
  LOSA_F32_FWD(128, 64, 64)
  LOSA_F32_FWD(128, 128, 128)
  LOSA_F32_FWD(64, 64, 32)
  LOSA_F32_FWD(64, 128, 32)
  LOSA_F32_FWD(128, 64, 32)
  LOSA_F32_FWD(128, 128, 32)
#undef LOSA_F32_FWD
  return hipErrorInvalidValue;
}

hipError_t launch_calibrate_f32(int d, int blk, int blk_k, const void* q, const void* k, int B,
                                int H, int N, int n_pad, float scale, float* mass, float* lse,
                                hipStream_t stream) {
#define LOSA_F32_CAL(DD, BB, KK)                                                              \
  if (d == DD && blk == BB && blk_k == KK)                                                    \
    return launch_cal_f32<DD, BB, KK>(q, k, B, H, N, n_pad, scale, mass, lse, stream);
  LOSA_F32_CAL(64, 64, 64)
  LOSA_F32_CAL(64, 128, 128)
  LOSA_F32_CAL(128, 64, 64)
  LOSA_F32_CAL(128, 128, 128)
  LOSA_F32_CAL(64, 64, 32)
  LOSA_F32_CAL(64, 128, 32)
  LOSA_F32_CAL(128, 64, 32)
  LOSA_F32_CAL(128, 128, 32)
#undef LOSA_F32_CAL
  return hipErrorInvalidValue;
}

}  // namespace losa
