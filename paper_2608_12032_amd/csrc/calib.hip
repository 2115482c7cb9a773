// Exact block attention masses of the dense construction step (Sec. 3.1,
// Eq. (1); Sec. 4.1), bf16 in, fp32 accumulation, gfx950 MFMA.
//
// For query block i of head (b, h), with R_i valid rows and all N valid keys:
//   mbar(i, j) = (1 / R_i) * sum_{q in B_i, q < N} sum_{k in B_j, k < N}
//                exp(s_qk - lse_q),     s = scale * q . k,
// i.e. Eq. (1)'s M(i, j) divided by R_i, so every row of mbar sums to one.
// Query blocks have BLK rows, key blocks BK keys (BK = BLK, or 32 for the
// paper's rectangular setting with 128-row query blocks and 32-key key blocks);
// the keys stream through LDS in tiles of BLK keys either way.
//
// The normaliser lse_q is known only after all keys are seen, so a workgroup
// (one query block, BLK/32 waves of 32 query rows) makes two sweeps over the
// key tiles of its head:
//   1. S^T = K Q^T per tile, running max and running sum -> lse_q (log2
//      domain) per query, kept in registers;
//   2. S^T again (identical MFMA order, so identical scores), p = exp2(x -
//      lse2_q), summed per lane, then across the wave; each wave parks its
//      per-tile partial in LDS and the workgroup adds the waves' partials in a
//      fixed order at the end.  No atomics: the result is bitwise repeatable.
// The MFMA orientation is the one of the sparse forward (one query per lane in
// the S^T accumulator), so the scores are bitwise those the forward computes.
// K tiles are double-buffered in LDS with direct 16-byte loads; one barrier per
// tile.  With LSE_IN the normaliser comes from the caller (the dense forward of
// the construction step already produced it) and only sweep 2 runs.
#include "common.hpp"
#include "launch.hpp"

namespace losa {

namespace {

template <int D, int BLK>
struct CalCfg {
  static constexpr int NW = BLK / 32;
  static constexpr int NT = NW * 64;
  static constexpr int KS = D / 16;
  static constexpr int KB = BLK / 32;                // 32-key sub-blocks of a tile
  static constexpr int KROW = D * 2;
  static constexpr int KCH = D / 8;
  static constexpr int TILE = BLK * D * 2;
  static constexpr int LOADS = TILE / (1024 * NW);
  static_assert(TILE % (1024 * NW) == 0, "tile must split into whole wave loads");
};

template <int D, int BLK>
__device__ __forceinline__ void issue_tile(char* buf, __amdgpu_buffer_rsrc_t rs, int j, int w,
                                           int lane) {
  using C = CalCfg<D, BLK>;
#pragma unroll
  for (int u = 0; u < C::LOADS; ++u) {
    const int base = (w * C::LOADS + u) * 1024;
    const int o = base + lane * 16;
    const int row = o / C::KROW;
    const int pch = (o % C::KROW) >> 4;
    const int c = pch ^ (row % C::KCH);
    load_lds_16(rs, buf + base, (uint32_t)(((j * BLK + row) * D + c * 8) * 2));
  }
}

template <int D, int BLK>
__device__ __forceinline__ void tile_scores(const char* buf, const bf16x8_t* qreg, int l32, int g,
                                            f32x16_t* sacc) {
  using C = CalCfg<D, BLK>;
  const int ksw = l32 % C::KCH;
#pragma unroll
  for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
    for (int t = 0; t < 16; ++t) sacc[kb][t] = 0.f;
#pragma unroll
  for (int s = 0; s < C::KS; ++s) {
    const int off = (((2 * s + g) ^ ksw) << 4);
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb) {
      const bf16x8_t a =
          *reinterpret_cast<const bf16x8_t*>(buf + (kb * 32 + l32) * C::KROW + off);
      sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[s], sacc[kb], 0, 0, 0);
    }
  }
}

template <int D, int BLK, int BK, bool LSE_IN>
__global__ void __launch_bounds__(BLK * 2, 2)
    calib_bf16_kernel(const __bf16* __restrict__ Q, const __bf16* __restrict__ K,
                      float* __restrict__ mass, float* __restrict__ lse, int rows_total, int n_q,
                      int n_k, int N, int n_pad, float scale_log2) {
  using C = CalCfg<D, BLK>;
  static_assert(BK % 32 == 0 && BLK % BK == 0, "key blocks split a tile into whole sub-blocks");
  constexpr int TB = BLK / BK;   // key blocks per tile
  constexpr int SPB = BK / 32;   // 32-key sub-blocks per key block
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  char* buf0 = smem;
  char* buf1 = smem + C::TILE;
  float* part = reinterpret_cast<float*>(smem + 2 * C::TILE);  // [NW][n_k]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31;
  const int g = lane >> 5;

  const int r = xcd_remap(blockIdx.x, rows_total);
  const int bh = r / n_q;
  const int i = r - bh * n_q;
  const size_t head = (size_t)bh * n_pad * D;
  const int rows_valid = min(BLK, N - i * BLK);
  float* mrow = mass + (size_t)r * n_k;

  if (rows_valid <= 0) {  // a query block made only of padding
    for (int j = tid; j < n_k; j += C::NT) mrow[j] = 0.f;
    if (!LSE_IN && lse != nullptr)
      for (int t = tid; t < BLK; t += C::NT) lse[(size_t)bh * n_pad + i * BLK + t] = -INFINITY;
    return;
  }

  const __amdgpu_buffer_rsrc_t krs = make_rsrc(K + head, (uint32_t)((size_t)n_pad * D * 2));
  const int qrow = i * BLK + w * 32 + l32;
  bf16x8_t qreg[C::KS];
  {
    const bf16x8_t* qp = reinterpret_cast<const bf16x8_t*>(Q + head + (size_t)qrow * D);
#pragma unroll
    for (int s = 0; s < C::KS; ++s) qreg[s] = qp[2 * s + g];
  }
  const int n_kv = (N + BLK - 1) / BLK;  // key tiles holding a real key

  const bool qvalid = qrow < N;
  float lse2;
  if constexpr (LSE_IN) {
    lse2 = qvalid ? lse[(size_t)bh * n_pad + qrow] * kLog2e : 0.f;
  } else {
  // ---- sweep 1: running max / sum -> lse (log2 units) ----------------------
  float m_run = kNegBig;
  float l_run = 0.f;
  issue_tile<D, BLK>(buf0, krs, 0, w, lane);
  for (int j = 0; j < n_kv; ++j) {
    char* cur = (j & 1) ? buf1 : buf0;
    char* nxt = (j & 1) ? buf0 : buf1;
    wait_vm_barrier<0>();  // tile j landed; every wave is done with tile j-1
    if (j + 1 < n_kv) issue_tile<D, BLK>(nxt, krs, j + 1, w, lane);
    f32x16_t sacc[C::KB];
    tile_scores<D, BLK>(cur, qreg, l32, g, sacc);
    const int kvalid = min(BLK, N - j * BLK);
    float mx = m_run;
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        const int key = kb * 32 + ((t >> 2) << 3) + (g << 2) + (t & 3);
        const float x = key < kvalid ? sacc[kb][t] * scale_log2 : -INFINITY;
        sacc[kb][t] = x;
        mx = fmaxf(mx, x);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    float lsum = 0.f;
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
      for (int t = 0; t < 16; ++t) lsum += fast_exp2(sacc[kb][t] - mx);
    l_run = l_run * fast_exp2(m_run - mx) + lsum;
    m_run = mx;
  }
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  lse2 = m_run + __log2f(l_tot);
  if (lse != nullptr && g == 0)
    lse[(size_t)bh * n_pad + qrow] = qvalid ? lse2 * kLn2 : -INFINITY;
  }
  // padding rows contribute exp2(x - inf) = 0 to every mass
  const float sub = qvalid ? lse2 : INFINITY;

  // ---- sweep 2: block masses -----------------------------------------------
  wait_vm_barrier<0>();  // all waves are done with the last tile of sweep 1 (or with nothing)
  issue_tile<D, BLK>(buf0, krs, 0, w, lane);
  for (int j = 0; j < n_kv; ++j) {
    char* cur = (j & 1) ? buf1 : buf0;
    char* nxt = (j & 1) ? buf0 : buf1;
    wait_vm_barrier<0>();
    if (j + 1 < n_kv) issue_tile<D, BLK>(nxt, krs, j + 1, w, lane);
    f32x16_t sacc[C::KB];
    tile_scores<D, BLK>(cur, qreg, l32, g, sacc);
    const int kvalid = min(BLK, N - j * BLK);
    float acc[TB];
#pragma unroll
    for (int b = 0; b < TB; ++b) acc[b] = 0.f;
#pragma unroll
    for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        const int key = kb * 32 + ((t >> 2) << 3) + (g << 2) + (t & 3);
        const float x = key < kvalid ? sacc[kb][t] * scale_log2 : -INFINITY;
        acc[kb / SPB] += fast_exp2(x - sub);
      }
#pragma unroll
    for (int b = 0; b < TB; ++b) {
      const float a = wave_sum(acc[b]);
      if (lane == 0) part[w * n_k + j * TB + b] = a;
    }
  }
  lds_read_barrier();  // partials written (lgkmcnt covers the LDS stores)
  const float inv_rows = 1.0f / (float)rows_valid;
  const int n_kb = n_kv * TB;  // key blocks inside the tiles swept (the rest hold no key)
  for (int j = tid; j < n_k; j += C::NT) {
    float s = 0.f;
    if (j < n_kb) {
#pragma unroll
      for (int ww = 0; ww < C::NW; ++ww) s += part[ww * n_k + j];
    }
    mrow[j] = s * inv_rows;
  }
}

template <int D, int BLK, int BK, bool LSE_IN>
hipError_t launch_cal(const void* q, const void* k, int B, int H, int N, int n_pad, float scale,
                      float* mass, float* lse, hipStream_t stream) {
  using C = CalCfg<D, BLK>;
  const int n_q = n_pad / BLK;
  const int n_k = n_pad / BK;
  const int rows = B * H * n_q;
  const size_t lds = 2 * (size_t)C::TILE + (size_t)C::NW * n_k * sizeof(float);
  hipError_t err =
      hipFuncSetAttribute(reinterpret_cast<const void*>(&calib_bf16_kernel<D, BLK, BK, LSE_IN>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL((calib_bf16_kernel<D, BLK, BK, LSE_IN>), dim3(rows), dim3(C::NT), lds, stream,
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(k), mass, lse,
                     rows, n_q, n_k, N, n_pad, scale * kLog2e);
  return hipGetLastError();
}

}  // namespace

size_t calib_bf16_lds_bytes(int d, int blk, int n_k) {
  return 2 * (size_t)blk * d * 2 + (size_t)(blk / 32) * n_k * sizeof(float);
}

hipError_t launch_calibrate_bf16(int d, int blk, int blk_k, const void* q, const void* k, int B,
                                 int H, int N, int n_pad, float scale, float* mass, float* lse,
                                 bool lse_in, hipStream_t stream) {
#define LOSA_CAL(DD, BB, KK)                                                              \
  if (d == DD && blk == BB && blk_k == KK)                                                \
    return lse_in ? launch_cal<DD, BB, KK, true>(q, k, B, H, N, n_pad, scale, mass, lse, stream) \
                  : launch_cal<DD, BB, KK, false>(q, k, B, H, N, n_pad, scale, mass, lse, stream);
  LOSA_CAL(128, 128, 128)
  LOSA_CAL(64, 128, 128)
  LOSA_CAL(128, 64, 64)
  LOSA_CAL(64, 64, 64)
  LOSA_CAL(128, 128, 32)
  LOSA_CAL(64, 128, 32)
  LOSA_CAL(128, 64, 32)
  LOSA_CAL(64, 64, 32)
#undef LOSA_CAL
  return hipErrorInvalidValue;
}

}  // namespace losa
