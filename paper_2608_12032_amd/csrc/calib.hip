// Exact block attention masses of the dense construction step (Sec. 3.1,
// Eq. (1); Sec. 4.1), bf16 in, fp32 accumulation, gfx950 MFMA.
//
// For query block i of head (b, h), with R_i valid rows and all N valid keys:
//   mbar(i, j) = (1 / R_i) * sum_{q in B_i, q < N} sum_{k in B_j, k < N}
//                exp(s_qk - lse_q),     s = scale * q . k,
// i.e. Eq. (1)'s M(i, j) divided by R_i, so every row of mbar sums to one.
// Query blocks have BLK rows, key blocks BK keys (BK = BLK, or 32 for the
// paper's rectangular setting with 128-row query blocks and 32-key key blocks);
// the keys stream through LDS in tiles of BLK keys (64 at d = 128 with
// 128-row blocks, where a 128-key block's sums are carried across its two
// tiles).
//
// The normaliser lse_q is known only after all keys are seen.  Two schemes:
//
// Two sweeps (no workspace): a workgroup (one query block, BLK/32 waves of 32
// query rows) sweeps the key tiles of its head twice:
//   1. S^T = K Q^T per tile and a running sum of 2^(x - m) -> lse_q (log2
//      domain) per query, kept in registers.  The reference m is raised only
//      when a lane's tile sum passes 2^20 (or is inf: the first tile), so a
//      score costs one fma, one exp2 and one add;
//   2. S^T again (identical MFMA order, so identical scores), p = exp2(x -
//      lse2_q), summed per lane, then across the wave; each wave parks its
//      per-key-block partial in LDS and the workgroup adds the waves' partials
//      in a fixed order at the end.  No atomics: the result is bitwise repeatable.
//
// One sweep with block statistics (STATS): sweep 1 alone, and for every
// query q and key block j it also stores
//   a(q, j) = log2( sum_{k in B_j, k < N} 2^(x_qk - m) ) + m,
// m being the reference the running sum used when block j went by.  a(q, j)
// is log2 of the block's unnormalised probability sum, so once lse2_q is
// known, mbar(i, j) = (1 / R_i) sum_q 2^(a(q, j) - lse2_q): stat_mass_kernel
// does that reduction.  The statistics cost 4 bytes per (query, key block),
// written once and read once, in place of a second pass of Q K^T and its
// exponentials.  The dense forward of the construction step writes the same
// statistics (sparse_fwd.hip), so its masses come from the same reduction.
//
// The MFMA orientation is the one of the sparse forward (one query per lane in
// the S^T accumulator), so the scores are bitwise those the forward computes.
// K tiles are double-buffered in LDS with direct 16-byte loads; one barrier per
// tile.
#include "common.hpp"
#include "launch.hpp"

namespace losa {

namespace {

// Keys per LDS tile: 64 at d = 128 with 128-row query blocks (a tile of scores
// then takes 32 registers instead of 64, and two 16 KiB tiles leave LDS for
// four workgroups per CU), else one query block's worth of keys.
constexpr int cal_tile_keys(int d, int blk) { return (d == 128 && blk == 128) ? 64 : blk; }

template <int D, int BLK>
struct CalCfg {
  static constexpr int NW = BLK / 32;
  static constexpr int NT = NW * 64;
  static constexpr int KS = D / 16;
  static constexpr int TK = cal_tile_keys(D, BLK);   // keys per tile
  static constexpr int KB = TK / 32;                 // 32-key sub-blocks of a tile
  static constexpr int KROW = D * 2;
  static constexpr int KCH = D / 8;
  static constexpr int TILE = TK * D * 2;
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
    load_lds_16(rs, buf + base, (uint32_t)(((j * C::TK + row) * D + c * 8) * 2));
  }
}

// S^T of a tile's KB 32-key sub-blocks, k-step by k-step (the sub-blocks'
// chains interleaved); each MFMA's K operand is read from LDS NPRE MFMAs ahead
// into a small register ring, an order fixed with sched_group_barrier (left to
// itself the compiler issued each read just before its MFMA, which then waited
// out the LDS latency: 2 % slower at the Wan shape).
template <int D, int BLK>
__device__ __forceinline__ void tile_scores(const char* buf, const bf16x8_t* qreg, int l32, int g,
                                            f32x16_t* sacc) {
  using C = CalCfg<D, BLK>;
  constexpr int NM = C::KS * C::KB;
  constexpr int NPRE = 4;  // MFMAs an operand read leads by
  const int ksw = l32 % C::KCH;
  auto rd = [&](int i) -> bf16x8_t {
    const int st = i / C::KB, kb = i % C::KB;
    const int off = (((2 * st + g) ^ ksw) << 4);
    return *reinterpret_cast<const bf16x8_t*>(buf + (kb * 32 + l32) * C::KROW + off);
  };
  bf16x8_t ring[NPRE];
#pragma unroll
  for (int i = 0; i < NPRE; ++i) ring[i] = rd(i);
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    const int st = i / C::KB, kb = i % C::KB;
    sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ring[i % NPRE], qreg[st],
                                                       st == 0 ? f32x16_t{} : sacc[kb], 0, 0, 0);
    if (i + NPRE < NM) ring[i % NPRE] = rd(i + NPRE);
  }
  __builtin_amdgcn_sched_group_barrier(0x100, NPRE, 0);
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i + NPRE < NM) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
}

// Scores of keys at or beyond kvalid (tile-relative) -> -inf: the ragged last
// key tile only.
template <int KB>
__device__ __forceinline__ void mask_tile(f32x16_t* s, int kvalid, int g) {
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const int key = kb * 32 + ((t >> 2) << 3) + (g << 2) + (t & 3);
      if (key >= kvalid) s[kb][t] = -INFINITY;
    }
}

// This lane's probabilities 2^(c*s - m) of a tile, summed per key block of the
// tile (bs, TB blocks of SPB 32-key sub-blocks; one partial per sub-block, for
// independent add chains); returns the lane's tile sum.
template <int KB, int TB>
__device__ __forceinline__ float tile_sums(const f32x16_t* s, float c, float m, float* bs) {
  constexpr int SPB = KB / TB;
  float acc[KB];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) {
    acc[kb] = 0.f;
#pragma unroll
    for (int t = 0; t < 16; ++t) acc[kb] += fast_exp2(__builtin_fmaf(s[kb][t], c, -m));
  }
  float l = 0.f;
#pragma unroll
  for (int b = 0; b < TB; ++b) {
    bs[b] = acc[b * SPB];
#pragma unroll
    for (int u = 1; u < SPB; ++u) bs[b] += acc[b * SPB + u];
    l += bs[b];
  }
  return l;
}

// tile_scores + tile_sums of a full tile in one interleaved stream, for d = 64:
// the sub-blocks' S^T accumulate one after the other, and the exponentials of
// sub-block kb-1 run under the MFMAs of sub-block kb.  At d = 64 a tile has
// half the MFMAs per exponential of d = 128, and leaving them to the other
// wave of the SIMD left the matrix cores idle (the interleave is 7-12 % faster
// there; at d = 128 it was 5 % slower, so d = 128 keeps the two-step form).
// Same scores, same summation order: bitwise the result of the two-step form.
template <int D, int BLK, int TB>
__device__ __forceinline__ float tile_fused(const char* buf, const bf16x8_t* qreg, int l32, int g,
                                            f32x16_t* sacc, float c, float m, float* bs) {
  using C = CalCfg<D, BLK>;
  constexpr int KB = C::KB;
  constexpr int SPB = KB / TB;
  constexpr int PM = 16 / C::KS;  // scores of the previous sub-block per MFMA
  const int ksw = l32 % C::KCH;
  float acc[KB];
#pragma unroll
  for (int kb = 0; kb <= KB; ++kb) {
#pragma unroll
    for (int s = 0; s < C::KS; ++s) {
      if (kb < KB) {
        const int off = (((2 * s + g) ^ ksw) << 4);
        const bf16x8_t a =
            *reinterpret_cast<const bf16x8_t*>(buf + (kb * 32 + l32) * C::KROW + off);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            a, qreg[s], s == 0 ? f32x16_t{} : sacc[kb], 0, 0, 0);
      }
      if (kb > 0) {
#pragma unroll
        for (int u = 0; u < PM; ++u) {
          const int t = s * PM + u;
          const float p = fast_exp2(__builtin_fmaf(sacc[kb - 1][t], c, -m));
          acc[kb - 1] = (t == 0) ? p : acc[kb - 1] + p;
        }
      }
    }
  }
  // per MFMA: its operand read, the MFMA, then PM (fma, add) pairs and PM exp
#pragma unroll
  for (int kb = 0; kb <= KB; ++kb)
#pragma unroll
    for (int s = 0; s < C::KS; ++s) {
      if (kb < KB) {
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      }
      if (kb > 0) {
        __builtin_amdgcn_sched_group_barrier(0x002, 2 * PM, 0);
        __builtin_amdgcn_sched_group_barrier(0x400, PM, 0);
      }
    }
  float l = 0.f;
#pragma unroll
  for (int b = 0; b < TB; ++b) {
    bs[b] = acc[b * SPB];
#pragma unroll
    for (int u = 1; u < SPB; ++u) bs[b] += acc[b * SPB + u];
    l += bs[b];
  }
  return l;
}

// Scores of tile `buf` (keys >= kvalid masked) and this lane's probability sums
// against m: per key block into bs, the lane's tile sum returned.
template <int D, int BLK, int TB>
__device__ __forceinline__ float tile_probs(const char* buf, const bf16x8_t* qreg, int l32, int g,
                                            int kvalid, float c, float m, f32x16_t* sacc,
                                            float* bs) {
  using C = CalCfg<D, BLK>;
  if constexpr (D == 64) {
    if (kvalid == C::TK) return tile_fused<D, BLK, TB>(buf, qreg, l32, g, sacc, c, m, bs);
  }
  tile_scores<D, BLK>(buf, qreg, l32, g, sacc);
  if (kvalid < C::TK) mask_tile<C::KB>(sacc, kvalid, g);
  return tile_sums<C::KB, TB>(sacc, c, m, bs);
}

// Bound on one lane's tile sum (so on each probability) before the running
// max must be raised: the max used trails the true one by at most 20 (log2
// units), and l stays far from fp32 overflow (2^20 per key, at most 2^19 keys).
constexpr float kCalSumBound = 1048576.0f;

// Waves per SIMD the register budget is cut for, so that the exponentials of
// some waves overlap the MFMAs of others: four with 128-row query blocks or at
// d = 64 (a 64-key tile of scores and the Q operands fit 128 registers; 32 KiB
// of tiles per workgroup), two otherwise.  The two-sweep scheme's partials add
// LDS and can lower the count the LDS allows.
template <int D, int BLK>
constexpr int cal_waves_per_simd() {
  return (D == 64 || BLK == 128) ? 4 : 2;
}

template <int D, int BLK, int BK, bool STATS>
__global__ void __launch_bounds__(BLK * 2)
    __attribute__((amdgpu_waves_per_eu(cal_waves_per_simd<D, BLK>())))
    calib_bf16_kernel(const __bf16* __restrict__ Q, const __bf16* __restrict__ K,
                      float* __restrict__ mass, float* __restrict__ lse,
                      float* __restrict__ stat, int rows_total, int n_q, int n_k, int N,
                      int n_pad, float scale_log2) {
  using C = CalCfg<D, BLK>;
  static_assert(BK % 32 == 0 && BLK % BK == 0, "key blocks split a query block's keys");
  static_assert(C::TK % BK == 0 || BK % C::TK == 0, "tiles and key blocks nest");
  constexpr int TB = C::TK >= BK ? C::TK / BK : 1;   // key blocks (or parts of one) per tile
  constexpr int TPB = BK > C::TK ? BK / C::TK : 1;   // tiles per key block
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

  if (rows_valid <= 0) {  // a query block made only of padding (STATS: stat_mass zeroes the row)
    if (!STATS)
      for (int j = tid; j < n_k; j += C::NT) mrow[j] = 0.f;
    if (lse != nullptr)
      for (int t = tid; t < BLK; t += C::NT) lse[(size_t)bh * n_pad + i * BLK + t] = -INFINITY;
    return;
  }

  const __amdgpu_buffer_rsrc_t krs = make_rsrc(K + head, (uint32_t)((size_t)n_pad * D * 2));
  const int qrow = i * BLK + w * 32 + l32;
  const bool qvalid = qrow < N;
  // padding query rows take Q = 0: their scores stay finite whatever the
  // padding holds, and they are never read into a mass
  bf16x8_t qreg[C::KS];
  {
    const bf16x8_t* qp = reinterpret_cast<const bf16x8_t*>(Q + head + (size_t)qrow * D);
#pragma unroll
    for (int s = 0; s < C::KS; ++s) qreg[s] = qvalid ? qp[2 * s + g] : bf16x8_t{};
  }
  const int n_kv = (N + C::TK - 1) / C::TK;  // key tiles holding a real key
  // a key block's sums are complete after its last tile, or after the last
  // tile swept (the block's remaining tiles hold no key)
  auto block_done = [&](int j) { return TPB == 1 || j % TPB == TPB - 1 || j == n_kv - 1; };
  auto first_block = [&](int j) { return TPB == 1 ? j * TB : j / TPB; };

  // ---- sweep 1: running max / sum -> lse (log2 units) ----------------------
  float m_run = kNegBig;
  float l_run = 0.f;
  float pend[TB];  // STATS: finished block statistics, stored one tile late
  int pend_blk = -1;  // first key block of pend (-1: nothing pending)
  float bacc[TB];  // block sums so far against m_run (TPB > 1: over the block's tiles)
#pragma unroll
  for (int b = 0; b < TB; ++b) bacc[b] = 0.f;
  issue_tile<D, BLK>(buf0, krs, 0, w, lane);
  for (int j = 0; j < n_kv; ++j) {
    char* cur = (j & 1) ? buf1 : buf0;
    char* nxt = (j & 1) ? buf0 : buf1;
    wait_vm_barrier<0>();  // tile j landed; every wave is done with tile j-1
    if (j + 1 < n_kv) issue_tile<D, BLK>(nxt, krs, j + 1, w, lane);
    if constexpr (STATS) {
      // the stores go out a whole tile before the next vmcnt(0) wait, which
      // then finds them done instead of waiting out their latency
      if (pend_blk >= 0 && g == 0) {
#pragma unroll
        for (int b = 0; b < TB; ++b)
          stat[((size_t)bh * n_k + pend_blk + b) * n_pad + qrow] = pend[b];
      }
      pend_blk = -1;
    }
    f32x16_t sacc[C::KB];
    const int kvalid = min(C::TK, N - j * C::TK);
    // Probabilities against the running max, without looking at this tile's
    // scores first.  If a lane's tile sum exceeds the bound (or is inf: the
    // first tile), the max is raised to the tile's and the sums redone; both
    // lanes of a query take the same max, so their sums stay comparable.
    float bs[TB];
    float lsum = tile_probs<D, BLK, TB>(cur, qreg, l32, g, kvalid, scale_log2, m_run, sacc, bs);
    if (__ballot(!(lsum <= kCalSumBound)) != 0) {
      float mx = sacc[0][0];
#pragma unroll
      for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
        for (int t = 0; t < 16; ++t) mx = fmaxf(mx, sacc[kb][t]);
      mx = fmaxf(mx, __shfl_xor(mx, 32)) * scale_log2;  // scale > 0: max commutes with it
      const float m_new = fmaxf(m_run, mx);
      const float alpha = fast_exp2(m_run - m_new);
      l_run *= alpha;
      if constexpr (TPB > 1) bacc[0] *= alpha;
      m_run = m_new;
      lsum = tile_sums<C::KB, TB>(sacc, scale_log2, m_run, bs);
    }
    l_run += lsum;
#pragma unroll
    for (int b = 0; b < TB; ++b) bacc[b] = TPB == 1 ? bs[b] : bacc[b] + bs[b];
    if (block_done(j)) {
      if constexpr (STATS) {
#pragma unroll
        for (int b = 0; b < TB; ++b) pend[b] = __log2f(bacc[b] + __shfl_xor(bacc[b], 32)) + m_run;
        pend_blk = first_block(j);
      }
#pragma unroll
      for (int b = 0; b < TB; ++b) bacc[b] = 0.f;
    }
  }
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float lse2 = m_run + __log2f(l_tot);
  if (lse != nullptr && g == 0)
    lse[(size_t)bh * n_pad + qrow] = qvalid ? lse2 * kLn2 : -INFINITY;
  if constexpr (STATS) {
    if (g == 0) {
#pragma unroll
      for (int b = 0; b < TB; ++b)
        stat[((size_t)bh * n_k + pend_blk + b) * n_pad + qrow] = pend[b];
    }
    return;
  }

  // padding rows (Q = 0, finite scores) contribute exp2(-inf) = 0 to every mass
  const float sub = qvalid ? lse2 : INFINITY;

  // ---- sweep 2: block masses -----------------------------------------------
#pragma unroll
  for (int b = 0; b < TB; ++b) bacc[b] = 0.f;
  wait_vm_barrier<0>();  // all waves are done with the last tile of sweep 1 (or with nothing)
  issue_tile<D, BLK>(buf0, krs, 0, w, lane);
  for (int j = 0; j < n_kv; ++j) {
    char* cur = (j & 1) ? buf1 : buf0;
    char* nxt = (j & 1) ? buf0 : buf1;
    wait_vm_barrier<0>();
    if (j + 1 < n_kv) issue_tile<D, BLK>(nxt, krs, j + 1, w, lane);
    f32x16_t sacc[C::KB];
    const int kvalid = min(C::TK, N - j * C::TK);
    float acc[TB];
    tile_probs<D, BLK, TB>(cur, qreg, l32, g, kvalid, scale_log2, sub, sacc, acc);
#pragma unroll
    for (int b = 0; b < TB; ++b) bacc[b] = TPB == 1 ? acc[b] : bacc[b] + acc[b];
    if (block_done(j)) {
      const int j0 = first_block(j);
#pragma unroll
      for (int b = 0; b < TB; ++b) {
        const float a = wave_sum(bacc[b]);
        if (lane == 0) part[w * n_k + j0 + b] = a;
        bacc[b] = 0.f;
      }
    }
  }
  lds_read_barrier();  // partials written (lgkmcnt covers the LDS stores)
  const float inv_rows = 1.0f / (float)rows_valid;
  const int n_kb = first_block(n_kv - 1) + TB;  // key blocks the sweep covered (the rest hold no key)
  for (int j = tid; j < n_k; j += C::NT) {
    float s = 0.f;
    if (j < n_kb) {
#pragma unroll
      for (int ww = 0; ww < C::NW; ++ww) s += part[ww * n_k + j];
    }
    mrow[j] = s * inv_rows;
  }
}

// mbar(i, j) = (1 / R_i) sum_{q in B_i, q < N} 2^(a(q, j) - lse2_q) from the
// block statistics a [BH][n_k][n_pad] (log2 units) and the natural-log
// normalisers lse [BH][n_pad].  One workgroup per mass row (bh, i); wave w
// takes groups of kStatGroup consecutive key blocks, each lane QPL adjacent
// queries of block i, so a wave reads BLK contiguous floats per key block and
// has kStatGroup such reads in flight.  Lanes 0..kStatGroup-1 then store the
// group's masses with one contiguous store.  Key blocks j >= n_kb hold no
// valid key and rows made only of padding get 0; padding queries are never
// read into the sum.  Fixed summation order: bitwise repeatable.
constexpr int kStatT = 256;
constexpr int kStatGroup = 8;

template <int BLK>
__global__ void __launch_bounds__(kStatT)
    stat_mass_kernel(const float* __restrict__ stat, const float* __restrict__ lse, int n_q,
                     int n_k, int n_kb, int N, int n_pad, float* __restrict__ mass) {
  constexpr int QPL = BLK / 64;
  constexpr int NWV = kStatT / 64;
  static_assert(QPL == 1 || QPL == 2, "64- or 128-row query blocks");
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int r = blockIdx.x;
  const int bh = r / n_q;
  const int i = r - bh * n_q;
  float* mrow = mass + (size_t)r * n_k;
  const int rows_valid = min(BLK, N - i * BLK);
  if (rows_valid <= 0) {
    for (int j = threadIdx.x; j < n_k; j += kStatT) mrow[j] = 0.f;
    return;
  }
  const int q0 = i * BLK + lane * QPL;
  bool ok[QPL];
  float sub[QPL];
#pragma unroll
  for (int e = 0; e < QPL; ++e) {
    ok[e] = q0 + e < N;
    sub[e] = ok[e] ? lse[(size_t)bh * n_pad + q0 + e] * kLog2e : 0.f;
  }
  const float inv = 1.0f / (float)rows_valid;
  const float* base = stat + (size_t)bh * n_k * n_pad + q0;
  for (int j0 = w * kStatGroup; j0 < n_k; j0 += NWV * kStatGroup) {
    float v[kStatGroup][QPL];
#pragma unroll
    for (int u = 0; u < kStatGroup; ++u) {
      const int j = j0 + u;
      if (j < n_kb) {
        const float* src = base + (size_t)j * n_pad;
        if constexpr (QPL == 2) {
          const f32x2_t t = *reinterpret_cast<const f32x2_t*>(src);
          v[u][0] = t[0];
          v[u][1] = t[1];
        } else {
          v[u][0] = *src;
        }
      } else {
#pragma unroll
        for (int e = 0; e < QPL; ++e) v[u][e] = 0.f;
      }
    }
    float mine = 0.f;
#pragma unroll
    for (int u = 0; u < kStatGroup; ++u) {
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < QPL; ++e) acc += ok[e] ? fast_exp2(v[u][e] - sub[e]) : 0.f;
      acc = wave_sum(acc);
      if (lane == u) mine = (j0 + u < n_kb) ? acc * inv : 0.f;
    }
    if (lane < kStatGroup && j0 + lane < n_k) mrow[j0 + lane] = mine;
  }
}

template <int D, int BLK, int BK, bool STATS>
hipError_t launch_cal(const void* q, const void* k, int B, int H, int N, int n_pad, float scale,
                      float* mass, float* lse, float* stat, hipStream_t stream) {
  using C = CalCfg<D, BLK>;
  const int n_q = n_pad / BLK;
  const int n_k = n_pad / BK;
  const int rows = B * H * n_q;
  const size_t lds = 2 * (size_t)C::TILE + (STATS ? 0 : (size_t)C::NW * n_k * sizeof(float));
  hipError_t err =
      hipFuncSetAttribute(reinterpret_cast<const void*>(&calib_bf16_kernel<D, BLK, BK, STATS>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL((calib_bf16_kernel<D, BLK, BK, STATS>), dim3(rows), dim3(C::NT), lds, stream,
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(k), mass, lse,
                     stat, rows, n_q, n_k, N, n_pad, scale * kLog2e);
  err = hipGetLastError();
  if (err != hipSuccess || !STATS) return err;
  return launch_stat_mass(BLK, BK, stat, lse, B * H, N, n_pad, mass, stream);
}

}  // namespace

hipError_t launch_stat_mass(int blk, int blk_k, const float* stat, const float* lse, int BH, int N,
                            int n_pad, float* mass, hipStream_t stream) {
  const int n_q = n_pad / blk;
  const int n_k = n_pad / blk_k;
  const int n_kb = (N + blk_k - 1) / blk_k;
  if (blk == 128)
    hipLaunchKernelGGL(stat_mass_kernel<128>, dim3(BH * n_q), dim3(kStatT), 0, stream, stat, lse,
                       n_q, n_k, n_kb, N, n_pad, mass);
  else if (blk == 64)
    hipLaunchKernelGGL(stat_mass_kernel<64>, dim3(BH * n_q), dim3(kStatT), 0, stream, stat, lse,
                       n_q, n_k, n_kb, N, n_pad, mass);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

size_t calib_bf16_lds_bytes(int d, int blk, int n_k) {
  return 2 * (size_t)cal_tile_keys(d, blk) * d * 2 + (size_t)(blk / 32) * n_k * sizeof(float);
}

hipError_t launch_calibrate_bf16(int d, int blk, int blk_k, const void* q, const void* k, int B,
                                 int H, int N, int n_pad, float scale, float* mass, float* lse,
                                 float* stat, hipStream_t stream) {
#define LOSA_CAL(DD, BB, KK)                                                                 \
  if (d == DD && blk == BB && blk_k == KK)                                                   \
    return stat ? launch_cal<DD, BB, KK, true>(q, k, B, H, N, n_pad, scale, mass, lse, stat,  \
                                                stream)                                      \
                : launch_cal<DD, BB, KK, false>(q, k, B, H, N, n_pad, scale, mass, lse, nullptr, \
                                                 stream);
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
