// Frozen-support block-sparse attention forward (Sec. 4.2, Eq. (4)), bf16 in,
// fp32 accumulation, on gfx950 MFMA.
//
// Work unit.  One workgroup owns one CSR row r = (b*H + h)*n_q + i: the BLK
// query rows of query block i, 32 per wave (BLK/32 waves, one per SIMD for
// BLK = 128), and walks only the key blocks the row retains.  Two workgroups
// share a CU at d = 128 and three at d = 64, so each SIMD runs two or three
// independent waves: while one waits at its workgroup barrier or on its
// exponentials, another keeps the matrix core busy.  The workgroup first
// turns its CSR entries into a sorted list of distinct valid block ids in LDS
// (per-block flags, then a ballot compaction), which realises Eq. (4)'s set
// semantics exactly: a repeated id counts once, ids outside [0, n_k) are
// dropped.
//
// Orientation.  Per 32-key sub-tile the wave computes S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16 (A = K rows from LDS, B = the wave's Q^T held in
// registers).  In the 32x32 accumulator a lane holds 16 scores of ONE query
// (column = lane % 32), so the online softmax (running max, running sum) is
// in-lane plus one exchange with lane ^ 32, which holds the other keys of the
// same query.  The exponentiated scores are already laid out as the B operand
// of O^T = V^T P^T, and the O^T accumulator again keeps one query per lane, so
// the per-query rescale and the final 1/l are in-lane too.
//
// Key order inside a 16-key MFMA step.  The B operand P^T of lane group g
// (lanes 32g..32g+31) holds, in register element e, the key
//   16*step + 4*g + e + (e >= 4 ? 4 : 0),
// which is where the S^T accumulator put it.  The A operand V^T must hold the
// same key in the same (lane group, element) slot; the transposed copy of V
// therefore stores, within every group of 16 keys, positions 4..7 and 8..11
// swapped (an involution), so each lane's 8 keys are 16 contiguous bytes.
//
// Streaming.  The row's keys are a stream of 32-key sub-tiles (NS = BK/32 per
// key block of BK keys; with BK = 32 the stream is padded to whole loop passes
// with sub-tiles whose keys are all masked).  K and V^T sub-tiles pass through
// two rings of kRing LDS slots, filled by 16-byte buffer loads that write LDS
// directly.  Sub-iteration s
// reads K sub-tile s+1 (scores of the next sub-tile) and V^T sub-tile s-1
// (P V of the previous one); after the barrier that opens it, the slots that
// sub-iteration s-1 finished with are refilled with K sub-tile s+kRing and V^T
// sub-tile s+kRing-2, both needed kRing-1 sub-iterations later.  Every
// sub-iteration issues the same number of loads (past the end of the stream
// they fetch the last block again), so one fixed vmcnt wait before each
// barrier is exact.  Inside a sub-iteration the matrix cores alternate the
// next scores with P V of the previous sub-tile while the VALU exponentiates
// the current one, and the loads leave one at a time between the MFMAs
// rather than in a burst; the instruction interleave is fixed with
// sched_group_barrier.
//
// LDS images.  A K sub-tile is 32 rows of D bf16, row-major, 16-byte chunks
// XOR-swizzled by 256-byte line; V^T is kept in global memory already in the
// LDS image of its sub-tiles (written by the transpose kernel), so its loads
// are plain contiguous copies.  Both swizzles make the 16 rows read by one
// 16-lane group of an operand read land in distinct banks.
//
// Softmax.  Probabilities are taken against the running max without looking
// at the sub-tile's scores first; only when a lane's sub-tile sum exceeds
// kSumBound (or is inf) is the max raised and the sub-tile redone, so every
// probability entering P V is at most kSumBound.
//
// Dense mode (template flag DENSE; the construction step).  Every row keeps
// every key block holding a valid key, rows run in id order, and per key block
// each query's probability sum is stored as a block statistic
// a(q, j) = log2(sum) + m (the reference m it was taken against), from which
// the block masses follow once lse is known (stat_mass_kernel).
//
// Dispatch order (sparse mode).  Rows run longest first inside chunks of
// neighbouring query blocks, each XCD on a contiguous range of rows
// (order_rows_kernel), so rows in flight share their key blocks in L2.
//
// Padding.  Keys >= N get score -inf (only the ragged last block needs it).
// Query rows >= N are written as 0 with lse = -inf; so are rows with an empty
// key set.  Row bounds are clamped to [0, col_idx_len], so a malformed CSR
// cannot make the kernel read outside col_idx.
#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace losa {

namespace {

// Entries of the in-LDS block list.
constexpr int kMaxList = kSparseFwdMaxNk;
// Sub-tile slots per operand ring.
constexpr int kRing = 4;

// Position <-> key permutation inside a group of 16 keys (swap of quads 1, 2).
__device__ __forceinline__ int perm16(int p) {
  const int quad = p >> 2;
  const int q2 = (quad == 1) ? 2 : (quad == 2 ? 1 : quad);
  return (q2 << 2) | (p & 3);
}

template <int D, int BLK, int BK>
struct FwdCfg {
  static constexpr int NW = BLK / 32;                // waves per workgroup
  static constexpr int NT = NW * 64;                 // threads
  static constexpr int KS = D / 16;                  // k-steps of S^T = K Q^T
  static constexpr int DB = D / 32;                  // 32-row d sub-blocks of O^T
  static constexpr int NS = BK / 32;                 // 32-key sub-tiles per key block
  static constexpr int R = kRing;                    // slots per ring
  static constexpr int LEAD = D == 64 ? 6 : 4;       // MFMAs an LDS operand read leads by
  static constexpr int BPI = R / NS;                 // key blocks per unrolled loop pass
  static constexpr int SUB = 32 * D * 2;             // bytes of a K or V^T sub-tile
  static constexpr int RING = R * SUB;               // bytes of one ring
  static constexpr int LPW = SUB / (1024 * NW);      // 1 KiB wave loads per sub-tile
  static constexpr int KROW = D * 2;                 // bytes of a K row
  static constexpr int KCPR = KROW / 16;             // 16-byte chunks per K row
  static constexpr int KRPL = 256 / KROW;            // K rows per 256-byte line
  static constexpr int VDB = 32 * 64;                // bytes of 32 V^T rows in a sub-tile
  static_assert(SUB % (1024 * NW) == 0, "sub-tile must split into whole wave loads");
  static_assert(R % NS == 0 && R >= 4 && (R & 1) == 0, "ring holds whole key blocks");
  static_assert(KS == 2 * DB, "QK and PV steps alternate one to one");
  static_assert(2 * RING >= kMaxList + 4 * NW, "list-building scratch fits the rings");
};

// Swizzled chunk of K chunk c in sub-tile row `row`.
template <int D, int BLK, int BK>
__device__ __forceinline__ int kswz(int row, int c) {
  using C = FwdCfg<D, BLK, BK>;
  return c ^ ((row / C::KRPL) % C::KCPR);
}

// Keep a per-lane LDS base address opaque inside the loop, so that every
// operand read stays "base + immediate" instead of the compiler hoisting one
// precomputed address per (slot, k-step) into its own register.
__device__ __forceinline__ void launder(uint32_t& x) { asm volatile("" : "+v"(x)); }

// Unpipelined S^T = K Q^T of one sub-tile (QK) and/or O^T += V^T P^T of one
// sub-tile (PV); the prologue and the drain of the pipeline.  ka[st] is this
// lane's LDS address of its chunk for k-step st in K slot 0, va[st] the same
// in V^T slot 0; kimm / vimm select the slot.
template <int D, int BLK, int BK, bool QK, bool PV>
__device__ __forceinline__ void mfma_pair(const uint32_t* ka, uint32_t kimm, const bf16x8_t* qreg,
                                          f32x16_t& snext, const uint32_t* va, uint32_t vimm,
                                          const bf16x8_t* pprev, f32x16_t* o) {
  using C = FwdCfg<D, BLK, BK>;
  constexpr int NPV = 2 * C::DB;
#pragma unroll
  for (int i = 0; i < C::KS; ++i) {
    if constexpr (QK) {
      const bf16x8_t a = lds_read16(ka[i] + kimm);
      snext = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[i], i == 0 ? f32x16_t{} : snext, 0,
                                                      0, 0);
    }
    if constexpr (PV) {
      if (i < NPV) {
        const int st = i / C::DB, db = i % C::DB;
        const bf16x8_t a = lds_read16(va[st] + vimm + db * C::VDB);
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pprev[st], o[db], 0, 0, 0);
      }
    }
  }
}

// Probabilities of one 32-key sub-tile for this lane's 16 scores against the
// running max m_run (log2 units): bf16-packed into pcur; returns their fp32 sum.
__device__ __forceinline__ float softmax_sub(const f32x16_t& cur, float scale_log2, float m_run,
                                             bf16x8_t* pcur) {
  f32x8_t p[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      p[h][e] = fast_exp2(__builtin_fmaf(cur[8 * h + e], scale_log2, -m_run));
    pcur[h] = __builtin_convertvector(p[h], bf16x8_t);
  }
  // two interleaved sums, started from the first two terms (the same values
  // and order as starting from +0, which the compiler cannot fold away)
  float ls0 = p[0][0], ls1 = p[0][1];
#pragma unroll
  for (int e = 2; e < 16; e += 2) {
    ls0 += p[e >> 3][e & 7];
    ls1 += p[e >> 3][(e & 7) + 1];
  }
  return ls0 + ls1;
}

// One pipelined sub-iteration, issued in a fixed order: NM = KS + 2*DB MFMAs
// alternate between S^T(next) = K Q^T (a KS-long dependent chain) and
// O^T += V^T P^T(prev) (2 k-steps x DB independent chains); each MFMA's LDS
// operand is read NPRE MFMAs ahead from a small register ring.  The softmax
// of the current sub-tile runs in their shadow: under each of the first NM/2
// MFMAs two scores are scaled (v_fma) and exponentiated (v_exp, a
// transcendental), under each of the last NM/2 the bf16 packs and the row
// sums.  The NL global->LDS loads of this sub-iteration (issue(t), t < NL)
// are spread evenly over the MFMAs instead of leaving in one burst, starting
// two MFMAs in, so that the sub-iteration's first operand reads reach LDS
// ahead of the loads' writes (1 % faster than starting at the first MFMA).
// sched_group_barrier fixes this order.
template <int D, int BLK, int BK, int NPRE, int NL, typename Issue>
__device__ __forceinline__ float pipeline_step(const uint32_t* ka, uint32_t kimm,
                                               const bf16x8_t* qreg, f32x16_t& snext,
                                               const uint32_t* va, uint32_t vimm,
                                               const bf16x8_t* pprev, f32x16_t* o, f32x16_t& cur,
                                               float scale_log2, float m_run, bf16x8_t* pcur,
                                               Issue&& issue) {
  using C = FwdCfg<D, BLK, BK>;
  constexpr int NM = C::KS + 2 * C::DB;
  static_assert(NM == 16 || NM == 8, "softmax split written for 8 or 16 MFMAs");
  static_assert(NL <= NM, "at most one load per MFMA");
  constexpr int EPM = 32 / NM;  // exponentials per MFMA in the first half
  auto read_op = [&](int i) -> bf16x8_t {
    if ((i & 1) == 0) return lds_read16(ka[i >> 1] + kimm);
    const int st = (i >> 1) / C::DB, db = (i >> 1) % C::DB;
    return lds_read16(va[st] + vimm + db * C::VDB);
  };
  // load t is issued right after MFMA OFF + t * SP
  static_assert(NM % NL == 0, "loads spread evenly");
  constexpr int SP = NM / NL;
  constexpr int OFF = SP > 2 ? 2 : SP - 1;
  auto has_load = [&](int i) { return i >= OFF && (i - OFF) % SP == 0; };
  bf16x8_t ring[NPRE];
#pragma unroll
  for (int i = 0; i < NPRE; ++i) ring[i] = read_op(i);
  f32x8_t p[2];
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    const bf16x8_t a = ring[i % NPRE];
    if ((i & 1) == 0) {
      const int st = i >> 1;
      snext = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[st], st == 0 ? f32x16_t{} : snext,
                                                      0, 0, 0);
    } else {
      const int st = (i >> 1) / C::DB, db = (i >> 1) % C::DB;
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pprev[st], o[db], 0, 0, 0);
    }
    if (i + NPRE < NM) ring[i % NPRE] = read_op(i + NPRE);
    if (has_load(i)) issue((i - OFF) / SP);
    if (i < NM / 2) {
#pragma unroll
      for (int u = 0; u < EPM; ++u) {
        const int e = i * EPM + u;
        p[e >> 3][e & 7] = fast_exp2(__builtin_fmaf(cur[e], scale_log2, -m_run));
      }
    }
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) pcur[h] = __builtin_convertvector(p[h], bf16x8_t);
  // two interleaved row sums, started from the first two terms (the same
  // values and order as starting from +0, which the compiler cannot fold)
  float ls0 = p[0][0], ls1 = p[0][1];
#pragma unroll
  for (int e = 2; e < 16; e += 2) {
    ls0 += p[e >> 3][e & 7];
    ls1 += p[e >> 3][(e & 7) + 1];
  }
  // fixed issue order: the NPRE lead reads; then per MFMA the next read, its
  // load if it has one, and either EPM (fma, exp) pairs or its share of the
  // 8 packs and 14 sums of the second half
  constexpr int TAIL = 22;
  __builtin_amdgcn_sched_group_barrier(0x100, NPRE, 0);
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i + NPRE < NM) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    if (has_load(i)) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read
    if (i < NM / 2) {
      __builtin_amdgcn_sched_group_barrier(0x002, EPM, 0);  // v_fma
      __builtin_amdgcn_sched_group_barrier(0x400, EPM, 0);  // v_exp
    } else {
      __builtin_amdgcn_sched_group_barrier(0x002, (2 * TAIL + NM - 1) / NM, 0);  // packs / sums
    }
  }
  // pin the softmax results here: otherwise the compiler sinks the exp2 work
  // next to its consumers in the following sub-iteration, out of the shadow
  // of these MFMAs
  float ls = ls0 + ls1;
  asm volatile("" : "+v"(ls), "+v"(pcur[0]), "+v"(pcur[1]));
  return ls;
}

// Raw-score maximum of a 32-key sub-tile for this lane's query (both halves).
__device__ __forceinline__ float sub_max(const f32x16_t& s) {
  float m = s[0];
#pragma unroll
  for (int t = 1; t < 16; ++t) m = fmaxf(m, s[t]);
  return max_with_partner(m);
}

// Scores of sub-tile `part`'s keys at or beyond kvalid (block-relative) -> -inf.
__device__ __forceinline__ void mask_sub(f32x16_t& s, int part, int kvalid, int g) {
#pragma unroll
  for (int t = 0; t < 16; ++t) {
    const int key = part * 32 + ((t >> 2) << 3) + (g << 2) + (t & 3);
    if (key >= kvalid) s[t] = -INFINITY;
  }
}

// Bound on one lane's sum of 16 probabilities of a sub-tile (so on each of
// them) before the running max must be raised.  The running max then trails
// the true one by at most log2 of it; l and O stay far from fp32 overflow
// (at most 2^20 per key over at most 2^19 keys).
constexpr float kSumBound = 1048576.0f;

// Waves per SIMD the register budget is cut for.  128-row query blocks: two at
// d = 128 (output accumulators, Q operands and two score tiles take ~250
// registers); three at d = 64, where a wave's VALU work per MFMA is twice that
// of d = 128 and a third wave hides more of it (168 registers; the rings and
// block list, 40 KiB per workgroup, allow four).  64-row blocks are limited by
// LDS instead.
template <int D, int BLK>
constexpr int fwd_waves_per_simd() {
  return BLK == 128 ? (D == 64 ? 3 : 2) : 1;
}

template <int D, int BLK, int BK, bool DENSE>
__global__ void __launch_bounds__(BLK * 2)
    __attribute__((amdgpu_waves_per_eu(fwd_waves_per_simd<D, BLK>())))
    sparse_fwd_bf16_kernel(const __bf16* __restrict__ Q, const __bf16* __restrict__ K,
                           const __bf16* __restrict__ Vt, const int32_t* __restrict__ row_ptr,
                           const int32_t* __restrict__ col_idx, int64_t col_len,
                           __bf16* __restrict__ O, float* __restrict__ lse,
                           float* __restrict__ bstat, const int* __restrict__ order, int n_q,
                           int n_k, int N, int n_pad, float scale_log2) {
  using C = FwdCfg<D, BLK, BK>;
  constexpr int NS = C::NS;
  constexpr int R = C::R;
  constexpr int BPI = C::BPI;
  // K ring at smem, V^T ring at smem + RING; slot x at + x*SUB
  __shared__ __attribute__((aligned(1024))) char smem[2 * C::RING];
  __shared__ uint16_t list[kMaxList];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31;
  const int g = lane >> 5;

  // DENSE: every row keeps every key block that holds a valid key (the dense
  // attention of the construction step); rows run in id order, each XCD on a
  // contiguous range of them.  A template flag, so that the two modes are
  // separate kernels in a trace.
  const int r = DENSE ? xcd_remap(blockIdx.x, gridDim.x) : order[blockIdx.x];
  const int bh = r / n_q;
  const int qb = r - bh * n_q;
  const size_t head = (size_t)bh * n_pad * D;
  const uint32_t head_bytes = (uint32_t)((size_t)n_pad * D * 2);
  const i32x4_t krs = rsrc_words(K + head, head_bytes);
  const i32x4_t vrs = rsrc_words(Vt + head, head_bytes);

  // ---- the row's distinct valid key blocks, ascending ---------------------
  // (flags and per-wave counts live in the rings, unused until the first load)
  int nb = 0;
  if constexpr (DENSE) {
    nb = (N + BK - 1) / BK;
    for (int j = tid; j < nb; j += C::NT) list[j] = (uint16_t)j;
    __syncthreads();
  } else {
    uint8_t* const flag = reinterpret_cast<uint8_t*>(smem);
    int* const wcount = reinterpret_cast<int*>(smem + kMaxList);
    for (int j = tid; j < n_k; j += C::NT) flag[j] = 0;
    __syncthreads();
    int64_t e0 = row_ptr[r], e1 = row_ptr[r + 1];
    e0 = e0 < 0 ? 0 : (e0 > col_len ? col_len : e0);
    e1 = e1 < e0 ? e0 : (e1 > col_len ? col_len : e1);
    for (int64_t e = e0 + tid; e < e1; e += C::NT) {
      const int j = col_idx[e];
      if (j >= 0 && j < n_k) flag[j] = 1;
    }
    __syncthreads();
    for (int c0 = 0; c0 < n_k; c0 += C::NT) {
      const int j = c0 + tid;
      const bool f = (j < n_k) && flag[j] != 0;
      const uint64_t bal = __ballot(f);
      const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
      if (lane == 0) wcount[w] = __popcll(bal);
      __syncthreads();
      int before = 0, total = 0;
#pragma unroll
      for (int x = 0; x < C::NW; ++x) {
        const int c = wcount[x];
        before += (x < w) ? c : 0;
        total += c;
      }
      if (f) list[nb + before + below] = (uint16_t)j;
      nb += total;
      __syncthreads();
    }
    nb = __builtin_amdgcn_readfirstlane(nb);
  }
  // sub-tiles in the stream.  With 32-key blocks (one sub-tile each) the
  // stream is padded to whole loop passes with sub-tiles whose keys are all
  // masked (they add nothing to O or l); larger blocks fill passes exactly,
  // or leave half a pass that the loop stops after.
  const int S_real = nb * NS;
  const int S = (NS == 1) ? (S_real + R - 1) / R * R : S_real;

  // this lane's query row and its Q^T operand (8 bf16 per k-step).  Padding
  // rows take Q = 0, so their scores stay finite whatever the padding holds
  // (their output is written as 0 in the epilogue).
  const int qrow = qb * BLK + w * 32 + l32;
  bf16x8_t qreg[C::KS];
  {
    const bf16x8_t* qp = reinterpret_cast<const bf16x8_t*>(Q + head + (size_t)qrow * D);
    const bool qvalid = qrow < N;
#pragma unroll
    for (int st = 0; st < C::KS; ++st) qreg[st] = qvalid ? qp[2 * st + g] : bf16x8_t{};
  }
  // per-lane LDS addresses of the operand reads in K slot 0 / V^T slot 0; the
  // slot and the d sub-block are immediates
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)smem;
  uint32_t ka[C::KS], va[2];
#pragma unroll
  for (int st = 0; st < C::KS; ++st)
    ka[st] = lds0 + l32 * C::KROW + (kswz<D, BLK, BK>(l32, 2 * st + g) << 4);
#pragma unroll
  for (int st = 0; st < 2; ++st)
    va[st] = lds0 + C::RING + (l32 >> 2) * 256 +
             (((l32 & 3) << 2) + ((2 * st + g) ^ ((l32 >> 2) & 3))) * 16;
  // per-lane global offsets of the direct loads (LDS position o of a K sub-tile
  // holds row o / KROW, chunk kswz(row, (o % KROW) / 16); V^T is stored as the
  // LDS image)
  uint32_t koffs[C::LPW];
#pragma unroll
  for (int u = 0; u < C::LPW; ++u) {
    const int o = (w * C::LPW + u) * 1024 + lane * 16;
    const int row = o / C::KROW;
    koffs[u] = (uint32_t)(row * C::KROW + (kswz<D, BLK, BK>(row, (o % C::KROW) >> 4) << 4));
  }
  const uint32_t voff0 = (uint32_t)(w * C::LPW * 1024 + lane * 16);

  // key sub-tile (block j, part) -> K slot x / V^T slot x
  auto load_k = [&](int x, int j, int part) {
#pragma unroll
    for (int u = 0; u < C::LPW; ++u)
      dma16(lds0 + x * C::SUB + (w * C::LPW + u) * 1024, krs, koffs[u],
            (uint32_t)((j * BK + part * 32) * C::KROW));
  };
  auto load_v = [&](int x, int j, int part) {
#pragma unroll
    for (int u = 0; u < C::LPW; ++u)
      dma16(lds0 + C::RING + x * C::SUB + (w * C::LPW + u) * 1024, vrs, voff0 + u * 1024,
            (uint32_t)((j * NS + part) * C::SUB));
  };
  // list entry x as a scalar, clamped into the list
  auto block_at = [&](int x) -> int {
    return __builtin_amdgcn_readfirstlane((int)list[x < nb ? x : nb - 1]);
  };

  f32x16_t oacc[C::DB];
#pragma unroll
  for (int db = 0; db < C::DB; ++db) oacc[db] = f32x16_t{};
  float m_run = kNegBig;  // max used for exp2 (scaled units)
  float l_run = 0.f;      // this lane's share of the row sum
  float b_run = 0.f;      // DENSE: this lane's share of the current key block's sum
  f32x16_t sc[2];         // raw scores of the sub-tiles with even / odd index
  bf16x8_t pb[2][2];      // bf16 probabilities of the sub-tiles with even / odd index

  if (S > 0) {
    int jc[BPI], jn[BPI];  // blocks of this loop pass's sub-tiles and the next pass's
    // prologue: K sub-tiles 0..R-1, V^T sub-tiles 0..R-3 (past the end of
    // the stream the last block again, so that no slot holds stale bytes);
    // zero V^T slot R-1 and the probabilities of "sub-tile -1"; scores of
    // sub-tile 0
#pragma unroll
    for (int x = 0; x < BPI; ++x) {
      jc[x] = block_at(x);
      jn[x] = block_at(BPI + x);
    }
#pragma unroll
    for (int y = 0; y < R; ++y) {
      const int jy = (y / NS < BPI) ? jc[y / NS] : jn[y / NS - BPI];
      load_k(y, jy, y % NS);
      if (y < R - 2) load_v(y, jy, y % NS);
    }
    for (int x = tid * 16; x < C::SUB; x += C::NT * 16)
      *reinterpret_cast<f32x4_t*>(smem + C::RING + (R - 1) * C::SUB + x) = f32x4_t{};
#pragma unroll
    for (int a2 = 0; a2 < 2; ++a2)
#pragma unroll
      for (int st = 0; st < 2; ++st) pb[a2][st] = bf16x8_t{};
    wait_vm_barrier<0>();
    mfma_pair<D, BLK, BK, true, false>(ka, 0, qreg, sc[0], va, 0, pb[1], oacc);

    // Sub-iteration s = R*u + H (H static).  On entry the raw scores of s are
    // in sc[H & 1] and the probabilities of s-1 in pb[(H + 1) & 1].  The
    // matrix cores compute the scores of s+1 (K slot (H+1) % R) alternating
    // with P V of s-1 (V^T slot (H-1) % R); the VALU exponentiates s.  A
    // rescale found necessary for s is applied after P V(s-1), before P V(s).
    // The scores computed for sub-tile S (after the last) are never used; the
    // first P V multiplies zero probabilities with the zeroed slot.
    auto sub_iter = [&](auto hh, int u) {
      constexpr int H = decltype(hh)::value;
      const int s = R * u + H;
      f32x16_t& cur = sc[H & 1];
      f32x16_t& nxt = sc[(H + 1) & 1];
#pragma unroll
      for (int st = 0; st < C::KS; ++st) launder(ka[st]);
      launder(va[0]);
      launder(va[1]);
      // K sub-tile s+1 and V^T sub-tile s-1 (both issued in sub-iteration
      // s-3, so not among the last two sub-iterations' loads that the count
      // leaves in flight) have landed for every wave, and every wave is done
      // with sub-iteration s-1.  Every sub-iteration issues the same loads
      // (past the end of the stream they fetch the last block again), so the
      // count is exact.
      wait_vm_barrier<(R - 2) * 2 * C::LPW>();
      constexpr int HV = H + R - 2;  // pass-relative index of sub-tile s+R-2
      const int jk = jn[H / NS];
      const int jv = (HV < R) ? jc[(HV < R ? HV : 0) / NS] : jn[(HV < R ? 0 : HV - R) / NS];
      // refill: K slot H <- K sub-tile s+R, V^T slot (H+R-2) % R <- sub-tile s+R-2
      auto issue = [&](int t) {
        if (t < C::LPW) {
          dma16(lds0 + H * C::SUB + (w * C::LPW + t) * 1024, krs, koffs[t],
                (uint32_t)((jk * BK + (H % NS) * 32) * C::KROW));
        } else {
          const int u = t - C::LPW;
          dma16(lds0 + C::RING + (HV % R) * C::SUB + (w * C::LPW + u) * 1024, vrs, voff0 + u * 1024,
                (uint32_t)((jv * NS + HV % NS) * C::SUB));
        }
      };
      // ragged last key block: mask the keys >= N of this sub-tile; a
      // padding sub-tile past the real stream is masked whole
      const int kvb = (R * u + H < S_real) ? N - jc[H / NS] * BK : 0;
      if (kvb < (H % NS + 1) * 32) mask_sub(cur, H % NS, kvb, g);
      // raised wave priority while the matrix cores are fed: when both waves
      // of a SIMD have instructions ready, the one inside its MFMA stream issues
      __builtin_amdgcn_s_setprio(1);
      float ls = pipeline_step<D, BLK, BK, C::LEAD, 2 * C::LPW>(ka, ((H + 1) % R) * C::SUB, qreg, nxt, va,
                                          ((H + R - 1) % R) * C::SUB, pb[(H + 1) & 1], oacc,
                                          cur, scale_log2, m_run, pb[H & 1], issue);
      __builtin_amdgcn_s_setprio(0);
      // The probabilities of s were taken against the running max without
      // looking at this sub-tile's scores.  If a lane's sum exceeds the bound
      // (or is inf: the first sub-tile, or a jump of the max), raise the max
      // to this sub-tile's and redo them; O^T, which now holds P V up to s-1,
      // and l move to the new reference.  Every probability that reaches P V
      // is therefore at most kSumBound.
      if (__ballot(!(ls <= kSumBound)) != 0) {
        const float ms = sub_max(cur) * scale_log2;
        const float m_new = fmaxf(m_run, ms);
        const float alpha = fast_exp2(m_run - m_new);
        m_run = m_new;
        l_run *= alpha;
        if constexpr (DENSE) b_run *= alpha;
#pragma unroll
        for (int db = 0; db < C::DB; ++db) oacc[db] *= alpha;
        ls = softmax_sub(cur, scale_log2, m_run, pb[H & 1]);
      }
      l_run += ls;
      if constexpr (DENSE) {
        // block statistic of the construction step: log2 of the query's
        // unnormalised probability sum over key block jc[H / NS] (its last
        // sub-tile is s), in absolute units, for the block-mass reduction
        b_run += ls;
        if constexpr (H % NS == NS - 1) {
          const float bt = add_partner(b_run);
          b_run = 0.f;
          if (bstat != nullptr && s < S_real && g == 0)
            bstat[((size_t)bh * n_k + jc[H / NS]) * n_pad + qrow] = __log2f(bt) + m_run;
        }
      }
    };

    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    static_assert(R == 4, "loop body written for a ring of 4");
    for (int u = 0;; ++u) {
      // block ids of the pass after next: the LDS read completes at the next
      // barrier and is consumed at the end of this pass
      int jf[BPI];
#pragma unroll
      for (int x = 0; x < BPI; ++x) {
        const int xi = (u + 2) * BPI + x;
        jf[x] = (int)list[xi < nb ? xi : nb - 1];
      }
      sub_iter(I0{}, u);
      sub_iter(I1{}, u);
      if constexpr (NS == 2) {
        if (R * u + 2 >= S) break;
      }
      sub_iter(I2{}, u);
      sub_iter(I3{}, u);
      if (R * (u + 1) >= S) break;
#pragma unroll
      for (int x = 0; x < BPI; ++x) {
        jc[x] = jn[x];
        jn[x] = __builtin_amdgcn_readfirstlane(jf[x]);
      }
    }
    // drain: P V of the last sub-tile S-1 (odd, so its probabilities are
    // pb[1]).  Its V^T slot was filled in sub-iteration S-3, one part by each
    // wave, and the last barrier only covered loads up to S-4: every wave
    // waits for all of its own loads (the later ones included, which nothing
    // reads, so that none lands after the workgroup's LDS is handed on), then
    // a barrier makes every wave's part visible.
    wait_vm_barrier<0>();
    mfma_pair<D, BLK, BK, false, true>(ka, 0, qreg, sc[0], va, (uint32_t)(((S - 1) % R) * C::SUB),
                                   pb[1], oacc);
  }

  // ---- epilogue: O = O^T / l, lse -----------------------------------------
  const float l_tot = add_partner(l_run);
  const bool row_ok = (qrow < N) && (l_tot > 0.f);
  const float inv = row_ok ? 1.0f / l_tot : 0.f;
  __bf16* orow = O + head + (size_t)qrow * D;
#pragma unroll
  for (int db = 0; db < C::DB; ++db)
#pragma unroll
    for (int qd = 0; qd < 4; ++qd) {
      f32x4_t v;
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = oacc[db][qd * 4 + u] * inv;
      const int d0 = db * 32 + qd * 8 + g * 4;
      *reinterpret_cast<bf16x4_t*>(orow + d0) = __builtin_convertvector(v, bf16x4_t);
    }
  if (lse != nullptr && g == 0) {
    lse[(size_t)bh * n_pad + qrow] = row_ok ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

// Dispatch order of the CSR rows.  Workgroup ids are dealt round-robin over
// the 8 XCDs, so id 8*k + x runs on XCD x as that XCD's k-th row.  XCD x gets
// a contiguous range of rows, cut into chunks of kOrderChunk consecutive rows
// (neighbouring query blocks of one head, which retain mostly the same key
// blocks).  The chunks run in order, so the rows in flight on an XCD at any
// time come from one or two chunks and share its L2; inside a chunk rows go
// longest first (longest-processing-time-first list scheduling), so the tail
// of the launch is made of short rows.  Ties keep the row order.  The order
// changes only the schedule, never a result.
constexpr int kOrderChunk = 128;

// One workgroup per (chunk c = blockIdx.x, XCD x = blockIdx.y): the chunk's
// row lengths go to LDS, then each thread ranks one row against them.
__global__ void __launch_bounds__(kOrderChunk)
    order_rows_kernel(const int32_t* __restrict__ row_ptr, int64_t col_len, int rows, int n_k,
                      int* __restrict__ order) {
  __shared__ int len[kOrderChunk];
  const int x = blockIdx.y;
  const int c0 = blockIdx.x * kOrderChunk;
  auto count_of = [&](int y) { return rows > y ? (rows - y + 7) / 8 : 0; };
  const int cnt = count_of(x);
  if (c0 >= cnt) return;  // this XCD has fewer chunks (uniform per workgroup)
  int start = 0;  // XCD x owns rows [start, start + cnt)
  for (int y = 0; y < x; ++y) start += count_of(y);
  const int n = min(cnt - c0, kOrderChunk);
  const int t = threadIdx.x;
  if (t < n) {
    const int r = start + c0 + t;
    int64_t e0 = row_ptr[r], e1 = row_ptr[r + 1];
    e0 = e0 < 0 ? 0 : (e0 > col_len ? col_len : e0);
    e1 = e1 < e0 ? e0 : (e1 > col_len ? col_len : e1);
    len[t] = (int)(e1 - e0 < n_k ? e1 - e0 : n_k);
  }
  __syncthreads();
  if (t < n) {
    const int mine = len[t];
    int rank = 0;  // rows of the chunk that go before this one
    for (int y = 0; y < n; ++y) rank += (len[y] > mine) || (len[y] == mine && y < t);
    order[(c0 + rank) * 8 + x] = start + c0 + t;
  }
}

// V [BH][n_pad][D] -> V^T in the LDS image of its 32-key sub-tiles: sub-tile y
// of a head is SUB contiguous bytes, 16-byte chunk p of it holds d = 4*(p/16) +
// (p/4)%4 and key positions 8c..8c+7 with c = (p%4) ^ ((p/16)%4); position q
// of a 32-key sub-tile holds key (q & ~15) | perm16(q & 15).  One workgroup
// transposes 64 keys (two sub-tiles) x D of one head through LDS.
template <int D>
__global__ void __launch_bounds__(256)
    transpose_v_kernel(const __bf16* __restrict__ V, __bf16* __restrict__ Vt, int n_pad) {
  constexpr int TK = 64;
  constexpr int LD = D + 2;  // padded LDS row (elements)
  __shared__ __bf16 tile[TK * LD];
  const int bh = blockIdx.y;
  const int n0 = blockIdx.x * TK;
  const __bf16* src = V + (size_t)bh * n_pad * D + (size_t)n0 * D;
  __bf16* dst = Vt + (size_t)bh * n_pad * D + (size_t)n0 * D;
  for (int c = threadIdx.x; c < TK * D / 8; c += 256) {
    const int row = c / (D / 8);
    const int col = (c % (D / 8)) * 8;
    const bf16x8_t v = *reinterpret_cast<const bf16x8_t*>(src + (size_t)row * D + col);
#pragma unroll
    for (int t = 0; t < 8; ++t) tile[row * LD + col + t] = v[t];
  }
  __syncthreads();
  // output chunk q: sub-tile q / (4D), chunk p = q % (4D) of it
  for (int q = threadIdx.x; q < TK * D / 8; q += 256) {
    const int y = q / (4 * D);
    const int p = q % (4 * D);
    const int line = p >> 4;
    const int d = line * 4 + ((p >> 2) & 3);
    const int c = (p & 3) ^ (line & 3);
    bf16x8_t v;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int pos = c * 8 + t;
      const int key = y * 32 + ((pos & ~15) | perm16(pos & 15));
      v[t] = tile[key * LD + d];
    }
    *reinterpret_cast<bf16x8_t*>(dst + (size_t)q * 8) = v;
  }
}

// Workspace layout: V^T (B*H*n_pad*D bf16), then the dispatch order (one int
// per row) at the next 256-byte boundary.
size_t vt_bytes(int BH, int n_pad, int d) { return ((size_t)BH * n_pad * d * 2 + 255) / 256 * 256; }

template <int D, int BLK, int BK>
hipError_t launch_fwd(const void* q, const void* k, const void* v, int B, int H, int N, int n_pad,
                      float scale, const int32_t* row_ptr, const int32_t* col_idx,
                      int64_t col_len, void* o, float* lse, void* workspace, hipStream_t stream) {
  const int BH = B * H;
  const int n_q = n_pad / BLK;
  const int n_k = n_pad / BK;
  const int rows = BH * n_q;
  __bf16* vt = static_cast<__bf16*>(workspace);
  int* order = reinterpret_cast<int*>(static_cast<char*>(workspace) + vt_bytes(BH, n_pad, D));
  const int per_xcd = (rows + 7) / 8;
  hipLaunchKernelGGL(order_rows_kernel, dim3((per_xcd + kOrderChunk - 1) / kOrderChunk, 8),
                     dim3(kOrderChunk), 0, stream, row_ptr, col_len, rows, n_k, order);
  dim3 tgrid(n_pad / 64, BH);
  hipLaunchKernelGGL(transpose_v_kernel<D>, tgrid, dim3(256), 0, stream,
                     static_cast<const __bf16*>(v), vt, n_pad);
  hipLaunchKernelGGL((sparse_fwd_bf16_kernel<D, BLK, BK, false>), dim3(rows),
                     dim3(FwdCfg<D, BLK, BK>::NT), 0, stream, static_cast<const __bf16*>(q),
                     static_cast<const __bf16*>(k), static_cast<const __bf16*>(vt), row_ptr,
                     col_idx, col_len, static_cast<__bf16*>(o), lse, nullptr, order, n_q, n_k, N,
                     n_pad, scale * kLog2e);
  return hipGetLastError();
}

// Dense attention of every query block over every valid key (the forward
// kernel with full rows): O, lse and, if stat is given, the block statistics
// of the construction step.
template <int D, int BLK, int BK>
hipError_t launch_dense(const void* q, const void* k, const void* v, int B, int H, int N,
                        int n_pad, float scale, void* o, float* lse, float* stat, void* workspace,
                        hipStream_t stream) {
  const int BH = B * H;
  const int n_q = n_pad / BLK;
  const int n_k = n_pad / BK;
  const int rows = BH * n_q;
  __bf16* vt = static_cast<__bf16*>(workspace);
  dim3 tgrid(n_pad / 64, BH);
  hipLaunchKernelGGL(transpose_v_kernel<D>, tgrid, dim3(256), 0, stream,
                     static_cast<const __bf16*>(v), vt, n_pad);
  hipLaunchKernelGGL((sparse_fwd_bf16_kernel<D, BLK, BK, true>), dim3(rows),
                     dim3(FwdCfg<D, BLK, BK>::NT), 0, stream, static_cast<const __bf16*>(q),
                     static_cast<const __bf16*>(k), static_cast<const __bf16*>(vt), nullptr,
                     nullptr, 0, static_cast<__bf16*>(o), lse, stat, nullptr, n_q, n_k, N, n_pad,
                     scale * kLog2e);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sparse_fwd_bf16(int d, int blk, int blk_k, const void* q, const void* k,
                                  const void* v, int B, int H, int N, int n_pad, float scale,
                                  const int32_t* row_ptr, const int32_t* col_idx,
                                  int64_t col_len, void* o, float* lse, void* workspace,
                                  hipStream_t stream) {
#define LOSA_FWD(DD, BB, KK)                                                                 \
  if (d == DD && blk == BB && blk_k == KK)                                                   \
    return launch_fwd<DD, BB, KK>(q, k, v, B, H, N, n_pad, scale, row_ptr, col_idx, col_len, \
                                  o, lse, workspace, stream);
  LOSA_FWD(128, 128, 128)
  LOSA_FWD(64, 128, 128)
  LOSA_FWD(128, 64, 64)
  LOSA_FWD(64, 64, 64)
  LOSA_FWD(128, 128, 32)
  LOSA_FWD(64, 128, 32)
  LOSA_FWD(128, 64, 32)
  LOSA_FWD(64, 64, 32)
#undef LOSA_FWD
  return hipErrorInvalidValue;
}

hipError_t launch_dense_bf16(int d, int blk, int blk_k, const void* q, const void* k,
                             const void* v, int B, int H, int N, int n_pad, float scale, void* o,
                             float* lse, float* stat, void* workspace, hipStream_t stream) {
#define LOSA_DENSE(DD, BB, KK)                                                                \
  if (d == DD && blk == BB && blk_k == KK)                                                    \
    return launch_dense<DD, BB, KK>(q, k, v, B, H, N, n_pad, scale, o, lse, stat, workspace, \
                                    stream);
  LOSA_DENSE(128, 128, 128)
  LOSA_DENSE(64, 128, 128)
  LOSA_DENSE(128, 64, 64)
  LOSA_DENSE(64, 64, 64)
  LOSA_DENSE(128, 128, 32)
  LOSA_DENSE(64, 128, 32)
  LOSA_DENSE(128, 64, 32)
  LOSA_DENSE(64, 64, 32)
#undef LOSA_DENSE
  return hipErrorInvalidValue;
}

size_t sparse_fwd_bf16_workspace(int B, int H, int n_pad, int d, int n_q) {
  // V^T in sub-tile LDS images, then the rows' dispatch order
  return vt_bytes(B * H, n_pad, d) + (size_t)B * H * n_q * sizeof(int);
}

}  // namespace losa
