// Frozen-support block-sparse attention forward (Sec. 4.2, Eq. (4)), bf16 in,
// fp32 accumulation, on gfx950 MFMA.
//
// One workgroup owns one CSR row r = (b*H + h)*n_q + i, i.e. the BLK query rows
// of query block i, and walks only the key blocks listed for it.  Each of its
// BLK/32 waves owns 32 query rows.
//
// Orientation.  Per 32-key sub-block the wave computes S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16 (A = K rows from LDS, B = the wave's Q^T held in
// registers).  In the 32x32 accumulator layout a lane holds 16 scores of ONE
// query (column = lane % 32), so the online softmax (running max m, running
// sum l) is in-lane, plus one exchange with lane ^ 32 which holds the other
// keys of the same query.  The exponentiated scores are already laid out as
// the B operand of O^T = V^T P^T, and the O^T accumulator again keeps one
// query per lane, so the per-query rescale by exp2(m_old - m_new) and the
// final 1/l are in-lane too.
//
// Key order inside a 16-key MFMA step.  The B operand P^T of lane group g
// (lanes 32g..32g+31) holds, in register element e, the key
//   16*step + 4*g + e + (e >= 4 ? 4 : 0),
// which is where the S^T accumulator put it.  The A operand V^T must hold the
// same key in the same (lane group, element) slot; the transposed copy of V
// therefore stores, within every group of 16 keys, positions 4..7 and 8..11
// swapped (an involution), so each lane's 8 keys are 16 contiguous bytes.
//
// Staging.  K tiles ([BLK keys][D]) and V^T tiles ([D][BLK keys]) are copied
// HBM -> LDS with 16-byte buffer loads that write LDS directly (no register
// round trip).  16-byte chunks are XOR-swizzled by row so that the MFMA operand
// reads (32 rows, one chunk column) hit distinct banks.  The K buffer is
// refilled as soon as all waves have finished S for the current tile, the V
// buffer as soon as P V is done, so the next tile's loads overlap the softmax
// and the P V product.  Two workgroups share a CU (64 KiB of LDS each).
//
// Padding.  Keys >= N get score -inf (only the ragged last block needs it).
// Query rows >= N are written as 0 with lse = -inf; so are rows with an empty
// key set.  Entries of col_idx outside [0, n_k) contribute nothing, and row
// bounds are clamped to [0, col_idx_len], so a corrupt CSR cannot read out of
// bounds.
#include "common.hpp"
#include "launch.hpp"

namespace losa {

namespace {

// Position <-> key permutation inside a group of 16 keys (swap of quads 1, 2).
__device__ __forceinline__ int perm16(int p) {
  const int quad = p >> 2;
  const int q2 = (quad == 1) ? 2 : (quad == 2 ? 1 : quad);
  return (q2 << 2) | (p & 3);
}

template <int D, int BLK>
struct FwdCfg {
  static constexpr int NW = BLK / 32;               // waves per workgroup
  static constexpr int NT = NW * 64;                // threads
  static constexpr int KS = D / 16;                 // k-steps of S^T = K Q^T
  static constexpr int KB = BLK / 32;               // 32-key sub-blocks per tile
  static constexpr int PS = BLK / 16;               // k-steps of O^T = V^T P^T
  static constexpr int DB = D / 32;                 // 32-row d sub-blocks
  static constexpr int KROW = D * 2;                // bytes of one K row in LDS
  static constexpr int KCH = D / 8;                 // 16-byte chunks per K row
  static constexpr int VROW = BLK * 2;              // bytes of one V^T row in LDS
  static constexpr int VCH = BLK / 8;               // 16-byte chunks per V^T row
  static constexpr int TILE = BLK * D * 2;          // bytes of a K or V^T tile
  static constexpr int LOADS = TILE / (1024 * NW);  // wave loads per tile per wave
  static_assert(TILE % (1024 * NW) == 0, "tile must split into whole wave loads");
  static_assert(KCH >= 8 && VCH >= 8, "swizzle needs >= 8 chunks per row");
};

// Issue the direct loads of K tile j (rows j*BLK.., all D) into LDS.
template <int D, int BLK>
__device__ __forceinline__ void issue_k_tile(char* Ks, __amdgpu_buffer_rsrc_t rs, int j, int w,
                                             int lane) {
  using C = FwdCfg<D, BLK>;
#pragma unroll
  for (int u = 0; u < C::LOADS; ++u) {
    const int base = (w * C::LOADS + u) * 1024;
    const int o = base + lane * 16;
    const int row = o / C::KROW;
    const int pch = (o % C::KROW) >> 4;
    const int c = pch ^ (row % C::KCH);
    const uint32_t voff = (uint32_t)(((j * BLK + row) * D + c * 8) * 2);
    load_lds_16(rs, Ks + base, voff);
  }
}

// Issue the direct loads of V^T tile j (all D rows, keys j*BLK..) into LDS.
template <int D, int BLK>
__device__ __forceinline__ void issue_v_tile(char* Vs, __amdgpu_buffer_rsrc_t rs, int j,
                                             int n_pad, int w, int lane) {
  using C = FwdCfg<D, BLK>;
#pragma unroll
  for (int u = 0; u < C::LOADS; ++u) {
    const int base = (w * C::LOADS + u) * 1024;
    const int o = base + lane * 16;
    const int row = o / C::VROW;
    const int pch = (o % C::VROW) >> 4;
    const int c = pch ^ (row % C::VCH);
    const uint32_t voff = (uint32_t)(((size_t)row * n_pad + j * BLK + c * 8) * 2);
    load_lds_16(rs, Vs + base, voff);
  }
}

template <int D, int BLK>
__global__ void __launch_bounds__(BLK * 2, 2)
    sparse_fwd_bf16_kernel(const __bf16* __restrict__ Q, const __bf16* __restrict__ K,
                           const __bf16* __restrict__ Vt, const int32_t* __restrict__ row_ptr,
                           const int32_t* __restrict__ col_idx, int64_t col_len,
                           __bf16* __restrict__ O, float* __restrict__ lse, int rows_total,
                           int n_q, int n_k, int N, int n_pad, float scale_log2) {
  using C = FwdCfg<D, BLK>;
  __shared__ __attribute__((aligned(1024))) char smem[2 * C::TILE];
  char* Ks = smem;
  char* Vs = smem + C::TILE;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31;
  const int g = lane >> 5;

  const int r = xcd_remap(blockIdx.x, rows_total);
  const int bh = r / n_q;
  const int i = r - bh * n_q;
  const size_t head = (size_t)bh * n_pad * D;
  const uint32_t head_bytes = (uint32_t)((size_t)n_pad * D * 2);
  const __amdgpu_buffer_rsrc_t krs = make_rsrc(K + head, head_bytes);
  const __amdgpu_buffer_rsrc_t vrs = make_rsrc(Vt + head, head_bytes);

  int64_t e0 = row_ptr[r];
  int64_t e1 = row_ptr[r + 1];
  e0 = e0 < 0 ? 0 : (e0 > col_len ? col_len : e0);
  e1 = e1 < e0 ? e0 : (e1 > col_len ? col_len : e1);

  // this lane's query row and its Q^T operand (8 bf16 per k-step)
  const int qrow = i * BLK + w * 32 + l32;
  bf16x8_t qreg[C::KS];
  {
    const bf16x8_t* qp = reinterpret_cast<const bf16x8_t*>(Q + head + (size_t)qrow * D);
#pragma unroll
    for (int s = 0; s < C::KS; ++s) qreg[s] = qp[2 * s + g];
  }

  // per-lane LDS byte offsets of the operand reads (row part added per sub-block)
  const int ksw = l32 % C::KCH;
  const int vsw = l32 % C::VCH;

  f32x16_t oacc[C::DB];
#pragma unroll
  for (int db = 0; db < C::DB; ++db)
#pragma unroll
    for (int t = 0; t < 16; ++t) oacc[db][t] = 0.f;
  float m_run = kNegBig;
  float l_run = 0.f;

  auto block_of = [&](int64_t e) -> int {
    const int j = __builtin_amdgcn_readfirstlane(col_idx[e]);
    return j;
  };

  int j_cur = 0;
  if (e0 < e1) {
    j_cur = block_of(e0);
    const int jl = (j_cur >= 0 && j_cur < n_k) ? j_cur : 0;
    issue_k_tile<D, BLK>(Ks, krs, jl, w, lane);
    issue_v_tile<D, BLK>(Vs, vrs, jl, n_pad, w, lane);
  }

  for (int64_t e = e0; e < e1; ++e) {
    const bool has_next = (e + 1 < e1);
    const int j_next = has_next ? block_of(e + 1) : 0;
    const bool j_ok = (j_cur >= 0 && j_cur < n_k);
    // keys of this tile that are real (< N); all masked for an invalid index
    const int kvalid = j_ok ? min(BLK, N - j_cur * BLK) : 0;

    // ---- S^T = K Q^T ------------------------------------------------------
    wait_vm_barrier<C::LOADS>();  // K(e) landed in LDS for every wave
    f32x16_t sacc[C::KB];
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
            *reinterpret_cast<const bf16x8_t*>(Ks + (kb * 32 + l32) * C::KROW + off);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[s], sacc[kb], 0, 0, 0);
      }
    }
    lds_read_barrier();  // every wave is done reading Ks
    if (has_next) {
      const int jl = (j_next >= 0 && j_next < n_k) ? j_next : 0;
      issue_k_tile<D, BLK>(Ks, krs, jl, w, lane);
    }

    // ---- online softmax (log2 domain) -------------------------------------
    float mx = m_run;
    if (kvalid >= BLK) {
#pragma unroll
      for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
        for (int t = 0; t < 16; ++t) {
          const float x = sacc[kb][t] * scale_log2;
          sacc[kb][t] = x;
          mx = fmaxf(mx, x);
        }
    } else {
#pragma unroll
      for (int kb = 0; kb < C::KB; ++kb)
#pragma unroll
        for (int t = 0; t < 16; ++t) {
          const int key = kb * 32 + ((t >> 2) << 3) + (g << 2) + (t & 3);
          const float x = key < kvalid ? sacc[kb][t] * scale_log2 : -INFINITY;
          sacc[kb][t] = x;
          mx = fmaxf(mx, x);
        }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float alpha = fast_exp2(m_run - mx);
    m_run = mx;
    float lsum = 0.f;
    bf16x8_t preg[C::PS];
#pragma unroll
    for (int s = 0; s < C::PS; ++s) {
      const int kb = s >> 1;
      const int h = (s & 1) * 8;
      f32x8_t p;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        p[t] = fast_exp2(sacc[kb][h + t] - mx);
        lsum += p[t];
      }
      preg[s] = __builtin_convertvector(p, bf16x8_t);
    }
    l_run = l_run * alpha + lsum;
#pragma unroll
    for (int db = 0; db < C::DB; ++db)
#pragma unroll
      for (int t = 0; t < 16; ++t) oacc[db][t] *= alpha;

    // ---- O^T += V^T P^T ---------------------------------------------------
    if (has_next) {
      wait_vm_barrier<C::LOADS>();  // V(e) landed; K(e+1) may still be in flight
    } else {
      wait_vm_barrier<0>();
    }
#pragma unroll
    for (int s = 0; s < C::PS; ++s) {
      const int off = (((2 * s + g) ^ vsw) << 4);
#pragma unroll
      for (int db = 0; db < C::DB; ++db) {
        const bf16x8_t a =
            *reinterpret_cast<const bf16x8_t*>(Vs + (db * 32 + l32) * C::VROW + off);
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, preg[s], oacc[db], 0, 0, 0);
      }
    }
    lds_read_barrier();  // every wave is done reading Vs
    if (has_next) {
      const int jl = (j_next >= 0 && j_next < n_k) ? j_next : 0;
      issue_v_tile<D, BLK>(Vs, vrs, jl, n_pad, w, lane);
    }
    j_cur = j_next;
  }

  // ---- epilogue: O = O^T / l, lse -----------------------------------------
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const bool row_ok = (qrow < N) && (l_tot > 0.f);
  const float inv = row_ok ? 1.0f / l_tot : 0.f;
  __bf16* orow = O + head + (size_t)qrow * D;
#pragma unroll
  for (int db = 0; db < C::DB; ++db)
#pragma unroll
    for (int qd = 0; qd < 4; ++qd) {
      f32x4_t v;
#pragma unroll
      for (int t = 0; t < 4; ++t) v[t] = oacc[db][qd * 4 + t] * inv;
      const int d0 = db * 32 + qd * 8 + g * 4;
      *reinterpret_cast<bf16x4_t*>(orow + d0) = __builtin_convertvector(v, bf16x4_t);
    }
  if (lse != nullptr && g == 0) {
    lse[(size_t)bh * n_pad + qrow] = row_ok ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

// V [BH][n_pad][D] -> V^T [BH][D][n_pad] with the 16-key position permutation.
// One workgroup transposes 64 keys x D of one head through LDS.
template <int D>
__global__ void __launch_bounds__(256)
    transpose_v_kernel(const __bf16* __restrict__ V, __bf16* __restrict__ Vt, int n_pad) {
  constexpr int TK = 64;
  constexpr int LD = D + 2;  // padded LDS row (elements)
  __shared__ __bf16 tile[TK * LD];
  const int bh = blockIdx.y;
  const int n0 = blockIdx.x * TK;
  const __bf16* src = V + (size_t)bh * n_pad * D + (size_t)n0 * D;
  __bf16* dst = Vt + (size_t)bh * D * n_pad + n0;
  // load: TK rows of D bf16, 8 bf16 per thread-step
  for (int c = threadIdx.x; c < TK * D / 8; c += 256) {
    const int row = c / (D / 8);
    const int col = (c % (D / 8)) * 8;
    const bf16x8_t v = *reinterpret_cast<const bf16x8_t*>(src + (size_t)row * D + col);
#pragma unroll
    for (int t = 0; t < 8; ++t) tile[row * LD + col + t] = v[t];
  }
  __syncthreads();
  // store: D rows of TK positions, 8 positions per thread-step
  for (int c = threadIdx.x; c < D * TK / 8; c += 256) {
    const int d = c / (TK / 8);
    const int p0 = (c % (TK / 8)) * 8;
    bf16x8_t v;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int p = p0 + t;
      const int key = (p & ~15) | perm16(p & 15);
      v[t] = tile[key * LD + d];
    }
    *reinterpret_cast<bf16x8_t*>(dst + (size_t)d * n_pad + p0) = v;
  }
}

template <int D, int BLK>
hipError_t launch_fwd(const void* q, const void* k, const void* v, int B, int H, int N, int n_pad,
                      float scale, const int32_t* row_ptr, const int32_t* col_idx,
                      int64_t col_len, void* o, float* lse, void* vt, hipStream_t stream) {
  const int BH = B * H;
  const int n_q = n_pad / BLK;
  const int n_k = n_pad / BLK;
  dim3 tgrid(n_pad / 64, BH);
  hipLaunchKernelGGL(transpose_v_kernel<D>, tgrid, dim3(256), 0, stream,
                     static_cast<const __bf16*>(v), static_cast<__bf16*>(vt), n_pad);
  const int rows = BH * n_q;
  hipLaunchKernelGGL((sparse_fwd_bf16_kernel<D, BLK>), dim3(rows), dim3(FwdCfg<D, BLK>::NT), 0,
                     stream, static_cast<const __bf16*>(q), static_cast<const __bf16*>(k),
                     static_cast<const __bf16*>(vt), row_ptr, col_idx, col_len,
                     static_cast<__bf16*>(o), lse, rows, n_q, n_k, N, n_pad, scale * kLog2e);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sparse_fwd_bf16(int d, int blk, const void* q, const void* k, const void* v,
                                  int B, int H, int N, int n_pad, float scale,
                                  const int32_t* row_ptr, const int32_t* col_idx,
                                  int64_t col_len, void* o, float* lse, void* workspace,
                                  hipStream_t stream) {
  if (d == 128 && blk == 128)
    return launch_fwd<128, 128>(q, k, v, B, H, N, n_pad, scale, row_ptr, col_idx, col_len, o,
                                lse, workspace, stream);
  if (d == 64 && blk == 128)
    return launch_fwd<64, 128>(q, k, v, B, H, N, n_pad, scale, row_ptr, col_idx, col_len, o, lse,
                               workspace, stream);
  if (d == 128 && blk == 64)
    return launch_fwd<128, 64>(q, k, v, B, H, N, n_pad, scale, row_ptr, col_idx, col_len, o, lse,
                               workspace, stream);
  if (d == 64 && blk == 64)
    return launch_fwd<64, 64>(q, k, v, B, H, N, n_pad, scale, row_ptr, col_idx, col_len, o, lse,
                              workspace, stream);
  return hipErrorInvalidValue;
}

size_t sparse_fwd_bf16_workspace(int B, int H, int n_pad, int d) {
  return (size_t)B * H * n_pad * d * 2;  // transposed V
}

}  // namespace losa
