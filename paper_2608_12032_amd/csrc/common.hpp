// Device-side primitives shared by the LoSA gfx950 kernels.
//
// Vector types for the bf16 MFMA operands, buffer resources (bounds-checked
// global loads: an offset outside the resource's byte range reads zero instead
// of faulting), 16-byte global->LDS direct loads, and explicit wait/barrier
// helpers that keep the compiler from moving LDS traffic across a barrier.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace losa {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// Finite stand-in for "no score seen yet": exp2(x - kNegBig) never overflows
// for a real score and exp2(kNegBig - m) is 0 for any real running max.
constexpr float kNegBig = -1.0e30f;

// Buffer resource over [base, base + bytes); stride 0 (raw addressing).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

// One wave-wide direct load: lane L copies 16 bytes from rsrc + voffset into
// LDS at lds_wave_base + 16 * L.  lds_wave_base must be wave-uniform.
__device__ __forceinline__ void load_lds_16(__amdgpu_buffer_rsrc_t rsrc, void* lds_wave_base,
                                            uint32_t voffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(
      rsrc, (__attribute__((address_space(3))) void*)lds_wave_base, 16, voffset, 0, 0, 0);
}

// Wait until at most N vector-memory operations of this wave are outstanding
// and all of its LDS operations have completed, then barrier.  After it the
// workgroup's direct loads issued before the last N are visible in LDS, and no
// wave still reads what it read before.  The "memory" clobber stops the
// compiler from moving LDS or global accesses across it.
template <int N>
__device__ __forceinline__ void wait_vm_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// All LDS reads of this wave have returned, then barrier: after it, every wave
// of the workgroup is done reading what it read before.
__device__ __forceinline__ void lds_read_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Workgroups are dispatched round-robin over the 8 XCDs (id % 8).  Map them so
// that each XCD walks a contiguous range of logical rows: neighbouring query
// blocks of one head then share that XCD's L2.  Ids past the last multiple of
// 8 keep their own number.
__device__ __forceinline__ int xcd_remap(int id, int total) {
  const int per = total >> 3;
  const int full = per << 3;
  if (id >= full) return id;
  return (id & 7) * per + (id >> 3);
}

}  // namespace losa
