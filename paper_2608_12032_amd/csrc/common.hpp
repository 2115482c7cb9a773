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

typedef int i32x4_t __attribute__((ext_vector_type(4)));

// Raw buffer descriptor over [base, base + bytes) in scalar registers (the
// fields make_rsrc fills): an offset outside the range reads zero.
__device__ __forceinline__ i32x4_t rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  i32x4_t r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;
  return r;
}

// One wave-wide 16-byte-per-lane buffer load straight into LDS: lane L's 16
// bytes at rs + voff + soff land at LDS byte lds + 16 L (lds wave-uniform).
// Written as inline assembly so that the compiler does not hold the LDS reads
// that follow it until it completes: the kernel guarantees they never touch
// the slot it writes, and waits for it explicitly (vmcnt) before the barrier
// that publishes the slot.  M0 carries the LDS address; the compiler emits
// no M0 use of its own in these kernels, so nothing it keeps there is lost.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"  // M0 is reserved: see above
__device__ __forceinline__ void dma16(uint32_t lds, const i32x4_t& rs, uint32_t voff, uint32_t soff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :: "s"(lds), "v"(voff), "s"(rs), "s"(soff) : "m0");
}
#pragma clang diagnostic pop

// max / sum of a value and the one held by lane ^ 32 (v_permlane32_swap gives
// each lane the pair {own, partner} in some order; max and + do not care).
__device__ __forceinline__ float max_with_partner(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float add_partner(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

typedef __attribute__((address_space(3))) const bf16x8_t lds_bf16x8_t;

// 16-byte LDS read at byte address `addr` (+ a compile-time immediate).
__device__ __forceinline__ bf16x8_t lds_read16(uint32_t addr) {
  return *reinterpret_cast<lds_bf16x8_t*>(addr);
}

}  // namespace losa
