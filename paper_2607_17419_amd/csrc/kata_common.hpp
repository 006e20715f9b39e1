// kata_common.hpp -- device helpers shared by the libkata kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kata {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

// Input element types: fp32 is `float`, bf16 travels as its 16-bit pattern.
struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) {
  return __uint_as_float(static_cast<uint32_t>(x.bits) << 16);
}

template <typename Tin>
__device__ __forceinline__ float load_f32(const Tin* p, size_t i) {
  return to_f32(p[i]);
}

// Two fp32 values -> packed bf16 pair (round to nearest even); hipcc lowers
// this to one v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  bf16x2 r;
  r[0] = static_cast<__bf16>(lo);
  r[1] = static_cast<__bf16>(hi);
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ float bf16lo_f32(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi_f32(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Row-major upper-triangle packed index of the pair (a, b), a <= b.
__host__ __device__ __forceinline__ int packed_index(int a, int b, int d) {
  return a * d - a * (a - 1) / 2 + (b - a);
}

// Wait until at most N vector-memory operations of this wave are in flight
// (lgkm and exp counters left alone).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (((N >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier that orders LDS only: this wave's LDS operations are
// complete (lgkmcnt 0), then s_barrier.  Unlike __syncthreads() it does not
// wait for outstanding vector-memory operations, so loads of later stages
// (global -> LDS copies among them) and global stores stay in flight; callers
// wait for a copied stage they consume with wait_vmcnt first.  The signal
// fences keep the compiler from moving memory accesses across the barrier.
__device__ __forceinline__ void lds_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0), vmcnt and expcnt unchanged
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

}  // namespace kata
