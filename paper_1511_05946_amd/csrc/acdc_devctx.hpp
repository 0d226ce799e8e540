// LDS synchronisation of the GPU kernels (the CPU emulation supplies its own
// context with the same two calls).
#pragma once

#include <hip/hip_runtime.h>

namespace acdc {

// LDS synchronisation for a row spread over T threads.  A row that fits in
// one wavefront only needs its LDS accesses kept in program order (LDS
// operations of a wavefront execute in order); wider rows use the workgroup
// barrier.
template <int T>
struct DevCtx {
  // Barriers order LDS only ("local" fences): global loads issued ahead of
  // a barrier stay in flight across it.
  __device__ __forceinline__ static void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
  }
  __device__ __forceinline__ void sync_row() {
    if constexpr (T > 64) {
      lds_barrier();
    } else {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
  }
  __device__ __forceinline__ void sync_all() { lds_barrier(); }

  // gfx950 cross-lane swaps of the pair (a, b), in place, per group of 16
  // lanes r0..r3 (lanes 0-15, 16-31, 32-47, 48-63 of the wave):
  //   swap16: a <- (a.r0, b.r0, a.r2, b.r2), b <- (a.r1, b.r1, a.r3, b.r3)
  //   swap32: a <- (a.lo, b.lo),             b <- (a.hi, b.hi)
  // (lo, hi = lanes 0-31, 32-63), so a + b afterwards holds pair sums of
  // a in one row (half) and of b in the other.
  __device__ __forceinline__ static void swap16(float& a, float& b) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
    a = __uint_as_float(r[0]);
    b = __uint_as_float(r[1]);
  }
  __device__ __forceinline__ static void swap32(float& a, float& b) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
    a = __uint_as_float(r[0]);
    b = __uint_as_float(r[1]);
  }
};

}  // namespace acdc
