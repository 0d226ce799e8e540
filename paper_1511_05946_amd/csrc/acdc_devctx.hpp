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
};

}  // namespace acdc
