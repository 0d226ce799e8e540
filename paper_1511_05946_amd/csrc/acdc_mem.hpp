// Global-memory views for the kernel bodies.
//
// On gfx950 a view is a buffer resource (4 SGPRs) and every access is
//   buffer_load/store  vdata, voffset (VGPR), rsrc, soffset (SGPR/const) offen
// so a thread keeps one 32-bit offset per access pattern and all per-chunk,
// per-slot and per-layer strides ride in the scalar offset.  This keeps
// loop-invariant 64-bit addresses out of the vector register file.  Views
// cover < 4 GiB from their base; callers rebase per row block / per layer.
//
// In the CPU emulation a view is a plain pointer.
#pragma once

#include <hip/hip_runtime.h>

#include <cstring>

namespace acdc {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

struct GView {
  // tables read through a GView are loaded one FFT pass ahead (cache latency)
  static constexpr bool kPrefetch = true;
#if defined(__HIP_DEVICE_COMPILE__)
  __amdgpu_buffer_rsrc_t r;
#endif
  char* p;  // stores: uniform base + 32-bit offset (global_store with an SGPR base)

  __host__ __device__ __forceinline__ static GView of(const void* base) {
    GView g;
#if defined(__HIP_DEVICE_COMPILE__)
    // raw buffer: stride 0, num_records = 4 GiB - 1, gfx9 dword3 (32-bit data)
    g.r = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)0xffffffff, 0x00020000);
#endif
    g.p = static_cast<char*>(const_cast<void*>(base));
    return g;
  }

  __host__ __device__ __forceinline__ float4 ld4(unsigned voff, unsigned soff) const {
#if defined(__HIP_DEVICE_COMPILE__)
    const f32x4 v = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
    return make_float4(v[0], v[1], v[2], v[3]);
#else
    float4 v;
    std::memcpy(&v, p + voff + soff, 16);
    return v;
#endif
  }
  __host__ __device__ __forceinline__ int4 ldi4(unsigned voff, unsigned soff) const {
#if defined(__HIP_DEVICE_COMPILE__)
    const i32x4 v = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
    return make_int4(v[0], v[1], v[2], v[3]);
#else
    int4 v;
    std::memcpy(&v, p + voff + soff, 16);
    return v;
#endif
  }
  __host__ __device__ __forceinline__ float2 ld2(unsigned voff, unsigned soff) const {
#if defined(__HIP_DEVICE_COMPILE__)
    const f32x2 v = __builtin_bit_cast(f32x2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
    return make_float2(v[0], v[1]);
#else
    float2 v;
    std::memcpy(&v, p + voff + soff, 8);
    return v;
#endif
  }
  __host__ __device__ __forceinline__ int2 ldi2(unsigned voff, unsigned soff) const {
#if defined(__HIP_DEVICE_COMPILE__)
    const u32x2 v = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
    return make_int2(int(v[0]), int(v[1]));
#else
    int2 v;
    std::memcpy(&v, p + voff + soff, 8);
    return v;
#endif
  }
  __host__ __device__ __forceinline__ int ldi1(unsigned voff, unsigned soff) const {
#if defined(__HIP_DEVICE_COMPILE__)
    return (int)__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
#else
    int v;
    std::memcpy(&v, p + voff + soff, 4);
    return v;
#endif
  }
  // 16 bytes per lane straight into LDS (buffer_load_dwordx4 ... lds): lane
  // l's bytes land at lds + 16 l, with lds the same for the whole wave.  No
  // register holds the data; the wave's vmcnt covers the copy.  The load is
  // device-coherent (sc1: it misses the L1), so it reads what this workgroup
  // stored earlier.
  __host__ __device__ __forceinline__ void ld_lds16(float* lds, unsigned lane, unsigned voff, unsigned soff) const {
#if defined(__HIP_DEVICE_COMPILE__)
    (void)lane;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voff, soff, 0,
                                             16 /* sc1 */);
#else
    std::memcpy(lds + 4 * lane, p + voff + soff, 16);
#endif
  }
  // Stores go through a plain global pointer: buffer stores fed from the
  // register arrays defeat register promotion of those arrays in this
  // compiler (they end up in private scratch), so only loads use the buffer
  // path.  The constant part of the offset goes to the uniform base first,
  // so that every store is (SGPR base + one 32-bit lane offset): written as
  // base + (voff + soff) the compiler forms a 64-bit address per store and
  // hoists them out of the layer loop (2 VGPRs per row chunk, spilled at
  // N = 9216).
  __host__ __device__ __forceinline__ void st4(float4 v, unsigned voff, unsigned soff) const {
    *reinterpret_cast<float4*>((p + soff) + voff) = v;
  }
  __host__ __device__ __forceinline__ void st4(float a, float b, float c, float d, unsigned voff,
                                               unsigned soff) const {
    *reinterpret_cast<float4*>((p + soff) + voff) = make_float4(a, b, c, d);
  }
  __host__ __device__ __forceinline__ void st2(float2 v, unsigned voff, unsigned soff) const {
    *reinterpret_cast<float2*>((p + soff) + voff) = v;
  }
};

// A read-only table copied into LDS, with the same (voffset, soffset)
// interface as GView's loads.
struct LdsView {
  static constexpr bool kPrefetch = false;  // LDS latency: load right before use
  const char* p;
  __host__ __device__ __forceinline__ static LdsView of(const void* base) {
    return LdsView{static_cast<const char*>(base)};
  }
  __host__ __device__ __forceinline__ float2 ld2(unsigned voff, unsigned soff) const {
    return *reinterpret_cast<const float2*>(p + voff + soff);
  }
  __host__ __device__ __forceinline__ float4 ld4(unsigned voff, unsigned soff) const {
    return *reinterpret_cast<const float4*>(p + voff + soff);
  }
};

}  // namespace acdc
