// LDS synchronisation of the GPU kernels (the CPU emulation supplies its own
// context with the same two calls).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

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

// LDS synchronisation for rows of W = T/64 > 1 waves that meet only each
// other, not the whole workgroup: the row's waves count arrivals in an LDS
// word.  A wave adds 1 once its LDS accesses have completed and leaves when
// the count reaches W times its own arrivals (the count only grows, so a
// partner already at its next sync keeps it there).  The waves of a row make
// the same sequence of sync_row calls and share a workgroup (resident, and
// saved and restored together), so the count always gets there within the
// time the slowest partner needs for the same work; the polling is also
// bounded (2^20 polls, tens of milliseconds), so every wave ends whatever
// happens.  sync_all stays the workgroup barrier.  `cnt` must be zero, and
// seen as zero by the whole workgroup, before the first sync_row.
template <int T>
struct GroupCtx {
  static_assert(T > 64 && T % 64 == 0, "rows of whole waves");
  static constexpr unsigned W = T / 64;
  // Each row owns two LDS words: [0] its arrival count, [1] the number of
  // its waits whose polling ran out (zero unless something is badly wrong;
  // report() adds those to a global count after the row work).
  static constexpr int kWords = 2;
  unsigned addr;  // LDS byte address of this row's two words
  unsigned gen;   // W times this wave's arrivals so far
  __device__ explicit GroupCtx(unsigned* c)
      : addr(unsigned(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) unsigned*)c))), gen(0) {}
  // One asm block (a single instruction to the register allocator, so the
  // polling loop adds no control flow around the row code).  The wave's LDS
  // accesses complete first (release), one lane adds 1 with the rest of the
  // exec mask saved and restored, then the wave polls until the count
  // reaches gen or the poll budget runs out; a run-out adds 1 to the row's
  // second word (on the fall-through path only, so the normal path is
  // unchanged).  The "memory" clobber keeps the compiler's LDS accesses on
  // their side of it (acquire).
  __device__ __forceinline__ void sync_row() {
    gen += W;
    unsigned long long save;
    unsigned tmp, seen, g, it;
    // Only VGPR inputs (they need not be known uniform, also at -O0); the
    // uniform copies live in SGPRs the block declares as outputs.
    asm volatile(
        "s_waitcnt lgkmcnt(0)\n"
        "v_readfirstlane_b32 %[g], %[genv]\n"
        "s_mov_b32 %[it], 0x100000\n"  // poll budget (2^20 polls, tens of ms)
        "s_mov_b64 %[save], exec\n"
        "s_mov_b64 exec, 1\n"
        "ds_add_u32 %[addr], %[one]\n"
        "s_mov_b64 exec, %[save]\n"
        "1:\n"
        "ds_read_b32 %[tmp], %[addr]\n"
        "s_waitcnt lgkmcnt(0)\n"
        "v_readfirstlane_b32 %[seen], %[tmp]\n"
        "s_cmp_ge_u32 %[seen], %[g]\n"
        "s_cbranch_scc1 2f\n"
        "s_sleep 1\n"
        "s_sub_u32 %[it], %[it], 1\n"
        "s_cbranch_scc0 1b\n"
        "s_mov_b64 exec, 1\n"
        "ds_add_u32 %[addr], %[one] offset:4\n"
        "s_mov_b64 exec, %[save]\n"
        "2:\n"
        : [save] "=&s"(save), [tmp] "=&v"(tmp), [seen] "=&s"(seen), [g] "=&s"(g), [it] "=&s"(it)
        : [addr] "v"(addr), [one] "v"(1u), [genv] "v"(gen)
        : "scc", "memory");
  }
  // After the workgroup's last row sync: adds the run-outs of its `rows`
  // rows (words laid out as above from `words`) to *count.
  __device__ static void report(const unsigned* words, int rows, int tid, unsigned long long* count) {
    DevCtx<T>::lds_barrier();
    if (tid < rows) {
      const unsigned n = words[kWords * tid + 1];
      if (n != 0u) __hip_atomic_fetch_add(count, (unsigned long long)n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __device__ __forceinline__ void sync_all() { DevCtx<T>::lds_barrier(); }
  __device__ __forceinline__ static void swap16(float& a, float& b) { DevCtx<T>::swap16(a, b); }
  __device__ __forceinline__ static void swap32(float& a, float& b) { DevCtx<T>::swap32(a, b); }
};

}  // namespace acdc
