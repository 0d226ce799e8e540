// Stockham FFT passes over one row held by T threads (registers + one LDS
// slab per row).
//
// Pass p with radix r and stride Ns = product of the earlier radices takes
// butterfly j's inputs j + i*(M/r), multiplies input i by W_{Ns r}^{i (j mod Ns)},
// applies the r-point DFT and writes output m to (j - j mod Ns) r + (j mod Ns)
// + m Ns.  The first pass reads registers, the last pass leaves its outputs in
// registers (output m of butterfly j is element j + m*Ns), and every pass in
// between goes through the slab.
//
// Which butterflies a thread owns in the first and last pass is a policy
// (KIND): 0 plain (j = t + T*beta), 1 mirrored pairs (p, T*B-1-p), 2 negated
// pairs (p, NB-p) with (0, NB/2) for p = 0, 3 adjacent pairs (2p, 2p+1),
// p = t + T*(beta/2).  The real path uses 1 and 2 so that whole float4
// chunks and Makhoul partners stay thread-local; the complex path uses 3
// where its plan allows, so that neighbouring elements share a thread and
// every row access is 16 bytes.
#pragma once

#include "acdc_dft.hpp"
#include "acdc_mem.hpp"

namespace acdc {

template <class PL, int KIND, int B>
__host__ __device__ __forceinline__ unsigned bfly(unsigned t, int beta) {
  if constexpr (KIND == 0) {
    return t + PL::T * beta;
  } else if constexpr (KIND == 1) {
    const unsigned p = t + PL::T * (beta >> 1);
    return (beta & 1) ? PL::T * B - 1 - p : p;
  } else if constexpr (KIND == 2) {
    const unsigned p = t + PL::T * (beta >> 1);
    return (beta & 1) ? (p == 0 ? PL::NB / 2 : PL::NB - p) : p;
  } else {
    static_assert(KIND == 3 && B % 2 == 0, "adjacent pairs need an even butterfly count");
    return 2u * (t + PL::T * unsigned(beta >> 1)) + unsigned(beta & 1);
  }
}

// Twiddles of one pass for the butterflies of thread t, held in registers.
// Input i of butterfly j takes W_{Ns r}^{i k}, k = j mod Ns, stored at
// [(i-1)/2][k][(i-1)%2] of the pass's table block (pairs of inputs share a
// 16-byte load; lanes with consecutive k read consecutive pairs).
// A pass's twiddles are loaded while the previous pass still computes, so
// the table latency hides behind its DFTs, LDS exchange and barrier.
template <class PL, bool INV, int PASS, int KF, int KL>
struct PassTw {
  static constexpr bool kLive = PASS > 0 && PASS < PL::NPASS && PL::ns(PASS, INV) > 1;
  static constexpr int r = kLive ? PL::radix(PASS, INV) : 2;
  static constexpr int b = PL::P / r;
  static constexpr int NW = kLive ? b * (r - 1) : 1;
  float2 w[NW];
  template <class TW>
  __host__ __device__ __forceinline__ void load(unsigned t, TW tw) {
    if constexpr (kLive) {
      constexpr int Ns = PL::ns(PASS, INV);
      constexpr int KIND = (PASS == PL::NPASS - 1) ? KL : 0;
      constexpr unsigned off = unsigned(PL::tw_off(PASS, INV)) * 8u;
#pragma unroll
      for (int beta = 0; beta < b; ++beta) {
        const unsigned vo = (bfly<PL, KIND, b>(t, beta) % Ns) * 16u;
#pragma unroll
        for (int i = 1; i < r; i += 2) {
          const unsigned so = off + unsigned((i - 1) * Ns) * 8u;  // pair (i-1)/2 starts at (i-1)*Ns float2
          if (i + 1 < r) {
            const float4 q = tw.ld4(vo, so);
            w[beta * (r - 1) + i - 1] = make_float2(q.x, q.y);
            w[beta * (r - 1) + i] = make_float2(q.z, q.w);
          } else {
            w[beta * (r - 1) + i - 1] = tw.ld2(vo, so);
          }
        }
      }
    }
  }
};

// The steps of one pass.  Pass p (radix r, stride Ns) owns butterflies j
// chosen by the KIND policy; it reads inputs j + i*(M/r) from the slab
// (except the first pass, which starts from registers), multiplies input i
// by W_{Ns r}^{i (j mod Ns)}, runs the r-point DFT and writes output m to
// (j - j mod Ns) r + (j mod Ns) + m Ns (except the last pass, whose outputs
// stay in registers).  Slab indices are padded: a -> a + (a >> PADSH).
template <class PL, bool INV, int PASS, int KF, int KL>
struct PassGeo {
  static constexpr int r = PL::radix(PASS, INV);
  static constexpr int Ns = PL::ns(PASS, INV);
  static constexpr int b = PL::P / r;
  static constexpr int stride = PL::M / r;
  static constexpr bool first = (PASS == 0);
  static constexpr bool last = (PASS == PL::NPASS - 1);
  static constexpr int KIND = first ? KF : (last ? KL : 0);
  static constexpr unsigned S = PL::PADSH;
  unsigned j[b];
  __host__ __device__ __forceinline__ explicit PassGeo(unsigned t) {
#pragma unroll
    for (int beta = 0; beta < b; ++beta) j[beta] = bfly<PL, KIND, b>(t, beta);
  }
  __host__ __device__ __forceinline__ void read(float2 (&v)[PL::P], const float2* slab) const {
    if constexpr (stride % (1 << S) == 0) {
      // stride is a multiple of 2^S: pad(j + i stride) = pad(j) + i (stride + stride/2^S)
      constexpr unsigned sp = stride + (stride >> S);
#pragma unroll
      for (int beta = 0; beta < b; ++beta) {
        const unsigned pj = j[beta] + (j[beta] >> S);
#pragma unroll
        for (int i = 0; i < r; ++i) v[beta * r + i] = slab[pj + i * sp];
      }
    } else {
#pragma unroll
      for (int beta = 0; beta < b; ++beta)
#pragma unroll
        for (int i = 0; i < r; ++i) {
          const unsigned a = j[beta] + i * stride;
          v[beta * r + i] = slab[a + (a >> S)];
        }
    }
  }
  __host__ __device__ __forceinline__ void twiddle(float2 (&v)[PL::P],
                                                   const PassTw<PL, INV, PASS, KF, KL>& tw) const {
    if constexpr (PassTw<PL, INV, PASS, KF, KL>::kLive) {
#pragma unroll
      for (int beta = 0; beta < b; ++beta)
#pragma unroll
        for (int i = 1; i < r; ++i) v[beta * r + i] = ctw<INV>(v[beta * r + i], tw.w[beta * (r - 1) + i - 1]);
    }
  }
  __host__ __device__ __forceinline__ static void dft(float2 (&v)[PL::P]) {
#pragma unroll
    for (int beta = 0; beta < b; ++beta) Dft<r, INV>::run(&v[beta * r]);
  }
  __host__ __device__ __forceinline__ void write(const float2 (&v)[PL::P], float2* slab) const {
#pragma unroll
    for (int beta = 0; beta < b; ++beta) {
      const unsigned k = j[beta] % Ns;
      const unsigned base = (j[beta] - k) * r + k;
      if constexpr (Ns % (1 << S) == 0 || (Ns == 1 && (1 << S) % r == 0)) {
        // no carry into the pad bits: pad(base + m Ns) = pad(base) + m (Ns + Ns/2^S)
        constexpr unsigned nsp = Ns + (Ns >> S);
        const unsigned pb = base + (base >> S);
#pragma unroll
        for (int m = 0; m < r; ++m) slab[pb + m * nsp] = v[beta * r + m];
      } else {
#pragma unroll
        for (int m = 0; m < r; ++m) {
          const unsigned a = base + m * Ns;
          slab[a + (a >> S)] = v[beta * r + m];
        }
      }
    }
  }
};

// One pass.  `next` is called once this pass no longer needs its own
// twiddles (it issues the next pass's loads); a scheduling fence keeps those
// loads ahead of this pass's arithmetic.
template <class PL, bool INV, int PASS, int KF, int KL, class Ctx, class Next>
__host__ __device__ __forceinline__ void stockham_pass(Ctx& ctx, float2 (&v)[PL::P], unsigned t, float2* slab,
                                                      const PassTw<PL, INV, PASS, KF, KL>& tw, Next&& next) {
  using G = PassGeo<PL, INV, PASS, KF, KL>;
  const G geo(t);
  if constexpr (!G::first) geo.read(v, slab);
  geo.twiddle(v, tw);
  next();
  ACDC_SCHED_FENCE();
  G::dft(v);
  if constexpr (!G::last) {
    ctx.sync_row();
    geo.write(v, slab);
    ctx.sync_row();
  }
}

// Two transforms of the same direction on arrays v and w that share the
// slab: pass by pass, both arrays use one set of twiddle registers, and
// the exchanges between passes run one array after the other through the
// slab (write v, read v, write w, read w).
template <class PL, bool INV, int PASS, int KF, int KL, class Ctx, class Next>
__host__ __device__ __forceinline__ void stockham_pass2(Ctx& ctx, float2 (&v)[PL::P], float2 (&w)[PL::P],
                                                       unsigned t, float2* slab,
                                                       const PassTw<PL, INV, PASS, KF, KL>& tw, Next&& next) {
  using G = PassGeo<PL, INV, PASS, KF, KL>;
  const G geo(t);
  geo.twiddle(v, tw);
  geo.twiddle(w, tw);
  ACDC_SCHED_FENCE();
  G::dft(v);
  next();  // the next pass's twiddles load while w's butterflies run
  ACDC_SCHED_FENCE();
  G::dft(w);
  if constexpr (!G::last) {
    // this pass's outputs go through the slab into the next pass's inputs
    using G1 = PassGeo<PL, INV, PASS + 1, KF, KL>;
    const G1 geo1(t);
    ctx.sync_row();
    geo.write(v, slab);
    ctx.sync_row();
    geo1.read(v, slab);
    ctx.sync_row();
    geo.write(w, slab);
    ctx.sync_row();
    geo1.read(w, slab);
  }
}

// Whole transform.  `tail` runs in the last pass right after its twiddle
// multiply: callers use it to issue the loads of what follows the FFT.
// `tab` is the twiddle table: the global constant table (GView) or its copy
// in LDS (LdsView).
template <class PL, bool INV, int KF, int KL, class Ctx, class TW, class Tail>
__host__ __device__ __forceinline__ void stockham_fft(Ctx& ctx, float2 (&v)[PL::P], unsigned t, float2* slab,
                                                     TW tab, Tail&& tail) {
  constexpr int NP = PL::NPASS;
  PassTw<PL, INV, 0, KF, KL> w0;
  PassTw<PL, INV, 1, KF, KL> w1;
  if constexpr (!TW::kPrefetch) {
    // each pass reads its own twiddles as it starts
    static_assert(NP <= 4, "up to four passes");
    PassTw<PL, INV, 2, KF, KL> w2;
    PassTw<PL, INV, 3, KF, KL> w3;
    stockham_pass<PL, INV, 0, KF, KL>(ctx, v, t, slab, w0, [&] { if constexpr (NP == 1) tail(); });
    if constexpr (NP > 1) {
      w1.load(t, tab);
      stockham_pass<PL, INV, 1, KF, KL>(ctx, v, t, slab, w1, [&] { if constexpr (NP == 2) tail(); });
    }
    if constexpr (NP > 2) {
      w2.load(t, tab);
      stockham_pass<PL, INV, 2, KF, KL>(ctx, v, t, slab, w2, [&] { if constexpr (NP == 3) tail(); });
    }
    if constexpr (NP > 3) {
      w3.load(t, tab);
      stockham_pass<PL, INV, 3, KF, KL>(ctx, v, t, slab, w3, tail);
    }
  } else if constexpr (NP == 1) {
    stockham_pass<PL, INV, 0, KF, KL>(ctx, v, t, slab, w0, tail);
  } else {
    stockham_pass<PL, INV, 0, KF, KL>(ctx, v, t, slab, w0, [&] { w1.load(t, tab); });
    PassTw<PL, INV, 2, KF, KL> w2;
    if constexpr (NP == 2) {
      stockham_pass<PL, INV, 1, KF, KL>(ctx, v, t, slab, w1, tail);
    } else {
      stockham_pass<PL, INV, 1, KF, KL>(ctx, v, t, slab, w1, [&] { w2.load(t, tab); });
      PassTw<PL, INV, 3, KF, KL> w3;
      if constexpr (NP == 3) {
        stockham_pass<PL, INV, 2, KF, KL>(ctx, v, t, slab, w2, tail);
      } else {
        stockham_pass<PL, INV, 2, KF, KL>(ctx, v, t, slab, w2, [&] { w3.load(t, tab); });
        stockham_pass<PL, INV, 3, KF, KL>(ctx, v, t, slab, w3, tail);
      }
    }
  }
}

template <class PL, bool INV, int KF, int KL, class Ctx, class TW>
__host__ __device__ __forceinline__ void stockham_fft(Ctx& ctx, float2 (&v)[PL::P], unsigned t, float2* slab,
                                                     TW tab) {
  stockham_fft<PL, INV, KF, KL>(ctx, v, t, slab, tab, [] {});
}

// Forward transforms of two arrays sharing each pass's twiddles (global
// table, loaded one pass ahead).  `tail` runs in the last pass right after
// its twiddle multiplies.
template <class PL, bool INV, int KF, int KL, class Ctx, class Tail>
__host__ __device__ __forceinline__ void stockham_fft2(Ctx& ctx, float2 (&v)[PL::P], float2 (&w)[PL::P],
                                                      unsigned t, float2* slab, GView tab, Tail&& tail) {
  constexpr int NP = PL::NPASS;
  static_assert(NP >= 2 && NP <= 4, "two to four passes");
  PassTw<PL, INV, 0, KF, KL> w0;
  PassTw<PL, INV, 1, KF, KL> w1;
  PassTw<PL, INV, 2, KF, KL> w2;
  PassTw<PL, INV, 3, KF, KL> w3;
  stockham_pass2<PL, INV, 0, KF, KL>(ctx, v, w, t, slab, w0, [&] { w1.load(t, tab); });
  if constexpr (NP == 2) {
    stockham_pass2<PL, INV, 1, KF, KL>(ctx, v, w, t, slab, w1, tail);
  } else {
    stockham_pass2<PL, INV, 1, KF, KL>(ctx, v, w, t, slab, w1, [&] { w2.load(t, tab); });
    if constexpr (NP == 3) {
      stockham_pass2<PL, INV, 2, KF, KL>(ctx, v, w, t, slab, w2, tail);
    } else {
      stockham_pass2<PL, INV, 2, KF, KL>(ctx, v, w, t, slab, w2, [&] { w3.load(t, tab); });
      stockham_pass2<PL, INV, 3, KF, KL>(ctx, v, w, t, slab, w3, tail);
    }
  }
}

// Sum the per-row images [rows][SLAB] of a workgroup in fixed row order and
// write the first NFL floats to out (float4 granularity).  With `old` (LDS,
// NFL floats) the sum is added to it afterwards: old + (row 0 + ... ).
// Called by every thread; the trip count is a compile-time constant.
template <int ROWS, int SLAB, int THREADS, int NFL>
__host__ __device__ __forceinline__ void sum_rows(const float* lds, GView out, int tid,
                                                  const float* old = nullptr) {
  constexpr int N4 = NFL / 4;
#pragma unroll
  for (int e0 = 0; e0 < N4; e0 += THREADS) {
    const unsigned e = unsigned(e0 + tid);
    if (N4 % THREADS == 0 || e < unsigned(N4)) {
      float4 s = reinterpret_cast<const float4*>(lds)[e];
#pragma unroll
      for (int r = 1; r < ROWS; ++r) {
        const float4 u = reinterpret_cast<const float4*>(lds + r * SLAB)[e];
        s.x += u.x;
        s.y += u.y;
        s.z += u.z;
        s.w += u.w;
      }
      if (old != nullptr) {
        const float4 o = reinterpret_cast<const float4*>(old)[e];
        s = make_float4(o.x + s.x, o.y + s.y, o.z + s.z, o.w + s.w);
      }
      out.st4(s, e * 16u, 0u);
    }
  }
}

// Copy NFL floats of global memory (view src, from its base) into LDS at
// dst, the workgroup's THREADS threads together, each wave 1 KiB blocks.  On
// the GPU these are direct-to-LDS loads that complete in the background;
// lds_fetch_wait() then the workgroup barrier publish them.
template <int NFL, int THREADS>
__host__ __device__ __forceinline__ void lds_fetch(float* dst, GView src, int tid) {
  constexpr int N4 = NFL / 4;
  static_assert(NFL % 4 == 0 && THREADS % 64 == 0, "whole waves of float4");
  const unsigned lane = unsigned(tid) % 64u;
#if defined(__HIP_DEVICE_COMPILE__)
  const unsigned w = __builtin_amdgcn_readfirstlane(unsigned(tid) / 64u);
#else
  const unsigned w = unsigned(tid) / 64u;
#endif
#pragma unroll
  for (int i = 0; i < (N4 + THREADS - 1) / THREADS; ++i) {
    const unsigned e0 = w * 64u + unsigned(i * THREADS);  // this wave's first float4
    if (N4 % THREADS == 0 || e0 < unsigned(N4)) {
      static_assert(N4 % 64 == 0, "blocks of 64 float4");
      src.ld_lds16(dst + e0 * 4u, lane, lane * 16u, e0 * 16u);
    }
  }
}
// Wait for this wave's outstanding vector-memory operations, the
// direct-to-LDS loads included (vmcnt(0); expcnt and lgkmcnt left open).
__host__ __device__ __forceinline__ void lds_fetch_wait() {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_s_waitcnt(0x0F70);
#endif
}

}  // namespace acdc
