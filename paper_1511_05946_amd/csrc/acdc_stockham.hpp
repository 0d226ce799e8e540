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
// pairs (p, NB-p) with (0, NB/2) for p = 0.  The real path uses 1 and 2 so
// that whole float4 chunks and Makhoul partners stay thread-local.
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
  } else {
    const unsigned p = t + PL::T * (beta >> 1);
    return (beta & 1) ? (p == 0 ? PL::NB / 2 : PL::NB - p) : p;
  }
}

template <class PL, bool INV, int PASS, int KF, int KL, class Ctx>
__host__ __device__ __forceinline__ void stockham_pass(Ctx& ctx, float2 (&v)[PL::P], unsigned t, float2* slab,
                                                      GView tw) {
  constexpr int P = PL::P;
  constexpr int r = PL::radix(PASS, INV);
  constexpr int Ns = PL::ns(PASS, INV);
  constexpr int b = P / r;
  constexpr int stride = PL::M / r;
  constexpr bool first = (PASS == 0);
  constexpr bool last = (PASS == PL::NPASS - 1);
  constexpr int KIND = first ? KF : (last ? KL : 0);
  unsigned j[b];
#pragma unroll
  for (int beta = 0; beta < b; ++beta) j[beta] = bfly<PL, KIND, b>(t, beta);
  if constexpr (!first) {
#pragma unroll
    for (int beta = 0; beta < b; ++beta)
#pragma unroll
      for (int i = 0; i < r; ++i) v[beta * r + i] = slab[j[beta] + i * stride];
  }
  if constexpr (Ns > 1) {
    // twiddles W_{Ns r}^{i k}, k = j mod Ns, from table row k of this pass
    constexpr unsigned off = unsigned(PL::tw_off(PASS, INV)) * 8u;
#pragma unroll
    for (int beta = 0; beta < b; ++beta) {
      const unsigned k = j[beta] % Ns;
      const unsigned vo = k * unsigned(r - 1) * 8u;
#pragma unroll
      for (int i = 1; i < r; ++i) v[beta * r + i] = ctw<INV>(v[beta * r + i], tw.ld2(vo, off + (i - 1) * 8u));
    }
  }
#pragma unroll
  for (int beta = 0; beta < b; ++beta) Dft<r, INV>::run(&v[beta * r]);
  if constexpr (!last) {
    ctx.sync_row();
#pragma unroll
    for (int beta = 0; beta < b; ++beta) {
      const unsigned k = j[beta] % Ns;
      const unsigned base = (j[beta] - k) * r + k;
#pragma unroll
      for (int m = 0; m < r; ++m) slab[base + m * Ns] = v[beta * r + m];
    }
    ctx.sync_row();
  }
}

template <class PL, bool INV, int KF, int KL, class Ctx>
__host__ __device__ __forceinline__ void stockham_fft(Ctx& ctx, float2 (&v)[PL::P], unsigned t, float2* slab,
                                                     GView tw) {
  stockham_pass<PL, INV, 0, KF, KL>(ctx, v, t, slab, tw);
  if constexpr (PL::NPASS > 1) stockham_pass<PL, INV, 1, KF, KL>(ctx, v, t, slab, tw);
  if constexpr (PL::NPASS > 2) stockham_pass<PL, INV, 2, KF, KL>(ctx, v, t, slab, tw);
  if constexpr (PL::NPASS > 3) stockham_pass<PL, INV, 3, KF, KL>(ctx, v, t, slab, tw);
}

// Sum the per-row images [rows][SLAB] of a workgroup in fixed row order and
// write nfl floats to out (float4 granularity).  Called by every thread.
template <int ROWS, int SLAB, int THREADS>
__host__ __device__ __forceinline__ void sum_rows(const float* lds, GView out, int nfl, int tid) {
  const unsigned n4 = unsigned(nfl) / 4;
  for (unsigned e = unsigned(tid); e < n4; e += THREADS) {
    float4 s = reinterpret_cast<const float4*>(lds)[e];
#pragma unroll
    for (int r = 1; r < ROWS; ++r) {
      const float4 u = reinterpret_cast<const float4*>(lds + r * SLAB)[e];
      s.x += u.x;
      s.y += u.y;
      s.z += u.z;
      s.w += u.w;
    }
    out.st4(s, e * 16u, 0u);
  }
}

}  // namespace acdc
