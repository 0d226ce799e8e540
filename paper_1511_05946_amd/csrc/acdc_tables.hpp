// Host construction of the per-plan constant tables.
//
// Every value is computed in double precision from an exactly reduced angle
// (integer octant reduction, then a series on |angle| <= pi/4) and rounded
// once to fp32.  Tables depend only on the plan, never on the data, so each
// device builds them once and keeps them until the process ends.
#pragma once

#include <cmath>
#include <cstring>
#include <vector>

#include "acdc_dft.hpp"
#include "acdc_plans.hpp"

namespace acdc {

struct HostC {
  double re, im;
};

// exp(-2 pi i e / L)
inline HostC w_pow(long long e, long long L) {
  const CS cs = cos_sin_2pi(e, L);
  return HostC{cs.c, -cs.s};
}

template <class PL>
inline void fill_fft_twiddles(float2* tw) {
  for (int d = 0; d < 2; ++d) {
    const bool inv = d == 1;
    for (int p = 1; p < PL::NPASS; ++p) {
      const int r = PL::radix(p, inv), Ns = PL::ns(p, inv), off = PL::tw_off(p, inv);
      for (int k = 0; k < Ns; ++k)
        for (int i = 1; i < r; ++i) {
          const HostC w = w_pow((long long)i * k, (long long)Ns * r);
          tw[off + k * (r - 1) + (i - 1)] = make_float2(float(w.re), float(w.im));
        }
    }
  }
}

// Spectrum index k handled by quartet slot `slot` of thread t, or -1 for the
// spare slot of every thread but thread 0.
template <class PL>
inline int real_slot_k(int t, int slot) {
  constexpr int RL = PL::RL, BL = PL::BL, NB = PL::NB, T = PL::T;
  if (slot == PL::NSL - 1) return t == 0 ? PL::M / 2 : -1;
  const int q = slot / RL, i = slot % RL;
  const int p = t + T * q;
  if (p != 0) return p + i * NB;
  return i < RL / 2 ? i * NB : NB / 2 + (i - RL / 2) * NB;
  (void)BL;
}

// Returns false if the quartet slots do not cover every DCT index exactly once.
template <class PL>
inline bool build_real_tables(std::vector<unsigned char>& buf) {
  constexpr int N = PL::N, M = PL::M, T = PL::T, NSL = PL::NSL;
  buf.assign(PL::TABLE_BYTES, 0);
  fill_fft_twiddles<PL>(reinterpret_cast<float2*>(buf.data()));
  float4* mk0 = reinterpret_cast<float4*>(buf.data() + PL::OFF_MK0);
  float4* mk1 = reinterpret_cast<float4*>(buf.data() + PL::OFF_MK1);
  int4* qidx = reinterpret_cast<int4*>(buf.data() + PL::OFF_QIDX);
  int* qmask = reinterpret_cast<int*>(buf.data() + PL::OFF_QMASK);
  std::vector<int> cover(N, 0);
  const double s0 = std::sqrt(1.0 / N), s = std::sqrt(2.0 / N);
  for (int slot = 0; slot < NSL; ++slot)
    for (int t = 0; t < T; ++t) {
      const int e = slot * T + t;
      const int k = real_slot_k<PL>(t, slot);
      if (k < 0) {
        mk0[e] = make_float4(0, 0, 0, 0);
        mk1[e] = make_float4(0, 0, 0, 0);
        qidx[e] = make_int4(0, 0, 0, 0);
        qmask[e] = 0;
        continue;
      }
      const double sk = (k == 0) ? s0 : s;
      const HostC w = w_pow(k, N);        // W_N^k
      const HostC q = w_pow(k, 4LL * N);  // W_4N^k
      const double fa = sk / 2, fb = s / (2 * std::sqrt(2.0)), fp = 1.0 / (2.0 * M * sk);
      mk0[e] = make_float4(float(w.re), float(w.im), float(fa * q.re), float(fa * q.im));
      mk1[e] = make_float4(float(fb * q.re), float(fb * q.im), float(fp * q.re), float(-fp * q.im));
      int idx[4] = {k, N - k, M - k, M + k};
      int dmask = 0, smask = 0;
      for (int c = 0; c < 4; ++c) {
        if (idx[c] < N) dmask |= 1 << c;
        else idx[c] = 0;
      }
      if (k == 0) smask = 0x5;              // X[0], X[M]
      else if (2 * k == M) smask = 0x3;     // X[M/2], X[3M/2]
      else smask = 0xF;
      for (int c = 0; c < 4; ++c)
        if (smask & (1 << c)) cover[idx[c]]++;
      qidx[e] = make_int4(idx[0], idx[1], idx[2], idx[3]);
      qmask[e] = dmask | (smask << 4);
    }
  for (int n = 0; n < N; ++n)
    if (cover[n] != 1) return false;
  return true;
}

template <class PL>
inline bool build_complex_tables(std::vector<unsigned char>& buf) {
  buf.assign(PL::TABLE_BYTES, 0);
  fill_fft_twiddles<PL>(reinterpret_cast<float2*>(buf.data()));
  return true;
}

}  // namespace acdc
