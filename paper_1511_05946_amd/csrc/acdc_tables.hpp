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
  for (int d = 0; d < PL::TW_DIRS; ++d) {
    const bool inv = d == 1;
    for (int p = 1; p < PL::NPASS; ++p) {
      const int r = PL::radix(p, inv), Ns = PL::ns(p, inv), off = PL::tw_off(p, inv);
      // [pair (i-1)/2][k][(i-1)%2]: one 16-byte load per lane reads the
      // twiddles of inputs i, i+1, and the lanes of a load read consecutive k
      for (int i = 1; i < r; ++i)
        for (int k = 0; k < Ns; ++k) {
          const HostC w = w_pow((long long)i * k, (long long)Ns * r);
          tw[off + ((i - 1) / 2) * 2 * Ns + 2 * k + (i - 1) % 2] = make_float2(float(w.re), float(w.im));
        }
    }
  }
}

// Spectrum index k handled by quartet slot `slot` of thread t, or -2 for
// slot 0 of thread 0, which carries the two self-paired values Z[0] and
// Z[M/2] and yields X[0], X[M], X[3M/2], X[M/2].
template <class PL>
inline int real_slot_k(int t, int slot) {
  constexpr int RL = PL::RL, NB = PL::NB, T = PL::T;
  const int q = slot / RL, i = slot % RL;
  const int p = t + T * q;
  if (p != 0) return p + i * NB;
  if (i == 0) return -2;
  return i < RL / 2 ? i * NB : NB / 2 + i * NB;
}

// Makhoul coefficients and DCT indices of the quartet of spectrum index k
// (k = -2: the self-paired quartet (Z[0], Z[M/2])), for width N.
inline void quartet_entry(int N, int k, float4& mk0, float4& mk1, int (&idx)[4]) {
  const int M = N / 2;
  const double s0 = std::sqrt(1.0 / N), s = std::sqrt(2.0 / N);
  if (k == -2) {
    // w = i turns the generic quartet into P1 = 2 Z[0], P2 = 2 conj(Z[M/2]).
    const HostC q8 = w_pow(1, 16);  // exp(-i pi/8)
    const double c8 = q8.re, s8 = -q8.im;
    mk0 = make_float4(0.f, 1.f, float(s0 / 2), float(-s0 / 2));
    mk1 = make_float4(float(s * (c8 + s8) / 4), float(s * (c8 - s8) / 4), float(s0 / 2), float(s0 / 2));
    idx[0] = 0;
    idx[1] = M;
    idx[2] = 3 * M / 2;
    idx[3] = M / 2;
  } else {
    const double sk = (k == 0) ? s0 : s;
    const HostC w = w_pow(k, N);        // W_N^k
    const HostC q = w_pow(k, 4LL * N);  // W_4N^k
    const double fa = sk / 2, fb = s / (2 * std::sqrt(2.0)), fp = 1.0 / (2.0 * M * sk);
    mk0 = make_float4(float(w.re), float(w.im), float(fa * q.re), float(fa * q.im));
    mk1 = make_float4(float(fb * q.re), float(fb * q.im), float(fp * q.re), float(-fp * q.im));
    idx[0] = k;
    idx[1] = N - k;
    idx[2] = M - k;
    idx[3] = M + k;
  }
}

// Returns false if the quartet slots do not cover every DCT index exactly once.
template <class PL>
inline bool build_real_tables(std::vector<unsigned char>& buf) {
  constexpr int N = PL::N, T = PL::T, NSL = PL::NSL;
  buf.assign(PL::TABLE_BYTES, 0);
  fill_fft_twiddles<PL>(reinterpret_cast<float2*>(buf.data()));
  float4* mk0 = reinterpret_cast<float4*>(buf.data() + PL::OFF_MK0);
  float4* mk1 = reinterpret_cast<float4*>(buf.data() + PL::OFF_MK1);
  int4* qidx = reinterpret_cast<int4*>(buf.data() + PL::OFF_QIDX);
  int* qmask = reinterpret_cast<int*>(buf.data() + PL::OFF_QMASK);
  std::vector<int> cover(N, 0);
  for (int slot = 0; slot < NSL; ++slot)
    for (int t = 0; t < T; ++t) {
      const int e = slot * T + t;
      int idx[4];
      quartet_entry(N, real_slot_k<PL>(t, slot), mk0[e], mk1[e], idx);
      for (int c = 0; c < 4; ++c) {
        if (idx[c] < 0 || idx[c] >= N) return false;
        cover[idx[c]]++;
      }
      qidx[e] = make_int4(idx[0], idx[1], idx[2], idx[3]);
      qmask[e] = 0xF | (0xF << 4);
    }
  for (int n = 0; n < N; ++n)
    if (cover[n] != 1) return false;
  return true;
}

// Tables of the multi-pass path for a power-of-two width N (M = N/2):
// W_M^e for e < M (DIF/DIT twiddles), then the quartet tables indexed by
// quartet e < M/2 (e = 0: the self-paired quartet, else spectrum index e).
struct MpTableLayout {
  size_t tw = 0, mk0 = 0, mk1 = 0, qidx = 0, qmask = 0, bytes = 0;
};
inline MpTableLayout mp_table_layout(long long N) {
  const size_t M = size_t(N / 2), NQ = M / 2;
  MpTableLayout l;
  l.tw = 0;
  l.mk0 = M * sizeof(float2);
  l.mk1 = l.mk0 + NQ * sizeof(float4);
  l.qidx = l.mk1 + NQ * sizeof(float4);
  l.qmask = l.qidx + NQ * sizeof(int4);
  l.bytes = l.qmask + NQ * sizeof(int);
  return l;
}
inline bool build_mp_tables(int N, std::vector<unsigned char>& buf) {
  const int M = N / 2, NQ = M / 2;
  const MpTableLayout l = mp_table_layout(N);
  buf.assign(l.bytes, 0);
  float2* tw = reinterpret_cast<float2*>(buf.data() + l.tw);
  for (int e = 0; e < M; ++e) {
    const HostC w = w_pow(e, M);
    tw[e] = make_float2(float(w.re), float(w.im));
  }
  float4* mk0 = reinterpret_cast<float4*>(buf.data() + l.mk0);
  float4* mk1 = reinterpret_cast<float4*>(buf.data() + l.mk1);
  int4* qidx = reinterpret_cast<int4*>(buf.data() + l.qidx);
  int* qmask = reinterpret_cast<int*>(buf.data() + l.qmask);
  std::vector<int> cover(N, 0);
  for (int e = 0; e < NQ; ++e) {
    int idx[4];
    quartet_entry(N, e == 0 ? -2 : e, mk0[e], mk1[e], idx);
    for (int c = 0; c < 4; ++c) {
      if (idx[c] < 0 || idx[c] >= N) return false;
      cover[idx[c]]++;
    }
    qidx[e] = make_int4(idx[0], idx[1], idx[2], idx[3]);
    qmask[e] = 0xF | (0xF << 4);
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
