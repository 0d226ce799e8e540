// Compile-time plans: how one row of width N is spread over threads and how
// its transforms are factored into Stockham passes.
//
// Real ACDC rows (DCT-II via Makhoul's reordering, Sec. 5 multi-call recipe
// and its Makhoul reference): a row of N reals is packed as M = N/2 complex
// values z[m] = v[2m] + i v[2m+1] and transformed by an M-point complex FFT.
// T threads share a row; each holds P = M/T complex values in registers.
// The FFT runs as NPASS Stockham passes with radices RAD[0..NPASS-1]; the
// inverse FFT runs the radices in reverse order so that its output lands in
// exactly the register layout the forward FFT reads.
//
// Complex AFDF rows (Sec. 3): N complex values, N-point FFT, same idea
// without the real-to-complex packing.
#pragma once

#include <cstdint>

#ifndef ACDC_TAB_PF
#define ACDC_TAB_PF 3  // quartet slots whose tables are loaded ahead
#endif
#ifndef ACDC_MQ_PF
#define ACDC_MQ_PF 3  // quartet-coefficient slots loaded ahead in the layer middles
#endif
#ifndef ACDC_MQ_PF_BWD
#define ACDC_MQ_PF_BWD 1  // the same in the backward middle (three float4 per slot; 1 beat 2 by 0.5-1.8 % at N = 4096)
#endif
#ifndef ACDC_CPLX_FWD_PF
#define ACDC_CPLX_FWD_PF 1  // complex forward: A and D loaded one step ahead of their use
#endif
#ifndef ACDC_PACKED_PERM
#define ACDC_PACKED_PERM 1  // fused real rows: perm as packed 16-bit slab offsets (N <= 16384)
#endif
#ifndef ACDC_FFT2
#define ACDC_FFT2 1  // backward: the h- and g-path FFTs share twiddle loads
#endif
#ifndef ACDC_CPLX_PAIRS
#define ACDC_CPLX_PAIRS 1  // complex rows: adjacent butterfly pairs where the plan allows
#endif
#ifndef ACDC_XLANE_SUM
#define ACDC_XLANE_SUM 0  // 1: rows of 16 lanes sum their images across the wave with lane swaps (measured slower)
#endif
#ifndef ACDC_LDS_PAD
#define ACDC_LDS_PAD 1
#endif

namespace acdc {

constexpr int cmax(int a, int b) { return a > b ? a : b; }
constexpr int cmin(int a, int b) { return a < b ? a : b; }
constexpr double csqrt(double x) {
  double r = x > 1 ? x : 1.0;
  for (int i = 0; i < 64; ++i) r = 0.5 * (r + x / r);
  return r;
}
constexpr int ilog2(int v) {
  int l = 0;
  while ((1 << (l + 1)) <= v) ++l;
  return l;
}

template <int N_, int T_, int R0_, int R1_, int R2_ = 1, int R3_ = 1>
struct RealPlan {
  static constexpr bool kComplex = false;
  static constexpr int N = N_;
  static constexpr int M = N_ / 2;  // complex points per row
  static constexpr int T = T_;      // threads per row
  static constexpr int P = M / T_;  // complex registers per thread
  static constexpr int NPASS = (R2_ == 1) ? 2 : ((R3_ == 1) ? 3 : 4);
  __host__ __device__ static constexpr int rad(int p) {
    return p == 0 ? R0_ : p == 1 ? R1_ : p == 2 ? R2_ : R3_;
  }
  // radix of pass p of the forward (INV=false) or inverse (INV=true) FFT
  __host__ __device__ static constexpr int radix(int p, bool inv) {
    return inv ? rad(NPASS - 1 - p) : rad(p);
  }
  // Stockham stride Ns before pass p: product of the earlier radices
  __host__ __device__ static constexpr int ns(int p, bool inv) {
    int s = 1;
    for (int q = 0; q < p; ++q) s *= radix(q, inv);
    return s;
  }
  static constexpr int R0 = R0_;
  static constexpr int RL = rad(NPASS - 1);
  static constexpr int B0 = P / R0;              // butterflies per thread, first pass
  static constexpr int BL = P / RL;              // butterflies per thread, last pass
  static constexpr int NB = M / RL;              // butterflies of the last pass
  static constexpr int NSL = (BL / 2) * RL;      // quartet slots per thread
  static constexpr int QF = NSL * T * 4;         // floats of one row's quartet image
  // FFT data in LDS: complex element a lives at a + (a >> PADSH), one pad
  // slot per 2^PADSH elements, so the stride-r writes of the first pass and
  // the stride-1 reads of the next spread over all banks.  Plans whose first
  // radix is not a power of two (N = 9216) go unpadded: there the padded
  // write addresses of the mixed-radix passes are not affine in the lane,
  // so each thread would hold one precomputed address per output (about 48
  // VGPRs, spilled) instead of one base per butterfly.
  static constexpr int PADSH =
      !ACDC_LDS_PAD ? 30 : (ilog2(R0_) >= 2 && (1 << ilog2(R0_)) == R0_ ? ilog2(R0_) : 30);
  static constexpr int FFT_FLOATS = 2 * (M + (M >> PADSH));
  static constexpr int SLAB = cmax(cmax(N, QF), FFT_FLOATS);  // LDS floats per row
  // twiddle table (float2) offsets: forward passes 1.., then inverse passes
  // 1.. -- unless the radix sequence is a palindrome, in which case the
  // inverse passes have the forward passes' radices and strides and share
  // their table.
  // Twiddles of a pass are stored in pairs (inputs i, i+1) so one 16-byte
  // load fetches two; an odd count is padded by one entry per k.
  __host__ __device__ static constexpr int tw_count(int p, bool inv) {
    return p == 0 ? 0 : ns(p, inv) * (radix(p, inv) - 1 + ((radix(p, inv) - 1) & 1));
  }
  __host__ __device__ static constexpr bool palindrome() {
    for (int p = 0; p < NPASS; ++p)
      if (rad(p) != rad(NPASS - 1 - p)) return false;
    return true;
  }
  static constexpr int TW_DIRS = palindrome() ? 1 : 2;  // table blocks stored
  __host__ __device__ static constexpr int tw_off(int p, bool inv) {
    const int dsel = (inv && TW_DIRS == 2) ? 1 : 0;
    int o = 0;
    for (int d = 0; d < TW_DIRS; ++d)
      for (int q = 0; q < NPASS; ++q) {
        if (d == dsel && q == p) return o;
        o += tw_count(q, d == 1);
      }
    return o;
  }
  __host__ __device__ static constexpr int tw_total() {
    int o = 0;
    for (int d = 0; d < TW_DIRS; ++d)
      for (int q = 0; q < NPASS; ++q) o += tw_count(q, d == 1);
    return o;
  }
  static constexpr int TW_FLOAT2 = tw_total();
  // table block layout in bytes: [fft twiddles][mk0 float4 NSL*T][mk1 float4 NSL*T]
  //                             [qidx int4 NSL*T][qmask int NSL*T]
  static constexpr int OFF_MK0 = ((TW_FLOAT2 * 8 + 255) / 256) * 256;
  static constexpr int OFF_MK1 = OFF_MK0 + NSL * T * 16;
  static constexpr int OFF_QIDX = OFF_MK1 + NSL * T * 16;
  static constexpr int OFF_QMASK = OFF_QIDX + NSL * T * 16;
  static constexpr int TABLE_BYTES = ((OFF_QMASK + NSL * T * 4 + 255) / 256) * 256;

  static_assert(N % 4 == 0, "N must be a multiple of 4");
  static_assert(M % T == 0, "threads must divide the row");
  static_assert(T <= 64 ? (64 % T == 0) : (T % 64 == 0), "rows tile whole waves");
  static_assert(R0_ * R1_ * R2_ * R3_ == M, "radices must multiply to N/2");
  static_assert(P % R0_ == 0 && P % R1_ == 0 && P % R2_ == 0 && P % R3_ == 0,
                "each radix must divide the per-thread register count");
  static_assert(B0 % 2 == 0, "first pass pairs mirrored butterflies");
  static_assert(BL % 2 == 0 && RL % 2 == 0, "last pass pairs negated butterflies");
  static_assert(R0 % 2 == 0, "first pass radix must be even");
};

template <int N_, int T_, int R0_, int R1_, int R2_ = 1, int R3_ = 1>
struct ComplexPlan {
  static constexpr bool kComplex = true;
  static constexpr int N = N_;  // complex points per row
  static constexpr int M = N_;
  static constexpr int T = T_;
  static constexpr int P = N_ / T_;
  static constexpr int NPASS = (R1_ == 1) ? 1 : ((R2_ == 1) ? 2 : ((R3_ == 1) ? 3 : 4));
  __host__ __device__ static constexpr int rad(int p) {
    return p == 0 ? R0_ : p == 1 ? R1_ : p == 2 ? R2_ : R3_;
  }
  __host__ __device__ static constexpr int radix(int p, bool inv) {
    return inv ? rad(NPASS - 1 - p) : rad(p);
  }
  __host__ __device__ static constexpr int ns(int p, bool inv) {
    int s = 1;
    for (int q = 0; q < p; ++q) s *= radix(q, inv);
    return s;
  }
  static constexpr int PADSH =
      !ACDC_LDS_PAD ? 30 : (ilog2(R0_) >= 2 && (1 << ilog2(R0_)) == R0_ ? ilog2(R0_) : 30);
  static constexpr int FFT_FLOATS = 2 * (N_ + (N_ >> PADSH));
  static constexpr int SLAB = FFT_FLOATS;  // LDS floats per row
  // Twiddles of a pass are stored in pairs (inputs i, i+1) so one 16-byte
  // load fetches two; an odd count is padded by one entry per k.
  __host__ __device__ static constexpr int tw_count(int p, bool inv) {
    return p == 0 ? 0 : ns(p, inv) * (radix(p, inv) - 1 + ((radix(p, inv) - 1) & 1));
  }
  __host__ __device__ static constexpr bool palindrome() {
    for (int p = 0; p < NPASS; ++p)
      if (rad(p) != rad(NPASS - 1 - p)) return false;
    return true;
  }
  static constexpr int TW_DIRS = palindrome() ? 1 : 2;
  __host__ __device__ static constexpr int tw_off(int p, bool inv) {
    const int dsel = (inv && TW_DIRS == 2) ? 1 : 0;
    int o = 0;
    for (int d = 0; d < TW_DIRS; ++d)
      for (int q = 0; q < NPASS; ++q) {
        if (d == dsel && q == p) return o;
        o += tw_count(q, d == 1);
      }
    return o;
  }
  __host__ __device__ static constexpr int tw_total() {
    int o = 0;
    for (int d = 0; d < TW_DIRS; ++d)
      for (int q = 0; q < NPASS; ++q) o += tw_count(q, d == 1);
    return o;
  }
  static constexpr int TW_FLOAT2 = tw_total();
  static constexpr int TABLE_BYTES = ((TW_FLOAT2 * 8 + 255) / 256) * 256 + 256;

  static_assert(N_ % T_ == 0, "threads must divide the row");
  static_assert(T <= 64 ? (64 % T == 0) : (T % 64 == 0), "rows tile whole waves");
  static_assert(R0_ * R1_ * R2_ * R3_ == N_, "radices must multiply to N");
  static_assert(P % R0_ == 0 && P % R1_ == 0 && P % R2_ == 0 && P % R3_ == 0,
                "each radix must divide the per-thread register count");
};

}  // namespace acdc
