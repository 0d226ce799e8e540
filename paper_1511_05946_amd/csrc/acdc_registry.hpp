// The supported row widths and their plans, plus the per-element helpers
// shared by the GPU kernels and the CPU emulation (parameter re-layout and
// the fixed-order batch reduction).
#pragma once

#include "acdc_complex.hpp"
#include "acdc_real.hpp"
#include "acdc_tables.hpp"

namespace acdc {

// Real ACDC plans: N -> (threads per row, Stockham radices of the N/2-point FFT).
using RP8 = RealPlan<8, 1, 2, 2>;
using RP16 = RealPlan<16, 1, 2, 4>;
using RP32 = RealPlan<32, 2, 4, 4>;
using RP64 = RealPlan<64, 2, 4, 8>;
using RP128 = RealPlan<128, 4, 8, 8>;
using RP256 = RealPlan<256, 4, 16, 8>;
using RP512 = RealPlan<512, 16, 8, 4, 8>;  // 16 complex values per thread
using RP1024 = RealPlan<1024, 32, 8, 8, 8>;  // 16 complex values per thread: 125 VGPRs forward, 4 waves per SIMD
using RP2048 = RealPlan<2048, 32, 16, 4, 16>;
using RP4096 = RealPlan<4096, 64, 16, 8, 16>;
using RP8192 = RealPlan<8192, 128, 16, 16, 16>;
using RP9216 = RealPlan<9216, 192, 12, 8, 4, 12>;
using RP16384 = RealPlan<16384, 256, 16, 32, 16>;
using RP32768 = RealPlan<32768, 512, 16, 8, 8, 16>;

// Complex AFDF plans: N -> (threads per row, radices of the N-point FFT).
using CP8 = ComplexPlan<8, 1, 2, 4>;
using CP16 = ComplexPlan<16, 1, 4, 4>;
using CP32 = ComplexPlan<32, 2, 4, 8>;
using CP64 = ComplexPlan<64, 4, 8, 8>;
using CP128 = ComplexPlan<128, 8, 16, 8>;
using CP256 = ComplexPlan<256, 8, 16, 16>;
using CP512 = ComplexPlan<512, 16, 32, 16>;
using CP1024 = ComplexPlan<1024, 32, 32, 32>;
using CP2048 = ComplexPlan<2048, 64, 32, 2, 32>;
using CP4096 = ComplexPlan<4096, 128, 16, 16, 16>;  // two butterflies per thread at both ends: adjacent pairs
using CP8192 = ComplexPlan<8192, 256, 32, 8, 32>;
using CP16384 = ComplexPlan<16384, 512, 32, 16, 32>;

// Rows per workgroup.  Forward rows are independent; backward rows of one
// workgroup are reduced together into one partial of dL/da, dL/dd.
//
// Real plans whose rows fit a wave (T <= 64) run 512-thread workgroups
// (8 waves) that also hold a copy of the FFT twiddle table in LDS when it
// fits next to the row slabs: every row of the workgroup then reads its
// twiddles from LDS instead of streaming them from the cache hierarchy.
// Such workgroups are persistent (each loops over row groups), so the
// table is copied once per workgroup.
#ifndef ACDC_FWD_THREADS
#define ACDC_FWD_THREADS 64
#endif
#ifndef ACDC_BWD_THREADS
#define ACDC_BWD_THREADS 512
#endif
#ifndef ACDC_TW_LDS
#define ACDC_TW_LDS 1
#endif
// Workgroup size for rows of at most 16 threads (small N): fewer rows per
// workgroup give more workgroups at a given batch.
#ifndef ACDC_NARROW_THREADS
#define ACDC_NARROW_THREADS 256
#endif
// A row width (threads) above one wave whose forward also keeps the twiddles
// in LDS (0: none).
#ifndef ACDC_TW_LDS_T
#define ACDC_TW_LDS_T 0
#endif
// Rows per backward workgroup for real rows of 32 threads (N = 1024, 2048):
// 8 (four waves, three workgroups per CU at 3 waves per SIMD) ran the
// backward 6-8 % faster than 16, more than the doubled partials cost.
#ifndef ACDC_BWD_ROWS_T32
#define ACDC_BWD_ROWS_T32 8
#endif
// Rows per backward workgroup for the three-wave rows of N = 9216.
#ifndef ACDC_BWD_ROWS_T192
#define ACDC_BWD_ROWS_T192 2
#endif
// Rows per backward workgroup for the two-wave complex rows of N = 4096.
// With the workgroup barrier for every FFT exchange, two 256-thread
// workgroups per CU beat one of 512 threads (backward 12 % faster, at twice
// the partials).  With each row's waves meeting only each other
// (GroupCtx), four rows per workgroup cost the backward 2 % and halve the
// partials: step 0.803 -> 0.765 ms.
#ifndef ACDC_BWD_ROWS_CPLX_T128
#define ACDC_BWD_ROWS_CPLX_T128 4
#endif
#ifndef ACDC_TW_LDS_BWD
#define ACDC_TW_LDS_BWD 0
#endif
// Rows of several waves in multi-row backward workgroups meet at an LDS
// counter of their own (GroupCtx) instead of the workgroup barrier at every
// FFT exchange: 0 turns that off.  Measured (same results bit for bit):
// backward 0.846 -> 0.774 ms at N = 9216, 0.775 -> 0.663 ms at N = 8192.
#ifndef ACDC_GROUP_SYNC
#define ACDC_GROUP_SYNC 1
#endif
// Persistent backward workgroups that add their tiles into one partial each
// (unbiased real rows, tiles of at most ACDC_BWD_ACC_MAX_ROWS rows): 0 turns
// them off.  Each added tile first fetches the slot's previous values, and
// the vector-memory counter completes in order, so every later load waits
// for that fetch too: at N = 4096 (8-row tiles) the backward lost more
// (0.087 ms) than the smaller reduction saved (0.059 ms); at N = 9216
// (2-row tiles, twice the partial bytes per row) the step gained 2.5 %.
#ifndef ACDC_BWD_ACC
#define ACDC_BWD_ACC 1
#endif
#ifndef ACDC_BWD_ACC_MAX_ROWS
#define ACDC_BWD_ACC_MAX_ROWS 2
#endif
constexpr int kLdsBytes = 160 * 1024;
template <class PL>
struct Launch {
  static constexpr int FWD_SLAB = PL::kComplex ? PL::SLAB : cmax(PL::N, PL::FFT_FLOATS);  // floats per row
  static constexpr int BWD_SLAB = PL::SLAB;
  static constexpr int WIDE_ROWS = PL::T <= 16 ? ACDC_NARROW_THREADS / PL::T : PL::T <= 64 ? 512 / PL::T : 1;
  static constexpr bool TW_LDS = ACDC_TW_LDS && !PL::kComplex && (PL::T <= 64 || PL::T == ACDC_TW_LDS_T) &&
                                 WIDE_ROWS * PL::SLAB * 4 + PL::TW_FLOAT2 * 8 <= kLdsBytes;
  static constexpr int FWD_ROWS =
      TW_LDS ? WIDE_ROWS : (PL::T >= ACDC_FWD_THREADS ? 1 : ACDC_FWD_THREADS / PL::T);
  static constexpr int BWD_ROWS =
      (PL::T == 32 && !PL::kComplex)    ? ACDC_BWD_ROWS_T32
      : PL::T == 192                    ? ACDC_BWD_ROWS_T192
      : (PL::kComplex && PL::T == 128)  ? ACDC_BWD_ROWS_CPLX_T128
                                        : (TW_LDS ? WIDE_ROWS : (PL::T >= ACDC_BWD_THREADS ? 1 : ACDC_BWD_THREADS / PL::T));
  static constexpr bool BWD_TW_LDS = TW_LDS && ACDC_TW_LDS_BWD;
  static constexpr bool BWD_GROUP_SYNC = ACDC_GROUP_SYNC && PL::T > 64 && PL::T % 64 == 0 && BWD_ROWS > 1;
  static constexpr int FWD_THREADS = FWD_ROWS * PL::T;
  static constexpr int BWD_THREADS = BWD_ROWS * PL::T;
  static constexpr int TW_FLOATS = TW_LDS ? PL::TW_FLOAT2 * 2 : 0;  // LDS copy of the twiddles
  static constexpr int BWD_TW_FLOATS = BWD_TW_LDS ? PL::TW_FLOAT2 * 2 : 0;
  static constexpr int FWD_LDS_FLOATS = FWD_ROWS * FWD_SLAB + TW_FLOATS;
  static constexpr int BWD_LDS_FLOATS = BWD_ROWS * BWD_SLAB + BWD_TW_FLOATS;
  static constexpr int FWD_LDS_BYTES = FWD_LDS_FLOATS * 4;
  static constexpr int BWD_LDS_BYTES = BWD_LDS_FLOATS * 4;
  // Occupancy the register allocator must reach (512 / WPE registers per lane).
  static constexpr int FWD_WPE = 2;
  static constexpr int BWD_WPE = 2;
  // Persistent accumulation keeps the previous partial values of one sum
  // (max(N, QF) floats) in LDS after the row slabs.  It is used where that
  // fits and does not cost a resident workgroup: the count that the LDS
  // allows stays at least the count that BWD_WPE waves per SIMD allow.
  static constexpr int ACC_FLOATS = cmax(PL::N, PL::QF);
  static constexpr int BWD_WAVE_WGS = (4 * BWD_WPE * 64) / BWD_THREADS;
  static constexpr int BWD_ACC_LDS_BYTES = BWD_LDS_BYTES + ACC_FLOATS * 4;
  static constexpr bool BWD_ACC = ACDC_BWD_ACC && !PL::kComplex && PL::N >= 1024 &&
                                  BWD_ROWS <= ACDC_BWD_ACC_MAX_ROWS && (PL::N / 4) % 64 == 0 &&
                                  (PL::QF / 4) % 64 == 0 && BWD_THREADS % 64 == 0 &&
                                  BWD_ACC_LDS_BYTES <= kLdsBytes &&
                                  kLdsBytes / BWD_ACC_LDS_BYTES >= cmin(kLdsBytes / BWD_LDS_BYTES, BWD_WAVE_WGS);
  static_assert(FWD_LDS_BYTES <= kLdsBytes && BWD_LDS_BYTES <= kLdsBytes, "LDS budget");
  static_assert(BWD_THREADS <= 1024 && FWD_THREADS <= 1024, "workgroup size");
};

// ACDC_ONLY_N=<width> instantiates a single real plan and ACDC_ONLY_CN a
// single complex plan (quick development builds); ACDC_PLAN_SUBSET
// instantiates real plans 8, 64, 1024, 4096, 9216 and complex plans 16, 256,
// 4096 (the sanitizer build of the tests).  Every other width then reports
// unsupported.
template <class PLn>
constexpr bool plan_built() {
#if defined(ACDC_ONLY_N)
  return PLn::N == ACDC_ONLY_N && !PLn::kComplex;
#elif defined(ACDC_ONLY_CN)
  return PLn::N == ACDC_ONLY_CN && PLn::kComplex;
#elif defined(ACDC_PLAN_SUBSET)
  return PLn::kComplex ? (PLn::N == 16 || PLn::N == 256 || PLn::N == 4096)
                       : (PLn::N == 8 || PLn::N == 64 || PLn::N == 1024 || PLn::N == 4096 || PLn::N == 9216);
#else
  return true;
#endif
}

template <class PLn, class F>
inline bool run_plan(F& f) {
  if constexpr (!plan_built<PLn>()) {
    return false;
  } else {
    f.template operator()<PLn>();
    return true;
  }
}

// Calls f.template operator()<Plan>() for the real plan of width N.
template <class F>
inline bool dispatch_real(int N, F&& f) {
  switch (N) {
    case 8: return run_plan<RP8>(f);
    case 16: return run_plan<RP16>(f);
    case 32: return run_plan<RP32>(f);
    case 64: return run_plan<RP64>(f);
    case 128: return run_plan<RP128>(f);
    case 256: return run_plan<RP256>(f);
    case 512: return run_plan<RP512>(f);
    case 1024: return run_plan<RP1024>(f);
    case 2048: return run_plan<RP2048>(f);
    case 4096: return run_plan<RP4096>(f);
    case 8192: return run_plan<RP8192>(f);
    case 9216: return run_plan<RP9216>(f);
    case 16384: return run_plan<RP16384>(f);
    case 32768: return run_plan<RP32768>(f);
    default: return false;
  }
}

template <class F>
inline bool dispatch_complex(int N, F&& f) {
  switch (N) {
    case 8: return run_plan<CP8>(f);
    case 16: return run_plan<CP16>(f);
    case 32: return run_plan<CP32>(f);
    case 64: return run_plan<CP64>(f);
    case 128: return run_plan<CP128>(f);
    case 256: return run_plan<CP256>(f);
    case 512: return run_plan<CP512>(f);
    case 1024: return run_plan<CP1024>(f);
    case 2048: return run_plan<CP2048>(f);
    case 4096: return run_plan<CP4096>(f);
    case 8192: return run_plan<CP8192>(f);
    case 16384: return run_plan<CP16384>(f);
    default: return false;
  }
}

// The per-entry quartet tables of a width N: Makhoul twiddle blocks mk0,
// mk1, the four DCT indices of each entry and their masks (low nibble: the
// d values to read; high nibble: the image values to store).  The fused
// plans index them by slot entry e = slot*T + t, the multi-pass path by the
// quartet number; entry 0 is the self-paired quartet (Z[0], Z[M/2]) in both.
struct QuartetTabs {
  const float4* mk0;
  const float4* mk1;
  const int4* qidx;
  const int* qmask;
  float qb0_re, qb0_im;  // entry 0's DCT-III pre-twiddle exp(i pi/8) / (2 sqrt(N))
};
template <class PL>
__host__ __device__ __forceinline__ QuartetTabs quartet_tabs(const char* tab) {
  return QuartetTabs{reinterpret_cast<const float4*>(tab + PL::OFF_MK0),
                     reinterpret_cast<const float4*>(tab + PL::OFF_MK1),
                     reinterpret_cast<const int4*>(tab + PL::OFF_QIDX),
                     reinterpret_cast<const int*>(tab + PL::OFF_QMASK), RealOps<PL>::kQbRe, RealOps<PL>::kQbIm};
}

// A layer vector (d or b) at the four quartet indices of entry e.
__host__ __device__ __forceinline__ float4 quartet_gather(const float* Vk, const QuartetTabs& q, int e) {
  const int4 idx = q.qidx[e];
  const int m = q.qmask[e] & 0xF;
  return make_float4((m & 1) ? Vk[idx.x] : 0.f, (m & 2) ? Vk[idx.y] : 0.f, (m & 4) ? Vk[idx.z] : 0.f,
                     (m & 8) ? Vk[idx.w] : 0.f);
}

// Quartet coefficients of layer k at slot entry e = slot*T + t.
//
// The middle of a layer takes one quartet's spectrum pair (Z[k], Z[M-k])
// through the DCT-II post-twiddle, the D diagonal and the DCT-III
// pre-twiddle (the steps listed in RealOps' Makhoul-quartet comment).  With
// the real-FFT split
//   E = Z[k] + conj Z[M-k],  O = (Z[k] - conj Z[M-k]) / i,
//   s1 = E + w O,  s2 = E - w O          (w = W_N^k)
// the post-twiddle, the four d values and the pre-twiddle act on s1 and s2
// separately, each as a 2x2 real matrix:
//   s1 -> qap * diag(d0, d1) * (qa s1)                (X[k], X[N-k] pair)
//   s2 -> conj(qb') * H^T diag(d2, d3) H * (qb s2)    (X[M-k], X[M+k] pair)
// with H = [[1,-1],[1,1]].  Both matrices are symmetric because qap and qb'
// point along conj(qa) and qb (also for thread 0's self-paired slot), so a
// slot needs w and 3 + 3 coefficients.  Output rows:
//   out[0] = (L1_00, L1_01, L1_11, L2_00)
//   out[1] = (L2_01, L2_11, w.x, w.y)
//   out[2] = (qa.x, qa.y, qbr.x, qbr.y) (the DCT-II outputs the backward needs)
//   out[3] = the D-domain bias through the pre-twiddle (zero without bias)
// Coefficients are formed in double from the fp32 twiddle tables and
// rounded once.
struct QuartetD {
  double x, y;
};
__host__ __device__ inline QuartetD qd_mul(QuartetD a, QuartetD w) {
  return QuartetD{a.x * w.x - a.y * w.y, a.x * w.y + a.y * w.x};
}
__host__ __device__ inline QuartetD qd_mulc(QuartetD a, QuartetD w) {  // a * conj(w)
  return QuartetD{a.x * w.x + a.y * w.y, a.y * w.x - a.x * w.y};
}
__host__ __device__ inline void quartet_coeffs(const float* Dk, const float* Bk, const QuartetTabs& q, int e,
                                               float4 (&out)[kMqRows]) {
  const float4 m0 = q.mk0[e];
  const float4 m1 = q.mk1[e];
  const float4 d = quartet_gather(Dk, q, e);
  const QuartetD qa{m0.z, m0.w}, qb{m1.x, m1.y}, qap{m1.z, m1.w};
  // thread 0's slot 0 carries the self-paired values; its pre-twiddle uses
  // exp(i pi/8) / (2 sqrt(N))
  const QuartetD qbp = e == 0 ? QuartetD{q.qb0_re, q.qb0_im} : qb;
  double L1[2][2], L2[2][2];
  for (int j = 0; j < 2; ++j) {
    const QuartetD s{double(j == 0), double(j == 1)};
    // s1 path: u1 = qa s1, (Y0, -Y1) = (d0 Re u1, d1 Im u1), Ap = (.) qap
    const QuartetD u1 = qd_mul(s, qa);
    const QuartetD ap = qd_mul(QuartetD{d.x * u1.x, d.y * u1.y}, qap);
    L1[0][j] = ap.x;
    L1[1][j] = ap.y;
    // s2 path: u2 = qb s2, X2 = u2.x - u2.y, X3 = u2.x + u2.y, Y = d X,
    // Bp = (Y2 + Y3, Y3 - Y2) conj(qb')
    const QuartetD u2 = qd_mul(s, qb);
    const double y2 = d.z * (u2.x - u2.y), y3 = d.w * (u2.x + u2.y);
    const QuartetD bp = qd_mulc(QuartetD{y2 + y3, y3 - y2}, qbp);
    L2[0][j] = bp.x;
    L2[1][j] = bp.y;
  }
  out[0] = make_float4(float(L1[0][0]), float(0.5 * (L1[0][1] + L1[1][0])), float(L1[1][1]), float(L2[0][0]));
  out[1] = make_float4(float(0.5 * (L2[0][1] + L2[1][0])), float(L2[1][1]), m0.x, m0.y);
  // qb rotated by (1 + i): the backward image then reads X[M-k], X[M+k] off
  // one complex product
  out[2] = make_float4(m0.z, m0.w, float(double(m1.x) - double(m1.y)), float(double(m1.x) + double(m1.y)));
  // D-domain bias: Y gains b, so Ap gains (b0 - i b1) qap and Bp gains
  // (b2 + b3 + i (b3 - b2)) conj(qb'); S = Ap + Bp, Dd = Ap - Bp give the
  // constant (zk, zm) = (S + i conj(w) Dd, conj(S - i conj(w) Dd)) added
  // after the 2x2 maps.
  out[3] = make_float4(0.f, 0.f, 0.f, 0.f);
  if (Bk != nullptr) {
    const float4 b = quartet_gather(Bk, q, e);
    const QuartetD ap = qd_mul(QuartetD{b.x, -double(b.y)}, qap);
    const QuartetD bp = qd_mulc(QuartetD{double(b.z) + b.w, double(b.w) - b.z}, qbp);
    const QuartetD S{ap.x + bp.x, ap.y + bp.y}, Dd{ap.x - bp.x, ap.y - bp.y};
    const QuartetD cw = qd_mulc(Dd, QuartetD{m0.x, m0.y});  // Dd conj(w)
    out[3] = make_float4(float(S.x - cw.y), float(S.y + cw.x), float(S.x + cw.y), float(cw.x - S.y));
  }
}

template <class PL>
__host__ __device__ inline void real_mq_entry(const float* Dk, const float* Bk, const char* tab, int e,
                                              float4 (&out)[kMqRows]) {
  quartet_coeffs(Dk, Bk, quartet_tabs<PL>(tab), e, out);
}

// Fixed-order batch reduction of the per-tile partials.  Entry e (a float4)
// of the reduced gradient is the sum over tiles t of partial[t][e]; tiles
// are split into PH phases (t mod PH), each phase is summed in increasing t,
// and the phase sums are added in phase order.  PH is 4, or 8 where the
// reduced gradient has fewer than kRedFewEntries float4 entries: with 4 the
// blocks would be too few to fill the chip (at N = 1024, K = 12, 6144
// entries, the reduction took 0.017 ms with 4 phases and 0.012 ms with 8;
// at N = 4096, K = 12, 24576 entries, 4 phases were the fastest).  The GPU
// kernel runs the phases on separate threads and combines them in LDS; the
// CPU emulation calls the same functions in the same order.
constexpr long long kRedFewEntries = 16384;
__host__ __device__ constexpr int red_phases(long long n4) { return n4 < kRedFewEntries ? 8 : 4; }
#ifndef ACDC_RED_GROUP
#define ACDC_RED_GROUP 4
#endif
// loads each thread issues ahead of their adds (at N = 4096, 4 beat 8 and 16)
constexpr int kRedGroup = ACDC_RED_GROUP;

__host__ __device__ __forceinline__ float4 add4(float4 a, float4 b) {
  return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

template <int PH>
__host__ __device__ __forceinline__ float4 tile_phase_sum4(const float4* partial, long long ntiles,
                                                           long long stride, long long e, int phase) {
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  long long t = phase;
  // loads in groups of kRedGroup ahead of their (in-order) adds
  for (; t + (kRedGroup - 1) * PH < ntiles; t += kRedGroup * PH) {
    float4 u[kRedGroup];
#pragma unroll
    for (int j = 0; j < kRedGroup; ++j) u[j] = partial[(t + j * PH) * stride + e];
#pragma unroll
    for (int j = 0; j < kRedGroup; ++j) s = add4(s, u[j]);
  }
  for (; t < ntiles; t += PH) s = add4(s, partial[t * stride + e]);
  return s;
}

template <int PH>
__host__ __device__ __forceinline__ float4 phases_total4(const float4 (&ph)[PH]) {
  float4 s = ph[0];
#pragma unroll
  for (int g = 1; g < PH; ++g) s = add4(s, ph[g]);
  return s;
}

__host__ __device__ __forceinline__ void put4(float4* p, float4 s, bool accumulate) {
  *p = accumulate ? add4(*p, s) : s;
}
__host__ __device__ __forceinline__ void put1(float* p, float s, bool accumulate) {
  *p = accumulate ? *p + s : s;
}

// Real path: float4 e4 of layer k of the reduced gradient.  The first N/4
// are dL/da in natural order; the next QF/4 are the dL/dd quartets of slot
// entries e = e4 - N/4, scattered to their indices; with a bias the last N/4
// are the batch sum of g (spatial), stored to gS for its DCT.
template <class PL>
__host__ __device__ __forceinline__ void real_reduce_store4(float4 s, int k, int e4, float* gA, float* gD,
                                                            float* gS, const char* tab, bool accumulate) {
  if (e4 < PL::N / 4) {
    put4(reinterpret_cast<float4*>(gA + (long long)k * PL::N) + e4, s, accumulate);
  } else if (e4 < (PL::N + PL::QF) / 4) {
    const int st = e4 - PL::N / 4;
    const int sm = (reinterpret_cast<const int*>(tab + PL::OFF_QMASK)[st] >> 4) & 0xF;
    const int4 idx = reinterpret_cast<const int4*>(tab + PL::OFF_QIDX)[st];
    float* gd = gD + (long long)k * PL::N;
    if (sm & 1) put1(gd + idx.x, s.x, accumulate);
    if (sm & 2) put1(gd + idx.y, s.y, accumulate);
    if (sm & 4) put1(gd + idx.z, s.z, accumulate);
    if (sm & 8) put1(gd + idx.w, s.w, accumulate);
  } else {
    reinterpret_cast<float4*>(gS + (long long)k * PL::N)[e4 - (PL::N + PL::QF) / 4] = s;
  }
}

// Complex path: float4 e4 in [0, N) of layer k (dL/da then dL/dd, natural).
template <class PL>
__host__ __device__ __forceinline__ void cplx_reduce_store4(float4 s, int k, int e4, float* gA, float* gD,
                                                            bool accumulate) {
  if (e4 < PL::N / 2) put4(reinterpret_cast<float4*>(gA + (long long)k * 2 * PL::N) + e4, s, accumulate);
  else put4(reinterpret_cast<float4*>(gD + (long long)k * 2 * PL::N) + (e4 - PL::N / 2), s, accumulate);
}

// Float4 entries per layer of one tile's partial.
template <class PL>
constexpr long long partial_entries4(bool bias = false) {
  if constexpr (PL::kComplex) return (long long)PL::N;
  else return (long long)(PL::N + PL::QF + (bias ? PL::N : 0)) / 4;
}

}  // namespace acdc
