// Complex AFDF cascade (Sec. 3: y = x A F D F^{-1} per layer, complex
// diagonals, F the unnormalised DFT with F^{-1} = conj(F)/N).
//
// A row of N complex values lives in the registers of T threads, P = N/T
// each.  Spatial layout: v[beta*R0 + i] is element t + T*(beta + i*B0);
// frequency layout: v[beta*RL + m] is element t + T*(beta + m*BL).  The
// forward FFT maps the first to the second and the inverse FFT (radices
// reversed) maps back, so D multiplies in place and nothing is reordered.
//
// Backward (PyTorch convention, grad = dL/dRe + i dL/dIm, so g_x = g_y W^H):
//   gh3 = FFT(g)/N, dd = sum conj(h2) gh3, gh1 = IFFT_unnorm(gh3 conj(d)),
//   da = sum conj(u) gh1, gu = gh1 conj(a).
#pragma once

#include "acdc_dft.hpp"
#include "acdc_plans.hpp"
#include "acdc_stockham.hpp"

namespace acdc {

template <class PL>
struct CplxOps {
  static constexpr int N = PL::N, T = PL::T, P = PL::P;
  static constexpr int R0 = PL::rad(0), RL = PL::rad(PL::NPASS - 1);
  static constexpr int B0 = P / R0, BL = P / RL;

  // f(element, v[s]) over the spatial layout
  template <class F>
  __host__ __device__ __forceinline__ static void for_spatial(float2 (&v)[P], int t, F&& f) {
#pragma unroll
    for (int beta = 0; beta < B0; ++beta)
#pragma unroll
      for (int i = 0; i < R0; ++i) f(t + T * (beta + i * B0), v[beta * R0 + i]);
  }
  template <class F>
  __host__ __device__ __forceinline__ static void for_spatial2(float2 (&v)[P], float2 (&w)[P], int t, F&& f) {
#pragma unroll
    for (int beta = 0; beta < B0; ++beta)
#pragma unroll
      for (int i = 0; i < R0; ++i) f(t + T * (beta + i * B0), v[beta * R0 + i], w[beta * R0 + i]);
  }
  template <class F>
  __host__ __device__ __forceinline__ static void for_freq(float2 (&v)[P], int t, F&& f) {
#pragma unroll
    for (int beta = 0; beta < BL; ++beta)
#pragma unroll
      for (int m = 0; m < RL; ++m) f(t + T * (beta + m * BL), v[beta * RL + m]);
  }

  __host__ __device__ __forceinline__ static void load(const float* row, float2 (&v)[P], int t, bool valid) {
    const float2* r = reinterpret_cast<const float2*>(row);
    for_spatial(v, t, [&](int e, float2& z) { z = valid ? r[e] : make_float2(0.f, 0.f); });
  }
  __host__ __device__ __forceinline__ static void store(float* row, float2 (&v)[P], int t) {
    float2* r = reinterpret_cast<float2*>(row);
    for_spatial(v, t, [&](int e, float2& z) { r[e] = z; });
  }
  template <bool CONJ>
  __host__ __device__ __forceinline__ static void scale(float2 (&v)[P], const float* a, int t) {
    const float2* ar = reinterpret_cast<const float2*>(a);
    for_spatial(v, t, [&](int e, float2& z) { z = CONJ ? cmulc(z, ar[e]) : cmul(z, ar[e]); });
  }
  template <bool CONJ>
  __host__ __device__ __forceinline__ static void scale_freq(float2 (&v)[P], const float* d, float f, int t) {
    const float2* dr = reinterpret_cast<const float2*>(d);
    for_freq(v, t, [&](int e, float2& z) {
      const float2 w = make_float2(dr[e].x * f, dr[e].y * f);
      z = CONJ ? cmulc(z, w) : cmul(z, w);
    });
  }

  template <class Ctx>
  __host__ __device__ __forceinline__ static void gather(Ctx& ctx, float2 (&v)[P], int t, float2* slab,
                                                         const int* perm) {
    ctx.sync_row();
    for_spatial(v, t, [&](int e, float2& z) { slab[e] = z; });
    ctx.sync_row();
    for_spatial(v, t, [&](int e, float2& z) { z = slab[perm[e]]; });
  }
  template <class Ctx>
  __host__ __device__ __forceinline__ static void scatter(Ctx& ctx, float2 (&v)[P], int t, float2* slab,
                                                          const int* perm) {
    ctx.sync_row();
    for_spatial(v, t, [&](int e, float2& z) { slab[perm[e]] = z; });
    ctx.sync_row();
    for_spatial(v, t, [&](int e, float2& z) { z = slab[e]; });
  }

  template <bool INV, class Ctx>
  __host__ __device__ __forceinline__ static void fft(Ctx& ctx, float2 (&v)[P], int t, float2* slab,
                                                      const float2* tw) {
    stockham_fft<PL, INV, 0, 0>(ctx, v, t, slab, tw);
  }
};

struct CplxArgs {
  const float* x;
  float* y;
  const float* A;
  const float* D;
  const int* perm;
  float* saved;
  const float* gy;
  float* gx;
  float* partial;  // [tiles][K][4N]: dA (2N floats) then dD (2N floats)
  const char* tab;
  long long batch;
  int K;
  unsigned flags;
};

template <class PL, class Ctx>
__host__ __device__ void cplx_forward_row(Ctx& ctx, const CplxArgs& a, int t, long long row, float* slab) {
  using O = CplxOps<PL>;
  constexpr int N = PL::N, P = PL::P;
  constexpr long long RS = 2LL * N;  // floats per row
  const bool valid = row < a.batch;
  const float2* tw = reinterpret_cast<const float2*>(a.tab);
  float2* slab2 = reinterpret_cast<float2*>(slab);
  const float invN = 1.0f / float(N);
  float2 v[P];
  O::load(a.x + row * RS, v, t, valid);
  for (int k = 0; k < a.K; ++k) {
    if (a.flags & 1u) O::gather(ctx, v, t, slab2, a.perm + (long long)k * N);
    if (a.saved != nullptr && k > 0 && valid) O::store(a.saved + ((long long)(k - 1) * a.batch + row) * RS, v, t);
    O::template scale<false>(v, a.A + k * RS, t);
    O::template fft<false>(ctx, v, t, slab2, tw);
    O::template scale_freq<false>(v, a.D + k * RS, invN, t);
    O::template fft<true>(ctx, v, t, slab2, tw);
  }
  if (a.y != nullptr && valid) O::store(a.y + row * RS, v, t);
}

template <class PL, int ROWS, class Ctx>
__host__ __device__ void cplx_backward_row(Ctx& ctx, const CplxArgs& a, int t, long long row, int tid,
                                           long long tile, float* lds, float* slab) {
  using O = CplxOps<PL>;
  constexpr int N = PL::N, P = PL::P, T = PL::T;
  constexpr int THREADS = ROWS * T;
  constexpr long long RS = 2LL * N;
  constexpr long long PS = 4LL * N;
  const bool valid = row < a.batch;
  const float2* tw = reinterpret_cast<const float2*>(a.tab);
  float2* slab2 = reinterpret_cast<float2*>(slab);
  const float invN = 1.0f / float(N);
  float2 g[P];
  O::load(a.gy + row * RS, g, t, valid);
  for (int k = a.K - 1; k >= 0; --k) {
    const float* urow = (k == 0) ? a.x + row * RS : a.saved + ((long long)(k - 1) * a.batch + row) * RS;
    float* part = a.partial + (tile * a.K + k) * PS;
    float2 h[P];
    O::load(urow, h, t, valid);
    O::template scale<false>(h, a.A + k * RS, t);
    O::template fft<false>(ctx, h, t, slab2, tw);          // h2
    O::template fft<false>(ctx, g, t, slab2, tw);
#pragma unroll
    for (int s = 0; s < P; ++s) g[s] = make_float2(g[s].x * invN, g[s].y * invN);  // gh3
    ctx.sync_row();
#pragma unroll
    for (int s = 0; s < P; ++s) h[s] = cmulc(g[s], h[s]);   // conj(h2) * gh3 in frequency layout
    O::for_freq(h, t, [&](int e, float2& z) { slab2[e] = z; });
    ctx.sync_all();
    sum_rows<ROWS, PL::SLAB, THREADS>(lds, part + RS, int(RS), tid);
    ctx.sync_all();
    O::template scale_freq<true>(g, a.D + k * RS, 1.0f, t);  // gh3 * conj(d)
    O::template fft<true>(ctx, g, t, slab2, tw);             // gh1 (unnormalised inverse)
    float2 u[P];
    O::load(urow, u, t, valid);
    ctx.sync_row();
    O::for_spatial2(u, g, t, [&](int e, float2& uu, float2& gg) { slab2[e] = cmulc(gg, uu); });
    ctx.sync_all();
    sum_rows<ROWS, PL::SLAB, THREADS>(lds, part, int(RS), tid);
    ctx.sync_all();
    O::template scale<true>(g, a.A + k * RS, t);            // gu = gh1 * conj(a)
    if (a.flags & 1u) O::scatter(ctx, g, t, slab2, a.perm + (long long)k * N);
  }
  if (valid) O::store(a.gx + row * RS, g, t);
}

}  // namespace acdc
