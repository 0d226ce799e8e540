// Complex AFDF cascade (Sec. 3: y = x A F D F^{-1} per layer, complex
// diagonals, F the unnormalised DFT with F^{-1} = conj(F)/N).
//
// A row of N complex values lives in the registers of T threads, P = N/T
// each.  Spatial layout: v[beta*R0 + i] is element t + T*(beta + i*B0);
// frequency layout: v[beta*RL + m] is element t + T*(beta + m*BL) -- or,
// with adjacent butterfly pairs (CplxOps::PAIRS), 2t + (beta&1) +
// 2T*(beta>>1) + i*T*B0 (resp. m*T*BL), so that each access moves two
// neighbouring elements.  The forward FFT maps the spatial layout to the
// frequency one and the inverse FFT (radices reversed) maps back, so D
// multiplies in place and nothing is reordered.
//
// Backward (PyTorch convention, grad = dL/dRe + i dL/dIm, so g_x = g_y W^H):
//   gh3 = FFT(g)/N, dd = sum conj(h2) gh3, gh1 = IFFT_unnorm(gh3 conj(d)),
//   da = sum conj(u) gh1, gu = gh1 conj(a).
#pragma once

#include "acdc_dft.hpp"
#include "acdc_mem.hpp"
#include "acdc_plans.hpp"
#include "acdc_stockham.hpp"

namespace acdc {

template <class PL>
struct CplxOps {
  static constexpr int N = PL::N, T = PL::T, P = PL::P;
  static constexpr int R0 = PL::rad(0), RL = PL::rad(PL::NPASS - 1);
  static constexpr int B0 = P / R0, BL = P / RL;
  // Butterfly ownership of the first and last pass (acdc_stockham.hpp): the
  // adjacent pairs (2p, 2p+1), p = t + T*(beta/2), when both passes give a
  // thread an even number of butterflies, else plain (t + T*beta).
  static constexpr bool PAIRS = ACDC_CPLX_PAIRS && B0 % 2 == 0 && BL % 2 == 0;
  static constexpr int KIND = PAIRS ? 3 : 0;

  // Element of v[beta*R0 + i] (spatial) or v[beta*RL + m] (frequency), as a
  // lane part plus a compile-time part:
  //   plain: t + T*(beta + i*B0)              (resp. t + T*(beta + m*BL))
  //   pairs: 2t + (beta&1) + 2T*(beta>>1) + i*T*B0   (resp. ... + m*T*BL)
  __host__ __device__ static constexpr unsigned lane_part(unsigned t) { return PAIRS ? 2u * t : t; }
  __host__ __device__ static constexpr unsigned cpart(int beta, int i, int B) {
    return PAIRS ? unsigned((beta & 1) + 2 * T * (beta >> 1) + i * T * B) : unsigned(T * (beta + i * B));
  }

  // f(lane_part, const_part, v[s]) with element = lane_part + const_part over
  // the spatial (resp. frequency) layout.
  template <class F>
  __host__ __device__ __forceinline__ static void for_spatial(float2 (&v)[P], unsigned t, F&& f) {
#pragma unroll
    for (int beta = 0; beta < B0; ++beta)
#pragma unroll
      for (int i = 0; i < R0; ++i) f(lane_part(t), cpart(beta, i, B0), v[beta * R0 + i]);
  }
  template <class F>
  __host__ __device__ __forceinline__ static void for_spatial2(float2 (&v)[P], float2 (&w)[P], unsigned t, F&& f) {
#pragma unroll
    for (int beta = 0; beta < B0; ++beta)
#pragma unroll
      for (int i = 0; i < R0; ++i) f(lane_part(t), cpart(beta, i, B0), v[beta * R0 + i], w[beta * R0 + i]);
  }
  template <class F>
  __host__ __device__ __forceinline__ static void for_freq(float2 (&v)[P], unsigned t, F&& f) {
#pragma unroll
    for (int beta = 0; beta < BL; ++beta)
#pragma unroll
      for (int m = 0; m < RL; ++m) f(lane_part(t), cpart(beta, m, BL), v[beta * RL + m]);
  }
  // With PAIRS: f(lane_part, const_part, z0, z1) over the spatial (resp.
  // frequency) layout's neighbouring elements (z1 = element + 1).
  template <class F>
  __host__ __device__ __forceinline__ static void for_spatial_pairs(float2 (&v)[P], unsigned t, F&& f) {
#pragma unroll
    for (int q = 0; q < B0 / 2; ++q)
#pragma unroll
      for (int i = 0; i < R0; ++i) f(lane_part(t), cpart(2 * q, i, B0), v[2 * q * R0 + i], v[(2 * q + 1) * R0 + i]);
  }
  template <class F>
  __host__ __device__ __forceinline__ static void for_freq_pairs(float2 (&v)[P], unsigned t, F&& f) {
#pragma unroll
    for (int q = 0; q < BL / 2; ++q)
#pragma unroll
      for (int m = 0; m < RL; ++m) f(lane_part(t), cpart(2 * q, m, BL), v[2 * q * RL + m], v[(2 * q + 1) * RL + m]);
  }

  // g views the workgroup's first row; roff = this row's offset (complex elements)
  // Rows past the batch end read the block's first row and are zeroed.
  __host__ __device__ __forceinline__ static void load(GView g, unsigned roff, float2 (&v)[P], unsigned t,
                                                       bool valid) {
    const unsigned ro = valid ? roff : 0u;
    const float zf = valid ? 1.0f : 0.0f;
    if constexpr (PAIRS) {
      for_spatial_pairs(v, t, [&](unsigned l, unsigned c, float2& z0, float2& z1) {
        const float4 h = g.ld4((l + ro) * 8u, c * 8u);
        z0 = make_float2(h.x * zf, h.y * zf);
        z1 = make_float2(h.z * zf, h.w * zf);
      });
    } else {
      for_spatial(v, t, [&](unsigned l, unsigned c, float2& z) {
        const float2 h = g.ld2((l + ro) * 8u, c * 8u);
        z = make_float2(h.x * zf, h.y * zf);
      });
    }
  }
  __host__ __device__ __forceinline__ static void store(GView g, unsigned roff, float2 (&v)[P], unsigned t) {
    if constexpr (PAIRS) {
      for_spatial_pairs(v, t, [&](unsigned l, unsigned c, float2& z0, float2& z1) {
        g.st4(z0.x, z0.y, z1.x, z1.y, (l + roff) * 8u, c * 8u);
      });
    } else {
      for_spatial(v, t, [&](unsigned l, unsigned c, float2& z) { g.st2(z, (l + roff) * 8u, c * 8u); });
    }
  }
  template <bool CONJ>
  __host__ __device__ __forceinline__ static void scale(float2 (&v)[P], GView a, unsigned t) {
    if constexpr (PAIRS) {
      for_spatial_pairs(v, t, [&](unsigned l, unsigned c, float2& z0, float2& z1) {
        const float4 w = a.ld4(l * 8u, c * 8u);
        z0 = CONJ ? cmulc(z0, make_float2(w.x, w.y)) : cmul(z0, make_float2(w.x, w.y));
        z1 = CONJ ? cmulc(z1, make_float2(w.z, w.w)) : cmul(z1, make_float2(w.z, w.w));
      });
    } else {
      for_spatial(v, t, [&](unsigned l, unsigned c, float2& z) {
        const float2 w = a.ld2(l * 8u, c * 8u);
        z = CONJ ? cmulc(z, w) : cmul(z, w);
      });
    }
  }
  template <bool CONJ>
  __host__ __device__ __forceinline__ static void scale_freq(float2 (&v)[P], GView d, float f, unsigned t) {
    if constexpr (PAIRS) {
      for_freq_pairs(v, t, [&](unsigned l, unsigned c, float2& z0, float2& z1) {
        const float4 dv = d.ld4(l * 8u, c * 8u);
        const float2 w0 = make_float2(dv.x * f, dv.y * f), w1 = make_float2(dv.z * f, dv.w * f);
        z0 = CONJ ? cmulc(z0, w0) : cmul(z0, w0);
        z1 = CONJ ? cmulc(z1, w1) : cmul(z1, w1);
      });
    } else {
      for_freq(v, t, [&](unsigned l, unsigned c, float2& z) {
        const float2 dv = d.ld2(l * 8u, c * 8u);
        const float2 w = make_float2(dv.x * f, dv.y * f);
        z = CONJ ? cmulc(z, w) : cmul(z, w);
      });
    }
  }

  // A row (segment) in the spatial or frequency layout, without the
  // validity zeroing of load(): offsets as in load().
  template <bool FREQ>
  __host__ __device__ __forceinline__ static void ld_row(GView g, unsigned roff, float2 (&v)[P], unsigned t) {
    if constexpr (PAIRS) {
      auto f = [&](unsigned l, unsigned c, float2& z0, float2& z1) {
        const float4 h = g.ld4((l + roff) * 8u, c * 8u);
        z0 = make_float2(h.x, h.y);
        z1 = make_float2(h.z, h.w);
      };
      if constexpr (FREQ) for_freq_pairs(v, t, f);
      else for_spatial_pairs(v, t, f);
    } else {
      auto f = [&](unsigned l, unsigned c, float2& z) { z = g.ld2((l + roff) * 8u, c * 8u); };
      if constexpr (FREQ) for_freq(v, t, f);
      else for_spatial(v, t, f);
    }
  }
  template <bool FREQ>
  __host__ __device__ __forceinline__ static void st_row(GView g, unsigned roff, float2 (&v)[P], unsigned t) {
    if constexpr (PAIRS) {
      auto f = [&](unsigned l, unsigned c, float2& z0, float2& z1) {
        g.st4(z0.x, z0.y, z1.x, z1.y, (l + roff) * 8u, c * 8u);
      };
      if constexpr (FREQ) for_freq_pairs(v, t, f);
      else for_spatial_pairs(v, t, f);
    } else {
      auto f = [&](unsigned l, unsigned c, float2& z) { g.st2(z, (l + roff) * 8u, c * 8u); };
      if constexpr (FREQ) for_freq(v, t, f);
      else for_spatial(v, t, f);
    }
  }

  // The thread's perm entries (spatial layout), loaded ahead of the gather.
  __host__ __device__ __forceinline__ static void load_idx(int (&idx)[P], GView perm, unsigned t) {
    if constexpr (PAIRS) {
#pragma unroll
      for (int q = 0; q < B0 / 2; ++q)
#pragma unroll
        for (int i = 0; i < R0; ++i) {
          const int2 p2 = perm.ldi2(lane_part(t) * 4u, cpart(2 * q, i, B0) * 4u);
          idx[2 * q * R0 + i] = p2.x;
          idx[(2 * q + 1) * R0 + i] = p2.y;
        }
    } else {
#pragma unroll
      for (int beta = 0; beta < B0; ++beta)
#pragma unroll
        for (int i = 0; i < R0; ++i) idx[beta * R0 + i] = perm.ldi1(t * 4u, cpart(beta, i, B0) * 4u);
    }
  }
  // u[n] = z[perm[n]] with the indices already in registers.
  template <class Ctx, class Hook>
  __host__ __device__ __forceinline__ static void gather_idx(Ctx& ctx, float2 (&v)[P], unsigned t, float2* slab,
                                                             const int (&idx)[P], Hook&& hook) {
    ctx.sync_row();
    for_spatial(v, t, [&](unsigned l, unsigned c, float2& z) { slab[l + c] = z; });
    ctx.sync_row();
    hook();
    ACDC_SCHED_FENCE();
#pragma unroll
    for (int s = 0; s < P; ++s) v[s] = slab[idx[s]];
  }

  template <class Ctx>
  __host__ __device__ __forceinline__ static void gather(Ctx& ctx, float2 (&v)[P], unsigned t, float2* slab,
                                                         GView perm) {
    ctx.sync_row();
    for_spatial(v, t, [&](unsigned l, unsigned c, float2& z) { slab[l + c] = z; });
    ctx.sync_row();
    for_spatial(v, t, [&](unsigned l, unsigned c, float2& z) { z = slab[perm.ldi1(l * 4u, c * 4u)]; });
  }
  template <class Ctx>
  __host__ __device__ __forceinline__ static void scatter(Ctx& ctx, float2 (&v)[P], unsigned t, float2* slab,
                                                          GView perm) {
    int idx[P];
    load_idx(idx, perm, t);
    ctx.sync_row();
#pragma unroll
    for (int s = 0; s < P; ++s) slab[idx[s]] = v[s];
    ctx.sync_row();
    for_spatial(v, t, [&](unsigned l, unsigned c, float2& z) { z = slab[l + c]; });
  }

  template <bool INV, class Ctx>
  __host__ __device__ __forceinline__ static void fft(Ctx& ctx, float2 (&v)[P], unsigned t, float2* slab,
                                                      GView tw) {
    stockham_fft<PL, INV, KIND, KIND>(ctx, v, t, slab, tw);
  }
  // `tail` runs in the last pass right after its twiddle multiplies.
  template <bool INV, class Ctx, class Tail>
  __host__ __device__ __forceinline__ static void fft(Ctx& ctx, float2 (&v)[P], unsigned t, float2* slab,
                                                      GView tw, Tail&& tail) {
    stockham_fft<PL, INV, KIND, KIND>(ctx, v, t, slab, tw, tail);
  }

  // A layer diagonal loaded ahead of its use (pairs layout: each float4 is
  // the two neighbouring elements of one pair), spatial or frequency order.
  static constexpr int NQ = P / 2;
  template <bool FREQ>
  __host__ __device__ __forceinline__ static void ld_diag(float4 (&r)[NQ], GView g, unsigned t) {
    static_assert(PAIRS, "pairs layout");
    int n = 0;
    auto f = [&](unsigned l, unsigned c, float2&, float2&) { r[n++] = g.ld4(l * 8u, c * 8u); };
    float2 dummy[P];
    if constexpr (FREQ) for_freq_pairs(dummy, t, f);
    else for_spatial_pairs(dummy, t, f);
  }
  // v *= diag (spatial) or v *= diag * f (frequency), diag from ld_diag
  template <bool FREQ, bool CONJ>
  __host__ __device__ __forceinline__ static void mul_diag(float2 (&v)[P], const float4 (&r)[NQ], float f, unsigned t) {
    int n = 0;
    auto g = [&](unsigned, unsigned, float2& z0, float2& z1) {
      const float4 w = r[n++];
      const float2 w0 = FREQ ? make_float2(w.x * f, w.y * f) : make_float2(w.x, w.y);
      const float2 w1 = FREQ ? make_float2(w.z * f, w.w * f) : make_float2(w.z, w.w);
      z0 = CONJ ? cmulc(z0, w0) : cmul(z0, w0);
      z1 = CONJ ? cmulc(z1, w1) : cmul(z1, w1);
    };
    if constexpr (FREQ) for_freq_pairs(v, t, g);
    else for_spatial_pairs(v, t, g);
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
__host__ __device__ void cplx_forward_row(Ctx& ctx, const CplxArgs& a, unsigned t, long long row0, unsigned rr,
                                          float* slab) {
  using O = CplxOps<PL>;
  constexpr int N = PL::N, P = PL::P;
  constexpr long long RS = 2LL * N;  // floats per row
  const long long row = row0 + rr;
  const bool valid = row < a.batch;
  const unsigned roff = rr * unsigned(N);
  const GView tab = GView::of(a.tab);
  float2* slab2 = reinterpret_cast<float2*>(slab);
  const float invN = 1.0f / float(N);
  float2 v[P];
  O::load(GView::of(a.x + row0 * RS), roff, v, t, valid);
  // With adjacent pairs on rows of two or more waves, a is loaded during
  // the gather and d in the forward FFT's last pass, one step ahead of their
  // use (smaller rows would lose a wave per SIMD to the 64 extra registers).
  constexpr bool AHEAD = ACDC_CPLX_FWD_PF && O::PAIRS && PL::T >= 128;
  for (int k = 0; k < a.K; ++k) {
    const GView ak = GView::of(a.A + k * RS), dk = GView::of(a.D + k * RS);
    float4 dg[O::NQ];
    auto load_a = [&] {
      if constexpr (AHEAD) O::template ld_diag<false>(dg, ak, t);
    };
    // the perm loads are issued before the gather's barriers
    if (a.flags & 1u) {
      int idx[P];
      O::load_idx(idx, GView::of(a.perm + (long long)k * N), t);
      O::gather_idx(ctx, v, t, slab2, idx, load_a);
    } else {
      load_a();
    }
    // stash u_k: u_1..u_{K-1} in slots 0..K-2, and with PERM u_0 in slot K-1
    if (a.saved != nullptr && (k > 0 || (a.flags & 1u)) && valid)
      O::store(GView::of(a.saved + ((long long)(k > 0 ? k - 1 : a.K - 1) * a.batch + row0) * RS), roff, v, t);
    if constexpr (AHEAD) {
      O::template mul_diag<false, false>(v, dg, 1.0f, t);
      O::template fft<false>(ctx, v, t, slab2, tab, [&] { O::template ld_diag<true>(dg, dk, t); });
      O::template mul_diag<true, false>(v, dg, invN, t);
    } else {
      O::template scale<false>(v, ak, t);
      O::template fft<false>(ctx, v, t, slab2, tab);
      O::template scale_freq<false>(v, dk, invN, t);
    }
    O::template fft<true>(ctx, v, t, slab2, tab);
  }
  if (a.y != nullptr && valid) O::store(GView::of(a.y + row0 * RS), roff, v, t);
}

template <class PL, int ROWS, class Ctx>
__host__ __device__ void cplx_backward_row(Ctx& ctx, const CplxArgs& a, unsigned t, long long row0, unsigned rr,
                                           int tid, long long tile, float* lds, float* slab) {
  using O = CplxOps<PL>;
  constexpr int N = PL::N, P = PL::P, T = PL::T;
  constexpr int THREADS = ROWS * T;
  constexpr long long RS = 2LL * N;
  constexpr long long PS = 4LL * N;
  const long long row = row0 + rr;
  const bool valid = row < a.batch;
  const unsigned roff = rr * unsigned(N);
  const GView tab = GView::of(a.tab);
  float2* slab2 = reinterpret_cast<float2*>(slab);
  const float invN = 1.0f / float(N);
  float2 g[P];
  O::load(GView::of(a.gy + row0 * RS), roff, g, t, valid);
  for (int k = a.K - 1; k >= 0; --k) {
    // u_k: stash slot k - 1; u_0 = x, or with PERM stash slot K - 1
    const long long slot = k > 0 ? k - 1 : a.K - 1;
    const GView ug = GView::of(k == 0 && !(a.flags & 1u) ? a.x + row0 * RS
                                                         : a.saved + (slot * a.batch + row0) * RS);
    const GView ak = GView::of(a.A + k * RS);
    float* part = a.partial + (tile * a.K + k) * PS;
    float2 h[P];
    O::load(ug, roff, h, t, valid);
    O::template scale<false>(h, ak, t);
    O::template fft<false>(ctx, h, t, slab2, tab);          // h2
    O::template fft<false>(ctx, g, t, slab2, tab);
#pragma unroll
    for (int s = 0; s < P; ++s) g[s] = make_float2(g[s].x * invN, g[s].y * invN);  // gh3
    ctx.sync_row();
#pragma unroll
    for (int s = 0; s < P; ++s) h[s] = cmulc(g[s], h[s]);   // conj(h2) * gh3 in frequency layout
    O::for_freq(h, t, [&](unsigned l, unsigned c, float2& z) { slab2[l + c] = z; });
    ctx.sync_all();
    sum_rows<ROWS, PL::SLAB, THREADS, 2 * N>(lds, GView::of(part + RS), tid);
    ctx.sync_all();
    O::template scale_freq<true>(g, GView::of(a.D + k * RS), 1.0f, t);  // gh3 * conj(d)
    O::template fft<true>(ctx, g, t, slab2, tab);                        // gh1 (unnormalised inverse)
    float2 u[P];
    O::load(ug, roff, u, t, valid);
    ctx.sync_row();
    O::for_spatial2(u, g, t, [&](unsigned l, unsigned c, float2& uu, float2& gg) { slab2[l + c] = cmulc(gg, uu); });
    ctx.sync_all();
    sum_rows<ROWS, PL::SLAB, THREADS, 2 * N>(lds, GView::of(part), tid);
    ctx.sync_all();
    O::template scale<true>(g, ak, t);            // gu = gh1 * conj(a)
    if (a.flags & 1u) O::scatter(ctx, g, t, slab2, GView::of(a.perm + (long long)k * N));
  }
  if (valid) O::store(GView::of(a.gx + row0 * RS), roff, g, t);
}

}  // namespace acdc
