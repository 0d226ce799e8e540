// Real ACDC cascade: per-thread building blocks and the forward / backward
// row bodies (Sec. 4 layer y = x A C D C^{-1}; Sec. 6.2 permutations + ReLU).
//
// A row of N reals lives in the registers of T threads as M = N/2 complex
// values (Makhoul's even/odd-reversed packing, so that the length-N DCT-II is
// an M-point complex FFT plus a pre/post twiddle).  Storage order in a thread:
//
//   spatial layout  v[2q*R0 + i], v[(2q+1)*R0 + i]   -- the inputs of the two
//                   mirrored first-pass butterflies p and T*B0-1-p,
//                   p = t + T*q.  Element m = j + i*(M/R0) of butterfly j is
//                   the complex value (h[4m], h[4m+2]) for m < M/2 and
//                   (h[4m'+3], h[4m'+1]), m' = M-1-m, otherwise; so a thread
//                   owns whole float4 chunks h[4c..4c+3] of the row.
//   frequency layout v[2q*RL + i], v[(2q+1)*RL + i]  -- the outputs of the
//                   two negated last-pass butterflies (p, NB-p), p = t+T*q
//                   ((0, NB/2) for p = 0).  Spectrum value Z[k] and its
//                   Makhoul partner Z[M-k] therefore sit in one thread.
//
// The inverse FFT runs the radices in reverse, so it reads the frequency
// layout and writes the spatial layout: a layer never moves data between
// threads except inside the FFT passes (and for the permutation).
//
// All functions are __host__ __device__ templates over a context type that
// supplies the LDS synchronisation, so the same code also runs as a CPU
// emulation (threads + barriers) in the tests.
#pragma once

#include "acdc_dft.hpp"
#include "acdc_mem.hpp"
#include "acdc_plans.hpp"
#include "acdc_stockham.hpp"

namespace acdc {

enum : unsigned { kFlagPerm = 1u, kFlagRelu = 2u, kFlagComplex = 4u };

__host__ __device__ __forceinline__ float2 sel2(bool c, float2 a, float2 b) {
  return make_float2(c ? a.x : b.x, c ? a.y : b.y);
}

template <class PL>
struct RealOps {
  static constexpr int N = PL::N, M = PL::M, T = PL::T, P = PL::P;
  static constexpr int R0 = PL::R0, RL = PL::RL, B0 = PL::B0, BL = PL::BL, NB = PL::NB;
  static constexpr int NSL = PL::NSL;

  // ---------------------------------------------------------------- chunks
  // Thread t owns the float4 chunks h[4c..4c+3] with
  //   side a: c = t + (T*q + i*T*B0)
  //   side b: c = (CB - t) + (T*(B0/2-1) - T*q + i*T*B0),  CB = T*B0 - 1 - T*(B0/2-1)
  // for q < B0/2, i < R0/2: a per-thread part plus a compile-time part.
  static constexpr unsigned CB = T * B0 - 1 - T * (B0 / 2 - 1);
  struct Lane {
    unsigned a, b;
  };
  __host__ __device__ __forceinline__ static Lane lane(unsigned t) { return Lane{t, CB - t}; }

  // Visit the chunks of a thread: f(lane_chunk, const_chunk, lo, hi) with
  // lo = (h0, h2), hi = (h3, h1) references into the spatial layout.
  template <class F>
  __host__ __device__ __forceinline__ static void for_chunks(float2 (&v)[P], Lane L, F&& f) {
#pragma unroll
    for (int q = 0; q < B0 / 2; ++q) {
#pragma unroll
      for (int i = 0; i < R0 / 2; ++i) {
        f(L.a, unsigned(T * q + i * T * B0), v[2 * q * R0 + i], v[(2 * q + 1) * R0 + R0 - 1 - i]);
        f(L.b, unsigned(T * (B0 / 2 - 1) - T * q + i * T * B0), v[(2 * q + 1) * R0 + i],
          v[2 * q * R0 + R0 - 1 - i]);
      }
    }
  }
  template <class F>
  __host__ __device__ __forceinline__ static void for_chunks2(float2 (&v)[P], float2 (&w)[P], Lane L, F&& f) {
#pragma unroll
    for (int q = 0; q < B0 / 2; ++q) {
#pragma unroll
      for (int i = 0; i < R0 / 2; ++i) {
        f(L.a, unsigned(T * q + i * T * B0), v[2 * q * R0 + i], v[(2 * q + 1) * R0 + R0 - 1 - i],
          w[2 * q * R0 + i], w[(2 * q + 1) * R0 + R0 - 1 - i]);
        f(L.b, unsigned(T * (B0 / 2 - 1) - T * q + i * T * B0), v[(2 * q + 1) * R0 + i],
          v[2 * q * R0 + R0 - 1 - i], w[(2 * q + 1) * R0 + i], w[2 * q * R0 + R0 - 1 - i]);
      }
    }
  }

  // Row loads/stores: g views the workgroup's first row, roff = this row's
  // offset from it in float4 chunks.
  // Rows past the batch end (valid == false) read the block's first row,
  // which always exists, and are zeroed: no branches around the loads.
  __host__ __device__ __forceinline__ static void load(GView g, unsigned roff, float2 (&v)[P], Lane L,
                                                       bool valid) {
    const unsigned ro = valid ? roff : 0u;
    const float z = valid ? 1.0f : 0.0f;
    for_chunks(v, L, [&](unsigned lc, unsigned cc, float2& lo, float2& hi) {
      const float4 h = g.ld4((lc + ro) * 16u, cc * 16u);
      lo = make_float2(h.x * z, h.z * z);
      hi = make_float2(h.w * z, h.y * z);
    });
  }
  __host__ __device__ __forceinline__ static void store(GView g, unsigned roff, float2 (&v)[P], Lane L) {
    for_chunks(v, L, [&](unsigned lc, unsigned cc, float2& lo, float2& hi) {
      g.st4(make_float4(lo.x, hi.y, lo.y, hi.x), (lc + roff) * 16u, cc * 16u);
    });
  }
  // v *= a (spatial diagonal of one layer)
  __host__ __device__ __forceinline__ static void scale(float2 (&v)[P], GView a, Lane L) {
    for_chunks(v, L, [&](unsigned lc, unsigned cc, float2& lo, float2& hi) {
      const float4 s = a.ld4(lc * 16u, cc * 16u);
      lo = make_float2(lo.x * s.x, lo.y * s.z);
      hi = make_float2(hi.x * s.w, hi.y * s.y);
    });
  }
  __host__ __device__ __forceinline__ static void relu(float2 (&v)[P]) {
#pragma unroll
    for (int s = 0; s < P; ++s) v[s] = make_float2(v[s].x > 0.f ? v[s].x : 0.f, v[s].y > 0.f ? v[s].y : 0.f);
  }

  // u[n] = z[perm[n]]: write z to LDS in natural order, read it back gathered.
  template <class Ctx>
  __host__ __device__ __forceinline__ static void gather(Ctx& ctx, float2 (&v)[P], Lane L, float* slab,
                                                         GView perm) {
    ctx.sync_row();
    for_chunks(v, L, [&](unsigned lc, unsigned cc, float2& lo, float2& hi) {
      reinterpret_cast<float4*>(slab)[lc + cc] = make_float4(lo.x, hi.y, lo.y, hi.x);
    });
    ctx.sync_row();
    for_chunks(v, L, [&](unsigned lc, unsigned cc, float2& lo, float2& hi) {
      const int4 pi = perm.ldi4(lc * 16u, cc * 16u);
      lo = make_float2(slab[pi.x], slab[pi.z]);
      hi = make_float2(slab[pi.w], slab[pi.y]);
    });
  }
  // g_z[perm[n]] = g_u[n]: the adjoint of gather.
  template <class Ctx>
  __host__ __device__ __forceinline__ static void scatter(Ctx& ctx, float2 (&v)[P], Lane L, float* slab,
                                                          GView perm) {
    ctx.sync_row();
    for_chunks(v, L, [&](unsigned lc, unsigned cc, float2& lo, float2& hi) {
      const int4 pi = perm.ldi4(lc * 16u, cc * 16u);
      slab[pi.x] = lo.x;
      slab[pi.y] = hi.y;
      slab[pi.z] = lo.y;
      slab[pi.w] = hi.x;
    });
    ctx.sync_row();
    for_chunks(v, L, [&](unsigned lc, unsigned cc, float2& lo, float2& hi) {
      const float4 h = reinterpret_cast<const float4*>(slab)[lc + cc];
      lo = make_float2(h.x, h.z);
      hi = make_float2(h.w, h.y);
    });
  }

  // ------------------------------------------------------------ FFT passes
  // Forward: mirrored first pass (chunk-local input), negated last pass
  // (Makhoul partners together); the inverse runs the mirror image.
  template <bool INV, class Ctx>
  __host__ __device__ __forceinline__ static void fft(Ctx& ctx, float2 (&v)[P], unsigned t, float2* slab,
                                                      GView tw) {
    if constexpr (INV) stockham_fft<PL, true, 2, 1>(ctx, v, t, slab, tw);
    else stockham_fft<PL, false, 1, 2>(ctx, v, t, slab, tw);
  }

  // ------------------------------------------------------ Makhoul quartets
  // One quartet: from Z[k], Z[M-k] produce the DCT-II outputs
  // X[k], X[N-k], X[M-k], X[M+k] (orthonormal scaling folded into qa, qb).
  __host__ __device__ __forceinline__ static void post_one(float2 zk, float2 zm, float4 m0, float4 m1,
                                                           float (&X)[4]) {
    const float2 w = make_float2(m0.x, m0.y), qa = make_float2(m0.z, m0.w);
    const float2 qb = make_float2(m1.x, m1.y);
    const float2 E = make_float2(zk.x + zm.x, zk.y - zm.y);  // Z[k] + conj Z[M-k]
    const float2 Od = make_float2(zk.y + zm.y, zm.x - zk.x); // (Z[k] - conj Z[M-k]) / i
    const float2 wO = cmul(Od, w);
    const float2 u1 = cmul(cadd(E, wO), qa);
    const float2 u2 = cmul(csub(E, wO), qb);
    X[0] = u1.x;
    X[1] = -u1.y;
    X[2] = u2.x - u2.y;
    X[3] = u2.x + u2.y;
  }
  // Inverse of post_one for the DCT-III (with the 1/M of the inverse FFT
  // folded into qap and conj(qb)).
  __host__ __device__ __forceinline__ static void pre_one(const float (&Y)[4], float4 m0, float4 m1,
                                                          float2& zk, float2& zm) {
    const float2 w = make_float2(m0.x, m0.y);
    const float2 qb = make_float2(m1.x, m1.y), qap = make_float2(m1.z, m1.w);
    const float2 Ap = cmul(make_float2(Y[0], -Y[1]), qap);
    const float2 Bp = cmulc(make_float2(Y[2] + Y[3], Y[3] - Y[2]), qb);
    const float2 S = cadd(Ap, Bp), Dd = csub(Ap, Bp);
    const float2 cw = cmulc(Dd, w);                 // conj(w) * Dd
    const float2 tt = make_float2(-cw.y, cw.x);     // i * conj(w) * Dd
    zk = cadd(S, tt);
    zm = make_float2(S.x - tt.x, tt.y - S.y);       // conj(S - tt)
  }

  // Makhoul twiddles of quartet slot `slot` for thread t (t16 = 16*t).
  __host__ __device__ __forceinline__ static float4 mk0(GView tab, unsigned t16, int slot) {
    return tab.ld4(t16, unsigned(PL::OFF_MK0 + slot * T * 16));
  }
  __host__ __device__ __forceinline__ static float4 mk1(GView tab, unsigned t16, int slot) {
    return tab.ld4(t16, unsigned(PL::OFF_MK1 + slot * T * 16));
  }

  __host__ __device__ __forceinline__ static void post(float2 (&v)[P], float (&X)[NSL][4], unsigned t,
                                                       GView tab) {
    const unsigned t16 = t * 16u;
    const bool sp = (t == 0);
#pragma unroll
    for (int q = 0; q < BL / 2; ++q) {
#pragma unroll
      for (int i = 0; i < RL; ++i) {
        const int slot = q * RL + i;
        float2 zk = v[2 * q * RL + i];
        float2 zm = v[(2 * q + 1) * RL + RL - 1 - i];
        if (q == 0) {
          if (i < RL / 2) {
            zm = sel2(sp, v[(RL - i) % RL], zm);
          } else {
            zk = sel2(sp, v[RL + i - RL / 2], zk);
            zm = sel2(sp, v[RL + 3 * RL / 2 - 1 - i], zm);
          }
        }
        post_one(zk, zm, mk0(tab, t16, slot), mk1(tab, t16, slot), X[slot]);
      }
    }
    post_one(v[RL / 2], v[RL / 2], mk0(tab, t16, NSL - 1), mk1(tab, t16, NSL - 1), X[NSL - 1]);
  }

  __host__ __device__ __forceinline__ static void pre(float (&X)[NSL][4], float2 (&v)[P], unsigned t,
                                                      GView tab) {
    const unsigned t16 = t * 16u;
    const bool sp = (t == 0);
    float2 ok[NSL], om[NSL];
#pragma unroll
    for (int s = 0; s < NSL; ++s) pre_one(X[s], mk0(tab, t16, s), mk1(tab, t16, s), ok[s], om[s]);
    place(ok, om, v, sp);
  }

  // Forward middle of a layer, fused per quartet slot so that no full DCT
  // image is held: Z (frequency layout) -> DCT-II quartet -> * d -> DCT-III
  // pre-twiddle -> Z' (frequency layout), written back into v.
  __host__ __device__ __forceinline__ static void mid(float2 (&v)[P], unsigned t, GView tab, GView dq) {
    const unsigned t16 = t * 16u;
    const bool sp = (t == 0);
    float2 ok[NSL], om[NSL];
#pragma unroll
    for (int q = 0; q < BL / 2; ++q) {
#pragma unroll
      for (int i = 0; i < RL; ++i) {
        const int slot = q * RL + i;
        float2 zk = v[2 * q * RL + i];
        float2 zm = v[(2 * q + 1) * RL + RL - 1 - i];
        if (q == 0) {
          if (i < RL / 2) {
            zm = sel2(sp, v[(RL - i) % RL], zm);
          } else {
            zk = sel2(sp, v[RL + i - RL / 2], zk);
            zm = sel2(sp, v[RL + 3 * RL / 2 - 1 - i], zm);
          }
        }
        const float4 m0 = mk0(tab, t16, slot), m1 = mk1(tab, t16, slot), d = dq.ld4(t16, unsigned(slot * T * 16));
        float X[4];
        post_one(zk, zm, m0, m1, X);
        X[0] *= d.x;
        X[1] *= d.y;
        X[2] *= d.z;
        X[3] *= d.w;
        pre_one(X, m0, m1, ok[slot], om[slot]);
      }
    }
    {
      const int slot = NSL - 1;
      const float4 m0 = mk0(tab, t16, slot), m1 = mk1(tab, t16, slot), d = dq.ld4(t16, unsigned(slot * T * 16));
      float X[4];
      post_one(v[RL / 2], v[RL / 2], m0, m1, X);
      X[0] *= d.x;
      X[1] *= d.y;
      X[2] *= d.z;
      X[3] *= d.w;
      pre_one(X, m0, m1, ok[slot], om[slot]);
    }
    place(ok, om, v, sp);
  }

  // Write the pre-twiddled pairs back to the frequency layout (thread 0's
  // first pair uses the special quartet order, see post()).
  __host__ __device__ __forceinline__ static void place(float2 (&ok)[NSL], float2 (&om)[NSL], float2 (&v)[P],
                                                        bool sp) {
#pragma unroll
    for (int q = 1; q < BL / 2; ++q) {
#pragma unroll
      for (int i = 0; i < RL; ++i) {
        v[2 * q * RL + i] = ok[q * RL + i];
        v[(2 * q + 1) * RL + RL - 1 - i] = om[q * RL + i];
      }
    }
#pragma unroll
    for (int rho = 0; rho < 2 * RL; ++rho) {
      const float2 gen = rho < RL ? ok[rho] : om[2 * RL - 1 - rho];
      float2 spc;
      if (rho < RL) {
        const int e = rho;
        spc = e < RL / 2 ? ok[e] : (e == RL / 2 ? ok[NSL - 1] : om[RL - e]);
      } else {
        const int e = rho - RL;
        spc = e < RL / 2 ? ok[e + RL / 2] : om[3 * RL / 2 - 1 - e];
      }
      v[rho] = sel2(sp, spc, gen);
    }
  }

  // X *= d in quartet layout (dq already holds d at the four indices, with
  // zeros where an index does not exist).
  __host__ __device__ __forceinline__ static void scale_q(float (&X)[NSL][4], GView dq, unsigned t) {
#pragma unroll
    for (int s = 0; s < NSL; ++s) {
      const float4 d = dq.ld4(t * 16u, unsigned(s * T * 16));
      X[s][0] *= d.x;
      X[s][1] *= d.y;
      X[s][2] *= d.z;
      X[s][3] *= d.w;
    }
  }
};

// ----------------------------------------------------------------- bodies
// Shared argument block of the row bodies (all pointers device pointers on
// the GPU, host pointers in the CPU emulation).
struct RealArgs {
  const float* x;
  float* y;            // forward output (may be null: stash-only forward)
  const float* A;
  const float4* Dq;    // [K][NSL*T] d in quartet layout
  const int* perm;     // [K][N] (PERM only)
  float* saved;        // [K-1][batch][N] layer inputs u_1..u_{K-1} (may be null)
  const float* gy;     // backward: upstream gradient
  float* gx;           // backward: input gradient
  float* partial;      // backward: [tiles][K][N + QF] per-tile sums
  const char* tab;     // plan tables
  long long batch;
  int K;
  unsigned flags;
};

template <class PL, class Ctx>
__host__ __device__ void real_forward_row(Ctx& ctx, const RealArgs& a, unsigned t, long long row0, unsigned rr,
                                          float* slab) {
  using O = RealOps<PL>;
  constexpr int N = PL::N, P = PL::P, NSL = PL::NSL, T = PL::T;
  const long long row = row0 + rr;
  const bool valid = row < a.batch;
  const unsigned roff = rr * unsigned(N / 4);
  const GView tab = GView::of(a.tab);
  const typename O::Lane L = O::lane(t);
  float2* slab2 = reinterpret_cast<float2*>(slab);
  float2 v[P];
  O::load(GView::of(a.x + row0 * N), roff, v, L, valid);
  for (int k = 0; k < a.K; ++k) {
    if (a.flags & kFlagPerm) O::gather(ctx, v, L, slab, GView::of(a.perm + (long long)k * N));
    if (a.saved != nullptr && k > 0 && valid)
      O::store(GView::of(a.saved + ((long long)(k - 1) * a.batch + row0) * N), roff, v, L);
    O::scale(v, GView::of(a.A + (long long)k * N), L);
    O::template fft<false>(ctx, v, t, slab2, tab);
    O::mid(v, t, tab, GView::of(a.Dq + (long long)k * NSL * T));
    O::template fft<true>(ctx, v, t, slab2, tab);
    if ((a.flags & kFlagRelu) && k < a.K - 1) O::relu(v);
  }
  if (a.y != nullptr && valid) O::store(GView::of(a.y + row0 * N), roff, v, L);
}

template <class PL, int ROWS, class Ctx>
__host__ __device__ void real_backward_row(Ctx& ctx, const RealArgs& a, unsigned t, long long row0, unsigned rr,
                                           int tid, long long tile, float* lds, float* slab) {
  using O = RealOps<PL>;
  constexpr int N = PL::N, P = PL::P, NSL = PL::NSL, T = PL::T, QF = PL::QF;
  constexpr int THREADS = ROWS * T;
  constexpr long long PS = N + QF;
  const long long row = row0 + rr;
  const bool valid = row < a.batch;
  const unsigned roff = rr * unsigned(N / 4);
  const GView tab = GView::of(a.tab);
  const typename O::Lane L = O::lane(t);
  float2* slab2 = reinterpret_cast<float2*>(slab);
  float2 g[P];
  O::load(GView::of(a.gy + row0 * N), roff, g, L, valid);
  for (int k = a.K - 1; k >= 0; --k) {
    const GView ug = GView::of(k == 0 ? a.x + row0 * N : a.saved + ((long long)(k - 1) * a.batch + row0) * N);
    const GView ak = GView::of(a.A + (long long)k * N);
    const GView dq = GView::of(a.Dq + (long long)k * NSL * T);
    float* part = a.partial + (tile * a.K + k) * PS;
    // h2 = DCT(u * a) (recomputed from the stored layer input)
    float H[NSL][4];
    {
      float2 v[P];
      O::load(ug, roff, v, L, valid);
      O::scale(v, ak, L);
      O::template fft<false>(ctx, v, t, slab2, tab);
      O::post(v, H, t, tab);
    }
    // gh3 = DCT(g)
    float G[NSL][4];
    O::template fft<false>(ctx, g, t, slab2, tab);
    O::post(g, G, t, tab);
    // dL/dd partial: sum over the workgroup's rows of h2 * gh3 (quartet layout)
    ctx.sync_row();
#pragma unroll
    for (int s = 0; s < NSL; ++s)
      reinterpret_cast<float4*>(slab)[s * T + t] =
          make_float4(H[s][0] * G[s][0], H[s][1] * G[s][1], H[s][2] * G[s][2], H[s][3] * G[s][3]);
    ctx.sync_all();
    sum_rows<ROWS, PL::SLAB, THREADS>(lds, GView::of(part + N), QF, tid);
    ctx.sync_all();
    // gh1 = DCT-III(gh3 * d)
    O::scale_q(G, dq, t);
    O::pre(G, g, t, tab);
    O::template fft<true>(ctx, g, t, slab2, tab);
    // dL/da partial: sum of u * gh1 (spatial, natural order)
    float2 u[P];
    O::load(ug, roff, u, L, valid);
    ctx.sync_row();
    O::for_chunks2(u, g, L, [&](unsigned lc, unsigned cc, float2& ulo, float2& uhi, float2& glo, float2& ghi) {
      reinterpret_cast<float4*>(slab)[lc + cc] =
          make_float4(ulo.x * glo.x, uhi.y * ghi.y, ulo.y * glo.y, uhi.x * ghi.x);
    });
    ctx.sync_all();
    sum_rows<ROWS, PL::SLAB, THREADS>(lds, GView::of(part), N, tid);
    ctx.sync_all();
    // dL/du = gh1 * a, through the ReLU of the previous layer, then un-permute
    O::scale(g, ak, L);
    if ((a.flags & kFlagRelu) && k > 0) {
      O::for_chunks2(u, g, L, [&](unsigned, unsigned, float2& ulo, float2& uhi, float2& glo, float2& ghi) {
        glo = make_float2(ulo.x > 0.f ? glo.x : 0.f, ulo.y > 0.f ? glo.y : 0.f);
        ghi = make_float2(uhi.x > 0.f ? ghi.x : 0.f, uhi.y > 0.f ? ghi.y : 0.f);
      });
    }
    if (a.flags & kFlagPerm) O::scatter(ctx, g, L, slab, GView::of(a.perm + (long long)k * N));
  }
  if (valid) O::store(GView::of(a.gx + row0 * N), roff, g, L);
}

}  // namespace acdc
