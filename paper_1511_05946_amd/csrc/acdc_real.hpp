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

enum : unsigned {
  kFlagPerm = 1u,
  kFlagRelu = 2u,
  kFlagComplex = 4u,
  kFlagBias = 8u,
  kFlagAccumulate = 16u,
  kFlagMultipass = 32u
};

// Rows of the per-layer quartet-coefficient table (real_mq_entry).
constexpr int kMqRows = 4;

// max(x, 0) as one integer max over the bit pattern: a float with the sign
// bit set is a negative int32, so -0 and every negative value become +0.
// (The float forms, max or compare-and-select, cost a second instruction
// that quiets NaNs first.)  A NaN keeps its sign's side: NaN or +0.
__host__ __device__ __forceinline__ float relu1(float x) {
  const int b = __builtin_bit_cast(int, x);
  return __builtin_bit_cast(float, b > 0 ? b : 0);
}

__host__ __device__ __forceinline__ float2 sel2(bool c, float2 a, float2 b) {
  return make_float2(c ? a.x : b.x, c ? a.y : b.y);
}

// ------------------------------------------------------ Makhoul quartets
// The per-quartet arithmetic shared by the fused row bodies and the
// multi-pass path (which holds the spectrum in HBM between passes).

// Real-FFT split of a Makhoul pair: E = Z[k] + conj Z[M-k],
// O = (Z[k] - conj Z[M-k]) / i, s1 = E + w O, s2 = E - w O.
struct Split {
  float2 s1, s2;
};
__host__ __device__ __forceinline__ Split quartet_split(float2 zk, float2 zm, float2 w) {
  const float2 E = make_float2(zk.x + zm.x, zk.y - zm.y);
  const float2 Od = make_float2(zk.y + zm.y, zm.x - zk.x);
  const float2 wO = cmul(Od, w);
  return Split{cadd(E, wO), csub(E, wO)};
}
// DCT-II outputs of a split, up to the sign of X[N-k]: returns
// (X[k], -X[N-k], X[M-k], X[M+k]), with the orthonormal scaling folded
// into qa and qbr = (1 + i) qb, so u1 = qa s1 = X[k] - i X[N-k] and
// u2 = qbr s2 = X[M-k] + i X[M+k].  The backward only forms products of
// two such images, where the sign cancels.
__host__ __device__ __forceinline__ void quartet_post(const Split& sp, float2 qa, float2 qbr, float (&X)[4]) {
  const float2 u1 = cmul(sp.s1, qa), u2 = cmul(sp.s2, qbr);
  X[0] = u1.x;
  X[1] = u1.y;
  X[2] = u2.x;
  X[3] = u2.y;
}
// From a split, the D diagonal and the DCT-III pre-twiddle as the two
// symmetric 2x2 maps L1 (on s1) and L2 (on s2), then the inverse split:
// S = L1 s1 + L2 s2, Dd = L1 s1 - L2 s2, zk = S + i conj(w) Dd,
// zm = conj(S - i conj(w) Dd).
__host__ __device__ __forceinline__ void quartet_back(const Split& sp, float4 c0, float4 c1, float2& zk,
                                                     float2& zm) {
  const float2 w = make_float2(c1.z, c1.w);
  const float2 s1 = sp.s1, s2 = sp.s2;
  const float2 p1 = make_float2(__builtin_fmaf(c0.y, s1.y, c0.x * s1.x), __builtin_fmaf(c0.z, s1.y, c0.y * s1.x));
  const float2 p2 = make_float2(__builtin_fmaf(c1.x, s2.y, c0.w * s2.x), __builtin_fmaf(c1.y, s2.y, c1.x * s2.x));
  const float2 S = cadd(p1, p2), Dd = csub(p1, p2);
  const float2 cw = cmulc(Dd, w);
  zk = make_float2(S.x - cw.y, S.y + cw.x);
  zm = make_float2(S.x + cw.y, cw.x - S.y);
}

template <class PL>
struct RealOps {
  static constexpr int N = PL::N, M = PL::M, T = PL::T, P = PL::P;
  static constexpr int R0 = PL::R0, RL = PL::RL, B0 = PL::B0, BL = PL::BL, NB = PL::NB;
  static constexpr int NSL = PL::NSL;

  // ---------------------------------------------------------------- chunks
  // Thread t owns NCH float4 chunks h[4c..4c+3] of the row.  Chunk ordinal
  // n = 2*(q*(R0/2) + i) + side, q < B0/2, i < R0/2, is at
  //   side a (n even): c = t + (T*q + i*T*B0)
  //   side b (n odd):  c = (CB - t) + (T*(B0/2-1) - T*q + i*T*B0),  CB = T*B0 - 1 - T*(B0/2-1)
  // a per-thread part plus a compile-time part; its complex values are
  // lo = (h0, h2) and hi = (h3, h1) of the spatial layout.
  static constexpr int NCH = P / 2;
  static_assert(NCH == B0 * (R0 / 2), "chunks cover the thread's registers");
  static constexpr unsigned CB = T * B0 - 1 - T * (B0 / 2 - 1);
  struct Lane {
    unsigned a, b;
  };
  __host__ __device__ __forceinline__ static Lane lane(unsigned t) { return Lane{t, CB - t}; }
  __host__ __device__ static constexpr int ch_q(int n) { return (n >> 1) / (R0 / 2); }
  __host__ __device__ static constexpr int ch_i(int n) { return (n >> 1) % (R0 / 2); }
  __host__ __device__ static constexpr unsigned ch_cc(int n) {
    return (n & 1) ? unsigned(T * (B0 / 2 - 1) - T * ch_q(n) + ch_i(n) * T * B0)
                   : unsigned(T * ch_q(n) + ch_i(n) * T * B0);
  }
  __host__ __device__ static constexpr int ch_lo(int n) {
    return (n & 1) ? (2 * ch_q(n) + 1) * R0 + ch_i(n) : 2 * ch_q(n) * R0 + ch_i(n);
  }
  __host__ __device__ static constexpr int ch_hi(int n) {
    return (n & 1) ? 2 * ch_q(n) * R0 + R0 - 1 - ch_i(n) : (2 * ch_q(n) + 1) * R0 + R0 - 1 - ch_i(n);
  }
  __host__ __device__ __forceinline__ static unsigned ch_lc(Lane L, int n) { return (n & 1) ? L.b : L.a; }

  // f(lane_chunk, const_chunk, lo, hi) for every chunk, in ordinal order.
  template <class F>
  __host__ __device__ __forceinline__ static void for_chunks(float2 (&v)[P], Lane L, F&& f) {
#pragma unroll
    for (int n = 0; n < NCH; ++n) f(ch_lc(L, n), ch_cc(n), v[ch_lo(n)], v[ch_hi(n)]);
  }
  template <class F>
  __host__ __device__ __forceinline__ static void for_chunks2(float2 (&v)[P], float2 (&w)[P], Lane L, F&& f) {
#pragma unroll
    for (int n = 0; n < NCH; ++n) f(ch_lc(L, n), ch_cc(n), v[ch_lo(n)], v[ch_hi(n)], w[ch_lo(n)], w[ch_hi(n)]);
  }

  // Row loads/stores: g views the workgroup's first row, roff = this row's
  // offset from it in float4 chunks.
  // Rows past the batch end (valid == false) read the block's first row,
  // which always exists, and are zeroed: no branches around the loads.
  __host__ __device__ __forceinline__ static void load_raw(float4 (&h)[NCH], GView g, unsigned roff, Lane L,
                                                           bool valid) {
    const unsigned ro = valid ? roff : 0u;
#pragma unroll
    for (int n = 0; n < NCH; ++n) h[n] = g.ld4((ch_lc(L, n) + ro) * 16u, ch_cc(n) * 16u);
  }
  __host__ __device__ __forceinline__ static void unpack(const float4 (&h)[NCH], float2 (&v)[P]) {
    int n = 0;
    for_chunks(v, Lane{0, 0}, [&](unsigned, unsigned, float2& lo, float2& hi) {
      lo = make_float2(h[n].x, h[n].z);
      hi = make_float2(h[n].w, h[n].y);
      ++n;
    });
  }
  __host__ __device__ __forceinline__ static void load(GView g, unsigned roff, float2 (&v)[P], Lane L,
                                                       bool valid) {
    float4 h[NCH];
    load_raw(h, g, roff, L, valid);
    const float z = valid ? 1.0f : 0.0f;
#pragma unroll
    for (int n = 0; n < NCH; ++n) h[n] = make_float4(h[n].x * z, h[n].y * z, h[n].z * z, h[n].w * z);
    unpack(h, v);
  }
  __host__ __device__ __forceinline__ static void store(GView g, unsigned roff, float2 (&v)[P], Lane L) {
    for_chunks(v, L, [&](unsigned lc, unsigned cc, float2& lo, float2& hi) {
      g.st4(make_float4(lo.x, hi.y, lo.y, hi.x), (lc + roff) * 16u, cc * 16u);
    });
  }
  // Per-thread chunks of a row-independent vector (a spatial diagonal).
  __host__ __device__ __forceinline__ static void load_vec(float4 (&s)[NCH], GView g, Lane L) {
#pragma unroll
    for (int n = 0; n < NCH; ++n) s[n] = g.ld4(ch_lc(L, n) * 16u, ch_cc(n) * 16u);
  }
  // Permutation indices.  Where a row's byte offsets fit 16 bits (N <=
  // 16384), k_real_mq repacks perm[k] per thread for the backward: for chunk
  // pair (2j, 2j+1) of lane t one int4 at [j][t] holds the eight slab byte
  // offsets 4 perm[.] of the two chunks, two per int (low half first), so a
  // thread loads NCH/2 int4 instead of NCH, and a 16-bit half feeds the LDS
  // address add directly.  Otherwise (and in the forward, where the packed
  // form measured slower) a thread loads its int4 chunks of perm[k].
  static constexpr bool kPackedPerm = ACDC_PACKED_PERM && N <= 16384 && NCH % 2 == 0;
  static constexpr int NIW = kPackedPerm ? NCH / 2 : NCH;  // int4 words per thread, packed table
  template <bool PK>
  static constexpr int niw() {
    return PK ? NIW : NCH;
  }
  // g: perm[k] (plain) or layer k of the packed table (PK)
  template <bool PK>
  __host__ __device__ __forceinline__ static void load_idx(int4 (&s)[niw<PK>()], GView g, Lane L, unsigned t) {
#pragma unroll
    for (int n = 0; n < niw<PK>(); ++n)
      s[n] = PK ? g.ldi4(t * 16u, unsigned(n * T * 16)) : g.ldi4(ch_lc(L, n) * 16u, ch_cc(n) * 16u);
  }
  // Slab byte offset of index c (0..3: perm of chunk element c) of chunk n.
  template <bool PK>
  __host__ __device__ __forceinline__ static unsigned idx_off(const int4 (&s)[niw<PK>()], int n, int c) {
    if constexpr (PK) {
      const int4 w = s[n >> 1];
      const unsigned u = unsigned((n & 1) ? (c < 2 ? w.z : w.w) : (c < 2 ? w.x : w.y));
      return (c & 1) ? (u >> 16) : (u & 0xffffu);
    } else {
      const int4 w = s[n];
      return 4u * unsigned(c == 0 ? w.x : c == 1 ? w.y : c == 2 ? w.z : w.w);
    }
  }
  // The packed int4 of lane t, chunk pair j, from layer k's perm (host or
  // device).  Indices outside [0, N) become 0.
  __host__ __device__ static int4 pack_perm_entry(const int* pk, int j, unsigned t) {
    const Lane L = lane(t);
    unsigned o[8];
    for (int h = 0; h < 2; ++h) {
      const int n = 2 * j + h;
      const unsigned base = (ch_lc(L, n) + ch_cc(n)) * 4u;
      for (int c = 0; c < 4; ++c) {
        const int p = pk[base + c];
        o[4 * h + c] = (p >= 0 && p < N) ? 4u * unsigned(p) : 0u;
      }
    }
    return make_int4(int(o[0] | (o[1] << 16)), int(o[2] | (o[3] << 16)), int(o[4] | (o[5] << 16)),
                     int(o[6] | (o[7] << 16)));
  }
  // v *= a (spatial diagonal of one layer, chunks from load_vec)
  __host__ __device__ __forceinline__ static void scale(float2 (&v)[P], const float4 (&s)[NCH]) {
    int n = 0;
    for_chunks(v, Lane{0, 0}, [&](unsigned, unsigned, float2& lo, float2& hi) {
      lo = make_float2(lo.x * s[n].x, lo.y * s[n].z);
      hi = make_float2(hi.x * s[n].w, hi.y * s[n].y);
      ++n;
    });
  }
  __host__ __device__ __forceinline__ static void relu(float2 (&v)[P]) {
#pragma unroll
    for (int s = 0; s < P; ++s) v[s] = make_float2(relu1(v[s].x), relu1(v[s].y));
  }

  // u[n] = z[perm[n]]: write z to LDS in natural order, read it back gathered
  // through the thread's index chunks (from load_idx).  `hook` runs between
  // the LDS write and the gathered reads.
  template <bool PK, class Ctx, class Hook>
  __host__ __device__ __forceinline__ static void gather(Ctx& ctx, float2 (&v)[P], Lane L, float* slab,
                                                         const int4 (&idx)[niw<PK>()], Hook&& hook) {
    ctx.sync_row();
    for_chunks(v, L, [&](unsigned lc, unsigned cc, float2& lo, float2& hi) {
      reinterpret_cast<float4*>(slab)[lc + cc] = make_float4(lo.x, hi.y, lo.y, hi.x);
    });
    ctx.sync_row();
    hook();
    ACDC_SCHED_FENCE();
    const char* sb = reinterpret_cast<const char*>(slab);
    auto at = [&](unsigned off) { return *reinterpret_cast<const float*>(sb + off); };
    int n = 0;
    for_chunks(v, L, [&](unsigned, unsigned, float2& lo, float2& hi) {
      lo = make_float2(at(idx_off<PK>(idx, n, 0)), at(idx_off<PK>(idx, n, 2)));
      hi = make_float2(at(idx_off<PK>(idx, n, 3)), at(idx_off<PK>(idx, n, 1)));
      ++n;
    });
  }
  // g_z[perm[n]] = g_u[n]: the adjoint of gather.
  template <bool PK, class Ctx, class Hook>
  __host__ __device__ __forceinline__ static void scatter(Ctx& ctx, float2 (&v)[P], Lane L, float* slab,
                                                          const int4 (&idx)[niw<PK>()], Hook&& hook) {
    ctx.sync_row();
    char* sb = reinterpret_cast<char*>(slab);
    auto at = [&](unsigned off) -> float& { return *reinterpret_cast<float*>(sb + off); };
    int n = 0;
    for_chunks(v, L, [&](unsigned, unsigned, float2& lo, float2& hi) {
      at(idx_off<PK>(idx, n, 0)) = lo.x;
      at(idx_off<PK>(idx, n, 1)) = hi.y;
      at(idx_off<PK>(idx, n, 2)) = lo.y;
      at(idx_off<PK>(idx, n, 3)) = hi.x;
      ++n;
    });
    ctx.sync_row();
    hook();
    ACDC_SCHED_FENCE();
    for_chunks(v, L, [&](unsigned lc, unsigned cc, float2& lo, float2& hi) {
      const float4 h = reinterpret_cast<const float4*>(slab)[lc + cc];
      lo = make_float2(h.x, h.z);
      hi = make_float2(h.w, h.y);
    });
  }

  // ------------------------------------------------------------ FFT passes
  // Forward: mirrored first pass (chunk-local input), negated last pass
  // (Makhoul partners together); the inverse runs the mirror image.
  template <bool INV, class Ctx, class TW, class Tail>
  __host__ __device__ __forceinline__ static void fft(Ctx& ctx, float2 (&v)[P], unsigned t, float2* slab,
                                                      TW tw, Tail&& tail) {
    if constexpr (INV) stockham_fft<PL, true, 2, 1>(ctx, v, t, slab, tw, tail);
    else stockham_fft<PL, false, 1, 2>(ctx, v, t, slab, tw, tail);
  }

  // Forward FFTs of two rows' arrays sharing twiddle loads (backward h- and
  // g-paths).
  template <class Ctx, class Tail>
  __host__ __device__ __forceinline__ static void fft2(Ctx& ctx, float2 (&v)[P], float2 (&w)[P], unsigned t,
                                                       float2* slab, GView tw, Tail&& tail) {
    stockham_fft2<PL, false, 1, 2>(ctx, v, w, t, slab, tw, tail);
  }

  // ------------------------------------------------------ Makhoul quartets
  // A quartet slot holds a spectrum pair Z[k], Z[M-k] of the packed row.
  // The DCT-II outputs of the quartet are (Makhoul's quarter-wave
  // post-twiddle, with the real-FFT split s1, s2 of `split` below)
  //   u1 = qa s1:  X[k] = Re u1,  X[N-k] = -Im u1
  //   u2 = qb s2:  X[M-k] = Re u2 - Im u2,  X[M+k] = Re u2 + Im u2
  // with qa, qb = W_4N^k times the orthonormal scales.  The DCT-III
  // pre-twiddle is the inverse map, with the 1/M of the inverse FFT folded
  // into its twiddles: Ap = (Y0 - i Y1) qap, Bp = (Y2 + Y3 + i (Y3 - Y2))
  // conj(qb'), S = Ap + Bp, Dd = Ap - Bp, Z'[k] = S + i conj(w) Dd,
  // Z'[M-k] = conj(S - i conj(w) Dd).  real_mq_entry folds post-twiddle, D
  // and pre-twiddle into the two symmetric 2x2 maps that sym_back applies.

  // Thread 0's first butterfly pair is (0, NB/2): both are self-negating,
  // so their Makhoul partners are not at the generic register positions.
  // With A = v[0..RL) the outputs of butterfly 0 (Z[j NB]) and B = v[RL..2RL)
  // those of butterfly NB/2 (Z[NB/2 + j NB]), partners are A_j, A_RL-j and
  // B_j, B_RL-1-j.  The permutation new[rho] = old[pi(rho)] below moves only
  // the blocks v[RL/2..RL) and v[3RL/2..2RL): slot i < RL/2 then pairs A_i
  // with A_RL-i (slot 0: the self-paired Z[0], Z[M/2], with their own table
  // entries) and slot i >= RL/2 pairs B_i with B_RL-1-i.
  __host__ __device__ static constexpr int perm_pi(int rho) {
    return rho < RL / 2       ? rho
           : rho < RL         ? RL + rho
           : rho < 3 * RL / 2 ? rho
           : rho < 2 * RL - 1 ? rho - RL + 1
                              : RL / 2;
  }
  __host__ __device__ static constexpr int perm_pi_inv(int o) {
    int r = 0;
    for (int rho = 0; rho < 2 * RL; ++rho)
      if (perm_pi(rho) == o) r = rho;
    return r;
  }
  // Every lane selects per moved register (thread 0 takes the permuted
  // value): one select per moved float.
  __host__ __device__ static constexpr bool moved(int rho) { return (rho % RL) >= RL / 2; }
  template <bool INV>
  __host__ __device__ __forceinline__ static void perm0(float2 (&v)[P], bool sp) {
    float2 nv[2 * RL];
#pragma unroll
    for (int rho = 0; rho < 2 * RL; ++rho) {
      const int src = INV ? perm_pi_inv(rho) : perm_pi(rho);
      nv[rho] = moved(rho) ? sel2(sp, v[src], v[rho]) : v[rho];
    }
#pragma unroll
    for (int rho = 0; rho < 2 * RL; ++rho) v[rho] = nv[rho];
  }
  __host__ __device__ __forceinline__ static void permute0(float2 (&v)[P], bool sp) { perm0<false>(v, sp); }
  __host__ __device__ __forceinline__ static void unpermute0(float2 (&v)[P], bool sp) { perm0<true>(v, sp); }
  static_assert([] {
    for (int rho = 0; rho < 2 * RL; ++rho)
      if (moved(rho) != (perm_pi(rho) != rho) || moved(perm_pi(rho)) != moved(rho) ||
          perm_pi(perm_pi_inv(rho)) != rho)
        return false;
    return true;
  }(), "thread 0's permutation moves exactly the blocks v[RL/2..RL), v[3RL/2..2RL)");
  // Rows of 16 lanes share a wave four at a time.  Their per-row images
  // are summed across the wave's four rows before they reach LDS, with the
  // gfx950 lane swaps (ctx.swap16 / swap32): for the float4 images f0..f3
  // of four consecutive slots (or chunks) 4s .. 4s+3, stage 1 pairs f0 with
  // f1 and f2 with f3 across rows (0,1), (2,3), stage 2 pairs the results
  // across the halves, and row j of the wave ends with the 4-row sum of f_j
  // (1.5 lane operations per float; the sum order is (r0 + r1) + (r2 + r3)).  Each row then writes one float4 in four,
  // into the image of its wave (the slab of the wave's first row), and the
  // cross-wave sum reads a quarter of the rows.
  static constexpr bool XL = ACDC_XLANE_SUM && T == 16 && NSL % 4 == 0 && (P / 2) % 4 == 0;
  // Stage 1 on (f0, f1) or (f2, f3): rows 0 / 2 get the first summed over
  // their row pair, rows 1 / 3 the second.
  template <class Ctx>
  __host__ __device__ __forceinline__ static float4 xlane_pair16(Ctx& ctx, float4 f0, float4 f1) {
    float a[4] = {f0.x, f0.y, f0.z, f0.w}, b[4] = {f1.x, f1.y, f1.z, f1.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      ctx.swap16(a[j], b[j]);
      a[j] += b[j];
    }
    return make_float4(a[0], a[1], a[2], a[3]);
  }
  // Stage 2 on the two stage-1 results: row j ends with f_j summed over the
  // wave's four rows.
  template <class Ctx>
  __host__ __device__ __forceinline__ static float4 xlane_pair32(Ctx& ctx, float4 h01, float4 h23) {
    float a[4] = {h01.x, h01.y, h01.z, h01.w}, c[4] = {h23.x, h23.y, h23.z, h23.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      ctx.swap32(a[j], c[j]);
      a[j] += c[j];
    }
    return make_float4(a[0], a[1], a[2], a[3]);
  }
  // The DCT-III pre-twiddle of thread 0's slot 0 needs its own qb':
  // exp(i pi/8) / (2 sqrt(N)).
  static constexpr float kQbRe = float(0.9238795325112867561 / (2.0 * csqrt(double(N))));
  static constexpr float kQbIm = float(0.3826834323650897717 / (2.0 * csqrt(double(N))));

  // Per-layer quartet coefficients (real_mq_entry), layout of one layer
  // [slot][kMqRows][T] float4, lane-contiguous:
  //   c0 = (L1_00, L1_01, L1_11, L2_00), c1 = (L2_01, L2_11, w.x, w.y),
  //   c2 = (qa.x, qa.y, qbr.x, qbr.y), qbr = (1 + i) qb   (backward only)
  //   c3 = (dzk.x, dzk.y, dzm.x, dzm.y)  D-domain bias through the
  //        pre-twiddle (forward with a bias only)
  // A loop over the slots loads NR of those rows (c0, c1 and, for NR = 3,
  // row R2) of slot s + PF while slot s computes; the first PF slots are
  // loaded ahead, in the tail of the preceding FFT.
  template <int NR, int R2 = 2>
  struct MqTabs {
    // slots loaded ahead: fewer when three rows are loaded per slot
    static constexpr int PF = NSL < (NR == 2 ? ACDC_MQ_PF : ACDC_MQ_PF_BWD) ? NSL
                              : (NR == 2 ? ACDC_MQ_PF : ACDC_MQ_PF_BWD);
    static constexpr int row(int r) { return r < 2 ? r : R2; }
    float4 m[NSL][NR];
  };
  template <int NR, int R2>
  __host__ __device__ __forceinline__ static void load_mslot(MqTabs<NR, R2>& tb, int slot, unsigned t, GView mq) {
#pragma unroll
    for (int r = 0; r < NR; ++r)
      tb.m[slot][r] = mq.ld4(t * 16u, unsigned((slot * kMqRows + MqTabs<NR, R2>::row(r)) * T * 16));
  }
  template <int NR, int R2>
  __host__ __device__ __forceinline__ static void load_mhead(MqTabs<NR, R2>& tb, unsigned t, GView mq) {
#pragma unroll
    for (int s = 0; s < MqTabs<NR, R2>::PF; ++s) load_mslot(tb, s, t, mq);
  }
  // Forward middle's table: c0, c1, plus c3 with a bias.
  template <bool BIAS>
  using FwdTabs = MqTabs<BIAS ? 3 : 2, 3>;

  using Split = acdc::Split;
  __host__ __device__ __forceinline__ static Split split(float2 zk, float2 zm, float2 w) {
    return quartet_split(zk, zm, w);
  }
  __host__ __device__ __forceinline__ static void post_x(const Split& sp, float2 qa, float2 qbr, float (&X)[4]) {
    quartet_post(sp, qa, qbr, X);
  }
  __host__ __device__ __forceinline__ static void sym_back(const Split& sp, float4 c0, float4 c1, float2& zk,
                                                           float2& zm) {
    quartet_back(sp, c0, c1, zk, zm);
  }

  // Forward middle of a layer, in place per quartet slot: Z (frequency
  // layout) -> DCT-II quartet -> * d (+ b) -> DCT-III pre-twiddle -> Z', as
  // split + sym_back (32 operations per slot; 4 more add the bias term).
  template <bool BIAS>
  __host__ __device__ __forceinline__ static void mid(float2 (&v)[P], unsigned t, GView mq, FwdTabs<BIAS>& tb) {
    constexpr int PFM = FwdTabs<BIAS>::PF;
    const bool sp = (t == 0);
    permute0(v, sp);
#pragma unroll
    for (int q = 0; q < BL / 2; ++q)
#pragma unroll
      for (int i = 0; i < RL; ++i) {
        const int slot = q * RL + i;
        if (slot + PFM < NSL) load_mslot(tb, slot + PFM, t, mq);
        ACDC_SCHED_FENCE();
        float2& zk = v[2 * q * RL + i];
        float2& zm = v[2 * q * RL + 2 * RL - 1 - i];
        const float4 c0 = tb.m[slot][0], c1 = tb.m[slot][1];
        sym_back(split(zk, zm, make_float2(c1.z, c1.w)), c0, c1, zk, zm);
        if constexpr (BIAS) {
          const float4 c3 = tb.m[slot][2];
          zk = make_float2(zk.x + c3.x, zk.y + c3.y);
          zm = make_float2(zm.x + c3.z, zm.y + c3.w);
        }
      }
    unpermute0(v, sp);
  }

  // Backward middle of a layer.  From H-side spectrum v (of u*a) and the
  // upstream spectrum g, per slot: H = DCT-II(v), G = DCT-II(g); the image
  // H*G (the dL/dd term of this row, quartet layout) goes to the slab; then
  // g <- DCT-III pre-twiddle of G*d, from g's split (sym_back).  v is
  // consumed.
  // One slot of the backward middle: returns the dL/dd image H*G and
  // updates g's quartet in place.
  __host__ __device__ __forceinline__ static float4 mid_bwd_slot(float2 (&v)[P], float2 (&g)[P], int slot,
                                                                 const float4 (&c)[3]) {
    const int q = slot / RL, i = slot % RL;
    const float4 c0 = c[0], c1 = c[1], c2 = c[2];
    const float2 w = make_float2(c1.z, c1.w), qa = make_float2(c2.x, c2.y), qbr = make_float2(c2.z, c2.w);
    float2& gk = g[2 * q * RL + i];
    float2& gm = g[2 * q * RL + 2 * RL - 1 - i];
    float H[4], G[4];
    post_x(split(v[2 * q * RL + i], v[2 * q * RL + 2 * RL - 1 - i], w), qa, qbr, H);
    const Split sg = split(gk, gm, w);
    post_x(sg, qa, qbr, G);
    sym_back(sg, c0, c1, gk, gm);
    return make_float4(H[0] * G[0], H[1] * G[1], H[2] * G[2], H[3] * G[3]);
  }
  // With XL each group of four consecutive slots' images is summed across
  // the wave's rows (xlane_pair16 / xlane_pair32), and row rw writes slot
  // 4s + rw of the sum into the wave image `wimg`.
  template <class Ctx>
  __host__ __device__ __forceinline__ static void mid_bwd(Ctx& ctx, float2 (&v)[P], float2 (&g)[P], unsigned t,
                                                          GView mq, MqTabs<3>& tb, float* slab, float* wimg,
                                                          unsigned rw) {
    constexpr int PFM = MqTabs<3>::PF;
    const bool sp = (t == 0);
    permute0(v, sp);
    permute0(g, sp);
    float4 im0, h01;
#pragma unroll
    for (int n = 0; n < NSL; ++n) {
      const int slot = n;
      if (n + PFM < NSL) load_mslot(tb, n + PFM, t, mq);
      ACDC_SCHED_FENCE();
      const float4 c[3] = {tb.m[slot][0], tb.m[slot][1], tb.m[slot][2]};
      const float4 im = mid_bwd_slot(v, g, slot, c);
      if constexpr (!XL) {
        reinterpret_cast<float4*>(slab)[slot * T + t] = im;
      } else if (n % 2 == 0) {
        im0 = im;
      } else if (n % 4 == 1) {
        h01 = xlane_pair16(ctx, im0, im);
      } else {
        const float4 sum = xlane_pair32(ctx, h01, xlane_pair16(ctx, im0, im));
        reinterpret_cast<float4*>(wimg)[(unsigned(n - 3) + rw) * T + t] = sum;
      }
    }
    unpermute0(g, sp);
  }
};

// ----------------------------------------------------------------- bodies
// Shared argument block of the row bodies (all pointers device pointers on
// the GPU, host pointers in the CPU emulation).
struct RealArgs {
  const float* x;
  float* y;            // forward output (may be null: stash-only forward)
  const float* A;
  const float4* Mq;    // [K][NSL][kMqRows][T] quartet coefficients (real_mq_entry)
  const int* perm;     // [K][N] (PERM only)
  float* saved;        // layer inputs [slots][batch][N]: u_1..u_{K-1} in slots 0..K-2, and with
                       // PERM u_0 in slot K-1 (may be null)
  const float* gy;     // backward: upstream gradient
  float* gx;           // backward: input gradient
  float* partial;      // backward: [slots][K][N + QF] sums, one slot per tile or per persistent workgroup
  const char* tab;     // plan tables
  long long batch;
  int K;
  unsigned flags;
  const int4* perm16 = nullptr;  // backward: [K][NCH/2][T] packed perm (PERM with RealOps::kPackedPerm)
};

// BIAS: the layers add the D-domain bias (Sec. 6.2), carried by row c3 of
// the quartet table.
template <class PL, bool BIAS, class Ctx, class TW>
__host__ __device__ void real_forward_row(Ctx& ctx, const RealArgs& a, unsigned t, long long row0, unsigned rr,
                                          float* slab, TW tab) {
  using O = RealOps<PL>;
  constexpr int N = PL::N, P = PL::P, NSL = PL::NSL, T = PL::T, NCH = O::NCH;
  const long long row = row0 + rr;
  const bool valid = row < a.batch;
  const bool permute = (a.flags & kFlagPerm) != 0;
  const unsigned roff = rr * unsigned(N / 4);
  const typename O::Lane L = O::lane(t);
  float2* slab2 = reinterpret_cast<float2*>(slab);
  float2 v[P];
  int4 idx[NCH];
  float4 av[NCH];
  O::load(GView::of(a.x + row0 * N), roff, v, L, valid);
  for (int k = 0; k < a.K; ++k) {
    const GView ak = GView::of(a.A + (long long)k * N);
    const GView mq = GView::of(a.Mq + (long long)k * NSL * kMqRows * T);
    if (permute) {
      O::template load_idx<false>(idx, GView::of(a.perm + (long long)k * N), L, t);
      O::template gather<false>(ctx, v, L, slab, idx, [&] { O::load_vec(av, ak, L); });
    } else {
      O::load_vec(av, ak, L);
    }
    // stash u_k for the backward: u_1..u_{K-1} in slots 0..K-2, and with
    // PERM u_0 = x gathered through perm[0] in slot K-1 (so the backward
    // needs no gather of x)
    if (a.saved != nullptr && valid && (k > 0 || permute))
      O::store(GView::of(a.saved + ((long long)(k > 0 ? k - 1 : a.K - 1) * a.batch + row0) * N), roff, v, L);
    O::scale(v, av);
    typename O::template FwdTabs<BIAS> tb;
    O::template fft<false>(ctx, v, t, slab2, tab, [&] { O::load_mhead(tb, t, mq); });
    O::template mid<BIAS>(v, t, mq, tb);
    O::template fft<true>(ctx, v, t, slab2, tab, [] {});
    if ((a.flags & kFlagRelu) && k < a.K - 1) O::relu(v);
  }
  if (a.y != nullptr && valid) O::store(GView::of(a.y + row0 * N), roff, v, L);
}

// Backward of one row of a tile (ROWS rows, one workgroup).  The tile's
// dL/da and dL/dd images go to partial slot `slot`.  With ACC the
// workgroup runs several tiles in turn and adds each one's images to the
// slot: `old` (LDS, max(N, QF) floats) is null on its first tile, and on
// the others receives the slot's previous values ahead of each sum
// (direct-to-LDS loads issued one phase early).
template <class PL, int ROWS, bool BIAS, bool ACC = false, class Ctx, class TW>
__host__ __device__ void real_backward_row(Ctx& ctx, const RealArgs& a, unsigned t, long long row0, unsigned rr,
                                           int tid, long long slot, float* lds, float* slab, TW tab,
                                           float* old = nullptr) {
  static_assert(!(ACC && BIAS), "the biased backward writes one partial per tile");
  using O = RealOps<PL>;
  constexpr int N = PL::N, P = PL::P, NSL = PL::NSL, T = PL::T, QF = PL::QF, NCH = O::NCH;
  constexpr int THREADS = ROWS * T;
  // tile partial per layer: [dL/da image N | dL/dd quartet image QF | row sum of g N (bias only)]
  constexpr long long PS = N + QF + (BIAS ? N : 0);
  const long long row = row0 + rr;
  const bool valid = row < a.batch;
  const bool permute = (a.flags & kFlagPerm) != 0;
  const unsigned roff = rr * unsigned(N / 4);
  const typename O::Lane L = O::lane(t);
  float2* slab2 = reinterpret_cast<float2*>(slab);
  // the images reach LDS one per row, or with XL one per wave (in the slab of
  // the wave's first row), and the cross-row sums add SROWS of them
  static_assert(!O::XL || ROWS % 4 == 0, "rows of 16 lanes fill whole waves");
  constexpr int SROWS = O::XL ? ROWS / 4 : ROWS;
  constexpr int SSTRIDE = O::XL ? 4 * PL::SLAB : PL::SLAB;
  const unsigned rw = rr % 4u;  // row within its wave (XL)
  float* const wimg = lds + (rr - rw) * PL::SLAB;
  // A row past the batch end reads the block's first row for u_k but starts
  // from g = 0, which every step keeps exactly zero (linear transforms,
  // diagonal scalings, masks); its images H * G and u * g therefore vanish
  // without masking u, as long as that first row is finite.
  // layer input u_k: stash slot k - 1 for k > 0; for k = 0 the block input
  // itself, or with PERM stash slot K - 1 (x gathered through perm[0])
  const float* const x0 = a.x + row0 * N;
  const float* const s0 = a.saved + (row0 - a.batch) * N;
  const float* const u0 = permute ? s0 + (long long)a.K * a.batch * N : x0;  // slot K-1 with PERM
  auto u_view = [&](int k) { return GView::of(k == 0 ? u0 : s0 + (long long)k * a.batch * N); };
  float2 g[P];
  float4 uv[NCH], av[NCH];
  int4 idx[O::NIW];
  O::load(GView::of(a.gy + row0 * N), roff, g, L, valid);
  O::load_raw(uv, u_view(a.K - 1), roff, L, valid);
  for (int k = a.K - 1; k >= 0; --k) {
    const GView ak = GView::of(a.A + (long long)k * N);
    const GView mq = GView::of(a.Mq + (long long)k * NSL * kMqRows * T);
    float* part = a.partial + (slot * a.K + k) * PS;
    // the slot's dL/dd values from earlier tiles, for the sum after the middle
    if constexpr (ACC)
      if (old != nullptr) lds_fetch<QF, THREADS>(old, GView::of(part + N), tid);
    if constexpr (BIAS) {
      // dL/db_k = sum over rows of DCT(g) = DCT(sum over rows of g): the
      // tile sums g here (spatial, natural order); one DCT per layer of the
      // batch sum follows the reduction.
      ctx.sync_row();
      O::for_chunks(g, L, [&](unsigned lc, unsigned cc, float2& lo, float2& hi) {
        reinterpret_cast<float4*>(slab)[lc + cc] = make_float4(lo.x, hi.y, lo.y, hi.x);
      });
      ctx.sync_all();
      sum_rows<ROWS, PL::SLAB, THREADS, N>(lds, GView::of(part + N + QF), tid);
      ctx.sync_all();
    }
    // h2 = DCT(u * a), gh3 = DCT(g); dL/dd image h2 * gh3; g <- pre(gh3 * d)
    {
      float2 v[P];
      O::load_vec(av, ak, L);
      O::unpack(uv, v);
      O::scale(v, av);
      typename O::template MqTabs<3> tb;
#if ACDC_FFT2
      O::fft2(ctx, v, g, t, slab2, tab, [&] { O::load_mhead(tb, t, mq); });
#else
      O::template fft<false>(ctx, v, t, slab2, tab, [] {});
      O::template fft<false>(ctx, g, t, slab2, tab, [&] { O::load_mhead(tb, t, mq); });
#endif
      ctx.sync_row();
      O::mid_bwd(ctx, v, g, t, mq, tb, slab, wimg, rw);
    }
    if constexpr (ACC)
      if (old != nullptr) lds_fetch_wait();
    ctx.sync_all();
    sum_rows<SROWS, SSTRIDE, THREADS, QF>(lds, GView::of(part + N), tid, ACC ? old : nullptr);
    ctx.sync_all();
    // and its dL/da values, for the sum after the inverse transform
    if constexpr (ACC)
      if (old != nullptr) lds_fetch<N, THREADS>(old, GView::of(part), tid);
    // gh1 = DCT-III(gh3 * d); u_k is reloaded meanwhile
    O::template fft<true>(ctx, g, t, slab2, tab, [&] { O::load_raw(uv, u_view(k), roff, L, valid); });
    {
      // Through the ReLU of the previous layer: u_k = 0 exactly where the
      // mask is off, so masking gh1 first leaves u * gh1 unchanged.  Then
      // the dL/da image u * gh1 (spatial, natural order) goes to the slab.
      const bool mask = (a.flags & kFlagRelu) && k > 0;
      ctx.sync_row();
      auto chunk = [&](int n) {
        float2& lo = g[O::ch_lo(n)];
        float2& hi = g[O::ch_hi(n)];
        const float4 u = uv[n];
        if (mask) {
          lo = make_float2(u.x > 0.f ? lo.x : 0.f, u.z > 0.f ? lo.y : 0.f);
          hi = make_float2(u.w > 0.f ? hi.x : 0.f, u.y > 0.f ? hi.y : 0.f);
        }
        return make_float4(u.x * lo.x, u.y * hi.y, u.z * lo.y, u.w * hi.x);
      };
      if constexpr (!O::XL) {
#pragma unroll
        for (int n = 0; n < NCH; ++n)
          reinterpret_cast<float4*>(slab)[O::ch_lc(L, n) + O::ch_cc(n)] = chunk(n);
      } else {
        // chunks in groups of four, summed across the wave's rows; row rw
        // writes the sum of chunk 4c + rw
#pragma unroll
        for (int c = 0; c < NCH / 4; ++c) {
          const int n0 = 4 * c, n1 = n0 + 1, n2 = n0 + 2, n3 = n0 + 3;
          const float4 h01 = O::xlane_pair16(ctx, chunk(n0), chunk(n1));
          const float4 sum = O::xlane_pair32(ctx, h01, O::xlane_pair16(ctx, chunk(n2), chunk(n3)));
          const unsigned p0 = O::ch_lc(L, n0) + O::ch_cc(n0), p1 = O::ch_lc(L, n1) + O::ch_cc(n1);
          const unsigned p2 = O::ch_lc(L, n2) + O::ch_cc(n2), p3 = O::ch_lc(L, n3) + O::ch_cc(n3);
          reinterpret_cast<float4*>(wimg)[rw == 0 ? p0 : rw == 1 ? p1 : rw == 2 ? p2 : p3] = sum;
          ACDC_SCHED_FENCE();
        }
      }
    }
    ACDC_SCHED_FENCE();  // the loads of a below stay behind the images (registers)
    if constexpr (ACC)
      if (old != nullptr) lds_fetch_wait();  // the fetch landed during the inverse transform
    O::load_vec(av, ak, L);
    ACDC_SCHED_FENCE();
    ctx.sync_all();
    sum_rows<SROWS, SSTRIDE, THREADS, N>(lds, GView::of(part), tid, ACC ? old : nullptr);
    ctx.sync_all();
    // dL/du = gh1 * a, then un-permute; the next layer's u loads meanwhile
    O::scale(g, av);
    const int kn = k > 0 ? k - 1 : 0;
    auto next = [&] { O::load_raw(uv, u_view(kn), roff, L, valid); };
    if (permute) {
      constexpr bool PK = O::kPackedPerm;
      O::template load_idx<PK>(idx, PK ? GView::of(a.perm16 + (long long)k * O::NIW * T)
                                       : GView::of(a.perm + (long long)k * N), L, t);
      O::template scatter<PK>(ctx, g, L, slab, idx, next);
    } else {
      next();
    }
  }
  if (valid) O::store(GView::of(a.gx + row0 * N), roff, g, L);
}

// DCT-II of one row (the bias gradient): out (+)= S C.  Forward FFT, then
// per quartet slot the real-FFT split and the post-twiddle of the backward's
// image (post_x), with w, qa, qbr from rows c1, c2 of a quartet table (they
// do not depend on d).  One row per T threads.
template <class PL, class Ctx, class TW>
__host__ __device__ void real_dct_row(Ctx& ctx, const float* S, float* out, const float4* Mq, bool accumulate,
                                      unsigned t, float* slab, TW tab, const char* tabc) {
  using O = RealOps<PL>;
  constexpr int P = PL::P, T = PL::T, RL = PL::RL, BL = PL::BL;
  const typename O::Lane L = O::lane(t);
  float2 v[P];
  O::load(GView::of(S), 0u, v, L, true);
  O::template fft<false>(ctx, v, t, reinterpret_cast<float2*>(slab), tab, [] {});
  O::permute0(v, t == 0);
  const GView mq = GView::of(Mq);
#pragma unroll
  for (int q = 0; q < BL / 2; ++q)
#pragma unroll
    for (int i = 0; i < RL; ++i) {
      const int slot = q * RL + i, e = slot * T + int(t);
      const float4 c1 = mq.ld4(t * 16u, unsigned((slot * kMqRows + 1) * T * 16));
      const float4 c2 = mq.ld4(t * 16u, unsigned((slot * kMqRows + 2) * T * 16));
      float X[4];
      O::post_x(O::split(v[2 * q * RL + i], v[2 * q * RL + 2 * RL - 1 - i], make_float2(c1.z, c1.w)),
                make_float2(c2.x, c2.y), make_float2(c2.z, c2.w), X);
      X[1] = -X[1];
      const int4 idx = reinterpret_cast<const int4*>(tabc + PL::OFF_QIDX)[e];
      const int sm = (reinterpret_cast<const int*>(tabc + PL::OFF_QMASK)[e] >> 4) & 0xF;
      const int id[4] = {idx.x, idx.y, idx.z, idx.w};
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (sm & (1 << j)) out[id[j]] = accumulate ? out[id[j]] + X[j] : X[j];
    }
}

}  // namespace acdc
