// Kernels of the multi-pass ACDC layers (declarations and the pass structure
// in acdc_multipass.hpp).  Elementwise passes use grid-stride loops over
// 64-bit indices; the segment FFTs reuse the complex row machinery.
#include <hip/hip_runtime.h>

#include "acdc_devctx.hpp"
#include "acdc_multipass.hpp"

namespace acdc {
namespace mp {
namespace {

constexpr int kThreads = 256;

// Workgroups go to the 8 XCDs (each with its own L2) in turn: workgroup w
// runs on XCD w mod 8.  Grids are a multiple of 8 workgroups, and gindex()
// hands XCD x the x-th contiguous eighth of the grid, so the workgroups
// that gather from one row share that XCD's L2.
constexpr int kXcds = 8;
constexpr int kPermThreads = 512;

dim3 grid_for(long long n) {
  long long blocks = (n + kThreads - 1) / kThreads;
  if (blocks > 65536) blocks = 65536;
  blocks = (blocks + kXcds - 1) / kXcds * kXcds;
  if (blocks < kXcds) blocks = kXcds;
  return dim3(unsigned(blocks));
}

__device__ __forceinline__ long long gstride() { return (long long)gridDim.x * blockDim.x; }
__device__ __forceinline__ long long gindex() {
  const unsigned per_xcd = gridDim.x / kXcds;
  const unsigned blk = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  return (long long)blk * blockDim.x + threadIdx.x;
}

// Makhoul packing by float4 chunks: chunk q of a row (floats 4q .. 4q+3)
// holds complex value m = q as (h.x, h.z) and m = M-1-q as (h.w, h.y).
__device__ __forceinline__ float2 chunk_even(float4 h) { return make_float2(h.x, h.z); }
__device__ __forceinline__ float2 chunk_odd(float4 h) { return make_float2(h.w, h.y); }
__device__ __forceinline__ float4 chunk_of(float2 even, float2 odd) { return make_float4(even.x, odd.y, even.y, odd.x); }
__device__ __forceinline__ float4 scale4(float4 h, float4 a) {
  return make_float4(h.x * a.x, h.y * a.y, h.z * a.z, h.w * a.w);
}
__device__ __forceinline__ float4 relu4(float4 h) { return make_float4(relu1(h.x), relu1(h.y), relu1(h.z), relu1(h.w)); }

// Chunk q (q < M/2) of row b: Z[q] and Z[M-1-q], scaled by a, stashed.
__global__ __launch_bounds__(kThreads) void k_pack(const float* __restrict__ src, const float* __restrict__ a,
                                                   float* __restrict__ stash, float2* __restrict__ Z, long long B,
                                                   long long N) {
  const long long M = N / 2, H = M / 2, total = B * H;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / H, q = i % H;
    float4 h = reinterpret_cast<const float4*>(src + b * N)[q];
    if (stash) reinterpret_cast<float4*>(stash + b * N)[q] = h;
    if (a) h = scale4(h, reinterpret_cast<const float4*>(a)[q]);
    Z[b * M + q] = chunk_even(h);
    Z[b * M + M - 1 - q] = chunk_odd(h);
  }
}

// Radix-R decimation in frequency on segments of length S (the row itself
// for the first pass): butterfly n of segment s reads x[n + j Q], Q = S/R,
// and writes y_r[n] = W_M^(n r M/S) sum_j x[n + j Q] W_R^(j r) to r Q + n.
template <int R>
__global__ __launch_bounds__(kThreads) void k_dif(float2* __restrict__ Z, long long B, long long M, long long S,
                                                  const float2* __restrict__ twM) {
  const long long Q = S / R, per_row = M / R, total = B * per_row, tws = M / S;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / per_row, q = i % per_row;
    const long long base = b * M + (q / Q) * S, n = q % Q;
    float2 x[R];
#pragma unroll
    for (int j = 0; j < R; ++j) x[j] = Z[base + n + j * Q];
    Dft<R, false>::run(x);
#pragma unroll
    for (int r = 1; r < R; ++r) x[r] = cmul(x[r], twM[n * r * tws]);
#pragma unroll
    for (int r = 0; r < R; ++r) Z[base + r * Q + n] = x[r];
  }
}

// The unnormalised inverse of k_dif: x'[n + j Q] = sum_r W_R^(-j r) W_M^(-n r M/S) y'_r[n].
template <int R>
__global__ __launch_bounds__(kThreads) void k_dit(float2* __restrict__ Z, long long B, long long M, long long S,
                                                  const float2* __restrict__ twM) {
  const long long Q = S / R, per_row = M / R, total = B * per_row, tws = M / S;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / per_row, q = i % per_row;
    const long long base = b * M + (q / Q) * S, n = q % Q;
    float2 y[R];
#pragma unroll
    for (int r = 0; r < R; ++r) y[r] = Z[base + r * Q + n];
#pragma unroll
    for (int r = 1; r < R; ++r) y[r] = cmulc(y[r], twM[n * r * tws]);
    Dft<R, true>::run(y);
#pragma unroll
    for (int j = 0; j < R; ++j) Z[base + n + j * Q] = y[j];
  }
}

// The first DIF pass (on whole rows, S = M) with the packing folded in.
// Butterfly n takes m = n + j Q (Q = M/R); for j < R/2 that is the even
// part of chunk n + j Q, for j >= R/2 the odd part of chunk
// nb + (R-1-j) Q, nb = Q-1-n.  So butterflies n and nb read the same R
// chunks, and one thread runs both (n < Q/2): every access contiguous.
template <int R>
__global__ __launch_bounds__(kThreads) void k_pack_dif(const float* __restrict__ src, const float* __restrict__ a,
                                                       float* __restrict__ stash, float2* __restrict__ Z, long long B,
                                                       long long M, const float2* __restrict__ twM) {
  const long long N = 2 * M, Q = M / R, H = Q / 2, total = B * H;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / H, n = i % H, nb = Q - 1 - n;
    const float4* row4 = reinterpret_cast<const float4*>(src + b * N);
    float4* st4 = stash ? reinterpret_cast<float4*>(stash + b * N) : nullptr;
    const float4* a4 = reinterpret_cast<const float4*>(a);
    float2 x[R], xb[R];
#pragma unroll
    for (int j = 0; j < R / 2; ++j) {
      const long long q = n + j * Q, qb = nb + j * Q;
      float4 h = row4[q], hb = row4[qb];
      if (st4) {
        st4[q] = h;
        st4[qb] = hb;
      }
      if (a4) {
        h = scale4(h, a4[q]);
        hb = scale4(hb, a4[qb]);
      }
      x[j] = chunk_even(h);
      xb[R - 1 - j] = chunk_odd(h);
      xb[j] = chunk_even(hb);
      x[R - 1 - j] = chunk_odd(hb);
    }
    Dft<R, false>::run(x);
    Dft<R, false>::run(xb);
#pragma unroll
    for (int r = 1; r < R; ++r) {
      x[r] = cmul(x[r], twM[n * r]);
      xb[r] = cmul(xb[r], twM[nb * r]);
    }
    float2* zrow = Z + b * M;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      zrow[r * Q + n] = x[r];
      zrow[r * Q + nb] = xb[r];
    }
  }
}

// The last DIT pass (S = M) with the unpacking (and ReLU) folded in: the
// mirror image of k_pack_dif, butterflies n and Q-1-n writing R chunks.
template <int R>
__global__ __launch_bounds__(kThreads) void k_dit_unpack(const float2* __restrict__ Z, float* __restrict__ dst,
                                                         long long B, long long M, const float2* __restrict__ twM,
                                                         int relu) {
  const long long N = 2 * M, Q = M / R, H = Q / 2, total = B * H;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / H, n = i % H, nb = Q - 1 - n;
    const float2* zrow = Z + b * M;
    float2 y[R], yb[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      y[r] = zrow[r * Q + n];
      yb[r] = zrow[r * Q + nb];
    }
#pragma unroll
    for (int r = 1; r < R; ++r) {
      y[r] = cmulc(y[r], twM[n * r]);
      yb[r] = cmulc(yb[r], twM[nb * r]);
    }
    Dft<R, true>::run(y);
    Dft<R, true>::run(yb);
    float4* out4 = reinterpret_cast<float4*>(dst + b * N);
#pragma unroll
    for (int j = 0; j < R / 2; ++j) {
      float4 h = chunk_of(y[j], yb[R - 1 - j]), hb = chunk_of(yb[j], y[R - 1 - j]);
      if (relu) {
        h = relu4(h);
        hb = relu4(hb);
      }
      out4[n + j * Q] = h;
      out4[nb + j * Q] = hb;
    }
  }
}

// Segment FFTs of L = CP::N points, in place, Launch<CP>::FWD_ROWS segments
// per workgroup.  Forward: natural-order input (spatial layout) to
// natural-order output (frequency layout); the inverse runs the mirror.
template <class CP, bool INV>
__global__ __launch_bounds__(Launch<CP>::FWD_THREADS) void k_seg(float2* __restrict__ Z, long long nseg,
                                                                 const char* __restrict__ tab) {
  using L = Launch<CP>;
  using O = CplxOps<CP>;
  constexpr int T = CP::T, P = CP::P;
  __shared__ float lds[L::FWD_ROWS * L::FWD_SLAB];
  const int tid = threadIdx.x;
  const unsigned t = unsigned(tid) % T;
  int r = tid / T;
  if constexpr (T >= 64) r = __builtin_amdgcn_readfirstlane(r);
  const long long seg0 = (long long)blockIdx.x * L::FWD_ROWS;
  const bool valid = seg0 + r < nseg;
  const unsigned roff = valid ? unsigned(r) * unsigned(CP::N) : 0u;
  const GView g = GView::of(Z + seg0 * CP::N);
  float2* slab = reinterpret_cast<float2*>(lds + r * L::FWD_SLAB);
  DevCtx<T> ctx;
  float2 v[P];
  O::template ld_row<INV>(g, roff, v, t);
  O::template fft<INV>(ctx, v, t, slab, GView::of(tab));
  if (valid) O::template st_row<!INV>(g, roff, v, t);
}

// Per-layer quartet coefficients [K][NQ][kMqRows] (entry-major).
__global__ __launch_bounds__(kThreads) void k_mq(const float* __restrict__ D, const float* __restrict__ Bias,
                                                 float4* __restrict__ Mq, int K, long long NQ, QuartetTabs q,
                                                 long long N) {
  const long long total = (long long)K * NQ;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long k = i / NQ;
    const int e = int(i % NQ);
    float4 row[kMqRows];
    quartet_coeffs(D + k * N, Bias ? Bias + k * N : nullptr, q, e, row);
#pragma unroll
    for (int r = 0; r < kMqRows; ++r) Mq[i * kMqRows + r] = row[r];
  }
}

// Positions of quartet entry e's pair: (Z[e], Z[M-e]), or (Z[0], Z[M/2]) for e = 0.
__device__ __forceinline__ void pair_pos(const Geo& g, long long e, long long& pa, long long& pb) {
  pa = pos(g, e);
  pb = pos(g, e == 0 ? g.M / 2 : g.M - e);
}

// Forward middle, kColRows rows per thread and quartet entry (the
// coefficients loaded once for them).
__global__ __launch_bounds__(kThreads) void k_mid_fwd(float2* __restrict__ Z, const float4* __restrict__ Mq,
                                                      long long B, Geo g, int bias) {
  const long long NQ = g.M / 2, P = (B + kColRows - 1) / kColRows, total = P * NQ;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long p = i / NQ, e = i % NQ;
    long long pa, pb;
    pair_pos(g, e, pa, pb);
    const float4 c0 = Mq[e * kMqRows], c1 = Mq[e * kMqRows + 1];
    const float4 c3 = bias ? Mq[e * kMqRows + 3] : make_float4(0.f, 0.f, 0.f, 0.f);
    const long long b0 = p * kColRows, b1 = b0 + kColRows < B ? b0 + kColRows : B;
    for (long long b = b0; b < b1; ++b) {
      float2* row = Z + b * g.M;
      float2 zk = row[pa], zm = row[pb];
      quartet_back(quartet_split(zk, zm, make_float2(c1.z, c1.w)), c0, c1, zk, zm);
      if (bias) {
        zk = make_float2(zk.x + c3.x, zk.y + c3.y);
        zm = make_float2(zm.x + c3.z, zm.y + c3.w);
      }
      row[pa] = zk;
      row[pb] = zm;
    }
  }
}

// Backward middle over a block of kColRows rows (in row order) per thread
// and quartet entry e: the images H*G (dL/dd) and, with a bias, G (dL/db),
// summed over the block's rows into partD/partB[p][4e + j] (quartet order);
// g's spectrum is replaced by the DCT-III pre-twiddle of G*d.  The
// coefficients are loaded once per block.
__global__ __launch_bounds__(kThreads) void k_mid_bwd(const float2* __restrict__ Zh, float2* __restrict__ Zg,
                                                      const float4* __restrict__ Mq, long long B, Geo g,
                                                      float* __restrict__ partD, float* __restrict__ partB) {
  const long long NQ = g.M / 2, P = (B + kColRows - 1) / kColRows, total = P * NQ, W = 2 * g.M;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long p = i / NQ, e = i % NQ;
    long long pa, pb;
    pair_pos(g, e, pa, pb);
    const float4 c0 = Mq[e * kMqRows], c1 = Mq[e * kMqRows + 1], c2 = Mq[e * kMqRows + 2];
    const float2 w = make_float2(c1.z, c1.w), qa = make_float2(c2.x, c2.y), qbr = make_float2(c2.z, c2.w);
    float4 sD = make_float4(0.f, 0.f, 0.f, 0.f), sB = sD;
    const long long b0 = p * kColRows, b1 = b0 + kColRows < B ? b0 + kColRows : B;
    for (long long b = b0; b < b1; ++b) {
      const float2* hrow = Zh + b * g.M;
      float2* grow = Zg + b * g.M;
      float2 gk = grow[pa], gm = grow[pb];
      float H[4], G[4];
      quartet_post(quartet_split(hrow[pa], hrow[pb], w), qa, qbr, H);
      const Split sg = quartet_split(gk, gm, w);
      quartet_post(sg, qa, qbr, G);
      sD = make_float4(sD.x + H[0] * G[0], sD.y + H[1] * G[1], sD.z + H[2] * G[2], sD.w + H[3] * G[3]);
      sB = make_float4(sB.x + G[0], sB.y - G[1], sB.z + G[2], sB.w + G[3]);
      quartet_back(sg, c0, c1, gk, gm);
      grow[pa] = gk;
      grow[pb] = gm;
    }
    reinterpret_cast<float4*>(partD + p * W)[e] = sD;
    if (partB) reinterpret_cast<float4*>(partB + p * W)[e] = sB;
  }
}

__global__ __launch_bounds__(kThreads) void k_unpack(const float2* __restrict__ Z, float* __restrict__ dst,
                                                     long long B, long long N, int relu) {
  const long long M = N / 2, H = M / 2, total = B * H;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / H, q = i % H;
    float4 h = chunk_of(Z[b * M + q], Z[b * M + M - 1 - q]);
    if (relu) h = relu4(h);
    reinterpret_cast<float4*>(dst + b * N)[q] = h;
  }
}

// dL/da image u * gh1 (gh1 masked where the previous layer's ReLU was off:
// u = 0 there), and dL/du = gh1 * a (no permutation).
__global__ __launch_bounds__(kThreads) void k_dA(const float* __restrict__ gh1, const float* __restrict__ u,
                                                 const float* __restrict__ a, int mask, float* __restrict__ imgA,
                                                 float* __restrict__ gnext, long long B, long long N) {
  const long long total = B * N;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long n = i % N;
    const float uu = u[i];
    float gh = gh1[i];
    if (mask && !(uu > 0.f)) gh = 0.f;
    imgA[i] = uu * gh;
    gnext[i] = gh * a[n];
  }
}

// ------------------------------------------------------------ permutations
// out[b][n] = in[b][src[n]] in chunks of C = min(N, kPermChunk) floats held
// in LDS (see acdc_multipass.hpp).  Pass A: workgroup (b, c) loads source
// chunk c and writes the C values it sources to tmp[b][cC + i], ordered by
// destination chunk, then destination.  Pass B: workgroup (b, d) reads the
// nC runs of tmp bound for chunk d into LDS (run-contiguous loads), then
// writes chunk d in order.  The backward runs the adjoint: the same tables
// with each pass's reads and writes exchanged.  Table entries are masked
// into range, so a malformed perm yields wrong values, never a stray access.

// Pass A table build, step 1: per block of kThreads destinations (all in
// one chunk d, as C is a multiple of kThreads), the count of each source
// chunk: cntS[blk][c].
__global__ __launch_bounds__(kThreads) void k_pt_count(const int* __restrict__ src, long long N, int C, int nC,
                                                       int* __restrict__ cntS, long long stride) {
  __shared__ int h[kPermMaxChunks];
  src += blockIdx.y * N;  // layer blockIdx.y
  cntS += blockIdx.y * stride;
  for (int c = threadIdx.x; c < nC; c += kThreads) h[c] = 0;
  __syncthreads();
  const long long n = (long long)blockIdx.x * kThreads + threadIdx.x;
  atomicAdd(&h[int((src[n] & (N - 1)) / C)], 1);
  __syncthreads();
  for (int c = threadIdx.x; c < nC; c += kThreads) cntS[(long long)blockIdx.x * nC + c] = h[c];
}

// Step 2, one thread per (d, c): the running count over chunk d's blocks
// (bpre[blk][c], exclusive) and the total cnt[d][c].
__global__ __launch_bounds__(kThreads) void k_pt_blocks(const int* __restrict__ cntS, int C, int nC,
                                                        int* __restrict__ bpre, int* __restrict__ cnt,
                                                        long long stride) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= nC * nC) return;
  cntS += blockIdx.y * stride;
  bpre += blockIdx.y * stride;
  cnt += blockIdx.y * stride;
  const int d = i / nC, c = i % nC, per = C / kThreads;
  int run = 0;
  for (int j = 0; j < per; ++j) {
    const long long blk = (long long)d * per + j;
    bpre[blk * nC + c] = run;
    run += cntS[blk * nC + c];
  }
  cnt[i] = run;
}

// Step 3, one workgroup: off[d][c] = c C + sum over d' < d of cnt[d'][c]
// (the tmp position of run (c, d)) and lst[d][c] = sum over c' < c of
// cnt[d][c'] (its LDS position in pass B).
__global__ __launch_bounds__(kThreads) void k_pt_offsets(const int* __restrict__ cnt, int C, int nC,
                                                         int* __restrict__ off, int* __restrict__ lst,
                                                         long long stride) {
  cnt += blockIdx.x * stride;  // one workgroup per layer
  off += blockIdx.x * stride;
  lst += blockIdx.x * stride;
  for (int c = threadIdx.x; c < nC; c += kThreads) {
    long long run = (long long)c * C;
    for (int d = 0; d < nC; ++d) {
      off[d * nC + c] = int(run);
      run += cnt[d * nC + c];
    }
  }
  for (int d = threadIdx.x; d < nC; d += kThreads) {
    int run = 0;
    for (int c = 0; c < nC; ++c) {
      lst[d * nC + c] = run;
      run += cnt[d * nC + c];
    }
  }
}

// Step 4: every destination n takes a place in its run (the order inside a
// block's share of a run is whatever the LDS counter hands out; the tables
// stay consistent, and the permuted values do not depend on it):
// srcA[tpos] = src[n] - c C, gposB[d C + slot] = tpos, locB[n] = slot.
__global__ __launch_bounds__(kThreads) void k_pt_place(const int* __restrict__ src, long long N, int C, int nC,
                                                       const int* __restrict__ bpre, const int* __restrict__ off,
                                                       const int* __restrict__ lst, int* __restrict__ srcA,
                                                       int* __restrict__ gposB, int* __restrict__ locB,
                                                       long long stride) {
  __shared__ int h[kPermMaxChunks];
  const long long ls = blockIdx.y * stride;
  src += blockIdx.y * N;
  bpre += ls;
  off += ls;
  lst += ls;
  srcA += ls;
  gposB += ls;
  locB += ls;
  for (int c = threadIdx.x; c < nC; c += kThreads) h[c] = 0;
  __syncthreads();
  const long long n = (long long)blockIdx.x * kThreads + threadIdx.x;
  const int sv = int(src[n] & (N - 1)), c = sv / C, d = int(n / C);
  const int p = bpre[(long long)blockIdx.x * nC + c] + atomicAdd(&h[c], 1);
  const long long tpos = ((long long)off[d * nC + c] + p) & (N - 1);
  const int slot = (lst[d * nC + c] + p) & (C - 1);
  srcA[tpos] = sv & (C - 1);
  gposB[(long long)d * C + slot] = int(tpos);
  locB[n] = slot;
}

// The pass kernels keep kPermBatch loads in flight per thread: with two
// 64 KB workgroups per CU, one load at a time would leave them bound by
// memory latency.  Element i of a chunk goes to thread i mod kPermThreads.
constexpr int kPermBatch = 8;
constexpr int kPermStep = kPermBatch * kPermThreads;
// With more than one chunk, C = kPermChunk and the loops of pass B and of
// the adjoint passes run whole steps; k_pt_a and k_pt_bt also serve a
// single chunk (C = N, any power of two from 256) and take plain loops when
// C is not a whole number of steps.
static_assert(kPermChunk % kPermStep == 0, "whole steps per chunk");

// Chunk copy HBM -> LDS (float4, contiguous).
__device__ __forceinline__ void chunk_to_lds(float4* __restrict__ lds4, const float4* __restrict__ g4, int C) {
  if ((C / 4) % kPermStep == 0) {
    for (int i0 = threadIdx.x; i0 < C / 4; i0 += kPermStep) {
      float4 v[kPermBatch];
#pragma unroll
      for (int u = 0; u < kPermBatch; ++u) v[u] = g4[i0 + u * kPermThreads];
#pragma unroll
      for (int u = 0; u < kPermBatch; ++u) lds4[i0 + u * kPermThreads] = v[u];
    }
  } else {
    for (int i = threadIdx.x; i < C / 4; i += kPermThreads) lds4[i] = g4[i];
  }
}
// Chunk copy LDS -> HBM (float4, contiguous).
__device__ __forceinline__ void chunk_from_lds(float4* __restrict__ g4, const float4* __restrict__ lds4, int C) {
  for (int i = threadIdx.x; i < C / 4; i += kPermThreads) g4[i] = lds4[i];
}

// Forward pass A (or, with one chunk, the whole permutation with tab = perm):
// out[b][cC + i] = in[b][cC + tab[cC + i]].  E is the element (float for
// real rows, float2 for complex ones); N and C count elements.
template <class E>
__global__ __launch_bounds__(kPermThreads) void k_pt_a(const E* __restrict__ in, E* __restrict__ out,
                                                       const int* __restrict__ tab, long long N, int C, int nC,
                                                       long long work) {
  constexpr int EW = int(sizeof(E) / sizeof(float));
  __shared__ float4 lds4[kPermChunk / 4];
  const E* lds = reinterpret_cast<const E*>(lds4);
  for (long long w = blockIdx.x; w < work; w += gridDim.x) {
    const long long b = w / nC, c = w % nC, base = b * N + c * C;
    chunk_to_lds(lds4, reinterpret_cast<const float4*>(in + base), C * EW);
    __syncthreads();
    const int* t = tab + c * C;
    if (C % kPermStep == 0) {
      for (int i0 = threadIdx.x; i0 < C; i0 += kPermStep) {
        int id[kPermBatch];
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u) id[u] = t[i0 + u * kPermThreads] & (C - 1);
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u) out[base + i0 + u * kPermThreads] = lds[id[u]];
      }
    } else {
      for (int i = threadIdx.x; i < C; i += kPermThreads) out[base + i] = lds[t[i] & (C - 1)];
    }
    __syncthreads();
  }
}

// Forward pass B: out[b][dC + j] = L[locB[dC + j]], L[j] = tmp[b][gposB[dC + j]].
template <class E>
__global__ __launch_bounds__(kPermThreads) void k_pt_b(const E* __restrict__ tmp, E* __restrict__ out,
                                                       const int* __restrict__ gposB, const int* __restrict__ locB,
                                                       long long N, int C, int nC, long long work) {
  __shared__ float4 lds4[kPermChunk / 4];
  E* lds = reinterpret_cast<E*>(lds4);
  for (long long w = blockIdx.x; w < work; w += gridDim.x) {
    const long long b = w / nC, d = w % nC, base = b * N + d * C;
    const int* gp = gposB + d * C;
    const int* lc = locB + d * C;
    const E* trow = tmp + b * N;
    for (int j0 = threadIdx.x; j0 < C; j0 += kPermStep) {
      int id[kPermBatch];
      E v[kPermBatch];
#pragma unroll
      for (int u = 0; u < kPermBatch; ++u) id[u] = gp[j0 + u * kPermThreads] & (N - 1);
#pragma unroll
      for (int u = 0; u < kPermBatch; ++u) v[u] = trow[id[u]];
#pragma unroll
      for (int u = 0; u < kPermBatch; ++u) lds[j0 + u * kPermThreads] = v[u];
    }
    __syncthreads();
    for (int j0 = threadIdx.x; j0 < C; j0 += kPermStep) {
      int id[kPermBatch];
#pragma unroll
      for (int u = 0; u < kPermBatch; ++u) id[u] = lc[j0 + u * kPermThreads] & (C - 1);
#pragma unroll
      for (int u = 0; u < kPermBatch; ++u) out[base + j0 + u * kPermThreads] = lds[id[u]];
    }
    __syncthreads();
  }
}

// The plain adjoint of pass B (or, with one chunk, of the whole
// permutation: loc = perm, no gpos): L[loc[dC + j]] = in[b][dC + j], then
// out[b][gpos[dC + j]] = L[j] (out[b][dC + j] without gpos).
template <class E>
__global__ __launch_bounds__(kPermThreads) void k_pt_btp(const E* __restrict__ in, E* __restrict__ out,
                                                         const int* __restrict__ gpos, const int* __restrict__ loc,
                                                         long long N, int C, int nC, long long work) {
  constexpr int EW = int(sizeof(E) / sizeof(float));
  __shared__ float4 lds4[kPermChunk / 4];
  E* lds = reinterpret_cast<E*>(lds4);
  for (long long w = blockIdx.x; w < work; w += gridDim.x) {
    const long long b = w / nC, d = w % nC, base = b * N + d * C;
    const int* lc = loc + d * C;
    if (C % kPermStep == 0) {
      for (int j0 = threadIdx.x; j0 < C; j0 += kPermStep) {
        int id[kPermBatch];
        E v[kPermBatch];
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u) {
          id[u] = lc[j0 + u * kPermThreads] & (C - 1);
          v[u] = in[base + j0 + u * kPermThreads];
        }
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u) lds[id[u]] = v[u];
      }
    } else {
      for (int j = threadIdx.x; j < C; j += kPermThreads) lds[lc[j] & (C - 1)] = in[base + j];
    }
    __syncthreads();
    if (gpos) {
      const int* gp = gpos + d * C;
      E* orow = out + b * N;
      for (int j0 = threadIdx.x; j0 < C; j0 += kPermStep) {
        int id[kPermBatch];
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u) id[u] = gp[j0 + u * kPermThreads] & (N - 1);
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u) orow[id[u]] = lds[j0 + u * kPermThreads];
      }
    } else {
      chunk_from_lds(reinterpret_cast<float4*>(out + base), lds4, C * EW);
    }
    __syncthreads();
  }
}

// Backward, first pass (the adjoint of pass B, or with one chunk of the
// whole permutation, loc = perm and no gpos), with the dL/da step folded
// in: for n in chunk d, gm = gh1 (0 where mask and u <= 0), imgA = u gm,
// L[loc[n]] = gm a[n]; then out[b][gpos[dC + j]] = L[j] (out[b][dC + j]
// without gpos).
__global__ __launch_bounds__(kPermThreads) void k_pt_bt(const float* __restrict__ gh1, const float* __restrict__ u,
                                                        const float* __restrict__ a, int mask,
                                                        float* __restrict__ imgA, float* __restrict__ out,
                                                        const int* __restrict__ gpos, const int* __restrict__ loc,
                                                        long long N, int C, int nC, long long work) {
  __shared__ float4 lds4[kPermChunk / 4];
  float* lds = reinterpret_cast<float*>(lds4);
  for (long long w = blockIdx.x; w < work; w += gridDim.x) {
    const long long b = w / nC, d = w % nC, base = b * N + d * C;
    const int* lc = loc + d * C;
    const float* ad = a + d * C;
    auto one = [&](int j, float uu, float gh, float av, int id) {
      const float g = (mask && !(uu > 0.f)) ? 0.f : gh;
      imgA[base + j] = uu * g;
      lds[id & (C - 1)] = g * av;
    };
    if (C % kPermStep == 0) {
      for (int j0 = threadIdx.x; j0 < C; j0 += kPermStep) {
        float uu[kPermBatch], gh[kPermBatch], av[kPermBatch];
        int id[kPermBatch];
#pragma unroll
        for (int q = 0; q < kPermBatch; ++q) {
          const int j = j0 + q * kPermThreads;
          uu[q] = u[base + j];
          gh[q] = gh1[base + j];
          av[q] = ad[j];
          id[q] = lc[j];
        }
#pragma unroll
        for (int q = 0; q < kPermBatch; ++q) one(j0 + q * kPermThreads, uu[q], gh[q], av[q], id[q]);
      }
    } else {
      for (int j = threadIdx.x; j < C; j += kPermThreads) one(j, u[base + j], gh1[base + j], ad[j], lc[j]);
    }
    __syncthreads();
    if (gpos) {
      const int* gp = gpos + d * C;
      float* orow = out + b * N;
      for (int j0 = threadIdx.x; j0 < C; j0 += kPermStep) {
        int id[kPermBatch];
#pragma unroll
        for (int q = 0; q < kPermBatch; ++q) id[q] = gp[j0 + q * kPermThreads] & (N - 1);
#pragma unroll
        for (int q = 0; q < kPermBatch; ++q) orow[id[q]] = lds[j0 + q * kPermThreads];
      }
    } else {
      chunk_from_lds(reinterpret_cast<float4*>(out + base), lds4, C);
    }
    __syncthreads();
  }
}

// Backward, second pass (the adjoint of pass A): L[srcA[cC + i]] =
// tmp[b][cC + i], then out[b][cC + i] = L[i].
template <class E>
__global__ __launch_bounds__(kPermThreads) void k_pt_at(const E* __restrict__ tmp, E* __restrict__ out,
                                                        const int* __restrict__ srcA, long long N, int C, int nC,
                                                        long long work) {
  constexpr int EW = int(sizeof(E) / sizeof(float));
  __shared__ float4 lds4[kPermChunk / 4];
  E* lds = reinterpret_cast<E*>(lds4);
  for (long long w = blockIdx.x; w < work; w += gridDim.x) {
    const long long b = w / nC, c = w % nC, base = b * N + c * C;
    const int* t = srcA + c * C;
    for (int i0 = threadIdx.x; i0 < C; i0 += kPermStep) {
      int id[kPermBatch];
      E v[kPermBatch];
#pragma unroll
      for (int q = 0; q < kPermBatch; ++q) {
        id[q] = t[i0 + q * kPermThreads] & (C - 1);
        v[q] = tmp[base + i0 + q * kPermThreads];
      }
#pragma unroll
      for (int q = 0; q < kPermBatch; ++q) lds[id[q]] = v[q];
    }
    __syncthreads();
    chunk_from_lds(reinterpret_cast<float4*>(out + base), lds4, C * EW);
    __syncthreads();
  }
}

// ------------------------------------------------------- complex (AFDF) rows
// A complex row is its own M = N point FFT input: no packing.  The steps
// follow the fused complex kernels' arithmetic (u * a, X * d / N, the
// unnormalised inverse; backward images g * conj(h) and gh1 * conj(u)).

// First DIF pass (S = M) on u * a, read from the layer input out of place
// (a may be null; with stash the input is stashed too).
template <int R>
__global__ __launch_bounds__(kThreads) void k_cdif_in(const float2* __restrict__ src, const float2* __restrict__ a,
                                                      float2* __restrict__ stash, float2* __restrict__ Z, long long B,
                                                      long long M, const float2* __restrict__ twM) {
  const long long Q = M / R, total = B * Q;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / Q, n = i % Q;
    float2 x[R];
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const long long m = b * M + n + j * Q;
      const float2 u = src[m];
      if (stash) stash[m] = u;
      x[j] = a ? cmul(u, a[n + j * Q]) : u;
    }
    Dft<R, false>::run(x);
#pragma unroll
    for (int r = 1; r < R; ++r) x[r] = cmul(x[r], twM[n * r]);
#pragma unroll
    for (int r = 0; r < R; ++r) Z[b * M + r * Q + n] = x[r];
  }
}

// Last DIT pass (S = M), written out of place to the layer output.
template <int R>
__global__ __launch_bounds__(kThreads) void k_cdit_out(const float2* __restrict__ Z, float2* __restrict__ dst,
                                                       long long B, long long M, const float2* __restrict__ twM) {
  const long long Q = M / R, total = B * Q;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / Q, n = i % Q;
    float2 y[R];
#pragma unroll
    for (int r = 0; r < R; ++r) y[r] = Z[b * M + r * Q + n];
#pragma unroll
    for (int r = 1; r < R; ++r) y[r] = cmulc(y[r], twM[n * r]);
    Dft<R, true>::run(y);
#pragma unroll
    for (int j = 0; j < R; ++j) dst[b * M + n + j * Q] = y[j];
  }
}

// Without DIF passes (one segment per row): Z = u * a (stashed), dst = Z.
__global__ __launch_bounds__(kThreads) void k_cscale(const float2* __restrict__ src, const float2* __restrict__ a,
                                                     float2* __restrict__ stash, float2* __restrict__ Z, long long B,
                                                     long long M) {
  const long long total = B * M;
  for (long long i = gindex(); i < total; i += gstride()) {
    const float2 u = src[i];
    if (stash) stash[i] = u;
    Z[i] = a ? cmul(u, a[i % M]) : u;
  }
}
__global__ __launch_bounds__(kThreads) void k_ccopy(const float2* __restrict__ Z, float2* __restrict__ dst,
                                                    long long total) {
  for (long long i = gindex(); i < total; i += gstride()) dst[i] = Z[i];
}

// Spectrum index of storage position q (the inverse of pos()).
__device__ __forceinline__ long long spec_index(const Geo& g, long long q) {
  const long long S1 = g.M / g.R1;
  const long long r1 = q / S1, rem = q % S1;
  const long long r2 = rem / g.L, k2 = rem % g.L;
  return r1 + (long long)g.R1 * (r2 + (long long)g.R2 * k2);
}

// Forward middle: X[k] *= d[k] / N, kColRows rows per thread and position.
__global__ __launch_bounds__(kThreads) void k_cmid_fwd(float2* __restrict__ Z, const float2* __restrict__ d,
                                                       long long B, Geo g, float invN) {
  const long long M = g.M, P = (B + kColRows - 1) / kColRows, total = P * M;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long p = i / M, q = i % M;
    const float2 dk = d[spec_index(g, q)];
    const float2 w = make_float2(dk.x * invN, dk.y * invN);
    const long long b0 = p * kColRows, b1 = b0 + kColRows < B ? b0 + kColRows : B;
    for (long long b = b0; b < b1; ++b) Z[b * M + q] = cmul(Z[b * M + q], w);
  }
}

// Backward middle: gh3 = FFT(g) / N, the dL/dd image gh3 * conj(h2) summed
// over blocks of kColRows rows into part[p][k] (complex, spectrum order),
// and g's spectrum replaced by gh3 * conj(d).
__global__ __launch_bounds__(kThreads) void k_cmid_bwd(const float2* __restrict__ Zh, float2* __restrict__ Zg,
                                                       const float2* __restrict__ d, long long B, Geo g, float invN,
                                                       float2* __restrict__ part) {
  const long long M = g.M, P = (B + kColRows - 1) / kColRows, total = P * M;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long p = i / M, q = i % M, k = spec_index(g, q);
    const float2 dk = d[k];
    float2 acc = make_float2(0.f, 0.f);
    const long long b0 = p * kColRows, b1 = b0 + kColRows < B ? b0 + kColRows : B;
    for (long long b = b0; b < b1; ++b) {
      const float2 gz = Zg[b * M + q];
      const float2 gh3 = make_float2(gz.x * invN, gz.y * invN);
      const float2 img = cmulc(gh3, Zh[b * M + q]);
      acc = make_float2(acc.x + img.x, acc.y + img.y);
      Zg[b * M + q] = cmulc(gh3, dk);
    }
    part[p * M + k] = acc;
  }
}

// The dL/da image gh1 * conj(u) and dL/du = gh1 * conj(a).
__global__ __launch_bounds__(kThreads) void k_cdA(const float2* __restrict__ gh1, const float2* __restrict__ u,
                                                  const float2* __restrict__ a, float2* __restrict__ imgA,
                                                  float2* __restrict__ gu, long long B, long long N) {
  const long long total = B * N;
  for (long long i = gindex(); i < total; i += gstride()) {
    const float2 gg = gh1[i];
    imgA[i] = cmulc(gg, u[i]);
    gu[i] = cmulc(gg, a[i % N]);
  }
}

// Column sums, stage 1: part[p][w] = sum of rows p*kColRows ... of img, in
// row order, four columns per thread.
__global__ __launch_bounds__(kThreads) void k_colsum1(const float* __restrict__ img, long long B, long long W,
                                                      float* __restrict__ part) {
  const long long W4 = W / 4, P = (B + kColRows - 1) / kColRows, total = P * W4;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long p = i / W4, w4 = i % W4;
    const long long b0 = p * kColRows, b1 = b0 + kColRows < B ? b0 + kColRows : B;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    const float4* col = reinterpret_cast<const float4*>(img) + w4;
#pragma unroll 4
    for (long long b = b0; b < b1; ++b) {
      const float4 v = col[b * W4];
      s = make_float4(s.x + v.x, s.y + v.y, s.z + v.z, s.w + v.w);
    }
    reinterpret_cast<float4*>(part)[p * W4 + w4] = s;
  }
}

// Stage 2: the block sums in block order, stored (or added) to the output.
__global__ __launch_bounds__(kThreads) void k_colsum2(const float* __restrict__ part, long long P, long long W,
                                                      float* __restrict__ out, QuartetTabs q, int quartet,
                                                      int accumulate) {
  for (long long w = gindex(); w < W; w += gstride()) {
    float s = 0.f;
    for (long long p = 0; p < P; ++p) s += part[p * W + w];
    long long o = w;
    if (quartet) {
      const long long e = w / 4;
      const int j = int(w % 4);
      if (!((q.qmask[e] >> (4 + j)) & 1)) continue;
      const int4 idx = q.qidx[e];
      o = j == 0 ? idx.x : j == 1 ? idx.y : j == 2 ? idx.z : idx.w;
    }
    out[o] = accumulate ? out[o] + s : s;
  }
}

template <class F>
bool with_seg_plan(int L, F&& f) {
  switch (L) {
    case 128: f.template operator()<CP128>(); return true;
    case 256: f.template operator()<CP256>(); return true;
    case 512: f.template operator()<CP512>(); return true;
    case 1024: f.template operator()<CP1024>(); return true;
    case 2048: f.template operator()<CP2048>(); return true;
    case 4096: f.template operator()<CP4096>(); return true;
    case 8192: f.template operator()<CP8192>(); return true;
    default: return false;
  }
}

}  // namespace

hipError_t pack(const float* src, const float* a, float* stash, float2* Z, long long B, long long N, hipStream_t s) {
  hipLaunchKernelGGL(k_pack, grid_for(B * (N / 4)), dim3(kThreads), 0, s, src, a, stash, Z, B, N);
  return hipGetLastError();
}

hipError_t dif(float2* Z, long long B, const Geo& g, long long S, int R, const float2* twM, hipStream_t s) {
  const dim3 grid = grid_for(B * (g.M / R)), block(kThreads);
  switch (R) {
    case 2: hipLaunchKernelGGL(k_dif<2>, grid, block, 0, s, Z, B, g.M, S, twM); break;
    case 4: hipLaunchKernelGGL(k_dif<4>, grid, block, 0, s, Z, B, g.M, S, twM); break;
    case 8: hipLaunchKernelGGL(k_dif<8>, grid, block, 0, s, Z, B, g.M, S, twM); break;
    case 16: hipLaunchKernelGGL(k_dif<16>, grid, block, 0, s, Z, B, g.M, S, twM); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t dit(float2* Z, long long B, const Geo& g, long long S, int R, const float2* twM, hipStream_t s) {
  const dim3 grid = grid_for(B * (g.M / R)), block(kThreads);
  switch (R) {
    case 2: hipLaunchKernelGGL(k_dit<2>, grid, block, 0, s, Z, B, g.M, S, twM); break;
    case 4: hipLaunchKernelGGL(k_dit<4>, grid, block, 0, s, Z, B, g.M, S, twM); break;
    case 8: hipLaunchKernelGGL(k_dit<8>, grid, block, 0, s, Z, B, g.M, S, twM); break;
    case 16: hipLaunchKernelGGL(k_dit<16>, grid, block, 0, s, Z, B, g.M, S, twM); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t pack_dif(const float* src, const float* a, float* stash, float2* Z, long long B, long long M, int R,
                    const float2* twM, hipStream_t s) {
  const dim3 grid = grid_for(B * (M / R / 2)), block(kThreads);
  switch (R) {
    case 2: hipLaunchKernelGGL(k_pack_dif<2>, grid, block, 0, s, src, a, stash, Z, B, M, twM); break;
    case 4: hipLaunchKernelGGL(k_pack_dif<4>, grid, block, 0, s, src, a, stash, Z, B, M, twM); break;
    case 8: hipLaunchKernelGGL(k_pack_dif<8>, grid, block, 0, s, src, a, stash, Z, B, M, twM); break;
    case 16: hipLaunchKernelGGL(k_pack_dif<16>, grid, block, 0, s, src, a, stash, Z, B, M, twM); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t dit_unpack(const float2* Z, float* dst, long long B, long long M, int R, const float2* twM, bool relu,
                      hipStream_t s) {
  const dim3 grid = grid_for(B * (M / R / 2)), block(kThreads);
  const int rl = relu ? 1 : 0;
  switch (R) {
    case 2: hipLaunchKernelGGL(k_dit_unpack<2>, grid, block, 0, s, Z, dst, B, M, twM, rl); break;
    case 4: hipLaunchKernelGGL(k_dit_unpack<4>, grid, block, 0, s, Z, dst, B, M, twM, rl); break;
    case 8: hipLaunchKernelGGL(k_dit_unpack<8>, grid, block, 0, s, Z, dst, B, M, twM, rl); break;
    case 16: hipLaunchKernelGGL(k_dit_unpack<16>, grid, block, 0, s, Z, dst, B, M, twM, rl); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t segments(float2* Z, long long nseg, int L, bool inverse, const char* seg_tab, hipStream_t s) {
  bool ok = with_seg_plan(L, [&]<class CP>() {
    using LC = Launch<CP>;
    const dim3 grid(unsigned((nseg + LC::FWD_ROWS - 1) / LC::FWD_ROWS));
    if (inverse) hipLaunchKernelGGL((k_seg<CP, true>), grid, dim3(LC::FWD_THREADS), 0, s, Z, nseg, seg_tab);
    else hipLaunchKernelGGL((k_seg<CP, false>), grid, dim3(LC::FWD_THREADS), 0, s, Z, nseg, seg_tab);
  });
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t mq(const float* D, const float* Bias, float4* Mq, int K, long long NQ, const QuartetTabs& q,
              hipStream_t s) {
  hipLaunchKernelGGL(k_mq, grid_for((long long)K * NQ), dim3(kThreads), 0, s, D, Bias, Mq, K, NQ, q, 4 * NQ);
  return hipGetLastError();
}

hipError_t mid_fwd(float2* Z, const float4* Mq, long long B, const Geo& g, bool bias, hipStream_t s) {
  const long long P = (B + kColRows - 1) / kColRows;
  hipLaunchKernelGGL(k_mid_fwd, grid_for(P * (g.M / 2)), dim3(kThreads), 0, s, Z, Mq, B, g, bias ? 1 : 0);
  return hipGetLastError();
}

hipError_t mid_bwd(const float2* Zh, float2* Zg, const float4* Mq, long long B, const Geo& g, float* partD,
                   float* partB, hipStream_t s) {
  const long long P = (B + kColRows - 1) / kColRows;
  hipLaunchKernelGGL(k_mid_bwd, grid_for(P * (g.M / 2)), dim3(kThreads), 0, s, Zh, Zg, Mq, B, g, partD, partB);
  return hipGetLastError();
}

hipError_t unpack(const float2* Z, float* dst, long long B, long long N, bool relu, hipStream_t s) {
  hipLaunchKernelGGL(k_unpack, grid_for(B * (N / 4)), dim3(kThreads), 0, s, Z, dst, B, N, relu ? 1 : 0);
  return hipGetLastError();
}

hipError_t dA(const float* gh1, const float* u, const float* a, bool mask, float* imgA, float* gnext, long long B,
              long long N, hipStream_t s) {
  hipLaunchKernelGGL(k_dA, grid_for(B * N), dim3(kThreads), 0, s, gh1, u, a, mask ? 1 : 0, imgA, gnext, B, N);
  return hipGetLastError();
}

PermGeo perm_geo(long long N, int ew) {
  const long long cap = kPermChunk / ew;
  PermGeo p;
  p.C = int(N < cap ? N : cap);
  p.nC = int(N / p.C);
  return p;
}

size_t perm_table_ints(long long N, int ew) {
  const PermGeo p = perm_geo(N, ew);
  if (p.nC == 1) return 0;
  return size_t(3 * N + 2 * (N / kThreads) * p.nC + 3LL * p.nC * p.nC);
}

PermTabs perm_tables_at(int* base, long long N, int ew) {
  const PermGeo p = perm_geo(N, ew);
  PermTabs t;
  if (p.nC == 1) return t;
  t.stride = (long long)perm_table_ints(N, ew);
  const long long nb = N / kThreads, nn = (long long)p.nC * p.nC;
  t.srcA = base;
  t.gposB = t.srcA + N;
  t.locB = t.gposB + N;
  t.cntS = t.locB + N;
  t.bpre = t.cntS + nb * p.nC;
  t.cnt = t.bpre + nb * p.nC;
  t.off = t.cnt + nn;
  t.lst = t.off + nn;
  return t;
}

PermTabs perm_layer(const PermTabs& t, int l) {
  if (t.srcA == nullptr) return t;
  const long long o = l * t.stride;
  PermTabs r = t;
  r.srcA += o;
  r.gposB += o;
  r.locB += o;
  r.cntS += o;
  r.bpre += o;
  r.cnt += o;
  r.off += o;
  r.lst += o;
  return r;
}

hipError_t perm_build(const int* perm, long long N, int layers, const PermTabs& t, hipStream_t s, int ew) {
  const PermGeo p = perm_geo(N, ew);
  if (p.nC == 1 || layers <= 0) return hipSuccess;
  const unsigned nb = unsigned(N / kThreads), nn = unsigned(p.nC * p.nC), L = unsigned(layers);
  hipLaunchKernelGGL(k_pt_count, dim3(nb, L), dim3(kThreads), 0, s, perm, N, p.C, p.nC, t.cntS, t.stride);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_pt_blocks, dim3((nn + kThreads - 1) / kThreads, L), dim3(kThreads), 0, s, t.cntS, p.C, p.nC,
                     t.bpre, t.cnt, t.stride);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_pt_offsets, dim3(L), dim3(kThreads), 0, s, t.cnt, p.C, p.nC, t.off, t.lst, t.stride);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_pt_place, dim3(nb, L), dim3(kThreads), 0, s, perm, N, p.C, p.nC, t.bpre, t.off, t.lst,
                     t.srcA, t.gposB, t.locB, t.stride);
  return hipGetLastError();
}

namespace {
dim3 perm_grid(long long work) { return dim3(unsigned(work < 65536 ? (work < 1 ? 1 : work) : 65536)); }
}  // namespace

hipError_t permute(const float* in, float* out, float* tmp, const int* perm, const PermTabs& t, long long B,
                   long long N, hipStream_t s) {
  const PermGeo p = perm_geo(N, 1);
  const long long work = B * p.nC;
  if (p.nC == 1) {
    hipLaunchKernelGGL(k_pt_a<float>, perm_grid(work), dim3(kPermThreads), 0, s, in, out, perm, N, p.C, p.nC, work);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_pt_a<float>, perm_grid(work), dim3(kPermThreads), 0, s, in, tmp, t.srcA, N, p.C, p.nC, work);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_pt_b<float>, perm_grid(work), dim3(kPermThreads), 0, s, tmp, out, t.gposB, t.locB, N, p.C, p.nC,
                     work);
  return hipGetLastError();
}

hipError_t dA_permute(const float* gh1, const float* u, const float* a, bool mask, float* imgA, float* gnext,
                      float* tmp, const int* perm, const PermTabs& t, long long B, long long N, hipStream_t s) {
  const PermGeo p = perm_geo(N, 1);
  const long long work = B * p.nC;
  const int mk = mask ? 1 : 0;
  if (p.nC == 1) {
    hipLaunchKernelGGL(k_pt_bt, perm_grid(work), dim3(kPermThreads), 0, s, gh1, u, a, mk, imgA, gnext,
                       static_cast<const int*>(nullptr), perm, N, p.C, p.nC, work);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_pt_bt, perm_grid(work), dim3(kPermThreads), 0, s, gh1, u, a, mk, imgA, tmp, t.gposB, t.locB,
                     N, p.C, p.nC, work);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_pt_at<float>, perm_grid(work), dim3(kPermThreads), 0, s, tmp, gnext, t.srcA, N, p.C, p.nC, work);
  return hipGetLastError();
}

// ---------------------------------------------------------- complex launchers
hipError_t cpermute(const float2* in, float2* out, float2* tmp, const int* perm, const PermTabs& t, long long B,
                    long long N, hipStream_t s) {
  const PermGeo p = perm_geo(N, 2);
  const long long work = B * p.nC;
  if (p.nC == 1) {
    hipLaunchKernelGGL(k_pt_a<float2>, perm_grid(work), dim3(kPermThreads), 0, s, in, out, perm, N, p.C, p.nC, work);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_pt_a<float2>, perm_grid(work), dim3(kPermThreads), 0, s, in, tmp, t.srcA, N, p.C, p.nC, work);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_pt_b<float2>, perm_grid(work), dim3(kPermThreads), 0, s, tmp, out, t.gposB, t.locB, N, p.C,
                     p.nC, work);
  return hipGetLastError();
}

hipError_t cpermute_adjoint(const float2* in, float2* out, float2* tmp, const int* perm, const PermTabs& t,
                            long long B, long long N, hipStream_t s) {
  const PermGeo p = perm_geo(N, 2);
  const long long work = B * p.nC;
  if (p.nC == 1) {
    hipLaunchKernelGGL(k_pt_btp<float2>, perm_grid(work), dim3(kPermThreads), 0, s, in, out,
                       static_cast<const int*>(nullptr), perm, N, p.C, p.nC, work);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_pt_btp<float2>, perm_grid(work), dim3(kPermThreads), 0, s, in, tmp, t.gposB, t.locB, N, p.C,
                     p.nC, work);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_pt_at<float2>, perm_grid(work), dim3(kPermThreads), 0, s, tmp, out, t.srcA, N, p.C, p.nC,
                     work);
  return hipGetLastError();
}

hipError_t cfft_in(const float2* src, const float2* a, float2* stash, float2* Z, long long B, const Geo& g,
                   const float2* twM, const char* seg_tab, hipStream_t s) {
  const dim3 block(kThreads);
  if (g.R1 > 1) {
    const dim3 grid = grid_for(B * (g.M / g.R1));
    switch (g.R1) {
      case 2: hipLaunchKernelGGL(k_cdif_in<2>, grid, block, 0, s, src, a, stash, Z, B, g.M, twM); break;
      case 4: hipLaunchKernelGGL(k_cdif_in<4>, grid, block, 0, s, src, a, stash, Z, B, g.M, twM); break;
      case 8: hipLaunchKernelGGL(k_cdif_in<8>, grid, block, 0, s, src, a, stash, Z, B, g.M, twM); break;
      case 16: hipLaunchKernelGGL(k_cdif_in<16>, grid, block, 0, s, src, a, stash, Z, B, g.M, twM); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    hipLaunchKernelGGL(k_cscale, grid_for(B * g.M), block, 0, s, src, a, stash, Z, B, g.M);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (g.R2 > 1 && (e = dif(Z, B, g, g.M / g.R1, g.R2, twM, s)) != hipSuccess) return e;
  return segments(Z, B * (g.M / g.L), g.L, false, seg_tab, s);
}

hipError_t cifft_out(float2* Z, float2* dst, long long B, const Geo& g, const float2* twM, const char* seg_tab,
                     hipStream_t s) {
  hipError_t e = segments(Z, B * (g.M / g.L), g.L, true, seg_tab, s);
  if (e != hipSuccess) return e;
  if (g.R2 > 1 && (e = dit(Z, B, g, g.M / g.R1, g.R2, twM, s)) != hipSuccess) return e;
  const dim3 block(kThreads);
  if (g.R1 > 1) {
    const dim3 grid = grid_for(B * (g.M / g.R1));
    switch (g.R1) {
      case 2: hipLaunchKernelGGL(k_cdit_out<2>, grid, block, 0, s, Z, dst, B, g.M, twM); break;
      case 4: hipLaunchKernelGGL(k_cdit_out<4>, grid, block, 0, s, Z, dst, B, g.M, twM); break;
      case 8: hipLaunchKernelGGL(k_cdit_out<8>, grid, block, 0, s, Z, dst, B, g.M, twM); break;
      case 16: hipLaunchKernelGGL(k_cdit_out<16>, grid, block, 0, s, Z, dst, B, g.M, twM); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    hipLaunchKernelGGL(k_ccopy, grid_for(B * g.M), block, 0, s, Z, dst, B * g.M);
  }
  return hipGetLastError();
}

hipError_t cmid_fwd(float2* Z, const float2* d, long long B, const Geo& g, float invN, hipStream_t s) {
  const long long P = (B + kColRows - 1) / kColRows;
  hipLaunchKernelGGL(k_cmid_fwd, grid_for(P * g.M), dim3(kThreads), 0, s, Z, d, B, g, invN);
  return hipGetLastError();
}

hipError_t cmid_bwd(const float2* Zh, float2* Zg, const float2* d, long long B, const Geo& g, float invN,
                    float2* part, hipStream_t s) {
  const long long P = (B + kColRows - 1) / kColRows;
  hipLaunchKernelGGL(k_cmid_bwd, grid_for(P * g.M), dim3(kThreads), 0, s, Zh, Zg, d, B, g, invN, part);
  return hipGetLastError();
}

hipError_t cdA(const float2* gh1, const float2* u, const float2* a, float2* imgA, float2* gu, long long B,
               long long N, hipStream_t s) {
  hipLaunchKernelGGL(k_cdA, grid_for(B * N), dim3(kThreads), 0, s, gh1, u, a, imgA, gu, B, N);
  return hipGetLastError();
}

hipError_t colsum_parts(const float* part, long long B, long long W, float* out, const QuartetTabs* q,
                        bool accumulate, hipStream_t s) {
  const long long P = (B + kColRows - 1) / kColRows;
  const QuartetTabs qq = q ? *q : QuartetTabs{};
  hipLaunchKernelGGL(k_colsum2, grid_for(W), dim3(kThreads), 0, s, part, P, W, out, qq, q ? 1 : 0,
                     accumulate ? 1 : 0);
  return hipGetLastError();
}

hipError_t colsum(const float* img, long long B, long long W, float* part, float* out, const QuartetTabs* q,
                  bool accumulate, hipStream_t s) {
  const long long P = (B + kColRows - 1) / kColRows;
  if (P > 0) {
    hipLaunchKernelGGL(k_colsum1, grid_for(P * (W / 4)), dim3(kThreads), 0, s, img, B, W, part);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return colsum_parts(part, B, W, out, q, accumulate, s);
}

}  // namespace mp
}  // namespace acdc
