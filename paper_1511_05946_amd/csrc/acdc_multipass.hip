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

__global__ __launch_bounds__(kThreads) void k_pack(const float* __restrict__ src, const int* __restrict__ perm,
                                                   const float* __restrict__ a, float* __restrict__ stash,
                                                   float2* __restrict__ Z, long long B, long long N) {
  const long long M = N / 2, total = B * M;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / M, m = i % M;
    long long i0, i1;
    pack_idx(m, M, i0, i1);
    const float* row = src + b * N;
    float u0 = row[perm ? (perm[i0] & (N - 1)) : i0];
    float u1 = row[perm ? (perm[i1] & (N - 1)) : i1];
    if (stash) {
      stash[b * N + i0] = u0;
      stash[b * N + i1] = u1;
    }
    if (a) {
      u0 *= a[i0];
      u1 *= a[i1];
    }
    Z[i] = make_float2(u0, u1);
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

// The first DIF pass (on whole rows, S = M) with the packing folded in:
// butterfly n gathers, scales and packs its R inputs m = n + j M/R straight
// from the spatial rows (stashing the gathered values), saving one pass.
__device__ __forceinline__ float2 packed_value(const float* row, const int* perm, const float* a, float* srow,
                                               long long m, long long M, long long N) {
  long long i0, i1;
  pack_idx(m, M, i0, i1);
  float u0 = row[perm ? (perm[i0] & (N - 1)) : i0];
  float u1 = row[perm ? (perm[i1] & (N - 1)) : i1];
  if (srow) {
    srow[i0] = u0;
    srow[i1] = u1;
  }
  if (a) {
    u0 *= a[i0];
    u1 *= a[i1];
  }
  return make_float2(u0, u1);
}

template <int R>
__global__ __launch_bounds__(kThreads) void k_pack_dif(const float* __restrict__ src, const int* __restrict__ perm,
                                                       const float* __restrict__ a, float* __restrict__ stash,
                                                       float2* __restrict__ Z, long long B, long long M,
                                                       const float2* __restrict__ twM) {
  const long long N = 2 * M, Q = M / R, total = B * Q;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / Q, n = i % Q;
    const float* row = src + b * N;
    float* srow = stash ? stash + b * N : nullptr;
    float2 x[R];
#pragma unroll
    for (int j = 0; j < R; ++j) x[j] = packed_value(row, perm, a, srow, n + j * Q, M, N);
    Dft<R, false>::run(x);
#pragma unroll
    for (int r = 1; r < R; ++r) x[r] = cmul(x[r], twM[n * r]);
#pragma unroll
    for (int r = 0; r < R; ++r) Z[b * M + r * Q + n] = x[r];
  }
}

// The last DIT pass (S = M) with the unpacking (and ReLU) folded in.
template <int R>
__global__ __launch_bounds__(kThreads) void k_dit_unpack(const float2* __restrict__ Z, float* __restrict__ dst,
                                                         long long B, long long M, const float2* __restrict__ twM,
                                                         int relu) {
  const long long N = 2 * M, Q = M / R, total = B * Q;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / Q, n = i % Q;
    float2 y[R];
#pragma unroll
    for (int r = 0; r < R; ++r) y[r] = Z[b * M + r * Q + n];
#pragma unroll
    for (int r = 1; r < R; ++r) y[r] = cmulc(y[r], twM[n * r]);
    Dft<R, true>::run(y);
    float* row = dst + b * N;
#pragma unroll
    for (int j = 0; j < R; ++j) {
      long long i0, i1;
      pack_idx(n + j * Q, M, i0, i1);
      row[i0] = relu ? (y[j].x > 0.f ? y[j].x : 0.f) : y[j].x;
      row[i1] = relu ? (y[j].y > 0.f ? y[j].y : 0.f) : y[j].y;
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
  if constexpr (!INV) {
    O::for_spatial(v, t, [&](unsigned l, unsigned c, float2& z) { z = g.ld2((l + roff) * 8u, c * 8u); });
    O::template fft<false>(ctx, v, t, slab, GView::of(tab));
    if (valid) O::for_freq(v, t, [&](unsigned l, unsigned c, float2& z) { g.st2(z, (l + roff) * 8u, c * 8u); });
  } else {
    O::for_freq(v, t, [&](unsigned l, unsigned c, float2& z) { z = g.ld2((l + roff) * 8u, c * 8u); });
    O::template fft<true>(ctx, v, t, slab, GView::of(tab));
    if (valid) O::for_spatial(v, t, [&](unsigned l, unsigned c, float2& z) { g.st2(z, (l + roff) * 8u, c * 8u); });
  }
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

__global__ __launch_bounds__(kThreads) void k_mid_fwd(float2* __restrict__ Z, const float4* __restrict__ Mq,
                                                      long long B, Geo g, int bias) {
  const long long NQ = g.M / 2, total = B * NQ;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / NQ, e = i % NQ;
    long long pa, pb;
    pair_pos(g, e, pa, pb);
    float2* row = Z + b * g.M;
    float2 zk = row[pa], zm = row[pb];
    const float4 c0 = Mq[e * kMqRows], c1 = Mq[e * kMqRows + 1];
    quartet_back(quartet_split(zk, zm, make_float2(c1.z, c1.w)), c0, c1, zk, zm);
    if (bias) {
      const float4 c3 = Mq[e * kMqRows + 3];
      zk = make_float2(zk.x + c3.x, zk.y + c3.y);
      zm = make_float2(zm.x + c3.z, zm.y + c3.w);
    }
    row[pa] = zk;
    row[pb] = zm;
  }
}

// Backward middle: images H*G (dL/dd) and, with a bias, G (dL/db) in
// quartet order [b][4e + j]; g's spectrum is replaced by the DCT-III
// pre-twiddle of G*d.
__global__ __launch_bounds__(kThreads) void k_mid_bwd(const float2* __restrict__ Zh, float2* __restrict__ Zg,
                                                      const float4* __restrict__ Mq, long long B, Geo g,
                                                      float* __restrict__ imgD, float* __restrict__ imgB) {
  const long long NQ = g.M / 2, total = B * NQ, W = 2 * g.M;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / NQ, e = i % NQ;
    long long pa, pb;
    pair_pos(g, e, pa, pb);
    const float2* hrow = Zh + b * g.M;
    float2* grow = Zg + b * g.M;
    float2 gk = grow[pa], gm = grow[pb];
    const float4 c0 = Mq[e * kMqRows], c1 = Mq[e * kMqRows + 1], c2 = Mq[e * kMqRows + 2];
    const float2 w = make_float2(c1.z, c1.w), qa = make_float2(c2.x, c2.y), qbr = make_float2(c2.z, c2.w);
    float H[4], G[4];
    quartet_post(quartet_split(hrow[pa], hrow[pb], w), qa, qbr, H);
    const Split sg = quartet_split(gk, gm, w);
    quartet_post(sg, qa, qbr, G);
    float4* d4 = reinterpret_cast<float4*>(imgD + b * W) + e;
    *d4 = make_float4(H[0] * G[0], H[1] * G[1], H[2] * G[2], H[3] * G[3]);
    if (imgB) *(reinterpret_cast<float4*>(imgB + b * W) + e) = make_float4(G[0], -G[1], G[2], G[3]);
    quartet_back(sg, c0, c1, gk, gm);
    grow[pa] = gk;
    grow[pb] = gm;
  }
}

__global__ __launch_bounds__(kThreads) void k_unpack(const float2* __restrict__ Z, float* __restrict__ dst,
                                                     long long B, long long N, int relu) {
  const long long M = N / 2, total = B * M;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / M, m = i % M;
    long long i0, i1;
    pack_idx(m, M, i0, i1);
    const float2 z = Z[i];
    dst[b * N + i0] = relu ? (z.x > 0.f ? z.x : 0.f) : z.x;
    dst[b * N + i1] = relu ? (z.y > 0.f ? z.y : 0.f) : z.y;
  }
}

// dL/da image u * gh1 (gh1 masked where the previous layer's ReLU was off:
// u = 0 there), and dL/du = gh1 * a scattered back through the gather.
__global__ __launch_bounds__(kThreads) void k_dA(const float* __restrict__ gh1, const float* __restrict__ u,
                                                 const float* __restrict__ a, const int* __restrict__ perm,
                                                 int mask, float* __restrict__ imgA, float* __restrict__ gnext,
                                                 long long B, long long N) {
  const long long total = B * N;
  for (long long i = gindex(); i < total; i += gstride()) {
    const long long b = i / N, n = i % N;
    const float uu = u[i];
    float gh = gh1[i];
    if (mask && !(uu > 0.f)) gh = 0.f;
    imgA[i] = uu * gh;
    gnext[b * N + (perm ? (perm[n] & (N - 1)) : n)] = gh * a[n];
  }
}

// Column sums, stage 1: part[p][w] = sum of rows p*kColRows ... of img.
__global__ __launch_bounds__(kThreads) void k_colsum1(const float* __restrict__ img, long long B, long long W,
                                                      float* __restrict__ part) {
  const long long w = (long long)blockIdx.x * kThreads + threadIdx.x;
  const long long p = blockIdx.y;
  if (w >= W) return;
  const long long b0 = p * kColRows;
  const long long b1 = b0 + kColRows < B ? b0 + kColRows : B;
  float s = 0.f;
  for (long long b = b0; b < b1; ++b) s += img[b * W + w];
  part[p * W + w] = s;
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

hipError_t pack(const float* src, const int* perm, const float* a, float* stash, float2* Z, long long B, long long N,
                hipStream_t s) {
  hipLaunchKernelGGL(k_pack, grid_for(B * (N / 2)), dim3(kThreads), 0, s, src, perm, a, stash, Z, B, N);
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

hipError_t pack_dif(const float* src, const int* perm, const float* a, float* stash, float2* Z, long long B,
                    long long M, int R, const float2* twM, hipStream_t s) {
  const dim3 grid = grid_for(B * (M / R)), block(kThreads);
  switch (R) {
    case 2: hipLaunchKernelGGL(k_pack_dif<2>, grid, block, 0, s, src, perm, a, stash, Z, B, M, twM); break;
    case 4: hipLaunchKernelGGL(k_pack_dif<4>, grid, block, 0, s, src, perm, a, stash, Z, B, M, twM); break;
    case 8: hipLaunchKernelGGL(k_pack_dif<8>, grid, block, 0, s, src, perm, a, stash, Z, B, M, twM); break;
    case 16: hipLaunchKernelGGL(k_pack_dif<16>, grid, block, 0, s, src, perm, a, stash, Z, B, M, twM); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t dit_unpack(const float2* Z, float* dst, long long B, long long M, int R, const float2* twM, bool relu,
                      hipStream_t s) {
  const dim3 grid = grid_for(B * (M / R)), block(kThreads);
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
  hipLaunchKernelGGL(k_mid_fwd, grid_for(B * (g.M / 2)), dim3(kThreads), 0, s, Z, Mq, B, g, bias ? 1 : 0);
  return hipGetLastError();
}

hipError_t mid_bwd(const float2* Zh, float2* Zg, const float4* Mq, long long B, const Geo& g, float* imgD,
                   float* imgB, hipStream_t s) {
  hipLaunchKernelGGL(k_mid_bwd, grid_for(B * (g.M / 2)), dim3(kThreads), 0, s, Zh, Zg, Mq, B, g, imgD, imgB);
  return hipGetLastError();
}

hipError_t unpack(const float2* Z, float* dst, long long B, long long N, bool relu, hipStream_t s) {
  hipLaunchKernelGGL(k_unpack, grid_for(B * (N / 2)), dim3(kThreads), 0, s, Z, dst, B, N, relu ? 1 : 0);
  return hipGetLastError();
}

hipError_t dA(const float* gh1, const float* u, const float* a, const int* perm, bool mask, float* imgA, float* gnext,
              long long B, long long N, hipStream_t s) {
  hipLaunchKernelGGL(k_dA, grid_for(B * N), dim3(kThreads), 0, s, gh1, u, a, perm, mask ? 1 : 0, imgA, gnext, B, N);
  return hipGetLastError();
}

hipError_t colsum(const float* img, long long B, long long W, float* part, float* out, const QuartetTabs* q,
                  bool accumulate, hipStream_t s) {
  const long long P = (B + kColRows - 1) / kColRows;
  if (P > 0) {
    hipLaunchKernelGGL(k_colsum1, dim3(unsigned((W + kThreads - 1) / kThreads), unsigned(P)), dim3(kThreads), 0, s,
                       img, B, W, part);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const QuartetTabs qq = q ? *q : QuartetTabs{};
  hipLaunchKernelGGL(k_colsum2, grid_for(W), dim3(kThreads), 0, s, part, P, W, out, qq, q ? 1 : 0,
                     accumulate ? 1 : 0);
  return hipGetLastError();
}

}  // namespace mp
}  // namespace acdc
