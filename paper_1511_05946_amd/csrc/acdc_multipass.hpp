// Multi-pass ACDC layers: the M = N/2 point FFT of each row runs through HBM
// in several kernel launches (the multiple-call implementation of Sec. 5.2,
// with hand-written passes in place of a vendor FFT).  Used for widths past
// the fused kernels' on-chip limit, or when ACDC_FLAG_MULTIPASS asks for it.
//
// Per layer and row, the steps of the fused kernels, one launch each:
//   pack     u = z[perm] (stashed for the backward), h1 = u * a, Makhoul's
//            even/odd-reversed packing into M complex values
//   DIF      zero, one or two radix-R passes (R <= 16) that split the M-point
//            FFT into segments of L <= 8192 points, each with its twiddle
//   segment  the L-point FFTs, one per workgroup, in registers and LDS
//   middle   per quartet: real-FFT split, post-twiddle, * d (+ b), DCT-III
//            pre-twiddle and inverse split (the fused kernels' quartet maps)
//   inverse  segment IFFTs, then the DIT passes in reverse
//   unpack   the inverse packing, ReLU, the layer output
// The spectrum stays in the digit-reversed order the DIF passes leave it in;
// the middle addresses it through pos() below.  The backward adds images of
// dL/dd, dL/da (and dL/db) per row, summed over the batch by fixed-order
// column sums.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "acdc_registry.hpp"

namespace acdc {
namespace mp {

// Geometry of one row's M-point FFT: M = R1 * R2 * L, R1, R2 in {1, 2, 4,
// 8, 16} (1 = no pass), L the in-LDS segment length.
struct Geo {
  long long M;
  int L, R1, R2;
};

// Storage position of spectrum value Z[k] after the DIF passes and the
// segment FFTs: k = r1 + R1 (r2 + R2 k2) sits at r1 (M/R1) + r2 L + k2.
__host__ __device__ __forceinline__ long long pos(const Geo& g, long long k) {
  const long long r1 = k % g.R1, j = k / g.R1;
  const long long r2 = j % g.R2, k2 = j / g.R2;
  return r1 * (g.M / g.R1) + r2 * g.L + k2;
}

// Makhoul packing: complex value m of a row holds the reals at spatial
// indices (4m, 4m+2) for m < M/2 and (4m'+3, 4m'+1), m' = M-1-m, otherwise.
__host__ __device__ __forceinline__ void pack_idx(long long m, long long M, long long& i0, long long& i1) {
  if (m < M / 2) {
    i0 = 4 * m;
    i1 = 4 * m + 2;
  } else {
    const long long q = M - 1 - m;
    i0 = 4 * q + 3;
    i1 = 4 * q + 1;
  }
}

// Launchers (acdc_multipass.hip).  All pointers are device pointers; every
// launcher enqueues on `s` and returns the launch status.  Index arrays
// (perm) are masked to [0, N), so a malformed permutation cannot address
// outside its row.
hipError_t pack(const float* src, const int* perm, const float* a, float* stash, float2* Z, long long B, long long N,
                hipStream_t s);
hipError_t dif(float2* Z, long long B, const Geo& g, long long S, int R, const float2* twM, hipStream_t s);
hipError_t dit(float2* Z, long long B, const Geo& g, long long S, int R, const float2* twM, hipStream_t s);
hipError_t segments(float2* Z, long long nseg, int L, bool inverse, const char* seg_tab, hipStream_t s);
// pack + the first DIF pass (radix R on whole rows), and the last DIT pass +
// unpack (+ ReLU): the same results as the separate launches, two passes
// over the batch fewer.
hipError_t pack_dif(const float* src, const int* perm, const float* a, float* stash, float2* Z, long long B,
                    long long M, int R, const float2* twM, hipStream_t s);
hipError_t dit_unpack(const float2* Z, float* dst, long long B, long long M, int R, const float2* twM, bool relu,
                      hipStream_t s);
hipError_t mq(const float* D, const float* Bias, float4* Mq, int K, long long NQ, const QuartetTabs& q,
              hipStream_t s);
hipError_t mid_fwd(float2* Z, const float4* Mq, long long B, const Geo& g, bool bias, hipStream_t s);
hipError_t mid_bwd(const float2* Zh, float2* Zg, const float4* Mq, long long B, const Geo& g, float* imgD,
                   float* imgB, hipStream_t s);
hipError_t unpack(const float2* Z, float* dst, long long B, long long N, bool relu, hipStream_t s);
hipError_t dA(const float* gh1, const float* u, const float* a, const int* perm, bool mask, float* imgA, float* gnext,
              long long B, long long N, hipStream_t s);
// out[w] (+)= sum over rows of img[b][w] in row order (blocks of kColRows
// rows, then the block sums in block order); with q, column w = 4e + j is
// the quartet value j of entry e, stored to its DCT index.
constexpr int kColRows = 64;
hipError_t colsum(const float* img, long long B, long long W, float* part, float* out, const QuartetTabs* q,
                  bool accumulate, hipStream_t s);

}  // namespace mp
}  // namespace acdc
