// Multi-pass ACDC layers: the M = N/2 point FFT of each row runs through HBM
// in several kernel launches (the multiple-call implementation of Sec. 5.2,
// with hand-written passes in place of a vendor FFT).  Used for widths past
// the fused kernels' on-chip limit, or when ACDC_FLAG_MULTIPASS asks for it.
//
// Per layer and row, the steps of the fused kernels, one launch each:
//   permute  u = z[perm] (into the stash slot for the backward), through LDS
//            chunks, below
//   pack     h1 = u * a, Makhoul's even/odd-reversed packing into M complex
//            values (folded into the first DIF pass when there is one)
//   DIF      zero, one or two radix-R passes (R <= 16) that split the M-point
//            FFT into segments of L <= 8192 points, each with its twiddle
//   segment  the L-point FFTs, one per workgroup, in registers and LDS
//   middle   per quartet: real-FFT split, post-twiddle, * d (+ b), DCT-III
//            pre-twiddle and inverse split (the fused kernels' quartet maps)
//   inverse  segment IFFTs, then the DIT passes in reverse
//   unpack   the inverse packing, ReLU, the layer output (folded into the
//            last DIT pass when there is one)
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
// (perm and the tables built from it) are masked into range, so a malformed
// permutation cannot address outside its row.
hipError_t pack(const float* src, const float* a, float* stash, float2* Z, long long B, long long N, hipStream_t s);
hipError_t dif(float2* Z, long long B, const Geo& g, long long S, int R, const float2* twM, hipStream_t s);
hipError_t dit(float2* Z, long long B, const Geo& g, long long S, int R, const float2* twM, hipStream_t s);
hipError_t segments(float2* Z, long long nseg, int L, bool inverse, const char* seg_tab, hipStream_t s);
// pack + the first DIF pass (radix R on whole rows), and the last DIT pass +
// unpack (+ ReLU): the same results as the separate launches, two passes
// over the batch fewer.
hipError_t pack_dif(const float* src, const float* a, float* stash, float2* Z, long long B, long long M, int R,
                    const float2* twM, hipStream_t s);
hipError_t dit_unpack(const float2* Z, float* dst, long long B, long long M, int R, const float2* twM, bool relu,
                      hipStream_t s);
hipError_t mq(const float* D, const float* Bias, float4* Mq, int K, long long NQ, const QuartetTabs& q,
              hipStream_t s);
hipError_t mid_fwd(float2* Z, const float4* Mq, long long B, const Geo& g, bool bias, hipStream_t s);
// The backward middle also sums the dL/dd (and dL/db) images over each
// block of kColRows rows into partD/partB[P][N] (P = ceil(B / kColRows)),
// for colsum_parts.
hipError_t mid_bwd(const float2* Zh, float2* Zg, const float4* Mq, long long B, const Geo& g, float* partD,
                   float* partB, hipStream_t s);
hipError_t unpack(const float2* Z, float* dst, long long B, long long N, bool relu, hipStream_t s);
hipError_t dA(const float* gh1, const float* u, const float* a, bool mask, float* imgA, float* gnext, long long B,
              long long N, hipStream_t s);

// Row permutations out[b][n] = in[b][perm[n]] for rows wider than one
// workgroup's LDS.  A gather straight from HBM pulls a cache line per
// element; here every access to HBM is contiguous, and the random accesses
// hit LDS.  The row is cut into nC = N / C chunks of C floats:
//   pass A  workgroup (b, c) loads source chunk c into LDS and writes the C
//           values sourced from it to tmp[b][cC ...], ordered by destination
//           chunk, then destination (nC runs, one per destination chunk)
//   pass B  workgroup (b, d) reads the nC runs bound for chunk d into LDS,
//           then writes chunk d of out in order
// With one chunk (N <= kPermChunk) pass A alone is the permutation.  The
// tables are built on the device from perm (perm_build, four small
// launches), so a call needs no host copy of perm.  The backward applies the
// adjoint (the inverse permutation) with the same tables, each pass's reads
// and writes exchanged.
constexpr int kPermChunk = 16384;                  // floats: 64 KB of LDS
constexpr int kPermMaxChunks = (1 << 22) / kPermChunk;  // the widest row
struct PermGeo {
  int C, nC;
};
// One layer's tables; layer l's sit stride ints further on.
struct PermTabs {
  int *srcA = nullptr, *gposB = nullptr, *locB = nullptr;  // [N] each
  int *cntS = nullptr, *bpre = nullptr;                    // [N / 256][nC]
  int *cnt = nullptr, *off = nullptr, *lst = nullptr;      // [nC][nC]
  long long stride = 0;
};
// ew: floats per element (1 for real rows, 2 for complex ones); a chunk
// holds kPermChunk / ew elements.
PermGeo perm_geo(long long N, int ew = 1);
size_t perm_table_ints(long long N, int ew = 1);              // per layer; 0 with one chunk
PermTabs perm_tables_at(int* base, long long N, int ew = 1);  // carve layer 0's tables from base
PermTabs perm_layer(const PermTabs& t, int l);                // layer l's tables
// Tables of the permutations perm[0 .. layers-1][N] into layers 0 .. layers-1.
hipError_t perm_build(const int* perm, long long N, int layers, const PermTabs& t, hipStream_t s, int ew = 1);
// out = in[perm] row by row; tmp is [B][N] scratch (unused with one chunk).
hipError_t permute(const float* in, float* out, float* tmp, const int* perm, const PermTabs& t, long long B,
                   long long N, hipStream_t s);
// The backward's dL/da step with the adjoint permutation: gm = gh1 masked
// (mask: where u <= 0), imgA = u gm, gnext[b][perm[n]] = gm[b][n] a[n].
hipError_t dA_permute(const float* gh1, const float* u, const float* a, bool mask, float* imgA, float* gnext,
                      float* tmp, const int* perm, const PermTabs& t, long long B, long long N, hipStream_t s);

// Complex (AFDF) rows of N complex elements: M = N points per row, no
// packing (acdc_multipass.hip).  The tables of cpermute come from
// perm_build(..., ew = 2).
hipError_t cpermute(const float2* in, float2* out, float2* tmp, const int* perm, const PermTabs& t, long long B,
                    long long N, hipStream_t s);
// out[b][perm[n]] = in[b][n] (the adjoint of cpermute, same tables)
hipError_t cpermute_adjoint(const float2* in, float2* out, float2* tmp, const int* perm, const PermTabs& t,
                            long long B, long long N, hipStream_t s);
// Z = FFT(src * a) (spectrum in pos() order); src is stashed when stash is
// set, a may be null.
hipError_t cfft_in(const float2* src, const float2* a, float2* stash, float2* Z, long long B, const Geo& g,
                   const float2* twM, const char* seg_tab, hipStream_t s);
// dst = unnormalised inverse FFT of Z (Z is overwritten).
hipError_t cifft_out(float2* Z, float2* dst, long long B, const Geo& g, const float2* twM, const char* seg_tab,
                     hipStream_t s);
// X[k] *= d[k] / N
hipError_t cmid_fwd(float2* Z, const float2* d, long long B, const Geo& g, float invN, hipStream_t s);
// gh3 = Zg / N; part[ceil(B / kColRows)][N] (complex) = row-block sums of
// gh3 * conj(Zh); Zg = gh3 * conj(d)
hipError_t cmid_bwd(const float2* Zh, float2* Zg, const float2* d, long long B, const Geo& g, float invN,
                    float2* part, hipStream_t s);
// imgA = gh1 * conj(u), gu = gh1 * conj(a)
hipError_t cdA(const float2* gh1, const float2* u, const float2* a, float2* imgA, float2* gu, long long B,
               long long N, hipStream_t s);
// out[w] (+)= sum over rows of img[b][w] in row order (blocks of kColRows
// rows, then the block sums in block order); with q, column w = 4e + j is
// the quartet value j of entry e, stored to its DCT index.  W is a
// multiple of 4; part holds [ceil(B / kColRows)][W].  colsum_parts runs the
// second stage alone, on block sums made elsewhere (mid_bwd).
constexpr int kColRows = 16;
hipError_t colsum(const float* img, long long B, long long W, float* part, float* out, const QuartetTabs* q,
                  bool accumulate, hipStream_t s);
hipError_t colsum_parts(const float* part, long long B, long long W, float* out, const QuartetTabs* q,
                        bool accumulate, hipStream_t s);

}  // namespace mp
}  // namespace acdc
