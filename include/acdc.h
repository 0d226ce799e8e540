/*
 * acdc.h -- C ABI of the MI355X (gfx950) ACDC / AFDF cascade library.
 *
 * Operation (Moczulski et al., "ACDC: A Structured Efficient Linear Layer",
 * arXiv:1511.05946).  One layer maps a row vector x of width N to
 *
 *     y = x A C D C^{-1}                      (Sec. 4, ACDC; A = diag(a), D = diag(d))
 *
 * with C the orthonormal DCT-II, c_nk = sqrt(2/N) eps_k cos(pi (2n+1) k / 2N),
 * n the spatial index, eps_0 = 1/sqrt(2), eps_k = 1 otherwise (Sec. 4), so
 * x C is the DCT-II of x and (.) C^{-1} = (.) C^T the DCT-III.  With
 * ACDC_FLAG_COMPLEX the layer is the complex AFDF of Sec. 3,
 *
 *     y = x A F D F^{-1},   F[n,k] = exp(-2 pi i n k / N),  F^{-1} = conj(F)/N.
 *
 * A cascade applies K layers in order, layer 0 first (the order-K product of
 * Sec. 3, made real in Sec. 4), optionally gathering each layer's input
 * through a fixed permutation and applying ReLU between layers (Sec. 6.2):
 *
 *     u_k = z_{k-1}[perm[k]]      (if ACDC_FLAG_PERM; z_{-1} = x)
 *     v_k = (u_k A_k C D_k + b_k) C^{-1}   (b_k only with ACDC_FLAG_BIAS)
 *     z_k = max(v_k, 0)           (if ACDC_FLAG_RELU and k < K-1), else v_k
 *     y   = z_{K-1}
 *
 * The bias b_k is added to the D-domain term of each layer, where Sec. 6.2
 * puts the additive biases of its cascade (on D, none on A), so that it
 * lands just before the ReLU.
 *
 * The backward pass gives dL/dx, dL/da_k, dL/dd_k (Sec. 4 derivative block)
 * and, with a bias, dL/db_k = sum over rows of the DCT-II of dL/dv_k, with
 * the parameter gradients summed over the batch.  Complex gradients use the
 * convention grad = dL/dRe + i dL/dIm (so dL/dx = dL/dy W^H).
 *
 * Memory.  Every pointer is a device pointer on the current HIP device unless
 * stated otherwise.  Arrays are contiguous, row-major, 16-byte aligned:
 *   x, y, grad_y, grad_x   [batch][N]   float (ACDC) or interleaved complex64
 *                                       (AFDF: 2N floats per row)
 *   A, D, grad_A, grad_D   [K][N]       same element type as x
 *   bias, grad_bias        [K][N]       float (ACDC_FLAG_BIAS, real layers only)
 *   perm                   [K][N]       int32, each row a permutation of 0..N-1
 *   saved                  [L][batch][N] layer inputs: u_1..u_{K-1} in slots 0..K-2, and with
 *                          ACDC_FLAG_PERM u_0 = x gathered through perm[0] in slot K-1
 *                          (L = K-1, or K with ACDC_FLAG_PERM)
 * The caller owns every buffer, including the workspaces; the library only
 * owns a small per-(device, N) table of constants built on first use (or by
 * acdc_prepare) and kept until the process ends.
 *
 * Errors.  Each call validates its arguments on the host before any HIP call
 * and returns a status; on error nothing is launched and no output is
 * touched.  Outputs must not alias inputs.  Launch failures return
 * ACDC_ERR_HIP (the HIP error code is kept per thread, see
 * acdc_last_hip_error); faults during execution surface asynchronously, as
 * for any HIP kernel.
 *
 * Streams.  Work is enqueued on `stream` (0 = the default stream) without any
 * host synchronisation, except that the very first use of a width N on a
 * device uploads its constant table synchronously.  Results are bitwise
 * reproducible for identical inputs on the same device.
 *
 * Supported widths (acdc_supported): ACDC N in {8, 16, ..., 32768} and 9216
 * with the fused kernels (one row per workgroup or wave, all K layers in one
 * launch); AFDF N in {8, 16, ..., 16384}.  Layers of power-of-two width also
 * run multi-pass (the multiple-call scheme of Sec. 5.2: each layer's FFT
 * goes through HBM in several launches, with hand-written passes): ACDC
 * 256 ... 2^22, AFDF 256 ... 2^21.  That path serves the widths past the
 * fused ones, and any such width with ACDC_FLAG_MULTIPASS; it needs more
 * workspace (see the *_workspace_size calls).
 * Batch sizes from 0 upward; K >= 1.
 *
 * Permutations.  Each row perm[k] must be a permutation of 0..N-1.  The
 * library does not check this (it would cost a pass over perm and a host
 * synchronisation per call); a row that is not a permutation gives
 * unspecified values in y, grad_x and the parameter gradients but never an
 * access outside the caller's buffers: the fused kernels use the entries
 * only as LDS indices within the workgroup (the backward's repacked copy
 * maps entries outside [0, N) to 0; in the forward an index past the
 * workgroup's LDS allocation reads 0, by the hardware's LDS bounds check),
 * and the multi-pass path reads every entry modulo N (the tables it builds
 * from perm are masked into range).
 */
#ifndef ACDC_H_
#define ACDC_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same type as hipStream_t, declared here so this header needs no HIP headers. */
typedef struct ihipStream_t* acdc_stream_t;

enum acdc_flags {
  ACDC_FLAG_PERM = 1u,       /* gather each layer's input through perm[k] */
  ACDC_FLAG_RELU = 2u,       /* ReLU after layers 0..K-2 (not with COMPLEX) */
  ACDC_FLAG_COMPLEX = 4u,    /* complex AFDF layers on interleaved complex64 */
  ACDC_FLAG_BIAS = 8u,       /* add b_k to each layer's D-domain term (not with COMPLEX) */
  ACDC_FLAG_ACCUMULATE = 16u, /* backward adds into grad_A, grad_D, grad_bias instead of overwriting */
  ACDC_FLAG_MULTIPASS = 32u   /* run the multi-pass path (below) even where a fused plan exists */
};

enum acdc_status {
  ACDC_OK = 0,
  ACDC_ERR_INVALID_ARG = -1, /* null/misaligned/aliased pointer, bad size or flag */
  ACDC_ERR_UNSUPPORTED = -2, /* width N not built, or COMPLEX with RELU or BIAS */
  ACDC_ERR_WORKSPACE = -3,   /* workspace missing or smaller than required */
  ACDC_ERR_HIP = -4,         /* a HIP runtime call failed */
  ACDC_ERR_NOT_PREPARED = -5 /* acdc_forward_noalloc: acdc_prepare(N, flags) not called on this device */
};

/* 1 if (N, flags) is supported by the compiled library, else 0.  Host only. */
int acdc_supported(int32_t N, uint32_t flags);

/* Build and upload the constant table for (N, flags) on the current device,
 * so that later calls enqueue without host synchronisation.  Optional. */
int acdc_prepare(int32_t N, uint32_t flags);

/* Bytes of the optional buffer `saved` that acdc_forward fills for
 * acdc_backward: the layer inputs u_1..u_{K-1}, [K-1][batch][N] elements,
 * plus u_0 (x gathered through perm[0]) in a last slot with ACDC_FLAG_PERM. */
size_t acdc_saved_bytes(int64_t batch, int32_t N, int32_t K, uint32_t flags);

/* Bytes of workspace acdc_forward needs (the per-layer quartet coefficients
 * built from D; on the multi-pass path also the packed spectra, a layer
 * buffer and, with ACDC_FLAG_PERM, a buffer for the permuted layer input and
 * the permutation tables that each call builds on the device from perm).
 * Host only. */
size_t acdc_forward_workspace_size(int64_t batch, int32_t N, int32_t K, uint32_t flags);

/* Bytes of workspace acdc_backward needs: per-workgroup partial sums of the
 * parameter gradients, the per-layer quartet coefficients (with
 * ACDC_FLAG_PERM followed by perm repacked as 16-bit offsets), the batch sums
 * behind the bias gradient (ACDC_FLAG_BIAS), and -- when have_saved is 0 and
 * acdc_saved_bytes(...) is not 0 -- room to recompute the layer inputs (the
 * paper's recompute policy, Sec. 5.3).  The multi-pass path adds its
 * spectra, layer buffers, row-block sums and permutation tables. */
size_t acdc_backward_workspace_size(int64_t batch, int32_t N, int32_t K, uint32_t flags, int have_saved);

/* Forward cascade: y = cascade(x).  `bias` is read with ACDC_FLAG_BIAS and
 * ignored (may be null) otherwise; `perm` likewise with ACDC_FLAG_PERM.  If
 * `saved` is non-null it also stores the layer inputs (see acdc_saved_bytes) there, for
 * acdc_backward; saved_bytes must be at least acdc_saved_bytes(...) (else
 * ACDC_ERR_WORKSPACE, nothing launched). */
int acdc_forward(const float* x, float* y, const float* A, const float* D, const float* bias,
                 const int32_t* perm, int64_t batch, int32_t N, int32_t K, uint32_t flags, float* saved,
                 size_t saved_bytes, void* workspace, size_t workspace_bytes, acdc_stream_t stream);

/* Forward cascade that allocates nothing, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments and results as
 * acdc_forward, bit for bit, without the workspace: the per-layer quartet
 * coefficients go to a file-scope device array of the library (16 MiB per
 * device, held until the process ends).
 *  - acdc_prepare(N, flags) must have been called on the current device
 *    first (it builds the constant table and finds that array's address);
 *    otherwise ACDC_ERR_NOT_PREPARED, nothing launched.
 *  - Fused widths only (ACDC_ERR_UNSUPPORTED for the multi-pass path, whose
 *    workspace grows with the batch), and K * acdc_forward_workspace_size
 *    per layer must fit the array: real rows need 16 N bytes per layer, so
 *    K * N <= 2^20 (else ACDC_ERR_WORKSPACE).  Complex rows need no scratch.
 *  - Every call on one device shares that device's array, and each call
 *    rewrites the part it uses before reading it: calls that overlap on one
 *    device (different streams or host threads without ordering) race.
 * No hipMalloc, hipFree or other allocation happens in this call. */
int acdc_forward_noalloc(const float* x, float* y, const float* A, const float* D, const float* bias,
                         const int32_t* perm, int64_t batch, int32_t N, int32_t K, uint32_t flags, float* saved,
                         size_t saved_bytes, acdc_stream_t stream);

/* Backward cascade (Sec. 4, the derivatives of a layer with respect to x,
 * a and d, chained through the cascade).  Given x and grad_y = dL/dy, writes
 * grad_x = dL/dx and grad_A, grad_D = dL/da_k, dL/dd_k summed over the
 * batch, in a fixed order that depends only on the call's shapes (batch,
 * N, K, flags) and the device (workgroups sum their rows, and the partials
 * are then added in 4 or 8 fixed tile phases, 8 for the smaller gradients;
 * at N = 9216 each resident workgroup first adds its tiles into one
 * partial), and with
 * ACDC_FLAG_BIAS grad_bias = dL/db_k (bias and grad_bias are then required,
 * and ignored otherwise).  The parameter gradients are overwritten, or with
 * ACDC_FLAG_ACCUMULATE added to what the arrays hold.  `saved` is the buffer
 * filled by acdc_forward for the same x, A, D, bias, perm (saved_bytes as
 * there), or null, in which case the layer inputs are recomputed into the
 * workspace first.  batch == 0 gives zero parameter gradients. */
int acdc_backward(const float* x, const float* grad_y, const float* A, const float* D, const float* bias,
                  const int32_t* perm, const float* saved, size_t saved_bytes, float* grad_x, float* grad_A,
                  float* grad_D, float* grad_bias, int64_t batch, int32_t N, int32_t K, uint32_t flags,
                  void* workspace, size_t workspace_bytes, acdc_stream_t stream);

/* Kernel timing for benchmarks (not for the callers' hot path).  While
 * enabled, each launch of the forward-cascade kernel (kind 0), the
 * backward-cascade kernel (kind 1) and the batch-reduction kernel (kind 2) is
 * bracketed by HIP events on its stream.  acdc_profile_read waits for the
 * recorded events, writes the summed durations in milliseconds to ms[0..2]
 * and the launch counts to launches[0..2] (host arrays of 3), and clears
 * the record.  Events are created once and reused. */
int acdc_profile_enable(int enable);
int acdc_profile_read(double* ms, int64_t* launches);

/* Static description of a status code. */
const char* acdc_status_string(int status);

/* hipError_t behind the calling thread's most recent ACDC_ERR_HIP (0 if none). */
int acdc_last_hip_error(void);

/* Health check of the backward kernels' row synchronisation.  Where one
 * batch row of the backward cascade (Sec. 4's gradients) spans several
 * wavefronts, those waves meet at a counter of their own instead of the
 * workgroup barrier, and each wait polls a bounded number of times (tens of
 * milliseconds) so that a wave can never spin forever.  A wait that runs out
 * of polls is counted on the device; its workgroup's results are then not
 * to be trusted.  acdc_sync_timeouts writes the count of the current device
 * (accumulated since the last clear) to *count and, when clear != 0, resets
 * it.  It copies synchronously on the null stream: synchronise the streams
 * that ran acdc_backward first.  Returns ACDC_ERR_INVALID_ARG for a null
 * count, ACDC_ERR_HIP when a copy fails (then *count is 0). */
int acdc_sync_timeouts(int64_t* count, int clear);

#ifdef __cplusplus
}
#endif

#endif /* ACDC_H_ */
