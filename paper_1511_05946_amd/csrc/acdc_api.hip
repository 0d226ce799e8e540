// HIP kernels for gfx950 and the C ABI declared in include/acdc.h.
//
// Kernels (one instantiation per supported width):
//   k_real_mq      per-layer quartet coefficients of the layer middle (tiny)
//   k_real_fwd     forward cascade, ROWS rows per workgroup, all K layers
//                  fused, rows kept in registers + one LDS slab per row
//   k_real_bwd     backward cascade with the reduction of dL/da, dL/dd over
//                  the workgroup's rows into one partial per tile, or
//                  (unbiased rows in tiles of at most two rows) persistent
//                  workgroups that add their tiles into one partial each
//   k_real_reduce  fixed-order sum of the partials over workgroups
//   k_real_dct     DCT-II of the batch sums of g (bias gradient, tiny)
// The multi-pass path (acdc_multipass.hip) serves widths beyond the fused
// plans and ACDC_FLAG_MULTIPASS; its host sequence is at the end of this file.
//   k_cplx_*       the same for the complex AFDF layers
#include <hip/hip_runtime.h>

#include <cstdio>
#include <map>
#include <mutex>
#include <tuple>
#include <vector>

#include "acdc.h"
#include "acdc_devctx.hpp"
#include "acdc_multipass.hpp"
#include "acdc_registry.hpp"

namespace acdc {

// Number of row syncs (GroupCtx) on this device whose polling budget ran out
// before the row's waves had all arrived; nonzero would mean wrong results.
// acdc_sync_timeouts reads and clears it.
static __device__ unsigned long long sync_timeouts;

// Threads past the K * NSL * T table entries repack perm for the row
// kernels (RealOps::pack_perm_entry), when P16 is given.
template <class PL>
__global__ __launch_bounds__(256) void k_real_mq(const float* __restrict__ D, const float* __restrict__ Bias,
                                                 float4* __restrict__ Mq, int K, const char* __restrict__ tab,
                                                 const int* __restrict__ perm, int4* __restrict__ P16) {
  constexpr int E = PL::NSL * PL::T;
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long long)K * E) {
    using O = RealOps<PL>;
    if constexpr (O::kPackedPerm) {
      constexpr int W = O::NIW * PL::T;
      const long long q = i - (long long)K * E;
      if (P16 == nullptr || q >= (long long)K * W) return;
      const int k = int(q / W), r = int(q % W);
      P16[q] = O::pack_perm_entry(perm + (long long)k * PL::N, r / PL::T, unsigned(r % PL::T));
    }
    return;
  }
  const int k = int(i / E), e = int(i % E);
  float4 row[kMqRows];
  real_mq_entry<PL>(D + (long long)k * PL::N, Bias != nullptr ? Bias + (long long)k * PL::N : nullptr, tab, e, row);
  // layout [k][slot][r][t]
  const int slot = e / PL::T, t = e % PL::T;
  float4* out = Mq + (long long)k * E * kMqRows + (long long)slot * kMqRows * PL::T + t;
#pragma unroll
  for (int r = 0; r < kMqRows; ++r) out[r * PL::T] = row[r];
}

// Copy of the FFT twiddle table (the first TW_FLOAT2 float2 of the plan's
// constant table) into LDS; the caller synchronises.
template <class PL>
__device__ __forceinline__ void copy_twiddles(float* dst, const char* tab, int tid, int nthreads) {
  const float2* src = reinterpret_cast<const float2*>(tab);
  float2* d2 = reinterpret_cast<float2*>(dst);
  for (int i = tid; i < PL::TW_FLOAT2; i += nthreads) d2[i] = src[i];
}

// The forward kernel is persistent: workgroup b handles row groups (tiles)
// b, b + gridDim.x, ...  Rows are independent, so results do not depend on
// the grid size.
template <class PL, bool BIAS>
__global__ __launch_bounds__(Launch<PL>::FWD_THREADS)
__attribute__((amdgpu_waves_per_eu(Launch<PL>::FWD_WPE))) void k_real_fwd(RealArgs a, long long ntiles) {
  using L = Launch<PL>;
  __shared__ float lds[L::FWD_LDS_FLOATS];
  DevCtx<PL::T> ctx;
  const int tid = threadIdx.x;
  const unsigned t = unsigned(tid) % PL::T;
  int r = tid / PL::T;
  if constexpr (PL::T >= 64) r = __builtin_amdgcn_readfirstlane(r);  // one row per whole wave
  // LDS: [twiddle copy (TW_FLOATS)][row slabs]; the table sits at offset 0
  // so that its loads address it through the instruction's immediate offset
  float* const rows = lds + L::TW_FLOATS;
  float* slab = rows + r * L::FWD_SLAB;
  if constexpr (L::TW_LDS) {
    float* twl = lds;
    copy_twiddles<PL>(twl, a.tab, tid, L::FWD_THREADS);
    ctx.sync_all();
    const LdsView tw = LdsView::of(twl);
    for (long long tile = blockIdx.x; tile < ntiles; tile += gridDim.x)
      real_forward_row<PL, BIAS>(ctx, a, t, tile * L::FWD_ROWS, unsigned(r), slab, tw);
  } else {
    const GView tw = GView::of(a.tab);
    for (long long tile = blockIdx.x; tile < ntiles; tile += gridDim.x)
      real_forward_row<PL, BIAS>(ctx, a, t, tile * L::FWD_ROWS, unsigned(r), slab, tw);
  }
}

template <class PL, bool BIAS>
__global__ __launch_bounds__(Launch<PL>::BWD_THREADS)
__attribute__((amdgpu_waves_per_eu(Launch<PL>::BWD_WPE))) void k_real_bwd(RealArgs a, long long ntiles) {
  using L = Launch<PL>;
  constexpr bool ACC = L::BWD_ACC && !BIAS;
  __shared__ float lds[L::BWD_LDS_FLOATS + (ACC ? L::ACC_FLOATS : 0)];
  const int tid = threadIdx.x;
  const unsigned t = unsigned(tid) % PL::T;
  int r = tid / PL::T;
  if constexpr (PL::T >= 64) r = __builtin_amdgcn_readfirstlane(r);  // one row per whole wave
  // LDS: [twiddle copy (TW_FLOATS)][row slabs][previous partial values (ACC)];
  // the table sits at offset 0 so that its loads address it through the
  // instruction's immediate offset
  float* const rows = lds + L::BWD_TW_FLOATS;
  float* slab = rows + r * L::BWD_SLAB;
  auto body = [&](auto& ctx) {
    if constexpr (ACC) {
      // persistent: workgroup w runs tiles w, w + G, ... (G = gridDim.x) and
      // adds them, in that order, into partial slot w
      static_assert(!L::BWD_TW_LDS, "persistent backward reads its twiddles from global memory");
      float* const old = lds + L::BWD_LDS_FLOATS;
      const unsigned w = blockIdx.x, nt = unsigned(ntiles);  // tiles < 2^31: batch <= 2^40 / N rows and N >= 1024
      for (unsigned tile = w; tile < nt; tile += gridDim.x)
        real_backward_row<PL, L::BWD_ROWS, BIAS, true>(ctx, a, t, (long long)tile * L::BWD_ROWS, unsigned(r), tid,
                                                       w, rows, slab, GView::of(a.tab), tile == w ? nullptr : old);
    } else if constexpr (L::BWD_TW_LDS) {
      // one tile per workgroup, one partial slot per tile
      const long long tile = blockIdx.x;
      float* twl = lds;
      copy_twiddles<PL>(twl, a.tab, tid, L::BWD_THREADS);
      ctx.sync_all();
      real_backward_row<PL, L::BWD_ROWS, BIAS>(ctx, a, t, tile * L::BWD_ROWS, unsigned(r), tid, tile, rows, slab,
                                               LdsView::of(twl));
    } else {
      const long long tile = blockIdx.x;
      real_backward_row<PL, L::BWD_ROWS, BIAS>(ctx, a, t, tile * L::BWD_ROWS, unsigned(r), tid, tile, rows, slab,
                                               GView::of(a.tab));
    }
  };
  if constexpr (L::BWD_GROUP_SYNC) {
    // rows of several waves meet at their own LDS counter (GroupCtx)
    using G = GroupCtx<PL::T>;
    __shared__ unsigned words[G::kWords * L::BWD_ROWS];
    if (tid < G::kWords * L::BWD_ROWS) words[tid] = 0u;
    DevCtx<PL::T>::lds_barrier();
    G ctx(&words[G::kWords * r]);
    body(ctx);
    G::report(words, L::BWD_ROWS, tid, &sync_timeouts);
  } else {
    DevCtx<PL::T> ctx;
    body(ctx);
  }
}

// Batch reduction: a block of kRedThreads threads owns kRedThreads / PH
// float4 entries of the reduced gradient (over all layers, entry index
// k * PS4 + e4) and sums them over the tiles with one thread per (entry,
// phase); phase sums meet in LDS and are added in phase order
// (tile_phase_sum4 / phases_total4).  128-thread blocks beat 256 and 64
// threads at N = 4096.
constexpr int kRedThreads = 128;

template <class PL, int PH>
__global__ __launch_bounds__(kRedThreads) void k_real_reduce(const float* __restrict__ partial, long long ntiles, int K,
                                                     float* __restrict__ gA, float* __restrict__ gD,
                                                     float* __restrict__ gS, const char* __restrict__ tab,
                                                     int bias, int accumulate) {
  const long long PS4 = partial_entries4<PL>(bias != 0);
  constexpr int E = kRedThreads / PH;
  __shared__ float4 ph[PH][E];
  const int lane = threadIdx.x % E, g = threadIdx.x / E;
  const long long i = (long long)blockIdx.x * E + lane;
  const long long n = (long long)K * PS4;
  ph[g][lane] = i < n ? tile_phase_sum4<PH>(reinterpret_cast<const float4*>(partial), ntiles, n, i, g)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
  __syncthreads();
  if (g == 0 && i < n) {
    float4 all[PH];
#pragma unroll
    for (int q = 0; q < PH; ++q) all[q] = ph[q][lane];
    real_reduce_store4<PL>(phases_total4<PH>(all), int(i / PS4), int(i % PS4), gA, gD, gS, tab, accumulate != 0);
  }
}

// Bias gradient: grad_b[k] (+)= DCT-II of the batch sum of g at layer k.
// One workgroup of T threads per layer.
template <class PL>
__global__ __launch_bounds__(PL::T) void k_real_dct(const float* __restrict__ S, float* __restrict__ gB,
                                                    const float4* __restrict__ Mq, const char* __restrict__ tab,
                                                    int accumulate) {
  __shared__ float lds[Launch<PL>::FWD_SLAB];
  DevCtx<PL::T> ctx;
  const long long k = blockIdx.x;
  real_dct_row<PL>(ctx, S + k * PL::N, gB + k * PL::N, Mq, accumulate != 0, threadIdx.x, lds, GView::of(tab), tab);
}

template <class PL>
__global__ __launch_bounds__(Launch<PL>::FWD_THREADS)
__attribute__((amdgpu_waves_per_eu(Launch<PL>::FWD_WPE))) void k_cplx_fwd(CplxArgs a) {
  using L = Launch<PL>;
  __shared__ float lds[L::FWD_ROWS * L::FWD_SLAB];
  DevCtx<PL::T> ctx;
  const int tid = threadIdx.x;
  const unsigned t = unsigned(tid) % PL::T;
  int r = tid / PL::T;
  if constexpr (PL::T >= 64) r = __builtin_amdgcn_readfirstlane(r);  // one row per whole wave
  cplx_forward_row<PL>(ctx, a, t, (long long)blockIdx.x * L::FWD_ROWS, unsigned(r), lds + r * L::FWD_SLAB);
}

template <class PL>
__global__ __launch_bounds__(Launch<PL>::BWD_THREADS)
__attribute__((amdgpu_waves_per_eu(Launch<PL>::BWD_WPE))) void k_cplx_bwd(CplxArgs a) {
  using L = Launch<PL>;
  __shared__ float lds[L::BWD_ROWS * L::BWD_SLAB];
  const int tid = threadIdx.x;
  const unsigned t = unsigned(tid) % PL::T;
  int r = tid / PL::T;
  if constexpr (PL::T >= 64) r = __builtin_amdgcn_readfirstlane(r);  // one row per whole wave
  if constexpr (L::BWD_GROUP_SYNC) {
    using G = GroupCtx<PL::T>;
    __shared__ unsigned words[G::kWords * L::BWD_ROWS];
    if (tid < G::kWords * L::BWD_ROWS) words[tid] = 0u;
    DevCtx<PL::T>::lds_barrier();
    G ctx(&words[G::kWords * r]);
    cplx_backward_row<PL, L::BWD_ROWS>(ctx, a, t, (long long)blockIdx.x * L::BWD_ROWS, unsigned(r), tid,
                                       (long long)blockIdx.x, lds, lds + r * L::BWD_SLAB);
    G::report(words, L::BWD_ROWS, tid, &sync_timeouts);
  } else {
    DevCtx<PL::T> ctx;
    cplx_backward_row<PL, L::BWD_ROWS>(ctx, a, t, (long long)blockIdx.x * L::BWD_ROWS, unsigned(r), tid,
                                       (long long)blockIdx.x, lds, lds + r * L::BWD_SLAB);
  }
}

template <class PL, int PH>
__global__ __launch_bounds__(kRedThreads) void k_cplx_reduce(const float* __restrict__ partial, long long ntiles, int K,
                                                     float* __restrict__ gA, float* __restrict__ gD,
                                                     int accumulate) {
  constexpr long long PS4 = partial_entries4<PL>();
  constexpr int E = kRedThreads / PH;
  __shared__ float4 ph[PH][E];
  const int lane = threadIdx.x % E, g = threadIdx.x / E;
  const long long i = (long long)blockIdx.x * E + lane;
  const long long n = (long long)K * PS4;
  ph[g][lane] = i < n ? tile_phase_sum4<PH>(reinterpret_cast<const float4*>(partial), ntiles, n, i, g)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
  __syncthreads();
  if (g == 0 && i < n) {
    float4 all[PH];
#pragma unroll
    for (int q = 0; q < PH; ++q) all[q] = ph[q][lane];
    cplx_reduce_store4<PL>(phases_total4<PH>(all), int(i / PS4), int(i % PS4), gA, gD, accumulate != 0);
  }
}

// Scratch of the no-allocation forward (acdc_forward_noalloc): the per-layer
// quartet coefficients that acdc_forward keeps in the caller's workspace.
// Each device holds its own copy until the process ends; host code reaches
// it only through the address hipGetSymbolAddress returns on that device.
constexpr size_t kNoAllocScratchBytes = size_t(16) << 20;
static __device__ __align__(256) float4 scratch[kNoAllocScratchBytes / sizeof(float4)];

// ------------------------------------------------------------------ host side

namespace {

thread_local int g_last_hip = 0;
std::mutex g_mu;
std::map<std::tuple<int, int, int>, void*> g_tables;  // (device, N, complex) -> device table

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

int hip_fail(hipError_t e) {
  g_last_hip = int(e);
  return ACDC_ERR_HIP;
}

// ----------------------------------------------------------- kernel timing
// While enabled, every main kernel launch is bracketed by HIP events on its
// stream (kind 0: forward cascade, 1: backward cascade, 2: batch reduction).
struct ProfRec {
  hipEvent_t a, b;
  int kind;
};
bool g_prof_on = false;
std::mutex g_prof_mu;
std::vector<ProfRec> g_prof_recs;
std::vector<hipEvent_t> g_prof_pool;

hipEvent_t prof_event() {
  if (!g_prof_pool.empty()) {
    hipEvent_t e = g_prof_pool.back();
    g_prof_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

struct ProfScope {
  int kind;
  hipStream_t s;
  hipEvent_t a = nullptr, b = nullptr;
  ProfScope(int k, hipStream_t st) : kind(k), s(st) {
    if (!g_prof_on) return;
    std::lock_guard<std::mutex> lock(g_prof_mu);
    a = prof_event();
    b = prof_event();
    if (a && b) (void)hipEventRecord(a, s);
  }
  ~ProfScope() {
    if (!a || !b) return;
    (void)hipEventRecord(b, s);
    std::lock_guard<std::mutex> lock(g_prof_mu);
    g_prof_recs.push_back(ProfRec{a, b, kind});
  }
};

bool fused_supported(int N, unsigned flags) {
  bool ok = false;
  auto probe = [&]<class PL>() { ok = true; };
  if (flags & kFlagComplex) dispatch_complex(N, probe);
  else dispatch_real(N, probe);
  return ok;
}

// Multi-pass path: power-of-two rows, real ones of width 256 ... 2^22 and
// complex ones of 256 ... 2^21 elements (the same M <= 2^21 point FFTs).
bool mp_width(long long N) { return N >= 256 && N <= (1LL << 22) && (N & (N - 1)) == 0; }
bool mp_width(long long N, unsigned flags) {
  return (flags & kFlagComplex) ? N <= (1LL << 21) && mp_width(N) : mp_width(N);
}
bool use_multipass(int N, unsigned flags) {
  return (flags & kFlagMultipass) != 0 || !fused_supported(N, flags);
}
bool supported(int N, unsigned flags) { return use_multipass(N, flags) ? mp_width(N, flags) : true; }

// Constant table of (N, complex) on the current device; built and uploaded
// on first use.
int get_table(int N, bool cplx, const char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e);
  std::lock_guard<std::mutex> lock(g_mu);
  auto key = std::make_tuple(dev, N, cplx ? 1 : 0);
  auto it = g_tables.find(key);
  if (it != g_tables.end()) {
    *out = static_cast<const char*>(it->second);
    return ACDC_OK;
  }
  std::vector<unsigned char> host;
  bool built = false, ok = false;
  auto build = [&]<class PL>() {
    built = true;
    if constexpr (PL::kComplex) ok = build_complex_tables<PL>(host);
    else ok = build_real_tables<PL>(host);
  };
  if (cplx) dispatch_complex(N, build);
  else dispatch_real(N, build);
  if (!built) return ACDC_ERR_UNSUPPORTED;
  if (!ok) return ACDC_ERR_UNSUPPORTED;
  void* d = nullptr;
  e = hipMalloc(&d, host.size());
  if (e != hipSuccess) return hip_fail(e);
  e = hipMemcpy(d, host.data(), host.size(), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(d);
    return hip_fail(e);
  }
  g_tables[key] = d;
  *out = static_cast<const char*>(d);
  return ACDC_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Workgroups of `kernel` (with `threads` threads) that fit on the current
// device at once; the persistent kernels launch min(tiles, this).  With
// `remember` false a value not yet cached is computed without caching it
// (the no-allocation entry point inserts nothing).
std::map<std::pair<const void*, int>, long long> g_resident;
long long resident_workgroups(const void* kernel, int threads, bool remember = true) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  std::lock_guard<std::mutex> lock(g_mu);
  auto key = std::make_pair(kernel, dev);
  auto it = g_resident.find(key);
  if (it != g_resident.end()) return it->second;
  int per_cu = 0, cus = 0;
  long long n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) == hipSuccess &&
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess)
    n = (long long)per_cu * cus;
  if (remember) g_resident[key] = n;
  return n;
}

long long persistent_grid(const void* kernel, int threads, long long tiles, bool remember = true) {
  const long long n = resident_workgroups(kernel, threads, remember);
  return (n > 0 && n < tiles) ? n : tiles;
}

// Per-device address of `scratch`, set by acdc_prepare (the library's set-up
// call) with the device current; null until then.
constexpr int kMaxDevices = 64;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_setup() {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e);
  if (dev < 0 || dev >= kMaxDevices) return ACDC_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch_ptr[dev] != nullptr) return ACDC_OK;
  void* p = nullptr;
  e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return hip_fail(e);
  g_scratch_ptr[dev] = p;
  return ACDC_OK;
}

// The constant table of (N, complex) on device `dev` if it exists (never
// builds one).
const char* find_table(int dev, int N, bool cplx) {
  std::lock_guard<std::mutex> lock(g_mu);
  auto it = g_tables.find(std::make_tuple(dev, N, cplx ? 1 : 0));
  return it == g_tables.end() ? nullptr : static_cast<const char*>(it->second);
}

constexpr uint32_t kAllFlags = kFlagPerm | kFlagRelu | kFlagComplex | kFlagBias | kFlagAccumulate | kFlagMultipass;

bool flags_supported(uint32_t flags) {
  return !((flags & kFlagComplex) && (flags & (kFlagRelu | kFlagBias)));
}

int check_common(int64_t batch, int32_t N, int32_t K, uint32_t flags) {
  if (flags & ~kAllFlags) return ACDC_ERR_INVALID_ARG;
  if (!flags_supported(flags)) return ACDC_ERR_UNSUPPORTED;
  if (batch < 0 || K < 1 || K > 65535 || N < 1) return ACDC_ERR_INVALID_ARG;
  if (!supported(N, flags)) return ACDC_ERR_UNSUPPORTED;
  if (batch > (int64_t(1) << 40) / N) return ACDC_ERR_INVALID_ARG;
  return ACDC_OK;
}

int check_ptrs(std::initializer_list<const void*> must, std::initializer_list<const void*> may) {
  for (const void* p : must)
    if (p == nullptr || !aligned16(p)) return ACDC_ERR_INVALID_ARG;
  for (const void* p : may)
    if (p != nullptr && !aligned16(p)) return ACDC_ERR_INVALID_ARG;
  return ACDC_OK;
}

bool distinct(std::initializer_list<const void*> outs, std::initializer_list<const void*> all) {
  for (const void* o : outs) {
    if (o == nullptr) continue;
    int seen = 0;
    for (const void* p : all)
      if (p == o) ++seen;
    if (seen != 1) return false;
  }
  return true;
}

template <class PL>
long long fwd_blocks(int64_t batch) {
  return (batch + Launch<PL>::FWD_ROWS - 1) / Launch<PL>::FWD_ROWS;
}
template <class PL>
long long bwd_tiles(int64_t batch) {
  return (batch + Launch<PL>::BWD_ROWS - 1) / Launch<PL>::BWD_ROWS;
}

size_t elem_floats(uint32_t flags) { return (flags & kFlagComplex) ? 2 : 1; }

// Floats of the `saved` buffer: the layer inputs u_1..u_{K-1}, preceded by
// u_0 (x gathered through perm[0]) with PERM.
size_t saved_layers(int32_t K, uint32_t flags) { return size_t(K - 1) + ((flags & kFlagPerm) ? 1 : 0); }
size_t saved_floats(int64_t batch, int32_t N, int32_t K, uint32_t flags) {
  return saved_layers(K, flags) * size_t(batch) * size_t(N) * elem_floats(flags);
}

struct WsLayout {
  size_t mq = 0, partial = 0, gs = 0, stash = 0, total = 0;
  size_t off_mq = 0, off_partial = 0, off_gs = 0, off_stash = 0;
};

// The quartet table, then for the backward (with PERM, where the plan packs
// it) the packed perm of every layer.
template <class PL>
size_t mq_table_bytes(int32_t K) {
  return align256(size_t(K) * PL::NSL * kMqRows * PL::T * sizeof(float4));
}
template <class PL>
size_t mq_bytes(int32_t K, uint32_t flags, bool backward) {
  using O = RealOps<PL>;
  const bool packed = backward && O::kPackedPerm && (flags & kFlagPerm) != 0;
  return mq_table_bytes<PL>(K) + (packed ? align256(size_t(K) * O::NIW * PL::T * sizeof(int4)) : 0);
}
template <class PL>
int4* perm16_of(float4* Mq, int32_t K, uint32_t flags) {
  if (!RealOps<PL>::kPackedPerm || !(flags & kFlagPerm)) return nullptr;
  return reinterpret_cast<int4*>(reinterpret_cast<char*>(Mq) + mq_table_bytes<PL>(K));
}

WsLayout bwd_layout(int64_t batch, int32_t N, int32_t K, uint32_t flags, bool have_saved) {
  WsLayout w;
  const bool bias = (flags & kFlagBias) != 0;
  auto f = [&]<class PL>() {
    const long long tiles = bwd_tiles<PL>(batch);
    w.partial = align256(size_t(tiles) * K * partial_entries4<PL>(bias) * sizeof(float4));
    if constexpr (!PL::kComplex) {
      // the bias gradient's DCT reads w, qa, qb' from the quartet table
      if (batch > 0 || bias) w.mq = mq_bytes<PL>(K, flags, true);
      if (bias) w.gs = align256(size_t(K) * PL::N * sizeof(float));
    }
  };
  if (flags & kFlagComplex) dispatch_complex(N, f);
  else dispatch_real(N, f);
  if (!have_saved) w.stash = align256(saved_floats(batch, N, K, flags) * 4);
  w.off_mq = 0;
  w.off_partial = w.off_mq + w.mq;
  w.off_gs = w.off_partial + w.partial;
  w.off_stash = w.off_gs + w.gs;
  w.total = w.off_stash + w.stash;
  return w;
}

size_t fwd_ws(int32_t N, int32_t K, uint32_t flags) {
  size_t b = 0;
  if (!(flags & kFlagComplex))
    dispatch_real(N, [&]<class PL>() { b = mq_bytes<PL>(K, flags, false); });
  return b;
}

// The quartet table into Mq, and the packed perm into P16 (if not null).
template <class PL>
int launch_real_mq(const float* D, const float* Bias, float4* Mq, int K, const char* tab, const int* perm,
                   int4* P16, hipStream_t s) {
  const long long n = (long long)K * PL::NSL * PL::T + (P16 != nullptr ? (long long)K * RealOps<PL>::NIW * PL::T : 0);
  hipLaunchKernelGGL(k_real_mq<PL>, dim3(unsigned((n + 255) / 256)), dim3(256), 0, s, D, Bias, Mq, K, tab, perm,
                     P16);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? ACDC_OK : hip_fail(e);
}

template <class PL, bool BIAS>
void launch_real_fwd_k(const RealArgs& a, hipStream_t s, bool remember) {
  const long long tiles = fwd_blocks<PL>(a.batch);
  const long long grid = persistent_grid(reinterpret_cast<const void*>(&k_real_fwd<PL, BIAS>),
                                         Launch<PL>::FWD_THREADS, tiles, remember);
  hipLaunchKernelGGL((k_real_fwd<PL, BIAS>), dim3(unsigned(grid)), dim3(Launch<PL>::FWD_THREADS), 0, s, a, tiles);
}

template <class PL>
int launch_real_fwd(const RealArgs& a, hipStream_t s, bool remember = true) {
  ProfScope prof(0, s);
  if (a.flags & kFlagBias) launch_real_fwd_k<PL, true>(a, s, remember);
  else launch_real_fwd_k<PL, false>(a, s, remember);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? ACDC_OK : hip_fail(e);
}

template <class PL>
int launch_cplx_fwd(const CplxArgs& a, hipStream_t s) {
  ProfScope prof(0, s);
  hipLaunchKernelGGL(k_cplx_fwd<PL>, dim3(unsigned(fwd_blocks<PL>(a.batch))), dim3(Launch<PL>::FWD_THREADS), 0,
                     s, a);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? ACDC_OK : hip_fail(e);
}

// ------------------------------------------------------ multi-pass path

mp::Geo mp_geo(long long N) {
  mp::Geo g;
  g.M = N / 2;
  g.L = int(g.M < 8192 ? g.M : 8192);
  const long long ratio = g.M / g.L;
  g.R1 = ratio == 1 ? 1 : int(ratio <= 16 ? ratio : 16);
  g.R2 = ratio <= 16 ? 1 : int(ratio / 16);
  return g;
}

struct MpTabs {
  const float2* tw = nullptr;
  QuartetTabs q{};
  const char* seg = nullptr;  // the complex plan table of the segment length
};
std::map<std::pair<int, int>, void*> g_mp_tables;  // (device, N) -> device table

int get_mp_tables(int N, MpTabs* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e);
  const mp::Geo g = mp_geo(N);
  int rc = get_table(g.L, true, &out->seg);
  if (rc != ACDC_OK) return rc;
  void* d = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    auto it = g_mp_tables.find({dev, N});
    if (it != g_mp_tables.end()) d = it->second;
  }
  if (d == nullptr) {
    std::vector<unsigned char> host;
    if (!build_mp_tables(N, host)) return ACDC_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_mu);
    auto it = g_mp_tables.find({dev, N});
    if (it != g_mp_tables.end()) {
      d = it->second;
    } else {
      e = hipMalloc(&d, host.size());
      if (e != hipSuccess) return hip_fail(e);
      e = hipMemcpy(d, host.data(), host.size(), hipMemcpyHostToDevice);
      if (e != hipSuccess) {
        (void)hipFree(d);
        return hip_fail(e);
      }
      g_mp_tables[{dev, N}] = d;
    }
  }
  const char* base = static_cast<const char*>(d);
  const MpTableLayout l = mp_table_layout(N);
  out->tw = reinterpret_cast<const float2*>(base + l.tw);
  const double qb = 1.0 / (2.0 * std::sqrt(double(N)));
  out->q = QuartetTabs{reinterpret_cast<const float4*>(base + l.mk0), reinterpret_cast<const float4*>(base + l.mk1),
                       reinterpret_cast<const int4*>(base + l.qidx), reinterpret_cast<const int*>(base + l.qmask),
                       float(0.9238795325112867561 * qb), float(0.3826834323650897717 * qb)};
  return ACDC_OK;
}

size_t mp_mq_bytes(long long N, int K) { return align256(size_t(K) * size_t(N / 4) * kMqRows * sizeof(float4)); }
size_t mp_rows_bytes(int64_t batch, long long N) { return align256(size_t(batch) * size_t(N) * sizeof(float)); }

// Floats per row element: 1, or 2 for complex (AFDF) rows.
int mp_ew(uint32_t flags) { return (flags & kFlagComplex) ? 2 : 1; }

// Permutation tables: all K layers' built at once (four launches per call)
// when they take at most 256 MB, else one layer's, rebuilt per layer.
int mp_perm_layers(long long N, int K, int ew) {
  const size_t per = mp::perm_table_ints(N, ew) * sizeof(int);
  return per * size_t(K) <= (size_t(256) << 20) ? K : 1;
}
size_t mp_perm_bytes(long long N, int K, uint32_t flags) {
  if (!(flags & kFlagPerm)) return 0;
  const int ew = mp_ew(flags);
  return align256(mp::perm_table_ints(N, ew) * sizeof(int) * size_t(mp_perm_layers(N, K, ew)));
}
// Layer k's tables, building them first when they are not all built.
hipError_t mp_perm_tabs(const int32_t* perm, long long N, int K, int k, const mp::PermTabs& pt, mp::PermTabs* out,
                        hipStream_t s, int ew = 1) {
  if (mp_perm_layers(N, K, ew) == K) {
    *out = mp::perm_layer(pt, k);
    return hipSuccess;
  }
  *out = pt;
  return mp::perm_build(perm + (long long)k * N, N, 1, pt, s, ew);
}
hipError_t mp_perm_prebuild(const int32_t* perm, long long N, int K, const mp::PermTabs& pt, hipStream_t s,
                            int ew = 1) {
  return mp_perm_layers(N, K, ew) == K ? mp::perm_build(perm, N, K, pt, s, ew) : hipSuccess;
}

// Forward workspace: quartet coefficients, the packed spectrum (also the
// permutation's scratch), the layer output; with PERM the permuted layer
// input (when no stash takes it) and the permutation tables.
struct MpFwdWs {
  size_t mq = 0, z = 0, zbuf = 0, ubuf = 0, ptab = 0, total = 0;
};
MpFwdWs mp_fwd_ws(int64_t batch, int32_t N, int32_t K, uint32_t flags) {
  MpFwdWs w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  const long long rowf = (long long)N * mp_ew(flags);  // floats per row
  w.mq = take((flags & kFlagComplex) ? 0 : mp_mq_bytes(N, K));
  w.z = take(mp_rows_bytes(batch, rowf));
  w.zbuf = take(mp_rows_bytes(batch, rowf));
  w.ubuf = take((flags & kFlagPerm) ? mp_rows_bytes(batch, rowf) : 0);
  w.ptab = take(mp_perm_bytes(N, K, flags));
  w.total = off;
  return w;
}

// Backward workspace: quartet coefficients, the h and g spectra (contiguous,
// transformed together), dL/dv of the current layer, the next layer's g,
// the dL/da image, the row-block sums (dL/dd, then dL/da; dL/db), the
// recompute stash and the permutation tables.
struct MpBwdWs {
  size_t mq = 0, zhg = 0, gh1 = 0, gbuf = 0, imgA = 0, gu = 0, part = 0, partB = 0, stash = 0, ptab = 0, total = 0;
};
MpBwdWs mp_bwd_ws(int64_t batch, int32_t N, int32_t K, uint32_t flags, bool have_saved) {
  MpBwdWs w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  const bool cplx = (flags & kFlagComplex) != 0;
  const size_t rowf = size_t(N) * size_t(mp_ew(flags));  // floats per row
  const size_t rows = size_t(batch) * rowf * sizeof(float);
  w.mq = take(cplx ? 0 : mp_mq_bytes(N, K));
  w.zhg = take(2 * rows);
  w.gh1 = take(rows);
  w.gbuf = take(rows);
  w.imgA = take(rows);
  w.gu = take(cplx && (flags & kFlagPerm) ? rows : 0);  // complex dL/du before the adjoint permutation
  const size_t parts = size_t((batch + mp::kColRows - 1) / mp::kColRows) * rowf * sizeof(float);
  w.part = take(parts);
  w.partB = take((flags & kFlagBias) ? parts : 0);
  w.stash = take(have_saved ? 0 : saved_floats(batch, N, K, flags) * sizeof(float));
  w.ptab = take(mp_perm_bytes(N, K, flags));
  w.total = off;
  return w;
}

#define MP_TRY(call)                          \
  do {                                        \
    const hipError_t e_ = (call);             \
    if (e_ != hipSuccess) return hip_fail(e_); \
  } while (0)

// Pack rows of src (stashed, scaled by a; each may be null) and run the
// forward FFT: the first DIF pass takes the packing.
int mp_pack_fft(const float* src, const float* a, float* stash, float2* Z, long long rows, long long N,
                const mp::Geo& g, const MpTabs& t, hipStream_t s) {
  if (g.R1 > 1) {
    MP_TRY(mp::pack_dif(src, a, stash, Z, rows, g.M, g.R1, t.tw, s));
  } else {
    MP_TRY(mp::pack(src, a, stash, Z, rows, N, s));
  }
  if (g.R2 > 1) MP_TRY(mp::dif(Z, rows, g, g.M / g.R1, g.R2, t.tw, s));
  MP_TRY(mp::segments(Z, rows * (g.M / g.L), g.L, false, t.seg, s));
  return ACDC_OK;
}

// Inverse FFT, then unpack (+ ReLU) into dst: the last DIT pass takes the unpacking.
int mp_ifft_unpack(float2* Z, float* dst, long long rows, long long N, bool relu, const mp::Geo& g, const MpTabs& t,
                   hipStream_t s) {
  MP_TRY(mp::segments(Z, rows * (g.M / g.L), g.L, true, t.seg, s));
  if (g.R2 > 1) MP_TRY(mp::dit(Z, rows, g, g.M / g.R1, g.R2, t.tw, s));
  if (g.R1 > 1) {
    MP_TRY(mp::dit_unpack(Z, dst, rows, g.M, g.R1, t.tw, relu, s));
  } else {
    MP_TRY(mp::unpack(Z, dst, rows, N, relu, s));
  }
  return ACDC_OK;
}

// Stash slot of layer input u_k (the fused path's layout): k - 1, or K - 1
// for u_0 with PERM.
float* mp_slot(float* saved, int k, int K, long long batch, long long N, bool perm_on) {
  if (saved == nullptr) return nullptr;
  if (k > 0) return saved + (long long)(k - 1) * batch * N;
  return perm_on ? saved + (long long)(K - 1) * batch * N : nullptr;
}

// The K forward layers.  With PERM, the permuted input u_k goes to its
// stash slot (or to ubuf without a stash), Z serving as the permutation's
// scratch; without, the packing stashes z itself.
int mp_forward_layers(const float* x, float* y, const float* A, const float4* Mq, const int32_t* perm,
                      int64_t batch, int32_t N, int32_t K, uint32_t flags, float* saved, float2* Z, float* zbuf,
                      float* ubuf, const mp::PermTabs& pt, bool tables_built, const MpTabs& t, hipStream_t s) {
  const mp::Geo g = mp_geo(N);
  const bool perm_on = (flags & kFlagPerm) != 0, relu = (flags & kFlagRelu) != 0;
  if (perm_on && !tables_built) MP_TRY(mp_perm_prebuild(perm, N, K, pt, s));
  for (int k = 0; k < K; ++k) {
    const float* src = k == 0 ? x : zbuf;
    float* slot = mp_slot(saved, k, K, batch, N, perm_on);
    const float* u = src;
    if (perm_on) {
      const int32_t* pk = perm + (long long)k * N;
      float* udst = slot != nullptr ? slot : ubuf;
      mp::PermTabs tk;
      MP_TRY(mp_perm_tabs(perm, N, K, k, pt, &tk, s));
      MP_TRY(mp::permute(src, udst, reinterpret_cast<float*>(Z), pk, tk, batch, N, s));
      u = udst;
      slot = nullptr;  // already stashed
    }
    int rc = mp_pack_fft(u, A + (long long)k * N, slot, Z, batch, N, g, t, s);
    if (rc != ACDC_OK) return rc;
    MP_TRY(mp::mid_fwd(Z, Mq + (long long)k * (N / 4) * kMqRows, batch, g, (flags & kFlagBias) != 0, s));
    rc = mp_ifft_unpack(Z, (k == K - 1 && y != nullptr) ? y : zbuf, batch, N, relu && k < K - 1, g, t, s);
    if (rc != ACDC_OK) return rc;
  }
  return ACDC_OK;
}

// ------------------------------------------------ complex (AFDF) multi-pass
// Rows of N complex elements are their own N-point FFT inputs (M = N, the
// geometry and twiddles of a real width 2N).  Per layer: u = z[perm] (into
// the stash slot), Z = FFT(u * a), Z *= d / N, z' = unnormalised IFFT(Z).
int mp_cplx_forward_layers(const float2* x, float2* y, const float2* A, const float2* D, const int32_t* perm,
                           int64_t batch, int32_t N, int32_t K, uint32_t flags, float* saved, float2* Z,
                           float2* zbuf, float2* ubuf, const mp::PermTabs& pt, bool tables_built, const MpTabs& t,
                           hipStream_t s) {
  const mp::Geo g = mp_geo(2LL * N);
  const bool perm_on = (flags & kFlagPerm) != 0;
  const float invN = 1.0f / float(N);
  if (perm_on && !tables_built) MP_TRY(mp_perm_prebuild(perm, N, K, pt, s, 2));
  for (int k = 0; k < K; ++k) {
    const float2* src = k == 0 ? x : zbuf;
    float2* slot = reinterpret_cast<float2*>(mp_slot(saved, k, K, batch, 2LL * N, perm_on));
    const float2* u = src;
    if (perm_on) {
      const int32_t* pk = perm + (long long)k * N;
      float2* udst = slot != nullptr ? slot : ubuf;
      mp::PermTabs tk;
      MP_TRY(mp_perm_tabs(perm, N, K, k, pt, &tk, s, 2));
      MP_TRY(mp::cpermute(src, udst, Z, pk, tk, batch, N, s));
      u = udst;
      slot = nullptr;  // already stashed
    }
    MP_TRY(mp::cfft_in(u, A + (long long)k * N, slot, Z, batch, g, t.tw, t.seg, s));
    MP_TRY(mp::cmid_fwd(Z, D + (long long)k * N, batch, g, invN, s));
    MP_TRY(mp::cifft_out(Z, (k == K - 1 && y != nullptr) ? y : zbuf, batch, g, t.tw, t.seg, s));
  }
  return ACDC_OK;
}

int mp_cplx_forward(const float* x, float* y, const float* A, const float* D, const int32_t* perm, int64_t batch,
                    int32_t N, int32_t K, uint32_t flags, float* saved, void* workspace, hipStream_t s) {
  MpTabs t;
  int rc = get_mp_tables(2 * N, &t);
  if (rc != ACDC_OK) return rc;
  const MpFwdWs w = mp_fwd_ws(batch, N, K, flags);
  char* ws = static_cast<char*>(workspace);
  const mp::PermTabs pt = mp::perm_tables_at(reinterpret_cast<int*>(ws + w.ptab), N, 2);
  ProfScope prof(0, s);
  if (batch == 0) return ACDC_OK;
  return mp_cplx_forward_layers(reinterpret_cast<const float2*>(x), reinterpret_cast<float2*>(y),
                                reinterpret_cast<const float2*>(A), reinterpret_cast<const float2*>(D), perm, batch,
                                N, K, flags, saved, reinterpret_cast<float2*>(ws + w.z),
                                reinterpret_cast<float2*>(ws + w.zbuf), reinterpret_cast<float2*>(ws + w.ubuf), pt,
                                false, t, s);
}

// Backward per layer (the fused complex kernels' steps): gh3 = FFT(g) / N,
// h2 = FFT(u * a), dL/dd += gh3 conj(h2), gh1 = IFFT(gh3 conj(d)),
// dL/da += gh1 conj(u), g_u = gh1 conj(a), scattered back through perm.
int mp_cplx_backward(const float* x, const float* grad_y, const float* A, const float* D, const int32_t* perm,
                     const float* saved, float* grad_x, float* grad_A, float* grad_D, int64_t batch, int32_t N,
                     int32_t K, uint32_t flags, bool have_saved, void* workspace, hipStream_t s) {
  MpTabs t;
  int rc = get_mp_tables(2 * N, &t);
  if (rc != ACDC_OK) return rc;
  const MpBwdWs w = mp_bwd_ws(batch, N, K, flags, have_saved);
  char* ws = static_cast<char*>(workspace);
  float2* Zh = reinterpret_cast<float2*>(ws + w.zhg);
  float2* Zg = Zh + batch * N;  // the g spectra follow the h spectra
  float2* gh1 = reinterpret_cast<float2*>(ws + w.gh1);
  float2* gbuf = reinterpret_cast<float2*>(ws + w.gbuf);
  float2* imgA = reinterpret_cast<float2*>(ws + w.imgA);
  float2* gu = reinterpret_cast<float2*>(ws + w.gu);
  float* part = reinterpret_cast<float*>(ws + w.part);
  float* stash = have_saved ? const_cast<float*>(saved) : reinterpret_cast<float*>(ws + w.stash);
  const mp::PermTabs pt = mp::perm_tables_at(reinterpret_cast<int*>(ws + w.ptab), N, 2);
  const mp::Geo g = mp_geo(2LL * N);
  const bool perm_on = (flags & kFlagPerm) != 0, acc = (flags & kFlagAccumulate) != 0;
  const float invN = 1.0f / float(N);
  const long long W = 2LL * N;  // floats per row
  const float2* x2 = reinterpret_cast<const float2*>(x);
  const float2* A2 = reinterpret_cast<const float2*>(A);
  const float2* D2 = reinterpret_cast<const float2*>(D);
  ProfScope prof(1, s);
  if (batch > 0) {
    if (perm_on) MP_TRY(mp_perm_prebuild(perm, N, K, pt, s, 2));
    if (!have_saved) {
      // recompute the layer inputs into the workspace (Zh, gh1 are free until the layer loop)
      rc = mp_cplx_forward_layers(x2, nullptr, A2, D2, perm, batch, N, K, flags, stash, Zh, gh1, nullptr, pt, true,
                                  t, s);
      if (rc != ACDC_OK) return rc;
    }
  }
  for (int k = K - 1; k >= 0; --k) {
    float* gA = grad_A + (long long)k * W;
    float* gD = grad_D + (long long)k * W;
    if (batch > 0) {
      const float2* u = k > 0 || perm_on ? reinterpret_cast<const float2*>(mp_slot(stash, k, K, batch, W, perm_on))
                                         : x2;
      const float2* ak = A2 + (long long)k * N;
      MP_TRY(mp::cfft_in(k == K - 1 ? reinterpret_cast<const float2*>(grad_y) : gbuf, nullptr, nullptr, Zg, batch, g,
                         t.tw, t.seg, s));
      MP_TRY(mp::cfft_in(u, ak, nullptr, Zh, batch, g, t.tw, t.seg, s));
      MP_TRY(mp::cmid_bwd(Zh, Zg, D2 + (long long)k * N, batch, g, invN, reinterpret_cast<float2*>(part), s));
      MP_TRY(mp::colsum_parts(part, batch, W, gD, nullptr, acc, s));
      MP_TRY(mp::cifft_out(Zg, gh1, batch, g, t.tw, t.seg, s));
      float2* gnext = reinterpret_cast<float2*>(k == 0 ? grad_x : reinterpret_cast<float*>(gbuf));
      if (perm_on) {
        const int32_t* pk = perm + (long long)k * N;
        mp::PermTabs tk;
        MP_TRY(mp_perm_tabs(perm, N, K, k, pt, &tk, s, 2));
        MP_TRY(mp::cdA(gh1, u, ak, imgA, gu, batch, N, s));
        MP_TRY(mp::cpermute_adjoint(gu, gnext, Zh, pk, tk, batch, N, s));  // Zh is free again
      } else {
        MP_TRY(mp::cdA(gh1, u, ak, imgA, gnext, batch, N, s));
      }
      MP_TRY(mp::colsum(reinterpret_cast<const float*>(imgA), batch, W, part, gA, nullptr, acc, s));
    } else {
      // no rows: zero (or unchanged, accumulating) parameter gradients
      MP_TRY(mp::colsum(nullptr, 0, W, part, gD, nullptr, acc, s));
      MP_TRY(mp::colsum(nullptr, 0, W, part, gA, nullptr, acc, s));
    }
  }
  return ACDC_OK;
}

int mp_forward(const float* x, float* y, const float* A, const float* D, const float* bias, const int32_t* perm,
               int64_t batch, int32_t N, int32_t K, uint32_t flags, float* saved, void* workspace, hipStream_t s) {
  if (flags & kFlagComplex) return mp_cplx_forward(x, y, A, D, perm, batch, N, K, flags, saved, workspace, s);
  MpTabs t;
  int rc = get_mp_tables(N, &t);
  if (rc != ACDC_OK) return rc;
  const MpFwdWs w = mp_fwd_ws(batch, N, K, flags);
  char* ws = static_cast<char*>(workspace);
  float4* Mq = reinterpret_cast<float4*>(ws + w.mq);
  float2* Z = reinterpret_cast<float2*>(ws + w.z);
  float* zbuf = reinterpret_cast<float*>(ws + w.zbuf);
  float* ubuf = reinterpret_cast<float*>(ws + w.ubuf);
  const mp::PermTabs pt = mp::perm_tables_at(reinterpret_cast<int*>(ws + w.ptab), N);
  ProfScope prof(0, s);
  MP_TRY(mp::mq(D, bias, Mq, K, N / 4, t.q, s));
  if (batch == 0) return ACDC_OK;
  return mp_forward_layers(x, y, A, Mq, perm, batch, N, K, flags, saved, Z, zbuf, ubuf, pt, false, t, s);
}

int mp_backward(const float* x, const float* grad_y, const float* A, const float* D, const float* bias,
                const int32_t* perm, const float* saved, float* grad_x, float* grad_A, float* grad_D,
                float* grad_bias, int64_t batch, int32_t N, int32_t K, uint32_t flags, bool have_saved,
                void* workspace, hipStream_t s) {
  if (flags & kFlagComplex)
    return mp_cplx_backward(x, grad_y, A, D, perm, saved, grad_x, grad_A, grad_D, batch, N, K, flags, have_saved,
                            workspace, s);
  MpTabs t;
  int rc = get_mp_tables(N, &t);
  if (rc != ACDC_OK) return rc;
  const MpBwdWs w = mp_bwd_ws(batch, N, K, flags, have_saved);
  char* ws = static_cast<char*>(workspace);
  float4* Mq = reinterpret_cast<float4*>(ws + w.mq);
  float2* Zh = reinterpret_cast<float2*>(ws + w.zhg);
  float2* Zg = Zh + batch * (N / 2);  // the g spectra follow the h spectra
  float* gh1 = reinterpret_cast<float*>(ws + w.gh1);
  float* gbuf = reinterpret_cast<float*>(ws + w.gbuf);
  float* imgA = reinterpret_cast<float*>(ws + w.imgA);
  float* part = reinterpret_cast<float*>(ws + w.part);
  float* partB = (flags & kFlagBias) ? reinterpret_cast<float*>(ws + w.partB) : nullptr;
  float* stash = have_saved ? const_cast<float*>(saved) : reinterpret_cast<float*>(ws + w.stash);
  const mp::PermTabs pt = mp::perm_tables_at(reinterpret_cast<int*>(ws + w.ptab), N);
  const mp::Geo g = mp_geo(N);
  const bool perm_on = (flags & kFlagPerm) != 0, relu = (flags & kFlagRelu) != 0;
  const bool acc = (flags & kFlagAccumulate) != 0;
  ProfScope prof(1, s);
  if (batch > 0) {
    MP_TRY(mp::mq(D, bias, Mq, K, N / 4, t.q, s));
    if (perm_on) MP_TRY(mp_perm_prebuild(perm, N, K, pt, s));
    if (!have_saved) {
      // recompute the layer inputs into the workspace (Zh, gh1 are free until the layer loop)
      rc = mp_forward_layers(x, nullptr, A, Mq, perm, batch, N, K, flags, stash, Zh, gh1, nullptr, pt, true, t, s);
      if (rc != ACDC_OK) return rc;
    }
  }
  for (int k = K - 1; k >= 0; --k) {
    float* gA = grad_A + (long long)k * N;
    float* gD = grad_D + (long long)k * N;
    float* gB = grad_bias ? grad_bias + (long long)k * N : nullptr;
    if (batch > 0) {
      const float* u = k > 0 || perm_on ? mp_slot(stash, k, K, batch, N, perm_on) : x;
      const float* ak = A + (long long)k * N;
      rc = mp_pack_fft(k == K - 1 ? grad_y : gbuf, nullptr, nullptr, Zg, batch, N, g, t, s);
      if (rc != ACDC_OK) return rc;
      rc = mp_pack_fft(u, ak, nullptr, Zh, batch, N, g, t, s);
      if (rc != ACDC_OK) return rc;
      MP_TRY(mp::mid_bwd(Zh, Zg, Mq + (long long)k * (N / 4) * kMqRows, batch, g, part, partB, s));
      MP_TRY(mp::colsum_parts(part, batch, N, gD, &t.q, acc, s));
      if (gB) MP_TRY(mp::colsum_parts(partB, batch, N, gB, &t.q, acc, s));
      rc = mp_ifft_unpack(Zg, gh1, batch, N, false, g, t, s);
      if (rc != ACDC_OK) return rc;
      float* gnext = k == 0 ? grad_x : gbuf;
      if (perm_on) {
        // Zh and Zg are free again: the permutation's scratch
        const int32_t* pk = perm + (long long)k * N;
        mp::PermTabs tk;
        MP_TRY(mp_perm_tabs(perm, N, K, k, pt, &tk, s));
        MP_TRY(mp::dA_permute(gh1, u, ak, relu && k > 0, imgA, gnext, reinterpret_cast<float*>(Zh), pk, tk, batch,
                              N, s));
      } else {
        MP_TRY(mp::dA(gh1, u, ak, relu && k > 0, imgA, gnext, batch, N, s));
      }
      MP_TRY(mp::colsum(imgA, batch, N, part, gA, nullptr, acc, s));
    } else {
      // no rows: zero (or unchanged, accumulating) parameter gradients
      MP_TRY(mp::colsum(nullptr, 0, N, part, gD, &t.q, acc, s));
      if (gB) MP_TRY(mp::colsum(nullptr, 0, N, part, gB, &t.q, acc, s));
      MP_TRY(mp::colsum(nullptr, 0, N, part, gA, nullptr, acc, s));
    }
  }
  return ACDC_OK;
}

// The fused forward's launches (per-layer quartet coefficients into
// `workspace`, then the cascade).  `remember` false: cache nothing on the host.
int fused_forward(const float* x, float* y, const float* A, const float* D, const float* bias, const int32_t* perm,
                  int64_t batch, int32_t N, int32_t K, uint32_t flags, float* saved, void* workspace,
                  const char* tab, hipStream_t s, bool remember) {
  int rc = ACDC_ERR_UNSUPPORTED;
  if (flags & kFlagComplex) {
    dispatch_complex(N, [&]<class PL>() {
      CplxArgs a{x, y, A, D, perm, saved, nullptr, nullptr, nullptr, tab, batch, K, flags};
      rc = launch_cplx_fwd<PL>(a, s);
    });
  } else {
    dispatch_real(N, [&]<class PL>() {
      float4* Mq = static_cast<float4*>(workspace);
      rc = launch_real_mq<PL>(D, bias, Mq, K, tab, perm, nullptr, s);
      if (rc != ACDC_OK) return;
      RealArgs a{x, y, A, Mq, perm, saved, nullptr, nullptr, nullptr, tab, batch, K, flags};
      rc = launch_real_fwd<PL>(a, s, remember);
    });
  }
  return rc;
}

}  // namespace
}  // namespace acdc

using namespace acdc;

extern "C" int acdc_supported(int32_t N, uint32_t flags) {
  if (flags & ~kAllFlags) return 0;
  if (!flags_supported(flags)) return 0;
  return supported(N, flags) ? 1 : 0;
}

extern "C" int acdc_prepare(int32_t N, uint32_t flags) {
  if (!acdc_supported(N, flags)) return ACDC_ERR_UNSUPPORTED;
  int rc = scratch_setup();
  if (rc != ACDC_OK) return rc;
  if (use_multipass(N, flags)) {
    MpTabs t;
    return get_mp_tables((flags & kFlagComplex) ? 2 * N : N, &t);
  }
  const char* tab = nullptr;
  rc = get_table(N, (flags & kFlagComplex) != 0, &tab);
  if (rc != ACDC_OK || (flags & kFlagComplex)) return rc;
  // cache the persistent grids, so that later calls look them up
  dispatch_real(N, [&]<class PL>() {
    (void)resident_workgroups(reinterpret_cast<const void*>(&k_real_fwd<PL, false>), Launch<PL>::FWD_THREADS);
    (void)resident_workgroups(reinterpret_cast<const void*>(&k_real_fwd<PL, true>), Launch<PL>::FWD_THREADS);
    if constexpr (Launch<PL>::BWD_ACC)
      (void)resident_workgroups(reinterpret_cast<const void*>(&k_real_bwd<PL, false>), Launch<PL>::BWD_THREADS);
  });
  return ACDC_OK;
}

extern "C" size_t acdc_saved_bytes(int64_t batch, int32_t N, int32_t K, uint32_t flags) {
  if (check_common(batch, N, K, flags) != ACDC_OK) return 0;
  return saved_floats(batch, N, K, flags) * sizeof(float);
}

extern "C" size_t acdc_forward_workspace_size(int64_t batch, int32_t N, int32_t K, uint32_t flags) {
  if (check_common(batch, N, K, flags) != ACDC_OK) return 0;
  if (use_multipass(N, flags)) return mp_fwd_ws(batch, N, K, flags).total;
  return fwd_ws(N, K, flags);
}

extern "C" size_t acdc_backward_workspace_size(int64_t batch, int32_t N, int32_t K, uint32_t flags,
                                                int have_saved) {
  if (check_common(batch, N, K, flags) != ACDC_OK) return 0;
  const bool hs = have_saved != 0 || saved_layers(K, flags) == 0;
  if (use_multipass(N, flags)) return mp_bwd_ws(batch, N, K, flags, hs).total;
  return bwd_layout(batch, N, K, flags, hs).total;
}

extern "C" int acdc_forward(const float* x, float* y, const float* A, const float* D, const float* bias,
                            const int32_t* perm, int64_t batch, int32_t N, int32_t K, uint32_t flags, float* saved,
                            size_t saved_bytes, void* workspace, size_t workspace_bytes, acdc_stream_t stream) {
  int rc = check_common(batch, N, K, flags);
  if (rc != ACDC_OK) return rc;
  if (saved != nullptr && saved_bytes < saved_floats(batch, N, K, flags) * sizeof(float)) return ACDC_ERR_WORKSPACE;
  const bool perm_on = (flags & kFlagPerm) != 0;
  const bool bias_on = (flags & kFlagBias) != 0;
  if (batch == 0) return ACDC_OK;
  rc = check_ptrs({x, y, A, D}, {perm_on ? (const void*)perm : nullptr, bias_on ? (const void*)bias : nullptr,
                                 saved, workspace});
  if (rc != ACDC_OK) return rc;
  if ((perm_on && perm == nullptr) || (bias_on && bias == nullptr)) return ACDC_ERR_INVALID_ARG;
  if (!bias_on) bias = nullptr;
  if (!distinct({y, saved}, {x, y, A, D, bias, perm, saved, workspace})) return ACDC_ERR_INVALID_ARG;
  const bool multipass = use_multipass(N, flags);
  const size_t need = multipass ? mp_fwd_ws(batch, N, K, flags).total : fwd_ws(N, K, flags);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return ACDC_ERR_WORKSPACE;
  if (multipass)
    return mp_forward(x, y, A, D, bias, perm, batch, N, K, flags, saved, workspace,
                      reinterpret_cast<hipStream_t>(stream));
  const bool cplx = (flags & kFlagComplex) != 0;
  const char* tab = nullptr;
  rc = get_table(N, cplx, &tab);
  if (rc != ACDC_OK) return rc;
  return fused_forward(x, y, A, D, bias, perm, batch, N, K, flags, saved, workspace, tab,
                       reinterpret_cast<hipStream_t>(stream), true);
}

extern "C" int acdc_forward_noalloc(const float* x, float* y, const float* A, const float* D, const float* bias,
                                    const int32_t* perm, int64_t batch, int32_t N, int32_t K, uint32_t flags,
                                    float* saved, size_t saved_bytes, acdc_stream_t stream) {
  int rc = check_common(batch, N, K, flags);
  if (rc != ACDC_OK) return rc;
  if (use_multipass(N, flags)) return ACDC_ERR_UNSUPPORTED;  // its workspace grows with the batch
  if (saved != nullptr && saved_bytes < saved_floats(batch, N, K, flags) * sizeof(float)) return ACDC_ERR_WORKSPACE;
  const size_t need = fwd_ws(N, K, flags);
  if (need > kNoAllocScratchBytes) return ACDC_ERR_WORKSPACE;
  const bool perm_on = (flags & kFlagPerm) != 0;
  const bool bias_on = (flags & kFlagBias) != 0;
  if (batch == 0) return ACDC_OK;
  rc = check_ptrs({x, y, A, D}, {perm_on ? (const void*)perm : nullptr, bias_on ? (const void*)bias : nullptr, saved});
  if (rc != ACDC_OK) return rc;
  if ((perm_on && perm == nullptr) || (bias_on && bias == nullptr)) return ACDC_ERR_INVALID_ARG;
  if (!bias_on) bias = nullptr;
  if (!distinct({y, saved}, {x, y, A, D, bias, perm, saved})) return ACDC_ERR_INVALID_ARG;
  int dev = 0;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e);
  if (dev < 0 || dev >= kMaxDevices) return ACDC_ERR_UNSUPPORTED;
  const bool cplx = (flags & kFlagComplex) != 0;
  const char* tab = find_table(dev, N, cplx);
  void* ws = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    ws = g_scratch_ptr[dev];
  }
  if (tab == nullptr || ws == nullptr) return ACDC_ERR_NOT_PREPARED;
  return fused_forward(x, y, A, D, bias, perm, batch, N, K, flags, saved, ws, tab,
                       reinterpret_cast<hipStream_t>(stream), false);
}

extern "C" int acdc_backward(const float* x, const float* grad_y, const float* A, const float* D,
                             const float* bias, const int32_t* perm, const float* saved, size_t saved_bytes,
                             float* grad_x, float* grad_A, float* grad_D, float* grad_bias, int64_t batch,
                             int32_t N, int32_t K, uint32_t flags, void* workspace, size_t workspace_bytes,
                             acdc_stream_t stream) {
  int rc = check_common(batch, N, K, flags);
  if (rc != ACDC_OK) return rc;
  if (saved != nullptr && saved_bytes < saved_floats(batch, N, K, flags) * sizeof(float)) return ACDC_ERR_WORKSPACE;
  const bool perm_on = (flags & kFlagPerm) != 0;
  const bool bias_on = (flags & kFlagBias) != 0;
  const int accumulate = (flags & kFlagAccumulate) != 0 ? 1 : 0;
  if (!bias_on) {
    bias = nullptr;
    grad_bias = nullptr;
  }
  rc = check_ptrs({A, D, grad_A, grad_D}, {perm_on ? (const void*)perm : nullptr, bias, grad_bias, saved, workspace});
  if (rc != ACDC_OK) return rc;
  if (bias_on && (bias == nullptr || grad_bias == nullptr)) return ACDC_ERR_INVALID_ARG;
  if (batch > 0) {
    rc = check_ptrs({x, grad_y, grad_x}, {});
    if (rc != ACDC_OK) return rc;
    if (perm_on && perm == nullptr) return ACDC_ERR_INVALID_ARG;
  }
  if (!distinct({grad_x, grad_A, grad_D, grad_bias},
                {x, grad_y, A, D, bias, perm, saved, grad_x, grad_A, grad_D, grad_bias, workspace}))
    return ACDC_ERR_INVALID_ARG;
  // nothing to recompute when no layer input needs storing (K == 1 without PERM)
  const bool have_saved = saved != nullptr || saved_layers(K, flags) == 0;
  if (use_multipass(N, flags)) {
    const size_t need = mp_bwd_ws(batch, N, K, flags, have_saved).total;
    if (workspace == nullptr || workspace_bytes < need) return ACDC_ERR_WORKSPACE;
    return mp_backward(x, grad_y, A, D, bias, perm, saved, grad_x, grad_A, grad_D, grad_bias, batch, N, K, flags,
                       have_saved, workspace, reinterpret_cast<hipStream_t>(stream));
  }
  const WsLayout w = bwd_layout(batch, N, K, flags, have_saved);
  if (w.total > 0 && (workspace == nullptr || workspace_bytes < w.total)) return ACDC_ERR_WORKSPACE;
  const bool cplx = (flags & kFlagComplex) != 0;
  const char* tab = nullptr;
  rc = get_table(N, cplx, &tab);
  if (rc != ACDC_OK) return rc;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  float* partial = reinterpret_cast<float*>(ws + w.off_partial);
  float* stash = have_saved ? const_cast<float*>(saved) : reinterpret_cast<float*>(ws + w.off_stash);
  if (cplx) {
    dispatch_complex(N, [&]<class PL>() {
      using L = Launch<PL>;
      const long long tiles = bwd_tiles<PL>(batch);
      if (batch > 0) {
        if (!have_saved) {
          CplxArgs f{x, nullptr, A, D, perm, stash, nullptr, nullptr, nullptr, tab, batch, K, flags};
          rc = launch_cplx_fwd<PL>(f, s);
          if (rc != ACDC_OK) return;
        }
        CplxArgs a{x, nullptr, A, D, perm, stash, grad_y, grad_x, partial, tab, batch, K, flags};
        hipError_t e;
        {
          ProfScope prof(1, s);
          hipLaunchKernelGGL(k_cplx_bwd<PL>, dim3(unsigned(tiles)), dim3(L::BWD_THREADS), 0, s, a);
          e = hipGetLastError();
        }
        if (e != hipSuccess) {
          rc = hip_fail(e);
          return;
        }
      }
      const long long n = (long long)K * partial_entries4<PL>();
      hipError_t e;
      {
        ProfScope prof(2, s);
        auto reduce = [&]<int PH>() {
          constexpr int E = kRedThreads / PH;
          hipLaunchKernelGGL((k_cplx_reduce<PL, PH>), dim3(unsigned((n + E - 1) / E)), dim3(kRedThreads), 0, s,
                             partial, tiles, K, grad_A, grad_D, accumulate);
        };
        if (red_phases(n) == 8) reduce.template operator()<8>();
        else reduce.template operator()<4>();
        e = hipGetLastError();
      }
      rc = e == hipSuccess ? ACDC_OK : hip_fail(e);
    });
  } else {
    dispatch_real(N, [&]<class PL>() {
      using L = Launch<PL>;
      const long long tiles = bwd_tiles<PL>(batch);
      // partial slots: one per tile, or one per resident workgroup of the
      // persistent (accumulating) unbiased backward
      const long long slots =
          (L::BWD_ACC && !bias_on)
              ? persistent_grid(reinterpret_cast<const void*>(&k_real_bwd<PL, false>), L::BWD_THREADS, tiles)
              : tiles;
      float4* Mq = reinterpret_cast<float4*>(ws + w.off_mq);
      int4* P16 = batch > 0 ? perm16_of<PL>(Mq, K, flags) : nullptr;
      float* gS = bias_on ? reinterpret_cast<float*>(ws + w.off_gs) : nullptr;
      if (batch > 0 || bias_on) {
        rc = launch_real_mq<PL>(D, bias, Mq, K, tab, perm, P16, s);
        if (rc != ACDC_OK) return;
      }
      if (batch > 0) {
        if (!have_saved) {
          RealArgs f{x, nullptr, A, Mq, perm, stash, nullptr, nullptr, nullptr, tab, batch, K, flags};
          rc = launch_real_fwd<PL>(f, s);
          if (rc != ACDC_OK) return;
        }
        RealArgs a{x, nullptr, A, Mq, perm, stash, grad_y, grad_x, partial, tab, batch, K, flags};
        a.perm16 = P16;
        hipError_t e;
        {
          ProfScope prof(1, s);
          if (bias_on)
            hipLaunchKernelGGL((k_real_bwd<PL, true>), dim3(unsigned(tiles)), dim3(L::BWD_THREADS), 0, s, a, tiles);
          else
            hipLaunchKernelGGL((k_real_bwd<PL, false>), dim3(unsigned(slots)), dim3(L::BWD_THREADS), 0, s, a, tiles);
          e = hipGetLastError();
        }
        if (e != hipSuccess) {
          rc = hip_fail(e);
          return;
        }
      }
      const long long n = (long long)K * partial_entries4<PL>(bias_on);
      hipError_t e;
      {
        ProfScope prof(2, s);
        auto reduce = [&]<int PH>() {
          constexpr int E = kRedThreads / PH;
          hipLaunchKernelGGL((k_real_reduce<PL, PH>), dim3(unsigned((n + E - 1) / E)), dim3(kRedThreads), 0, s,
                             partial, slots, K, grad_A, grad_D, gS, tab, bias_on ? 1 : 0, accumulate);
        };
        if (red_phases(n) == 8) reduce.template operator()<8>();
        else reduce.template operator()<4>();
        e = hipGetLastError();
        if (e == hipSuccess && bias_on) {
          hipLaunchKernelGGL(k_real_dct<PL>, dim3(unsigned(K)), dim3(PL::T), 0, s, gS, grad_bias, Mq, tab,
                             accumulate);
          e = hipGetLastError();
        }
      }
      rc = e == hipSuccess ? ACDC_OK : hip_fail(e);
    });
  }
  return rc;
}

extern "C" int acdc_profile_enable(int enable) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  g_prof_on = enable != 0;
  return ACDC_OK;
}

extern "C" int acdc_profile_read(double* ms, int64_t* launches) {
  if (ms == nullptr || launches == nullptr) return ACDC_ERR_INVALID_ARG;
  for (int i = 0; i < 3; ++i) {
    ms[i] = 0.0;
    launches[i] = 0;
  }
  std::lock_guard<std::mutex> lock(g_prof_mu);
  int rc = ACDC_OK;
  for (const ProfRec& r : g_prof_recs) {
    float t = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&t, r.a, r.b);
    if (e != hipSuccess) rc = hip_fail(e);
    ms[r.kind] += t;
    launches[r.kind] += 1;
    g_prof_pool.push_back(r.a);
    g_prof_pool.push_back(r.b);
  }
  g_prof_recs.clear();
  return rc;
}

extern "C" const char* acdc_status_string(int status) {
  switch (status) {
    case ACDC_OK: return "ok";
    case ACDC_ERR_INVALID_ARG: return "invalid argument";
    case ACDC_ERR_UNSUPPORTED: return "unsupported width or flag combination";
    case ACDC_ERR_WORKSPACE: return "workspace missing or too small";
    case ACDC_ERR_HIP: return "HIP runtime error";
    case ACDC_ERR_NOT_PREPARED: return "width not prepared on this device (call acdc_prepare first)";
    default: return "unknown status";
  }
}

extern "C" int acdc_last_hip_error(void) { return g_last_hip; }

extern "C" int acdc_sync_timeouts(int64_t* count, int clear) {
  if (count == nullptr) return ACDC_ERR_INVALID_ARG;
  *count = 0;
  unsigned long long n = 0;
  hipError_t e = hipMemcpyFromSymbol(&n, HIP_SYMBOL(sync_timeouts), sizeof(n), 0, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e);
  *count = (int64_t)n;
  if (clear != 0 && n != 0) {
    const unsigned long long zero = 0;
    e = hipMemcpyToSymbol(HIP_SYMBOL(sync_timeouts), &zero, sizeof(zero), 0, hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e);
  }
  return ACDC_OK;
}
