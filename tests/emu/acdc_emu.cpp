// CPU emulation of the HIP kernels' row bodies (test infrastructure).
//
// The same __host__ __device__ templates that the GPU kernels instantiate are
// run here with one OS thread per GPU thread and a std::barrier standing in
// for every LDS synchronisation, on host memory.  This checks the index
// algebra, the plan tables and the reduction order on the CPU; the GPU tests
// then check the real kernels.  Built by tests/emu/build_emu.py.
#include <barrier>
#include <cstring>
#include <cstdio>
#include <thread>
#include <vector>

#include "../../paper_1511_05946_amd/csrc/acdc_registry.hpp"

using namespace acdc;

namespace {

struct HostCtx {
  std::barrier<>* bar;
  int tid;
  float* xa;  // per-thread exchange slots of the cross-lane swaps
  float* xb;
  void sync_row() { bar->arrive_and_wait(); }
  void sync_all() { bar->arrive_and_wait(); }
  // The GPU's permlane16 / permlane32 swaps (acdc_devctx.hpp), through
  // shared slots between two barriers.
  template <int W>
  void swap(float& a, float& b) {
    xa[tid] = a;
    xb[tid] = b;
    bar->arrive_and_wait();
    const int lane = tid % 64, base = tid - lane;
    const bool upper = (lane / W) % 2 == 1;  // odd row (W = 16) or upper half (W = 32)
    const int partner = base + (upper ? lane - W : lane + W);
    const float na = upper ? xb[partner] : xa[tid];
    const float nb = upper ? xb[tid] : xa[partner];
    bar->arrive_and_wait();
    a = na;
    b = nb;
  }
  void swap16(float& a, float& b) { swap<16>(a, b); }
  void swap32(float& a, float& b) { swap<32>(a, b); }
};

template <class F>
void run_wg(int threads, F&& body) {
  std::barrier<> bar(threads);
  std::vector<float> xa(threads), xb(threads);
  std::vector<std::thread> th;
  th.reserve(threads);
  for (int tid = 0; tid < threads; ++tid)
    th.emplace_back([&, tid] {
      HostCtx ctx{&bar, tid, xa.data(), xb.data()};
      body(ctx, tid);
    });
  for (auto& x : th) x.join();
}

// The batch reduction in the GPU kernel's order: per entry, the phase sums
// in phase order.
template <class PL, class Store>
void reduce_all(const float* partial, long long ntiles, int K, long long PS4, Store&& store) {
  const long long n = (long long)K * PS4;
  auto run = [&]<int PH>() {
    for (long long i = 0; i < n; ++i) {
      float4 ph[PH];
      for (int g = 0; g < PH; ++g)
        ph[g] = tile_phase_sum4<PH>(reinterpret_cast<const float4*>(partial), ntiles, n, i, g);
      store(phases_total4<PH>(ph), int(i / PS4), int(i % PS4));
    }
  };
  if (red_phases(n) == 8) run.template operator()<8>();
  else run.template operator()<4>();
}

// Per-layer quartet coefficients in the kernel's [k][slot][kMqRows][T] layout.
template <class PL>
std::vector<float4> quartet_coefficients(const float* D, const float* B, int K, const std::vector<unsigned char>& tab) {
  constexpr int E = PL::NSL * PL::T;
  std::vector<float4> mq((size_t)K * E * kMqRows);
  for (int k = 0; k < K; ++k)
    for (int e = 0; e < E; ++e) {
      float4 row[kMqRows];
      real_mq_entry<PL>(D + (size_t)k * PL::N, B ? B + (size_t)k * PL::N : nullptr, (const char*)tab.data(), e, row);
      const int slot = e / PL::T, t = e % PL::T;
      for (int r = 0; r < kMqRows; ++r)
        mq[(size_t)k * E * kMqRows + (size_t)(slot * kMqRows + r) * PL::T + t] = row[r];
    }
  return mq;
}

// The packed perm the backward reads where the plan packs it (k_real_mq's
// extra threads on the GPU); empty otherwise.
template <class PL>
std::vector<int4> packed_perm(const int* perm, int K, unsigned flags) {
  using O = RealOps<PL>;
  std::vector<int4> p;
  if (!O::kPackedPerm || !(flags & kFlagPerm) || perm == nullptr) return p;
  p.resize((size_t)K * O::NIW * PL::T);
  for (int k = 0; k < K; ++k)
    for (int j = 0; j < O::NIW; ++j)
      for (int t = 0; t < PL::T; ++t)
        p[((size_t)k * O::NIW + j) * PL::T + t] = O::pack_perm_entry(perm + (size_t)k * PL::N, j, unsigned(t));
  return p;
}

template <class PL, bool BIAS>
void real_fwd_k(const RealArgs& a, const std::vector<unsigned char>& tab) {
  using L = Launch<PL>;
  const long long nwg = (a.batch + L::FWD_ROWS - 1) / L::FWD_ROWS;
  std::vector<float> lds((size_t)L::FWD_LDS_FLOATS);
  float* twl = lds.data();
  float* rows = lds.data() + L::TW_FLOATS;
  if (L::TW_LDS) std::memcpy(twl, tab.data(), (size_t)PL::TW_FLOAT2 * 8);
  for (long long wg = 0; wg < nwg; ++wg)
    run_wg(L::FWD_THREADS, [&](HostCtx& ctx, int tid) {
      const int r = tid / PL::T, t = tid % PL::T;
      float* slab = rows + (size_t)r * L::FWD_SLAB;
      if constexpr (L::TW_LDS)
        real_forward_row<PL, BIAS>(ctx, a, unsigned(t), wg * L::FWD_ROWS, unsigned(r), slab, LdsView::of(twl));
      else
        real_forward_row<PL, BIAS>(ctx, a, unsigned(t), wg * L::FWD_ROWS, unsigned(r), slab, GView::of(tab.data()));
    });
}

template <class PL>
void real_fwd(const float* x, float* y, const float* A, const float* D, const float* B, const int* perm,
              long long batch, int K, unsigned flags, float* saved, const std::vector<unsigned char>& tab) {
  const std::vector<float4> mq = quartet_coefficients<PL>(D, (flags & kFlagBias) ? B : nullptr, K, tab);
  RealArgs a{x, y, A, mq.data(), perm, saved, nullptr, nullptr, nullptr, (const char*)tab.data(), batch, K, flags};
  if (flags & kFlagBias) real_fwd_k<PL, true>(a, tab);
  else real_fwd_k<PL, false>(a, tab);
}

// Persistent backward workgroups to emulate (0: one workgroup per tile, as
// the GPU runs plans without persistent accumulation or with at least as
// many resident workgroups as tiles).
long long g_bwd_slots = 0;

template <class PL, bool BIAS>
constexpr bool emu_acc() {
  return Launch<PL>::BWD_ACC && !BIAS;
}

// Partial slots of a backward over ntiles tiles.
template <class PL, bool BIAS>
long long bwd_slots(long long ntiles) {
  return (emu_acc<PL, BIAS>() && g_bwd_slots > 0 && g_bwd_slots < ntiles) ? g_bwd_slots : ntiles;
}

template <class PL, bool BIAS>
void real_bwd_k(const RealArgs& a, long long ntiles, float* lds, const std::vector<unsigned char>& tab) {
  using L = Launch<PL>;
  const long long slots = bwd_slots<PL, BIAS>(ntiles);
  // workgroup w runs tiles w, w + slots, ... in turn, as the persistent
  // kernel does, adding them into slot w (its LDS kept across its tiles)
  for (long long w = 0; w < slots; ++w)
    for (long long tile = w; tile < ntiles; tile += slots)
      run_wg(L::BWD_THREADS, [&](HostCtx& ctx, int tid) {
        const int r = tid / PL::T, t = tid % PL::T;
        float* slab = lds + (size_t)r * L::BWD_SLAB;
        if constexpr (emu_acc<PL, BIAS>())
          real_backward_row<PL, L::BWD_ROWS, BIAS, true>(ctx, a, unsigned(t), tile * L::BWD_ROWS, unsigned(r), tid, w,
                                                         lds, slab, GView::of(tab.data()),
                                                         tile == w ? nullptr : lds + L::BWD_LDS_FLOATS);
        else
          real_backward_row<PL, L::BWD_ROWS, BIAS>(ctx, a, unsigned(t), tile * L::BWD_ROWS, unsigned(r), tid, w, lds,
                                                   slab, GView::of(tab.data()));
      });
}

template <class PL>
void real_bwd(const float* x, const float* gy, const float* A, const float* D, const float* B, const int* perm,
              const float* saved_in, float* gx, float* gA, float* gD, float* gB, long long batch, int K,
              unsigned flags, const std::vector<unsigned char>& tab) {
  using L = Launch<PL>;
  static_assert(!L::BWD_TW_LDS, "the emulation follows the global-twiddle backward");
  const bool bias = (flags & kFlagBias) != 0;
  const bool acc = (flags & kFlagAccumulate) != 0;
  std::vector<float> saved_buf;
  const float* saved = saved_in;
  const size_t layers = size_t(K - 1) + ((flags & kFlagPerm) ? 1 : 0);  // u_0 too with PERM
  if (saved == nullptr && layers > 0) {
    saved_buf.resize(layers * batch * PL::N);
    real_fwd<PL>(x, nullptr, A, D, B, perm, batch, K, flags, saved_buf.data(), tab);
    saved = saved_buf.data();
  }
  const std::vector<float4> mq = quartet_coefficients<PL>(D, bias ? B : nullptr, K, tab);
  const long long ntiles = (batch + L::BWD_ROWS - 1) / L::BWD_ROWS;
  const long long slots = bias ? bwd_slots<PL, true>(ntiles) : bwd_slots<PL, false>(ntiles);
  const long long PS4 = partial_entries4<PL>(bias);
  std::vector<float> partial((size_t)slots * K * PS4 * 4);
  const std::vector<int4> p16 = packed_perm<PL>(perm, K, flags);
  RealArgs a{x, nullptr, A, mq.data(), perm, const_cast<float*>(saved), gy, gx, partial.data(),
             (const char*)tab.data(), batch, K, flags};
  a.perm16 = p16.empty() ? nullptr : p16.data();
  std::vector<float> lds((size_t)L::BWD_LDS_FLOATS + L::ACC_FLOATS);
  if (bias) real_bwd_k<PL, true>(a, ntiles, lds.data(), tab);
  else real_bwd_k<PL, false>(a, ntiles, lds.data(), tab);
  std::vector<float> gS(bias ? (size_t)K * PL::N : 0);
  reduce_all<PL>(partial.data(), slots, K, PS4, [&](float4 s, int k, int e4) {
    real_reduce_store4<PL>(s, k, e4, gA, gD, gS.data(), (const char*)tab.data(), acc);
  });
  if (bias) {
    std::vector<float> lds1((size_t)L::FWD_SLAB);
    for (int k = 0; k < K; ++k)
      run_wg(PL::T, [&](HostCtx& ctx, int t) {
        real_dct_row<PL>(ctx, gS.data() + (size_t)k * PL::N, gB + (size_t)k * PL::N, mq.data(), acc, unsigned(t),
                         lds1.data(), GView::of(tab.data()), (const char*)tab.data());
      });
  }
}

template <class PL>
void cplx_fwd(const float* x, float* y, const float* A, const float* D, const int* perm, long long batch,
              int K, unsigned flags, float* saved, const std::vector<unsigned char>& tab) {
  using L = Launch<PL>;
  CplxArgs a{x, y, A, D, perm, saved, nullptr, nullptr, nullptr, (const char*)tab.data(), batch, K, flags};
  const long long nwg = (batch + L::FWD_ROWS - 1) / L::FWD_ROWS;
  std::vector<float> lds((size_t)L::FWD_ROWS * L::FWD_SLAB);
  for (long long wg = 0; wg < nwg; ++wg)
    run_wg(L::FWD_THREADS, [&](HostCtx& ctx, int tid) {
      const int r = tid / PL::T, t = tid % PL::T;
      cplx_forward_row<PL>(ctx, a, unsigned(t), wg * L::FWD_ROWS, unsigned(r), lds.data() + (size_t)r * L::FWD_SLAB);
    });
}

template <class PL>
void cplx_bwd(const float* x, const float* gy, const float* A, const float* D, const int* perm,
              const float* saved_in, float* gx, float* gA, float* gD, long long batch, int K, unsigned flags,
              const std::vector<unsigned char>& tab) {
  using L = Launch<PL>;
  std::vector<float> saved_buf;
  const float* saved = saved_in;
  const size_t layers = size_t(K - 1) + ((flags & kFlagPerm) ? 1 : 0);  // u_0 too with PERM
  if (saved == nullptr && layers > 0) {
    saved_buf.resize(layers * batch * 2 * PL::N);
    cplx_fwd<PL>(x, nullptr, A, D, perm, batch, K, flags, saved_buf.data(), tab);
    saved = saved_buf.data();
  }
  const long long ntiles = (batch + L::BWD_ROWS - 1) / L::BWD_ROWS;
  const long long PS = 4LL * PL::N;
  std::vector<float> partial((size_t)ntiles * K * PS);
  CplxArgs a{x, nullptr, A, D, perm, const_cast<float*>(saved), gy, gx, partial.data(),
             (const char*)tab.data(), batch, K, flags};
  std::vector<float> lds((size_t)L::BWD_ROWS * L::BWD_SLAB);
  for (long long wg = 0; wg < ntiles; ++wg)
    run_wg(L::BWD_THREADS, [&](HostCtx& ctx, int tid) {
      const int r = tid / PL::T, t = tid % PL::T;
      cplx_backward_row<PL, L::BWD_ROWS>(ctx, a, unsigned(t), wg * L::BWD_ROWS, unsigned(r), tid, wg, lds.data(),
                                         lds.data() + (size_t)r * L::BWD_SLAB);
    });
  reduce_all<PL>(partial.data(), ntiles, K, partial_entries4<PL>(), [&](float4 s, int k, int e4) {
    cplx_reduce_store4<PL>(s, k, e4, gA, gD, (flags & kFlagAccumulate) != 0);
  });
}

}  // namespace

extern "C" int acdc_emu_forward(const float* x, float* y, const float* A, const float* D, const float* B,
                                const int* perm, long long batch, int N, int K, unsigned flags, float* saved) {
  int rc = -2;
  if (flags & kFlagComplex) {
    dispatch_complex(N, [&]<class PL>() {
      std::vector<unsigned char> tab;
      build_complex_tables<PL>(tab);
      cplx_fwd<PL>(x, y, A, D, perm, batch, K, flags, saved, tab);
      rc = 0;
    });
  } else {
    dispatch_real(N, [&]<class PL>() {
      std::vector<unsigned char> tab;
      if (!build_real_tables<PL>(tab)) {
        rc = -5;
        return;
      }
      real_fwd<PL>(x, y, A, D, B, perm, batch, K, flags, saved, tab);
      rc = 0;
    });
  }
  return rc;
}

extern "C" int acdc_emu_backward(const float* x, const float* gy, const float* A, const float* D,
                                 const float* B, const int* perm, const float* saved, float* gx, float* gA,
                                 float* gD, float* gB, long long batch, int N, int K, unsigned flags) {
  int rc = -2;
  if (flags & kFlagComplex) {
    dispatch_complex(N, [&]<class PL>() {
      std::vector<unsigned char> tab;
      build_complex_tables<PL>(tab);
      cplx_bwd<PL>(x, gy, A, D, perm, saved, gx, gA, gD, batch, K, flags, tab);
      rc = 0;
    });
  } else {
    dispatch_real(N, [&]<class PL>() {
      std::vector<unsigned char> tab;
      if (!build_real_tables<PL>(tab)) {
        rc = -5;
        return;
      }
      real_bwd<PL>(x, gy, A, D, B, perm, saved, gx, gA, gD, gB, batch, K, flags, tab);
      rc = 0;
    });
  }
  return rc;
}

// Emulate `slots` persistent backward workgroups where the plan accumulates
// (0: one per tile).  Returns whether the unbiased backward of real rows of
// width N accumulates with the compiled launch settings.
extern "C" int acdc_emu_set_backward_slots(long long slots, int N) {
  g_bwd_slots = slots;
  int acc = 0;
  dispatch_real(N, [&]<class PL>() { acc = Launch<PL>::BWD_ACC ? 1 : 0; });
  return acc;
}

// The fixed-order batch reduction alone: out[e] (float4 e < n4) = the sum
// over ntiles tiles of partial[t][e], in the kernels' order (red_phases(n4)
// tile phases, grouped loads, phases added in order).  Returns the number of
// phases used.
extern "C" int acdc_emu_reduce4(const float* partial, long long ntiles, long long n4, float* out) {
  auto run = [&]<int PH>() {
    for (long long e = 0; e < n4; ++e) {
      float4 ph[PH];
      for (int g = 0; g < PH; ++g)
        ph[g] = tile_phase_sum4<PH>(reinterpret_cast<const float4*>(partial), ntiles, n4, e, g);
      reinterpret_cast<float4*>(out)[e] = phases_total4<PH>(ph);
    }
    return PH;
  };
  return red_phases(n4) == 8 ? run.template operator()<8>() : run.template operator()<4>();
}
