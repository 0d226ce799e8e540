// Sanitizer driver (test infrastructure, CPU only).
//
// Built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/emu/build_sanitize.py, it runs
//   1. the kernels' __host__ __device__ row bodies in the CPU emulation
//      (acdc_emu.cpp) on small cascades of every flag combination, ragged
//      last workgroups included (and persistent backward workgroups that
//      add several tiles into one partial), and checks determinism and that
//      the saved and recompute backwards agree bit for bit;
//   2. the C ABI's host-side argument validation and size arithmetic
//      (acdc_api.hip, compiled for the host only) on bad, extreme and
//      boundary arguments, which must return the documented status codes.
// Any sanitizer report or failed check makes the process exit non-zero.
#include "acdc_emu.cpp"

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>

#include "acdc.h"

namespace {

int g_fail = 0;
#define CHECK(cond)                                                     \
  do {                                                                  \
    if (!(cond)) {                                                      \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++g_fail;                                                         \
    }                                                                   \
  } while (0)

struct Case {
  int N, K;
  long long B;
  unsigned flags;
};

void fill(std::vector<float>& v, std::mt19937& g, float mean, float sd) {
  std::normal_distribution<float> d(mean, sd);
  for (float& f : v) f = d(g);
}

void run_case(const Case& c) {
  const bool cplx = (c.flags & kFlagComplex) != 0;
  const size_t ew = cplx ? 2 : 1;
  const size_t rowf = size_t(c.N) * ew, layf = size_t(c.K) * c.N * ew;
  std::mt19937 g(unsigned(c.N * 131 + c.K * 7 + c.flags));
  std::vector<float> x(c.B * rowf), gy(c.B * rowf), A(layf), D(layf), bias(size_t(c.K) * c.N);
  fill(x, g, 0.f, 1.f);
  fill(gy, g, 0.f, 1.f);
  fill(A, g, 1.f, .1f);
  fill(D, g, 1.f, .1f);
  fill(bias, g, 0.f, .1f);
  std::vector<int> perm(size_t(c.K) * c.N);
  for (int k = 0; k < c.K; ++k) {
    for (int n = 0; n < c.N; ++n) perm[size_t(k) * c.N + n] = n;
    std::shuffle(perm.begin() + size_t(k) * c.N, perm.begin() + size_t(k + 1) * c.N, g);
  }
  const float* B = (c.flags & kFlagBias) ? bias.data() : nullptr;
  const size_t slots = size_t(c.K - 1) + ((c.flags & kFlagPerm) ? 1 : 0);
  std::vector<float> y(c.B * rowf), y2(c.B * rowf), saved(std::max<size_t>(slots, 1) * c.B * rowf);
  CHECK(acdc_emu_forward(x.data(), y.data(), A.data(), D.data(), B, perm.data(), c.B, c.N, c.K, c.flags,
                         saved.data()) == 0);
  CHECK(acdc_emu_forward(x.data(), y2.data(), A.data(), D.data(), B, perm.data(), c.B, c.N, c.K, c.flags,
                         nullptr) == 0);
  CHECK(std::memcmp(y.data(), y2.data(), y.size() * 4) == 0);
  for (float f : y) CHECK(std::isfinite(f));
  std::vector<float> gx1(c.B * rowf), gx2(c.B * rowf), gA1(layf), gA2(layf), gD1(layf), gD2(layf);
  std::vector<float> gB1(size_t(c.K) * c.N), gB2(size_t(c.K) * c.N);
  CHECK(acdc_emu_backward(x.data(), gy.data(), A.data(), D.data(), B, perm.data(), slots ? saved.data() : nullptr,
                          gx1.data(), gA1.data(), gD1.data(), B ? gB1.data() : nullptr, c.B, c.N, c.K,
                          c.flags) == 0);
  CHECK(acdc_emu_backward(x.data(), gy.data(), A.data(), D.data(), B, perm.data(), nullptr, gx2.data(),
                          gA2.data(), gD2.data(), B ? gB2.data() : nullptr, c.B, c.N, c.K, c.flags) == 0);
  CHECK(std::memcmp(gx1.data(), gx2.data(), gx1.size() * 4) == 0);
  CHECK(std::memcmp(gA1.data(), gA2.data(), gA1.size() * 4) == 0);
  CHECK(std::memcmp(gD1.data(), gD2.data(), gD1.size() * 4) == 0);
  CHECK(std::memcmp(gB1.data(), gB2.data(), gB1.size() * 4) == 0);
  for (float f : gx1) CHECK(std::isfinite(f));
  std::printf("emulation N=%d K=%d B=%lld flags=%u ok\n", c.N, c.K, c.B, c.flags);
}

void abi_checks() {
  alignas(256) static float buf[4096];
  float* p = buf;
  float* q = buf + 1024;
  float* r = buf + 2048;
  float* s = buf + 3072;
  const int32_t* perm = reinterpret_cast<const int32_t*>(buf + 512);
  // supported widths and flags
  CHECK(acdc_supported(4096, ACDC_FLAG_PERM | ACDC_FLAG_RELU) == 1);
  CHECK(acdc_supported(9216, 0) == 1);
  CHECK(acdc_supported(-4096, 0) == 0);
  CHECK(acdc_supported(INT32_MAX, 0) == 0);
  CHECK(acdc_supported(4096, 1u << 31) == 0);
  CHECK(acdc_supported(4096, ACDC_FLAG_COMPLEX | ACDC_FLAG_RELU) == 0);
  // sizes at the extremes: no overflow, 0 for rejected arguments
  CHECK(acdc_saved_bytes(-1, 4096, 12, 0) == 0);
  CHECK(acdc_saved_bytes(int64_t(1) << 62, 4096, 12, 0) == 0);
  CHECK(acdc_saved_bytes(8192, 4096, 65535, ACDC_FLAG_PERM) == size_t(65535) * 8192 * 4096 * 4);
  CHECK(acdc_saved_bytes(8192, 4096, 65536, 0) == 0);
  CHECK(acdc_backward_workspace_size(int64_t(1) << 28, 4096, 12, ACDC_FLAG_PERM, 1) > 0);
  CHECK(acdc_backward_workspace_size(int64_t(1) << 62, 4096, 12, 0, 0) == 0);
  CHECK(acdc_forward_workspace_size(1 << 10, 1 << 22, 4, ACDC_FLAG_PERM | ACDC_FLAG_RELU) > 0);
  CHECK(acdc_forward_workspace_size(1 << 20, 1 << 22, 4, 0) == 0);  // past the 2^40-element cap
  CHECK(acdc_forward_workspace_size(1 << 20, (1 << 22) + 2, 4, 0) == 0);
  CHECK(acdc_backward_workspace_size(0, 4096, 12, ACDC_FLAG_BIAS, 1) > 0);
  // argument validation before any HIP call
  CHECK(acdc_forward(p, q, r, s, nullptr, nullptr, 4, 64, 1, 1u << 20, nullptr, 0, nullptr, 0, nullptr) ==
        ACDC_ERR_INVALID_ARG);
  CHECK(acdc_forward(p, q, r, s, nullptr, nullptr, 4, 100, 1, 0, nullptr, 0, nullptr, 0, nullptr) ==
        ACDC_ERR_UNSUPPORTED);
  CHECK(acdc_forward(p, q, r, s, nullptr, nullptr, -1, 64, 1, 0, nullptr, 0, nullptr, 0, nullptr) ==
        ACDC_ERR_INVALID_ARG);
  CHECK(acdc_forward(p, q, r, s, nullptr, nullptr, 4, 64, 0, 0, nullptr, 0, nullptr, 0, nullptr) ==
        ACDC_ERR_INVALID_ARG);
  CHECK(acdc_forward(p + 1, q, r, s, nullptr, nullptr, 4, 64, 1, 0, nullptr, 0, nullptr, 0, nullptr) ==
        ACDC_ERR_INVALID_ARG);  // misaligned x
  CHECK(acdc_forward(p, p, r, s, nullptr, nullptr, 4, 64, 1, 0, nullptr, 0, nullptr, 0, nullptr) ==
        ACDC_ERR_INVALID_ARG);  // y aliases x
  CHECK(acdc_forward(p, q, r, s, nullptr, nullptr, 4, 64, 1, ACDC_FLAG_PERM, nullptr, 0, nullptr, 0, nullptr) ==
        ACDC_ERR_INVALID_ARG);  // PERM without perm
  CHECK(acdc_forward(p, q, r, s, nullptr, perm, 4, 64, 2, ACDC_FLAG_PERM, s, 16, nullptr, 0, nullptr) ==
        ACDC_ERR_WORKSPACE);  // saved too small
  CHECK(acdc_forward(p, q, r, s, nullptr, nullptr, 4, 64, 2, 0, nullptr, 0, nullptr, 0, nullptr) ==
        ACDC_ERR_WORKSPACE);  // no forward workspace
  CHECK(acdc_forward(p, q, r, s, nullptr, nullptr, 0, 64, 2, 0, nullptr, 0, nullptr, 0, nullptr) == ACDC_OK);
  CHECK(acdc_backward(p, q, r, s, nullptr, nullptr, nullptr, 0, p, r, s, nullptr, 4, 64, 1, 0, nullptr, 0,
                      nullptr) == ACDC_ERR_INVALID_ARG);  // outputs alias inputs
  CHECK(acdc_backward(p, q, r, s, nullptr, nullptr, nullptr, 0, buf + 256, buf + 384, buf + 448, nullptr, 4, 64,
                      1, ACDC_FLAG_BIAS, nullptr, 0, nullptr) == ACDC_ERR_INVALID_ARG);  // BIAS without bias
  CHECK(acdc_backward(p, q, r, s, nullptr, nullptr, nullptr, 0, buf + 256, buf + 384, buf + 448, nullptr, 4, 64,
                      1, 0, nullptr, 0, nullptr) == ACDC_ERR_WORKSPACE);
  CHECK(acdc_backward(p, q, r, s, nullptr, nullptr, nullptr, 0, buf + 256, buf + 384, buf + 448, nullptr, 4,
                      1 << 22, 1, ACDC_FLAG_COMPLEX, nullptr, 0, nullptr) == ACDC_ERR_UNSUPPORTED);
  for (int st = 1; st >= -5; --st) CHECK(acdc_status_string(st) != nullptr);
  CHECK(acdc_last_hip_error() == 0);
  std::printf("abi checks done\n");
}

}  // namespace

int main() {
  const Case cases[] = {
      {8, 2, 300, kFlagPerm | kFlagRelu},              // 256 rows per tile: a ragged second tile
      {64, 3, 70, kFlagPerm | kFlagRelu | kFlagBias},
      {64, 2, 67, 0},
      {1024, 3, 19, kFlagPerm | kFlagRelu | kFlagBias},
      {4096, 2, 9, kFlagPerm | kFlagRelu},
      {9216, 2, 3, kFlagPerm | kFlagRelu},
      {16, 2, 11, kFlagComplex | kFlagPerm},
      {256, 3, 5, kFlagComplex | kFlagPerm},
      {4096, 1, 3, kFlagComplex},
  };
  for (const Case& c : cases) run_case(c);
  // the persistent accumulating backward: 3 tiles of 2 rows over 2 slots
  CHECK(acdc_emu_set_backward_slots(2, 9216) == 1);
  run_case({9216, 2, 5, kFlagPerm});
  acdc_emu_set_backward_slots(0, 9216);
  abi_checks();
  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("sanitize driver ok\n");
  return 0;
}
