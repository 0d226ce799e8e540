// In-register DFT codelets for gfx950 (complex fp32 as float2).
//
// dft<R, INV>(x) replaces x[0..R-1] by its R-point DFT in natural order,
//   X[m] = sum_i x[i] * exp(-+2 pi i i m / R)   (minus sign forward, plus inverse),
// unnormalised.  Composite sizes split R = R1 * R2 (Cooley-Tukey, four-step
// in registers) with compile-time twiddles, so every index is a constant and
// the whole transform stays in VGPRs.  Multiplications by 1, -1 and +-i are
// done as moves and sign flips.
//
// The constant twiddles are evaluated at compile time in double precision
// (octant reduction + Taylor series on |angle| <= pi/4) and rounded once to
// fp32.
#pragma once

#include <hip/hip_runtime.h>

namespace acdc {

// Scheduling fence: keeps the instruction scheduler from hoisting the loads
// of later steps above this point (bounds register pressure).  No-op on the
// host.
#if defined(__HIP_DEVICE_COMPILE__)
#define ACDC_SCHED_FENCE() __builtin_amdgcn_sched_barrier(0)
#else
#define ACDC_SCHED_FENCE() ((void)0)
#endif

// ----------------------------------------------------------- compile-time trig

constexpr double kPi = 3.141592653589793238462643383279502884;

constexpr double taylor_sin(double x) {
  double term = x, sum = x;
  for (int n = 1; n < 16; ++n) {
    term *= -x * x / double((2 * n) * (2 * n + 1));
    sum += term;
  }
  return sum;
}

constexpr double taylor_cos(double x) {
  double term = 1.0, sum = 1.0;
  for (int n = 1; n < 16; ++n) {
    term *= -x * x / double((2 * n - 1) * (2 * n));
    sum += term;
  }
  return sum;
}

// cos and sin of 2*pi*e/L with exact integer octant reduction.
struct CS {
  double c, s;
};

constexpr CS cos_sin_2pi(long long e, long long L) {
  e %= L;
  if (e < 0) e += L;
  const long long num = 8 * e;
  const long long o = num / L;                    // octant 0..7
  const double f = double(num - o * L) / double(L);  // [0, 1)
  double ca = 0, sa = 0;
  if ((o & 1) == 0) {
    const double a = (kPi / 4) * f;
    ca = taylor_cos(a);
    sa = taylor_sin(a);
  } else {
    const double a = (kPi / 4) * (1.0 - f);
    ca = taylor_sin(a);
    sa = taylor_cos(a);
  }
  switch (o >> 1) {
    case 0: return CS{ca, sa};
    case 1: return CS{-sa, ca};
    case 2: return CS{-ca, -sa};
    default: return CS{sa, -ca};
  }
}

// ----------------------------------------------------------- complex helpers

__host__ __device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__host__ __device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }

// a * w
__host__ __device__ __forceinline__ float2 cmul(float2 a, float2 w) {
  return make_float2(__builtin_fmaf(a.x, w.x, -a.y * w.y), __builtin_fmaf(a.x, w.y, a.y * w.x));
}
// a * conj(w)
__host__ __device__ __forceinline__ float2 cmulc(float2 a, float2 w) {
  return make_float2(__builtin_fmaf(a.x, w.x, a.y * w.y), __builtin_fmaf(a.y, w.x, -a.x * w.y));
}
// a * w for forward twiddles, a * conj(w) for the inverse direction
template <bool INV>
__host__ __device__ __forceinline__ float2 ctw(float2 a, float2 w) {
  if constexpr (INV) return cmulc(a, w);
  else return cmul(a, w);
}

// Multiply by exp(-+2 pi i E / R) known at compile time.
template <int E, int R, bool INV>
__host__ __device__ __forceinline__ float2 cmul_const(float2 v) {
  constexpr int e = ((E % R) + R) % R;
  if constexpr (e == 0) {
    return v;
  } else if constexpr (2 * e == R) {
    return make_float2(-v.x, -v.y);
  } else if constexpr (4 * e == R) {
    // forward: * (-i); inverse: * (+i)
    if constexpr (INV) return make_float2(-v.y, v.x);
    else return make_float2(v.y, -v.x);
  } else if constexpr (4 * e == 3 * R) {
    if constexpr (INV) return make_float2(v.y, -v.x);
    else return make_float2(-v.y, v.x);
  } else {
    constexpr CS cs = cos_sin_2pi(e, R);
    constexpr float c = float(cs.c);
    constexpr float s = INV ? float(cs.s) : float(-cs.s);
    return make_float2(__builtin_fmaf(v.x, c, -v.y * s), __builtin_fmaf(v.x, s, v.y * c));
  }
}

// ----------------------------------------------------------- base codelets

template <int R, bool INV>
struct Dft;

template <bool INV>
struct Dft<1, INV> {
  __host__ __device__ __forceinline__ static void run(float2*) {}
};

template <bool INV>
struct Dft<2, INV> {
  __host__ __device__ __forceinline__ static void run(float2* x) {
    const float2 a = x[0], b = x[1];
    x[0] = cadd(a, b);
    x[1] = csub(a, b);
  }
};

template <bool INV>
struct Dft<3, INV> {
  __host__ __device__ __forceinline__ static void run(float2* x) {
    // X0 = a + b + c; X1,2 = a - (b+c)/2 -+ i sqrt(3)/2 (b - c)  (forward)
    constexpr float h = 0.8660254037844386467637231707529362f;
    const float2 a = x[0], b = x[1], c = x[2];
    const float2 s = cadd(b, c), d = csub(b, c);
    const float2 t = make_float2(__builtin_fmaf(-0.5f, s.x, a.x), __builtin_fmaf(-0.5f, s.y, a.y));
    x[0] = cadd(a, s);
    // forward: -i*h*d = (h*d.y, -h*d.x)
    const float sg = INV ? -1.0f : 1.0f;
    const float2 r = make_float2(sg * h * d.y, -sg * h * d.x);
    x[1] = cadd(t, r);
    x[2] = csub(t, r);
  }
};

template <bool INV>
struct Dft<4, INV> {
  __host__ __device__ __forceinline__ static void run(float2* x) {
    const float2 t0 = cadd(x[0], x[2]), t1 = csub(x[0], x[2]);
    const float2 t2 = cadd(x[1], x[3]), t3 = csub(x[1], x[3]);
    x[0] = cadd(t0, t2);
    x[2] = csub(t0, t2);
    // forward: X1 = t1 - i t3, X3 = t1 + i t3
    const float2 it3 = INV ? make_float2(-t3.y, t3.x) : make_float2(t3.y, -t3.x);
    x[1] = cadd(t1, it3);
    x[3] = csub(t1, it3);
  }
};

// Composite: R = R1 * R2, input index i = R2*i1 + i2, output m = m1 + R1*m2.
template <int R>
constexpr int split_first() {
  return (R % 4 == 0 && R > 4) ? 4 : ((R % 2 == 0 && R > 2) ? 2 : ((R % 3 == 0 && R > 3) ? 3 : 1));
}

template <int R1, int R2, int R, bool INV, int I2, int M1>
struct TwiddleStep {
  __host__ __device__ __forceinline__ static void run(float2* y) {
    y[I2 * R1 + M1] = cmul_const<I2 * M1, R, INV>(y[I2 * R1 + M1]);
    if constexpr (M1 + 1 < R1) TwiddleStep<R1, R2, R, INV, I2, M1 + 1>::run(y);
    else if constexpr (I2 + 1 < R2) TwiddleStep<R1, R2, R, INV, I2 + 1, 0>::run(y);
  }
};

template <int R, bool INV>
struct Dft {
  static_assert(R > 4, "base codelets cover R <= 4");
  static constexpr int R1 = split_first<R>();
  static constexpr int R2 = R / R1;
  static_assert(R1 > 1 && R1 * R2 == R, "unsupported radix");
  __host__ __device__ __forceinline__ static void run(float2* x) {
    float2 y[R];
#pragma unroll
    for (int i2 = 0; i2 < R2; ++i2) {
      float2 t[R1];
#pragma unroll
      for (int i1 = 0; i1 < R1; ++i1) t[i1] = x[R2 * i1 + i2];
      Dft<R1, INV>::run(t);
#pragma unroll
      for (int m1 = 0; m1 < R1; ++m1) y[i2 * R1 + m1] = t[m1];
    }
    TwiddleStep<R1, R2, R, INV, 0, 0>::run(y);
#pragma unroll
    for (int m1 = 0; m1 < R1; ++m1) {
      float2 t[R2];
#pragma unroll
      for (int i2 = 0; i2 < R2; ++i2) t[i2] = y[i2 * R1 + m1];
      Dft<R2, INV>::run(t);
#pragma unroll
      for (int m2 = 0; m2 < R2; ++m2) x[m1 + R1 * m2] = t[m2];
    }
  }
};

}  // namespace acdc
