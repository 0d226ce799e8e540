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

// ----------------------------------------------------- radix 8 and 16
// Specialised codelets.  The constant twiddles W_16^e of the composite split
// are written as W = C (1 -+ i tau) (tau = tan(pi/8), C = cos(pi/8)) and
// W_8^1 = c (1 -+ i) (c = 1/sqrt 2): the products with (1 -+ i tau) and
// (1 -+ i) take two fused multiply-adds or two additions, and the real
// factors C, c ride in the fused multiply-adds of the butterfly that
// follows.  Radix 16: 144 operations instead of 160; radix 8: 52 instead of
// 56.  Index conventions as in the composite: input i = R2*i1 + i2, output
// m = m1 + R1*m2.

// v * (-i) forward, v * (+i) inverse
template <bool INV>
__host__ __device__ __forceinline__ float2 mul_mi(float2 v) {
  return INV ? make_float2(-v.y, v.x) : make_float2(v.y, -v.x);
}
// v * (1 -+ i)
template <bool INV>
__host__ __device__ __forceinline__ float2 mul_1mi(float2 v) {
  return INV ? make_float2(v.x - v.y, v.y + v.x) : make_float2(v.x + v.y, v.y - v.x);
}
// v * (-1 -+ i)
template <bool INV>
__host__ __device__ __forceinline__ float2 mul_m1mi(float2 v) {
  return INV ? make_float2(-v.x - v.y, v.x - v.y) : make_float2(v.y - v.x, -v.y - v.x);
}
// v * (1 -+ i tau)
template <bool INV>
__host__ __device__ __forceinline__ float2 mul_1mt(float2 v, float tau) {
  return INV ? make_float2(__builtin_fmaf(-tau, v.y, v.x), __builtin_fmaf(tau, v.x, v.y))
             : make_float2(__builtin_fmaf(tau, v.y, v.x), __builtin_fmaf(-tau, v.x, v.y));
}
// v * (tau -+ i)
template <bool INV>
__host__ __device__ __forceinline__ float2 mul_tmi(float2 v, float tau) {
  return INV ? make_float2(__builtin_fmaf(tau, v.x, -v.y), __builtin_fmaf(tau, v.y, v.x))
             : make_float2(__builtin_fmaf(tau, v.x, v.y), __builtin_fmaf(tau, v.y, -v.x));
}

// 4-point DFT of (z0, k1 v1, z2, k1 v3) with k1 real, z2 = k2 u2 (k2 real;
// k2 == 1 means z2 = u2 exactly).  Writes X[0..3] to out[0], out[s], ...
template <bool INV>
__host__ __device__ __forceinline__ void dft4_scaled(float2 z0, float2 u2, float k2, bool k2one, float2 v1,
                                                     float2 v3, float k1, float2* out, int s) {
  float2 t0, t1;
  if (k2one) {
    t0 = cadd(z0, u2);
    t1 = csub(z0, u2);
  } else {
    t0 = make_float2(__builtin_fmaf(k2, u2.x, z0.x), __builtin_fmaf(k2, u2.y, z0.y));
    t1 = make_float2(__builtin_fmaf(-k2, u2.x, z0.x), __builtin_fmaf(-k2, u2.y, z0.y));
  }
  const float2 sm = cadd(v1, v3), df = mul_mi<INV>(csub(v1, v3));
  out[0] = make_float2(__builtin_fmaf(k1, sm.x, t0.x), __builtin_fmaf(k1, sm.y, t0.y));
  out[2 * s] = make_float2(__builtin_fmaf(-k1, sm.x, t0.x), __builtin_fmaf(-k1, sm.y, t0.y));
  out[s] = make_float2(__builtin_fmaf(k1, df.x, t1.x), __builtin_fmaf(k1, df.y, t1.y));
  out[3 * s] = make_float2(__builtin_fmaf(-k1, df.x, t1.x), __builtin_fmaf(-k1, df.y, t1.y));
}

constexpr float kC16 = 0.92387953251128675613f;   // cos(pi/8)
constexpr float kT16 = 0.41421356237309504880f;   // tan(pi/8)
constexpr float kC8 = 0.70710678118654752440f;    // 1/sqrt(2)

template <bool INV>
struct Dft<16, INV> {
  __host__ __device__ __forceinline__ static void run(float2* x) {
    float2 y[4][4];  // y[i2][m1]
#pragma unroll
    for (int i2 = 0; i2 < 4; ++i2) {
      float2 t[4] = {x[i2], x[4 + i2], x[8 + i2], x[12 + i2]};
      Dft<4, INV>::run(t);
#pragma unroll
      for (int m1 = 0; m1 < 4; ++m1) y[i2][m1] = t[m1];
    }
    // column m1 = 0: no twiddles
    {
      float2 t[4] = {y[0][0], y[1][0], y[2][0], y[3][0]};
      Dft<4, INV>::run(t);
#pragma unroll
      for (int m2 = 0; m2 < 4; ++m2) x[4 * m2] = t[m2];
    }
    // m1 = 1: W^1 = C(1 -+ i tau), W^2 = c(1 -+ i), W^3 = C(tau -+ i)
    dft4_scaled<INV>(y[0][1], mul_1mi<INV>(y[2][1]), kC8, false, mul_1mt<INV>(y[1][1], kT16),
                     mul_tmi<INV>(y[3][1], kT16), kC16, x + 1, 4);
    // m1 = 2: W^2 = c(1 -+ i), W^4 = -+i, W^6 = c(-1 -+ i)
    dft4_scaled<INV>(y[0][2], mul_mi<INV>(y[2][2]), 1.0f, true, mul_1mi<INV>(y[1][2]), mul_m1mi<INV>(y[3][2]), kC8,
                     x + 2, 4);
    // m1 = 3: W^3 = C(tau -+ i), W^6 = c(-1 -+ i), W^9 = -C(1 -+ i tau)
    {
      const float2 w9 = mul_1mt<INV>(y[3][3], kT16);
      dft4_scaled<INV>(y[0][3], mul_m1mi<INV>(y[2][3]), kC8, false, mul_tmi<INV>(y[1][3], kT16),
                       make_float2(-w9.x, -w9.y), kC16, x + 3, 4);
    }
  }
};

template <bool INV>
struct Dft<8, INV> {
  __host__ __device__ __forceinline__ static void run(float2* x) {
    float2 a[4] = {x[0], x[2], x[4], x[6]};  // i2 = 0
    float2 b[4] = {x[1], x[3], x[5], x[7]};  // i2 = 1
    Dft<4, INV>::run(a);
    Dft<4, INV>::run(b);
    // m1 = 0: plain; m1 = 2: * (-+i)
    x[0] = cadd(a[0], b[0]);
    x[4] = csub(a[0], b[0]);
    const float2 b2 = mul_mi<INV>(b[2]);
    x[2] = cadd(a[2], b2);
    x[6] = csub(a[2], b2);
    // m1 = 1: * c(1 -+ i); m1 = 3: * c(-1 -+ i)
    const float2 u1 = mul_1mi<INV>(b[1]), u3 = mul_m1mi<INV>(b[3]);
    x[1] = make_float2(__builtin_fmaf(kC8, u1.x, a[1].x), __builtin_fmaf(kC8, u1.y, a[1].y));
    x[5] = make_float2(__builtin_fmaf(-kC8, u1.x, a[1].x), __builtin_fmaf(-kC8, u1.y, a[1].y));
    x[3] = make_float2(__builtin_fmaf(kC8, u3.x, a[3].x), __builtin_fmaf(kC8, u3.y, a[3].y));
    x[7] = make_float2(__builtin_fmaf(-kC8, u3.x, a[3].x), __builtin_fmaf(-kC8, u3.y, a[3].y));
  }
};

}  // namespace acdc
