// Complex arithmetic on float2 and compile-time roots of unity.
//
// Twiddle constants are evaluated at compile time in double precision from
// the exact rational angle 2*pi*m/N (octant reduction in integer arithmetic,
// then a Taylor series on |x| <= pi/4), and rounded once to float.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

#define LR_HD __host__ __device__ __forceinline__

namespace lr {

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E).
// Guarantees full unrolling with constant indices, so small arrays stay in
// registers and twiddle exponents are constant expressions.
template <int B, int E, class F>
LR_HD void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

LR_HD float2 c2(float x, float y) { float2 r; r.x = x; r.y = y; return r; }
LR_HD float2 cadd(float2 a, float2 b) { return c2(a.x + b.x, a.y + b.y); }
LR_HD float2 csub(float2 a, float2 b) { return c2(a.x - b.x, a.y - b.y); }
LR_HD float2 cscale(float2 a, float s) { return c2(a.x * s, a.y * s); }
LR_HD float2 cconj(float2 a) { return c2(a.x, -a.y); }
// a * b
LR_HD float2 cmul(float2 a, float2 b) {
  return c2(fmaf(a.x, b.x, -a.y * b.y), fmaf(a.x, b.y, a.y * b.x));
}
// a * conj(b)
LR_HD float2 cmulc(float2 a, float2 b) {
  return c2(fmaf(a.x, b.x, a.y * b.y), fmaf(a.y, b.x, -a.x * b.y));
}
// conj(a) * b
LR_HD float2 cconjmul(float2 a, float2 b) {
  return c2(fmaf(a.x, b.x, a.y * b.y), fmaf(a.x, b.y, -a.y * b.x));
}
LR_HD float cabs2(float2 a) { return fmaf(a.x, a.x, a.y * a.y); }

// Multiply by the quarter-turn root exp(SIGN * i*pi/2) = SIGN * i.
template <int SIGN>
LR_HD float2 mul_qturn(float2 a) {
  return SIGN < 0 ? c2(a.y, -a.x) : c2(-a.y, a.x);
}

// ---- compile-time roots of unity ----------------------------------------
struct cdbl { double re, im; };

constexpr double kPi = 3.14159265358979323846264338327950288;

constexpr double sin_taylor(double x) {
  double x2 = x * x, t = x, s = x;
  for (int i = 1; i < 13; ++i) { t *= -x2 / ((2.0 * i) * (2.0 * i + 1.0)); s += t; }
  return s;
}
constexpr double cos_taylor(double x) {
  double x2 = x * x, t = 1.0, s = 1.0;
  for (int i = 1; i < 13; ++i) { t *= -x2 / ((2.0 * i - 1.0) * (2.0 * i)); s += t; }
  return s;
}

// exp(sign * 2*pi*i * m / N), double precision, for any integer m.
constexpr cdbl unit_root(long long m, long long N, int sign) {
  m %= N;
  if (m < 0) m += N;
  const long long q = (4 * m) / N;      // quadrant
  const long long r = 4 * m - q * N;    // angle within quadrant = (pi/2) * r / N
  double c = 1.0, s = 0.0;
  if (2 * r <= N) {
    const double p = kPi / 2.0 * static_cast<double>(r) / static_cast<double>(N);
    c = cos_taylor(p);
    s = sin_taylor(p);
  } else {
    const double p = kPi / 2.0 * static_cast<double>(N - r) / static_cast<double>(N);
    c = sin_taylor(p);
    s = cos_taylor(p);
  }
  for (long long i = 0; i < q; ++i) { const double t = c; c = -s; s = t; }
  return cdbl{c, sign * s};
}

// Table of exp(-2*pi*i*k/N), k <= N (entry N repeats entry 0), as floats.
template <int N>
struct RootTable { float2 w[N + 1]; };

template <int N>
constexpr RootTable<N> make_root_table() {
  RootTable<N> t{};
  for (int k = 0; k <= N; ++k) {
    const cdbl z = unit_root(k, N, -1);
    t.w[k].x = static_cast<float>(z.re);
    t.w[k].y = static_cast<float>(z.im);
  }
  return t;
}

// Multiply a by W_N^E0 with W_N = exp(SIGN*2*pi*i/N), E0 a compile-time
// constant: the trivial rotations are exact and the general root is an
// immediate evaluated in double precision at compile time.
template <int N, int SIGN, int E0>
LR_HD float2 twiddle_const(float2 a) {
  constexpr int e = ((E0 % N) + N) % N;
  if constexpr (e == 0) {
    return a;
  } else if constexpr ((4 * e) % N == 0) {
    constexpr int q = (4 * e) / N;  // 1, 2, 3 quarter turns
    if constexpr (q == 2) return c2(-a.x, -a.y);
    const float2 b = mul_qturn<SIGN>(a);
    if constexpr (q == 1) return b;
    return c2(-b.x, -b.y);
  } else if constexpr ((8 * e) % N == 0) {
    // odd multiple of pi/4: (+-1 +- i)/sqrt(2) rotations
    const float h = 0.70710678118654752440f;
    constexpr int o = (8 * e) / N;  // 1, 3, 5, 7
    const float2 r1 = SIGN < 0 ? c2((a.x + a.y) * h, (a.y - a.x) * h)
                               : c2((a.x - a.y) * h, (a.x + a.y) * h);
    if constexpr (o == 1) return r1;
    if constexpr (o == 3) return mul_qturn<SIGN>(r1);
    if constexpr (o == 5) return c2(-r1.x, -r1.y);
    const float2 t = mul_qturn<SIGN>(r1);
    return c2(-t.x, -t.y);
  } else {
    constexpr cdbl z = unit_root(e, N, SIGN);
    constexpr float wr = static_cast<float>(z.re);
    constexpr float wi = static_cast<float>(z.im);
    return cmul(a, c2(wr, wi));
  }
}

// exp(SIGN*2*pi*i*E/N) = scale * (1 + i*r) where |cos| >= |sin| (scale =
// cos, r = tan), else scale * (r + i) (scale = sin, r = cot).  split_root
// multiplies by the unit-scale factor with two FMAs; the caller applies the
// scale, which is then at least 1/sqrt(2) in magnitude and r at most 1.
// Quarter turns: SIGN*i (scale 1), -1 (scale -1, nothing to multiply) and
// -SIGN*i (scale -1), all exact.
constexpr double dabs(double x) { return x < 0 ? -x : x; }
constexpr bool split_root_cos(long long e, long long N, int sign) {
  return dabs(unit_root(e, N, sign).re) >= dabs(unit_root(e, N, sign).im);
}
constexpr double split_root_scale(long long e, long long N, int sign) {
  e %= N;
  if (e < 0) e += N;
  if (e == 0) return 1.0;
  if ((4 * e) % N == 0) return (4 * e) / N == 1 ? 1.0 : -1.0;
  return split_root_cos(e, N, sign) ? unit_root(e, N, sign).re : unit_root(e, N, sign).im;
}
template <int N, int SIGN, int E0>
LR_HD float2 split_root(float2 a) {
  constexpr int e = ((E0 % N) + N) % N;
  if constexpr (e == 0) {
    return a;
  } else if constexpr ((4 * e) % N == 0) {
    if constexpr ((4 * e) / N == 2) return a;
    return mul_qturn<SIGN>(a);
  } else {
    constexpr cdbl z = unit_root(e, N, SIGN);
    if constexpr (split_root_cos(e, N, SIGN)) {
      constexpr float r = static_cast<float>(z.im / z.re);
      return c2(fmaf(-r, a.y, a.x), fmaf(r, a.x, a.y));
    } else {
      constexpr float r = static_cast<float>(z.re / z.im);
      return c2(fmaf(r, a.x, -a.y), fmaf(r, a.y, a.x));
    }
  }
}

}  // namespace lr
