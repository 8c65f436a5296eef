// Register-resident small DFTs ("codelets") on float2 arrays.
//
// Dft<R, SIGN>::run(a) replaces a[0..R) (natural order) by its DFT
// X[k] = sum_n a[n] * exp(SIGN*2*pi*i*n*k/R), natural order, unnormalised.
// Radices 2, 3, 4, 5 and 7 are written out; larger sizes are composed at compile
// time by Cooley-Tukey (with constant twiddles) or, for coprime factors, by
// the Good-Thomas prime-factor map (no twiddles).  Every index is a
// compile-time constant after unrolling, so the arrays live in registers.
#pragma once

#include "cplx.hpp"

namespace lr {

template <int R, int SIGN>
struct Dft;

template <int SIGN>
struct Dft<1, SIGN> {
  LR_HD static void run(float2*) {}
};

template <int SIGN>
struct Dft<2, SIGN> {
  LR_HD static void run(float2* a) {
    const float2 t = a[1];
    a[1] = csub(a[0], t);
    a[0] = cadd(a[0], t);
  }
};

template <int SIGN>
struct Dft<3, SIGN> {
  LR_HD static void run(float2* a) {
    const float s = 0.86602540378443864676f;  // sin(2*pi/3)
    const float2 t = cadd(a[1], a[2]);
    const float2 d = csub(a[1], a[2]);
    const float2 m = c2(fmaf(-0.5f, t.x, a[0].x), fmaf(-0.5f, t.y, a[0].y));
    const float2 r = mul_qturn<SIGN>(c2(s * d.x, s * d.y));
    a[0] = cadd(a[0], t);
    a[1] = cadd(m, r);
    a[2] = csub(m, r);
  }
};

template <int SIGN>
struct Dft<4, SIGN> {
  LR_HD static void run(float2* a) {
    const float2 t0 = cadd(a[0], a[2]);
    const float2 t1 = csub(a[0], a[2]);
    const float2 t2 = cadd(a[1], a[3]);
    const float2 t3 = mul_qturn<SIGN>(csub(a[1], a[3]));
    a[0] = cadd(t0, t2);
    a[2] = csub(t0, t2);
    a[1] = cadd(t1, t3);
    a[3] = csub(t1, t3);
  }
};

// Radix 2 and 4 on inputs given up to constant factors, as Dft5 below:
// element p of the input is G::g(p) * a[p] (g(0) = 1).  Same instruction
// counts as the plain codelets; the factors ride in FMA constants.
template <int SIGN, class G>
struct Dft2S {
  LR_HD static void run(float2* a) {
    constexpr float g1 = static_cast<float>(G::g(1));
    const float2 t = a[1];
    a[1] = c2(fmaf(-g1, t.x, a[0].x), fmaf(-g1, t.y, a[0].y));
    a[0] = c2(fmaf(g1, t.x, a[0].x), fmaf(g1, t.y, a[0].y));
  }
};

template <int SIGN, class G>
struct Dft4S {
  LR_HD static void run(float2* a) {
    constexpr double g1 = G::g(1), g2 = G::g(2), g3 = G::g(3);
    constexpr float f2 = static_cast<float>(g2), r31 = static_cast<float>(g3 / g1);
    constexpr float f1 = static_cast<float>(g1);
    // SIGN*i*g1*v = (-SIGN*g1*v.y, SIGN*g1*v.x)
    constexpr float h1 = static_cast<float>(SIGN < 0 ? g1 : -g1);
    const float2 t0 = c2(fmaf(f2, a[2].x, a[0].x), fmaf(f2, a[2].y, a[0].y));
    const float2 t1 = c2(fmaf(-f2, a[2].x, a[0].x), fmaf(-f2, a[2].y, a[0].y));
    const float2 T2 = c2(fmaf(r31, a[3].x, a[1].x), fmaf(r31, a[3].y, a[1].y));
    const float2 T3 = c2(fmaf(-r31, a[3].x, a[1].x), fmaf(-r31, a[3].y, a[1].y));
    a[0] = c2(fmaf(f1, T2.x, t0.x), fmaf(f1, T2.y, t0.y));
    a[2] = c2(fmaf(-f1, T2.x, t0.x), fmaf(-f1, T2.y, t0.y));
    a[1] = c2(fmaf(h1, T3.y, t1.x), fmaf(-h1, T3.x, t1.y));
    a[3] = c2(fmaf(-h1, T3.y, t1.x), fmaf(h1, T3.x, t1.y));
  }
};

// Radix 5 on inputs given up to constant factors: element p of the input is
// G::g(p) * a[p] (g(0) = 1), so that a Cooley-Tukey stage can leave the
// magnitude of its twiddles to this step.  With t1 = g1 T1, t3 = g1 T3,
// t2 = g2 T2, t4 = g2 T4 (T1, T3 = a[1] +- (g4/g1) a[4], T2, T4 likewise),
//   X0 = a0 + t1 + t2,  X1, X4 = b1 +- SIGN i (s1 t3 + s2 t4),
//   X2, X3 = b2 +- SIGN i (s2 t3 - s1 t4),
// b1 = a0 + c1 t1 + c2 t2, b2 = a0 + c2 t1 + c1 t2.  Every factor g_p and
// sine folds into a constant of an FMA: 32 instructions, scaled or not.
struct UnitScale {
  static constexpr double g(int) { return 1.0; }
};

template <int SIGN, class G>
struct Dft5 {
  LR_HD static void run(float2* a) {
    constexpr double c1 = 0.30901699437494742410;   // cos(2*pi/5)
    constexpr double c2v = -0.80901699437494742410; // cos(4*pi/5)
    constexpr double s1 = 0.95105651629515357212;   // sin(2*pi/5)
    constexpr double s2 = 0.58778525229247312917;   // sin(4*pi/5)
    constexpr double g1 = G::g(1), g2 = G::g(2), g3 = G::g(3), g4 = G::g(4);
    constexpr float r14 = static_cast<float>(g4 / g1);
    constexpr float r23 = static_cast<float>(g3 / g2);
    const float2 T1 = c2(fmaf(r14, a[4].x, a[1].x), fmaf(r14, a[4].y, a[1].y));
    const float2 T3 = c2(fmaf(-r14, a[4].x, a[1].x), fmaf(-r14, a[4].y, a[1].y));
    const float2 T2 = c2(fmaf(r23, a[3].x, a[2].x), fmaf(r23, a[3].y, a[2].y));
    const float2 T4 = c2(fmaf(-r23, a[3].x, a[2].x), fmaf(-r23, a[3].y, a[2].y));
    constexpr float e11 = static_cast<float>(c1 * g1), e12 = static_cast<float>(c2v * g2);
    constexpr float e21 = static_cast<float>(c2v * g1), e22 = static_cast<float>(c1 * g2);
    const float2 b1 = c2(fmaf(e12, T2.x, fmaf(e11, T1.x, a[0].x)), fmaf(e12, T2.y, fmaf(e11, T1.y, a[0].y)));
    const float2 b2 = c2(fmaf(e22, T2.x, fmaf(e21, T1.x, a[0].x)), fmaf(e22, T2.y, fmaf(e21, T1.y, a[0].y)));
    // s1 t3 + s2 t4 = k1 (T3 + q1 T4), s2 t3 - s1 t4 = k2 (T3 - q2 T4)
    constexpr double k1 = s1 * g1, k2 = s2 * g1;
    constexpr float q1 = static_cast<float>(s2 * g2 / k1), q2 = static_cast<float>(s1 * g2 / k2);
    const float2 v1 = c2(fmaf(q1, T4.x, T3.x), fmaf(q1, T4.y, T3.y));
    const float2 v2 = c2(fmaf(-q2, T4.x, T3.x), fmaf(-q2, T4.y, T3.y));
    // SIGN*i*k*v = (-SIGN*k*v.y, SIGN*k*v.x)
    constexpr float f1 = static_cast<float>(SIGN < 0 ? k1 : -k1);
    constexpr float f2 = static_cast<float>(SIGN < 0 ? k2 : -k2);
    constexpr float h1 = static_cast<float>(g1), h2 = static_cast<float>(g2);
    a[0] = c2(fmaf(h2, T2.x, fmaf(h1, T1.x, a[0].x)), fmaf(h2, T2.y, fmaf(h1, T1.y, a[0].y)));
    a[1] = c2(fmaf(f1, v1.y, b1.x), fmaf(-f1, v1.x, b1.y));
    a[4] = c2(fmaf(-f1, v1.y, b1.x), fmaf(f1, v1.x, b1.y));
    a[2] = c2(fmaf(f2, v2.y, b2.x), fmaf(-f2, v2.x, b2.y));
    a[3] = c2(fmaf(-f2, v2.y, b2.x), fmaf(f2, v2.x, b2.y));
  }
};

template <int SIGN>
struct Dft<5, SIGN> : Dft5<SIGN, UnitScale> {};

// Radix 7 as three conjugate pairs: with t_k = a[k] + a[7-k] and
// d_k = a[k] - a[7-k] (k = 1, 2, 3),
//   X[m], X[7-m] = a[0] + sum_k cos(2 pi k m / 7) t_k  +-  SIGN i sum_k sin(2 pi k m / 7) d_k.
// Each odd sum is written as its first sine times a two-FMA combination, and
// that sine is applied in the output FMA.
template <int SIGN>
struct Dft<7, SIGN> {
  LR_HD static void run(float2* a) {
    const float c1 = 0.62348980185873359439f;   // cos(2*pi/7)
    const float c2v = -0.22252093395631433737f;  // cos(4*pi/7)
    const float c3 = -0.90096886790241903498f;   // cos(6*pi/7)
    const float s1 = 0.78183148246802980363f;   // sin(2*pi/7)
    const float s2 = 0.97492791218182361934f;   // sin(4*pi/7)
    const float s3 = 0.43388373911755823142f;   // sin(6*pi/7)
    const float2 t1 = cadd(a[1], a[6]);
    const float2 t2 = cadd(a[2], a[5]);
    const float2 t3 = cadd(a[3], a[4]);
    const float2 d1 = csub(a[1], a[6]);
    const float2 d2 = csub(a[2], a[5]);
    const float2 d3 = csub(a[3], a[4]);
    auto re = [&](float x1, float x2, float x3) {
      return c2(fmaf(x3, t3.x, fmaf(x2, t2.x, fmaf(x1, t1.x, a[0].x))),
                fmaf(x3, t3.y, fmaf(x2, t2.y, fmaf(x1, t1.y, a[0].y))));
    };
    // d1 + q2*d2 + q3*d3
    auto odd = [&](float q2, float q3) {
      return c2(fmaf(q3, d3.x, fmaf(q2, d2.x, d1.x)), fmaf(q3, d3.y, fmaf(q2, d2.y, d1.y)));
    };
    constexpr float g = SIGN < 0 ? 1.f : -1.f;
    // b +- SIGN*i*s*v
    auto out = [&](float2 b, float s, float2 v, float2& hi, float2& lo) {
      hi = c2(fmaf(g * s, v.y, b.x), fmaf(-g * s, v.x, b.y));
      lo = c2(fmaf(-g * s, v.y, b.x), fmaf(g * s, v.x, b.y));
    };
    const float2 b1 = re(c1, c2v, c3);
    const float2 b2 = re(c2v, c3, c1);
    const float2 b3 = re(c3, c1, c2v);
    // sums s1 d1 + s2 d2 + s3 d3, s2 d1 - s3 d2 - s1 d3, s3 d1 - s1 d2 + s2 d3
    const float2 v1 = odd(1.24697960371746706105f, 0.55495813208737119142f);
    const float2 v2 = odd(-0.44504186791262880858f, -0.80193773580483825247f);
    const float2 v3 = odd(-1.80193773580483825247f, 2.24697960371746706105f);
    a[0] = cadd(a[0], cadd(t1, cadd(t2, t3)));
    out(b1, s1, v1, a[1], a[6]);
    out(b2, s2, v2, a[2], a[5]);
    out(b3, s3, v3, a[3], a[4]);
  }
};

// Cooley-Tukey N = P*Q: P transforms of length Q on the stride-P
// subsequences, twiddle exp(SIGN*2*pi*i*p*k2/N), then Q transforms of length P;
// output X[k2 + Q*k1].  With P = 2, 4 or 5 each twiddle is applied as
// split_root (two FMAs, or none for the quarter turns) and its magnitude
// factor is folded into the length-P step of column k2 (the scaled codelets
// with TwiddleScale).
template <int N, int SIGN, int K2>
struct TwiddleScale {
  static constexpr double g(int p) { return (p * K2) % N == 0 ? 1.0 : split_root_scale(p * K2, N, SIGN); }
};

template <int P, int Q, int SIGN>
struct DftCT {
  LR_HD static void run(float2* a) {
    constexpr int N = P * Q;
    constexpr bool SPLIT = P == 2 || P == 4 || P == 5;
    float2 t[N];
    static_for<0, P>([&](auto pc) {
      constexpr int p = decltype(pc)::value;
      float2 s[Q];
      static_for<0, Q>([&](auto mc) { s[mc.value] = a[P * mc.value + p]; });
      Dft<Q, SIGN>::run(s);
      static_for<0, Q>([&](auto kc) {
        constexpr int k2 = decltype(kc)::value;
        if constexpr (SPLIT) {
          t[p * Q + k2] = split_root<N, SIGN, p * k2>(s[k2]);
        } else {
          t[p * Q + k2] = twiddle_const<N, SIGN, p * k2>(s[k2]);
        }
      });
    });
    static_for<0, Q>([&](auto kc) {
      constexpr int k2 = decltype(kc)::value;
      float2 u[P];
      static_for<0, P>([&](auto pc) { u[pc.value] = t[pc.value * Q + k2]; });
      if constexpr (P == 2) {
        Dft2S<SIGN, TwiddleScale<N, SIGN, k2>>::run(u);
      } else if constexpr (P == 4) {
        Dft4S<SIGN, TwiddleScale<N, SIGN, k2>>::run(u);
      } else if constexpr (P == 5) {
        Dft5<SIGN, TwiddleScale<N, SIGN, k2>>::run(u);
      } else {
        Dft<P, SIGN>::run(u);
      }
      static_for<0, P>([&](auto jc) { a[k2 + Q * jc.value] = u[jc.value]; });
    });
  }
};

constexpr int inv_mod(int a, int m) {
  for (int x = 1; x < m; ++x)
    if ((a * x) % m == 1) return x;
  return m == 1 ? 0 : -1;
}

// Good-Thomas N = P*Q with gcd(P, Q) = 1: input map n = (Q*p + P*q) mod N,
// output map k = CRT(k mod P, k mod Q); no twiddles.
template <int P, int Q, int SIGN>
struct DftPFA {
  LR_HD static void run(float2* a) {
    constexpr int N = P * Q;
    constexpr int E1 = Q * inv_mod(Q % P, P);
    constexpr int E2 = P * inv_mod(P % Q, Q);
    static_assert(inv_mod(Q % P, P) >= 0 && inv_mod(P % Q, Q) >= 0, "factors must be coprime");
    float2 t[N];
    static_for<0, P>([&](auto pc) {
      constexpr int p = decltype(pc)::value;
      float2 s[Q];
      static_for<0, Q>([&](auto qc) { s[qc.value] = a[(Q * p + P * qc.value) % N]; });
      Dft<Q, SIGN>::run(s);
      static_for<0, Q>([&](auto kc) { t[p * Q + kc.value] = s[kc.value]; });
    });
    static_for<0, Q>([&](auto kc) {
      constexpr int k2 = decltype(kc)::value;
      float2 u[P];
      static_for<0, P>([&](auto pc) { u[pc.value] = t[pc.value * Q + k2]; });
      Dft<P, SIGN>::run(u);
      static_for<0, P>([&](auto jc) { a[(jc.value * E1 + k2 * E2) % N] = u[jc.value]; });
    });
  }
};

template <int SIGN> struct Dft<8, SIGN> : DftCT<2, 4, SIGN> {};
template <int SIGN> struct Dft<10, SIGN> : DftPFA<2, 5, SIGN> {};
template <int SIGN> struct Dft<16, SIGN> : DftCT<4, 4, SIGN> {};
template <int SIGN> struct Dft<20, SIGN> : DftPFA<4, 5, SIGN> {};
template <int SIGN> struct Dft<25, SIGN> : DftCT<5, 5, SIGN> {};
template <int SIGN> struct Dft<32, SIGN> : DftCT<4, 8, SIGN> {};
template <int SIGN> struct Dft<40, SIGN> : DftPFA<8, 5, SIGN> {};
template <int SIGN> struct Dft<14, SIGN> : DftPFA<2, 7, SIGN> {};

}  // namespace lr
