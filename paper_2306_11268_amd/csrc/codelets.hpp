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

template <int SIGN>
struct Dft<5, SIGN> {
  LR_HD static void run(float2* a) {
    const float c1 = 0.30901699437494742410f;   // cos(2*pi/5)
    const float c2v = -0.80901699437494742410f; // cos(4*pi/5)
    const float s1 = 0.95105651629515357212f;   // sin(2*pi/5)
    const float s2 = 0.58778525229247312917f;   // sin(4*pi/5)
    const float2 t1 = cadd(a[1], a[4]);
    const float2 t2 = cadd(a[2], a[3]);
    const float2 t3 = csub(a[1], a[4]);
    const float2 t4 = csub(a[2], a[3]);
    const float2 b1 = c2(fmaf(c2v, t2.x, fmaf(c1, t1.x, a[0].x)), fmaf(c2v, t2.y, fmaf(c1, t1.y, a[0].y)));
    const float2 b2 = c2(fmaf(c1, t2.x, fmaf(c2v, t1.x, a[0].x)), fmaf(c1, t2.y, fmaf(c2v, t1.y, a[0].y)));
    const float2 u1 = mul_qturn<SIGN>(c2(fmaf(s1, t3.x, s2 * t4.x), fmaf(s1, t3.y, s2 * t4.y)));
    const float2 u2 = mul_qturn<SIGN>(c2(fmaf(s2, t3.x, -s1 * t4.x), fmaf(s2, t3.y, -s1 * t4.y)));
    a[0] = cadd(a[0], cadd(t1, t2));
    a[1] = cadd(b1, u1);
    a[4] = csub(b1, u1);
    a[2] = cadd(b2, u2);
    a[3] = csub(b2, u2);
  }
};

// Radix 7 as three conjugate pairs: with t_k = a[k] + a[7-k] and
// d_k = a[k] - a[7-k] (k = 1, 2, 3),
//   X[m], X[7-m] = a[0] + sum_k cos(2 pi k m / 7) t_k  +-  SIGN i sum_k sin(2 pi k m / 7) d_k.
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
    auto im = [&](float y1, float y2, float y3) {
      return mul_qturn<SIGN>(c2(fmaf(y3, d3.x, fmaf(y2, d2.x, y1 * d1.x)), fmaf(y3, d3.y, fmaf(y2, d2.y, y1 * d1.y))));
    };
    const float2 b1 = re(c1, c2v, c3);
    const float2 b2 = re(c2v, c3, c1);
    const float2 b3 = re(c3, c1, c2v);
    const float2 u1 = im(s1, s2, s3);
    const float2 u2 = im(s2, -s3, -s1);
    const float2 u3 = im(s3, -s1, s2);
    a[0] = cadd(a[0], cadd(t1, cadd(t2, t3)));
    a[1] = cadd(b1, u1);
    a[6] = csub(b1, u1);
    a[2] = cadd(b2, u2);
    a[5] = csub(b2, u2);
    a[3] = cadd(b3, u3);
    a[4] = csub(b3, u3);
  }
};

// Cooley-Tukey N = P*Q: P transforms of length Q on the stride-P
// subsequences, twiddle exp(SIGN*2*pi*i*p*k2/N), then Q transforms of length P;
// output X[k2 + Q*k1].
template <int P, int Q, int SIGN>
struct DftCT {
  LR_HD static void run(float2* a) {
    constexpr int N = P * Q;
    float2 t[N];
    static_for<0, P>([&](auto pc) {
      constexpr int p = decltype(pc)::value;
      float2 s[Q];
      static_for<0, Q>([&](auto mc) { s[mc.value] = a[P * mc.value + p]; });
      Dft<Q, SIGN>::run(s);
      static_for<0, Q>([&](auto kc) {
        constexpr int k2 = decltype(kc)::value;
        t[p * Q + k2] = twiddle_const<N, SIGN, p * k2>(s[k2]);
      });
    });
    static_for<0, Q>([&](auto kc) {
      constexpr int k2 = decltype(kc)::value;
      float2 u[P];
      static_for<0, P>([&](auto pc) { u[pc.value] = t[pc.value * Q + k2]; });
      Dft<P, SIGN>::run(u);
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
