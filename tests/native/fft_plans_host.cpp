// Host-side check of the register codelets and the two-step tile plans.
//
// Each supported FFT length is run through the same A-step / B-step
// sequence the GPU tile kernels use (here as plain loops over items) and
// compared with a direct double-precision DFT sum.  Prints one line per
// case and exits non-zero on any failure.
#include <cmath>
#include <complex>
#include <cstdio>
#include <random>
#include <vector>

#include "../../paper_2306_11268_amd/csrc/plan.hpp"

using cd = std::complex<double>;

static std::vector<cd> naive_dft(const std::vector<cd>& x, int sign) {
  const int n = (int)x.size();
  std::vector<cd> y(n);
  for (int k = 0; k < n; ++k) {
    cd s = 0;
    for (int j = 0; j < n; ++j) {
      const long long e = (1LL * j * k) % n;
      s += x[j] * std::polar(1.0, sign * 2.0 * M_PI * (double)e / n);
    }
    y[k] = s;
  }
  return y;
}

static double rel_err(const std::vector<cd>& a, const std::vector<cd>& b) {
  double num = 0, den = 0;
  for (size_t i = 0; i < a.size(); ++i) { num += std::norm(a[i] - b[i]); den += std::norm(b[i]); }
  return std::sqrt(num / den);
}

template <int R>
static bool check_codelet(std::mt19937& g) {
  std::normal_distribution<double> nd;
  bool ok = true;
  for (int sign : {-1, 1}) {
    std::vector<cd> x(R);
    float2 a[R];
    for (int i = 0; i < R; ++i) { x[i] = cd((float)nd(g), (float)nd(g)); a[i] = lr::c2((float)x[i].real(), (float)x[i].imag()); }
    if (sign < 0) lr::Dft<R, -1>::run(a); else lr::Dft<R, 1>::run(a);
    std::vector<cd> y(R);
    for (int i = 0; i < R; ++i) y[i] = cd(a[i].x, a[i].y);
    const double e = rel_err(y, naive_dft(x, sign));
    const bool pass = e < 1e-6;
    std::printf("codelet R=%d sign=%+d rel=%.3e %s\n", R, sign, e, pass ? "ok" : "FAIL");
    ok &= pass;
  }
  return ok;
}

// Forward transform through the tile steps: natural positions in, natural frequencies out.
template <class PL>
static std::vector<cd> plan_forward(const std::vector<cd>& x) {
  std::vector<float2> lds(PL::N);
  for (int p = 0; p < PL::N; ++p) lds[PL::slot_of_pos(p)] = lr::c2((float)x[p].real(), (float)x[p].imag());
  for (int j = 0; j < PL::N2; ++j) {
    float2 a[PL::N1];
    for (int k = 0; k < PL::N1; ++k) {
      a[k] = lds[PL::a_slot(j, k)];
      if (PL::slot_of_pos(PL::pos(k, j)) != PL::a_slot(j, k)) { std::printf("slot/pos mismatch\n"); std::exit(2); }
    }
    lr::Dft<PL::N1, -1>::run(a);
    for (int k = 0; k < PL::N1; ++k) lds[PL::a_slot(j, k)] = a[k];
  }
  std::vector<cd> out(PL::N);
  for (int k1 = 0; k1 < PL::N1; ++k1) {
    float2 b[PL::N2];
    for (int j = 0; j < PL::N2; ++j) {
      b[j] = lds[PL::b_slot(k1, j)];
      if (!PL::PFA) b[j] = lr::cmul(b[j], PL::twiddle(k1, j));
    }
    lr::Dft<PL::N2, -1>::run(b);
    for (int k2 = 0; k2 < PL::N2; ++k2) {
      out[PL::freq(k1, k2)] = cd(b[k2].x, b[k2].y);
      if (PL::slot_of_freq(PL::freq(k1, k2)) != PL::b_slot(k1, k2)) { std::printf("slot_of_freq mismatch\n"); std::exit(2); }
    }
  }
  return out;
}

// Inverse transform through the tile steps: natural frequencies in, natural positions out (times N).
template <class PL>
static std::vector<cd> plan_inverse(const std::vector<cd>& f) {
  std::vector<float2> lds(PL::N);
  for (int k1 = 0; k1 < PL::N1; ++k1) {
    float2 b[PL::N2];
    for (int k2 = 0; k2 < PL::N2; ++k2) { const cd v = f[PL::freq(k1, k2)]; b[k2] = lr::c2((float)v.real(), (float)v.imag()); }
    lr::Dft<PL::N2, 1>::run(b);
    for (int j = 0; j < PL::N2; ++j) {
      if (!PL::PFA) b[j] = lr::cmulc(b[j], PL::twiddle(k1, j));
      lds[PL::b_slot(k1, j)] = b[j];
    }
  }
  for (int j = 0; j < PL::N2; ++j) {
    float2 a[PL::N1];
    for (int k = 0; k < PL::N1; ++k) a[k] = lds[PL::a_slot(j, k)];
    lr::Dft<PL::N1, 1>::run(a);
    for (int k = 0; k < PL::N1; ++k) lds[PL::a_slot(j, k)] = a[k];
  }
  std::vector<cd> out(PL::N);
  for (int p = 0; p < PL::N; ++p) { const float2 v = lds[PL::slot_of_pos(p)]; out[p] = cd(v.x, v.y); }
  return out;
}

template <class PL>
static bool check_plan_type(std::mt19937& g) {
  constexpr int N = PL::N;
  std::normal_distribution<double> nd;
  std::vector<cd> x(N);
  for (auto& v : x) v = cd((float)nd(g), (float)nd(g));
  const double ef = rel_err(plan_forward<PL>(x), naive_dft(x, -1));
  const double ei = rel_err(plan_inverse<PL>(x), naive_dft(x, +1));
  // every slot is visited exactly once by the A-items and by the B-items, and
  // the position map is a bijection
  std::vector<int> ca(N, 0), cb(N, 0), cp(N, 0);
  for (int j = 0; j < PL::N2; ++j) for (int k = 0; k < PL::N1; ++k) { ca[PL::a_slot(j, k)]++; cp[PL::pos(k, j)]++; }
  for (int k1 = 0; k1 < PL::N1; ++k1) for (int j = 0; j < PL::N2; ++j) cb[PL::b_slot(k1, j)]++;
  bool cover = true;
  for (int p = 0; p < N; ++p) cover &= (ca[p] == 1 && cb[p] == 1 && cp[p] == 1);
  // the incremental slot walk agrees with slot_of_pos from every start
  for (int p0 = 0; p0 < N; p0 += 7) {
    auto w = PL::walk(p0);
    for (int p = p0; p < N; ++p) {
      cover &= PL::walk_slot(w) == PL::slot_of_pos(p);
      PL::walk_next(w);
    }
  }
  const bool pass = ef < 2e-6 && ei < 2e-6 && cover;
  std::printf("plan N=%d (%dx%d %s) fwd=%.3e inv=%.3e cover=%d %s\n", N, PL::N1, PL::N2,
              PL::PFA ? "pfa" : "ct", ef, ei, (int)cover, pass ? "ok" : "FAIL");
  return pass;
}

template <int N>
static bool check_plan(std::mt19937& g) {
  bool ok = check_plan_type<typename lr::PlanFor<N>::type>(g);
  if (lr::PlanFor<N>::type::PFA) ok &= check_plan_type<typename lr::RowPlanFor<N>::type>(g);
  return ok;
}

int main() {
  std::mt19937 g(1234);
  bool ok = true;
  ok &= check_codelet<2>(g); ok &= check_codelet<3>(g); ok &= check_codelet<4>(g);
  ok &= check_codelet<5>(g); ok &= check_codelet<8>(g); ok &= check_codelet<10>(g);
  ok &= check_codelet<16>(g); ok &= check_codelet<20>(g); ok &= check_codelet<25>(g);
  ok &= check_codelet<32>(g); ok &= check_codelet<40>(g); ok &= check_codelet<7>(g);
  ok &= check_codelet<14>(g);
  ok &= check_plan<64>(g); ok &= check_plan<100>(g); ok &= check_plan<128>(g);
  ok &= check_plan<200>(g); ok &= check_plan<256>(g); ok &= check_plan<350>(g); ok &= check_plan<400>(g);
  ok &= check_plan<500>(g); ok &= check_plan<512>(g); ok &= check_plan<1000>(g);
  ok &= check_plan<1024>(g);
  std::printf(ok ? "ALL OK\n" : "FAILURES\n");
  return ok ? 0 : 1;
}
