// Host-side check of the shared-memory layout of the tile kernels: for every
// FFT length and tile width the kernels can use, the entry of (slot, vector)
// -- including the table column v = T -- is distinct and inside the buffer
// (below the spare slot), the spare slot fits, and the workgroup's shared
// memory fits a CU, and the register budget (waves per SIMD the kernels ask
// the compiler for) lets one workgroup's waves fit the CU's four SIMDs.  The bank spread of the A- and B-step accesses (lanes per
// 8-byte bank pair; two is the minimum for 8-byte accesses) is printed for
// the record.  Runs on the host only; no kernel is launched.
#include <cstdio>
#include <vector>

#include "../../paper_2306_11268_amd/csrc/tile.hpp"

template <class PL, int T>
static bool check_cfg() {
  using C = lr::Cfg<PL, T>;
  bool ok = true;
  std::vector<int> seen(C::LDS_ELEMS, 0);
  for (int slot = 0; slot < C::N; ++slot) {
    for (int v = 0; v <= T; ++v) {
      const int idx = slot * C::TP + v;
      if (idx < 0 || idx >= C::SPARE) { ok = false; continue; }
      if (seen[idx]++) ok = false;
    }
  }
  if (C::SPARE + C::TP > C::LDS_ELEMS) ok = false;
  if (C::LDS_BYTES > 160 * 1024) ok = false;
  // the register budget the kernels ask for lets one workgroup fit a CU: its
  // waves spread over 4 SIMDs need ceil(waves / 4) per SIMD (512 / that
  // registers), with and without gradient accumulators
  const int waves = C::P / 64;
  const int need = (waves + 3) / 4;
  if (C::WAVES < need || C::WAVES_ACC < need) ok = false;
  // B-step access: lane l of a wave works on B-item k1 = l / T (+ wave offset)
  // and vector v = l % T, all at the same element j
  int worst = 0;
  for (int j = 0; j < C::N2; ++j) {
    int count[32] = {0};
    for (int l = 0; l < 64; ++l) {
      const int k1 = l / T, v = l % T;
      if (k1 >= C::N1) continue;
      ++count[((C::N2 * k1 + j) * C::TP + v) % 32];
    }
    for (int b = 0; b < 32; ++b) worst = count[b] > worst ? count[b] : worst;
  }
  // A-step access (lane l: vector l % T, A-item l / T), for the record
  int worst_a = 0;
  {
    int count[32] = {0};
    for (int l = 0; l < 64; ++l) {
      const int j = l / T, v = l % T;
      if (j >= C::N2) continue;
      const int c = ++count[(j * C::TP + v) % 32];
      worst_a = c > worst_a ? c : worst_a;
    }
  }
  std::printf("N=%4d T=%2d TP=%2d LDS=%6d lanes per bank pair: B %d, A %d  %s\n", C::N, T, C::TP, C::LDS_BYTES,
              worst, worst_a, ok ? "ok" : "FAIL");
  return ok;
}

template <int N>
static bool check_size() {
  using PL = typename lr::PlanFor<N>::type;
  bool ok = true;
  // the widths for which T * N2 is whole waves and the buffer fits a CU
  lr::static_for<0, 4>([&](auto i) {
    constexpr int T = 4 << decltype(i)::value;
    if constexpr ((T * PL::N2) % 64 == 0 && T * PL::N2 <= 1024) {
      if constexpr (lr::Cfg<PL, T>::LDS_BYTES <= 160 * 1024) ok &= check_cfg<PL, T>();
    }
  });
  return ok;
}

int main() {
  bool ok = true;
  ok &= check_size<64>(); ok &= check_size<100>(); ok &= check_size<128>(); ok &= check_size<200>();
  ok &= check_size<256>(); ok &= check_size<350>(); ok &= check_size<400>(); ok &= check_size<500>(); ok &= check_size<512>();
  ok &= check_size<1000>(); ok &= check_size<1024>();
  ok &= check_cfg<lr::PlanFor<200>::type, 24>();
  // the ten-wave forward tiles of 500 and 1000 points
  ok &= check_cfg<lr::PlanFor<500>::type, 32>();
  ok &= check_cfg<lr::PlanFor<1000>::type, 16>();
  std::printf(ok ? "ALL OK\n" : "FAILURES\n");
  return ok ? 0 : 1;
}
