// Device-side tile machinery: a workgroup transforms T vectors of length N
// at once, held in shared memory as lds[slot][vector] (pitch T+1).
//
// Thread tid works on vector v = tid % T in "slot" s = tid / T; slot s owns
// A-items i2 = s, s+S, ... and B-items k1 = s, s+S, ...  Consecutive lanes
// therefore touch consecutive vectors, which keeps shared-memory accesses
// conflict free and makes column loads from global memory coalesced.
#pragma once

#include "plan.hpp"

namespace lr {

template <class PL, int T_, int S_>
struct Cfg {
  using Plan = PL;
  static constexpr int N = PL::N;
  static constexpr int N1 = PL::N1;
  static constexpr int N2 = PL::N2;
  static constexpr int T = T_;
  static constexpr int S = S_;
  static constexpr int P = T_ * S_;
  static constexpr int TP = T_ + 1;
  static constexpr int IA = (N2 + S_ - 1) / S_;
  static constexpr int IB = (N1 + S_ - 1) / S_;
  static constexpr bool A_FULL = (N2 % S_) == 0;
  static constexpr bool B_FULL = (N1 % S_) == 0;
  static constexpr int LDS_ELEMS = N * TP;
  static constexpr int LDS_BYTES = LDS_ELEMS * 8 + (P / 64) * 4;
  // Waves per SIMD that shared memory (160 KiB per CU) allows; the kernels
  // ask the compiler to fit their registers to this occupancy.
  static constexpr int WG_PER_CU = (160 * 1024) / LDS_BYTES;
  static constexpr int WAVES_RAW = (WG_PER_CU * (P / 64)) / 4;
  static constexpr int WAVES = WAVES_RAW < 1 ? 1 : (WAVES_RAW > 8 ? 8 : WAVES_RAW);
  static_assert(P % 64 == 0, "workgroup must be whole wavefronts");
};

template <class C>
struct Tile {
  float2* lds;
  int v;
  int s;
  __device__ __forceinline__ float2& at(int slot) const { return lds[slot * C::TP + v]; }
};

// ---- A-items -------------------------------------------------------------

template <class C>
__device__ __forceinline__ void read_a(const Tile<C>& t, int j, float2 (&x)[C::N1]) {
  const float2* p = &t.at(j);
  static_for<0, C::N1>([&](auto k) { x[k.value] = p[k.value * C::N2 * C::TP]; });
}
template <class C>
__device__ __forceinline__ void write_a(const Tile<C>& t, int j, const float2 (&x)[C::N1]) {
  float2* p = &t.at(j);
  static_for<0, C::N1>([&](auto k) { p[k.value * C::N2 * C::TP] = x[k.value]; });
}

// Run f(ii, i2) for this thread's A-items; ii is a compile-time constant
// (std::integral_constant) so per-item register arrays can be indexed by it.
template <class C, class F>
__device__ __forceinline__ void for_a_items_static(const Tile<C>& t, F&& f) {
  static_for<0, C::IA>([&](auto ic) {
    const int i2 = t.s + C::S * decltype(ic)::value;
    if (C::A_FULL || i2 < C::N2) f(ic, i2);
  });
}
// Same with a run-time item loop (smaller code, no per-item state).
template <class C, class F>
__device__ __forceinline__ void for_a_items(const Tile<C>& t, F&& f) {
#pragma unroll 1
  for (int ii = 0; ii < C::IA; ++ii) {
    const int i2 = t.s + C::S * ii;
    if (!C::A_FULL && i2 >= C::N2) break;
    f(i2);
  }
}

// ---- B-items -------------------------------------------------------------

template <class C>
__device__ __forceinline__ void read_b(const Tile<C>& t, int k1, float2 (&y)[C::N2]) {
  const float2* p = &t.at(C::N2 * k1);
  static_for<0, C::N2>([&](auto j) { y[j.value] = p[j.value * C::TP]; });
}
template <class C>
__device__ __forceinline__ void write_b(const Tile<C>& t, int k1, const float2 (&y)[C::N2]) {
  float2* p = &t.at(C::N2 * k1);
  static_for<0, C::N2>([&](auto j) { p[j.value * C::TP] = y[j.value]; });
}

// Forward half of the B-step: twiddles (Cooley-Tukey only), then DFT over j.
template <class C>
__device__ __forceinline__ void b_forward(int k1, float2 (&y)[C::N2]) {
  using PL = typename C::Plan;
  if constexpr (!PL::PFA) {
    static_for<1, C::N2>([&](auto j) { y[j.value] = cmul(y[j.value], PL::twiddle(k1, j.value)); });
  }
  Dft<C::N2, -1>::run(y);
}
// Inverse half of the B-step: inverse DFT over k2, then conjugate twiddles.
template <class C>
__device__ __forceinline__ void b_inverse(int k1, float2 (&y)[C::N2]) {
  using PL = typename C::Plan;
  Dft<C::N2, 1>::run(y);
  if constexpr (!PL::PFA) {
    static_for<1, C::N2>([&](auto j) { y[j.value] = cmulc(y[j.value], PL::twiddle(k1, j.value)); });
  }
}

// B-step "forward, multiply by a per-frequency table, inverse" used by every
// propagation: tab is ordered [k1][k2] (B-item major), conj selects conj(tab).
template <class C>
__device__ __forceinline__ void b_spectral(const Tile<C>& t, const float2* __restrict__ tab, bool conj_tab) {
#pragma unroll 1
  for (int ii = 0; ii < C::IB; ++ii) {
    const int k1 = t.s + C::S * ii;
    if (!C::B_FULL && k1 >= C::N1) break;
    float2 y[C::N2];
    read_b(t, k1, y);
    b_forward<C>(k1, y);
    const float2* tk = tab + k1 * C::N2;
    if (conj_tab) {
      static_for<0, C::N2>([&](auto k) { y[k.value] = cmulc(y[k.value], tk[k.value]); });
    } else {
      static_for<0, C::N2>([&](auto k) { y[k.value] = cmul(y[k.value], tk[k.value]); });
    }
    b_inverse<C>(k1, y);
    write_b(t, k1, y);
  }
}

// ---- reductions ------------------------------------------------------------

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// Sum over the workgroup in a fixed order; red must hold P/64 floats.
template <int P>
__device__ __forceinline__ float block_sum(float x, float* red) {
  x = wave_sum(x);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = x;
  __syncthreads();
  float r = 0.f;
#pragma unroll
  for (int i = 0; i < P / 64; ++i) r += red[i];
  __syncthreads();
  return r;
}

}  // namespace lr
