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

// T vectors per workgroup; slot s = tid / T owns A-item j = s (one per
// thread, S = N2 slots) and B-items k1 = s, s + S, ...
template <class PL, int T_>
struct Cfg {
  using Plan = PL;
  static constexpr int N = PL::N;
  static constexpr int N1 = PL::N1;
  static constexpr int N2 = PL::N2;
  static constexpr int T = T_;
  static constexpr int S = PL::N2;
  static constexpr int P = T_ * S;
  static constexpr int TP = T_ + 1;
  static constexpr int IB = (N1 + S - 1) / S;
  static constexpr bool B_FULL = (N1 % S) == 0;
  // N slots of T+1 entries, then a spare slot that absorbs the shared-memory
  // writes of walk positions outside the tile
  static constexpr int SPARE = N * TP;
  static constexpr int LDS_ELEMS = (N + 1) * TP;
  static constexpr int LDS_BYTES = LDS_ELEMS * 8 + (P / 64) * 4;
  // Waves per SIMD that shared memory (160 KiB per CU) allows; the kernels
  // ask the compiler to fit their registers to this occupancy, and to at
  // least 2 waves (256 registers): allowed 512 at one wave per SIMD, the
  // large-N kernels took them all and hid no latency.
  static constexpr int WG_PER_CU = (160 * 1024) / LDS_BYTES;
  static constexpr int WAVES_RAW = (WG_PER_CU * (P / 64)) / 4;
  // one workgroup must fit: ten waves put three on some SIMD (168 registers)
  static constexpr int WAVES_MIN = (P / 64 + 3) / 4;
  static constexpr int WAVES_FIT = WAVES_RAW < WAVES_MIN ? WAVES_MIN : WAVES_RAW;
  static constexpr int WAVES = WAVES_FIT < 2 ? 2 : (WAVES_FIT > 4 ? 4 : WAVES_FIT);
  // kernels that also carry per-element gradient accumulators
  static constexpr int WAVES_ACC = WAVES > 2 ? (WAVES_MIN > 2 ? WAVES_MIN : 2) : WAVES;
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

// Root exp(-2*pi*i*m/N), m <= N, read at a 32-bit offset from the table's
// uniform base (one address register per load, nothing to keep live).
template <int N>
__device__ __forceinline__ float2 root_at(unsigned m) {
  return *reinterpret_cast<const float2*>(reinterpret_cast<const char*>(Roots<N>::table.w) + m * 8u);
}

// Forward half of the B-step: twiddles exp(-2*pi*i*k1*j/N) (Cooley-Tukey
// only), then DFT over j.
// Twiddles of long B-items as products of two roots, w^(k1*j) =
// w^(k1*(j mod 8)) * w^(8*k1*(j/8)): 7 + (N2/8 - 1) loads instead of N2 - 1.
template <class C, bool INV>
__device__ __forceinline__ void b_twiddle_split(int k1, float2 (&y)[C::N2]) {
  constexpr int NB = (C::N2 + 7) / 8;
  float2 lo[8];
  float2 hi[NB];
  static_for<1, 8>([&](auto j) {
    lo[j.value] = root_at<C::N>(INV ? (unsigned)(C::N - k1 * j.value) : (unsigned)(k1 * j.value));
  });
  static_for<1, NB>([&](auto b) {
    hi[b.value] = root_at<C::N>(INV ? (unsigned)(C::N - 8 * k1 * b.value) : (unsigned)(8 * k1 * b.value));
  });
  static_for<1, C::N2>([&](auto jc) {
    constexpr int j = decltype(jc)::value;
    constexpr int jl = j % 8;
    constexpr int jh = j / 8;
    if constexpr (jh == 0) {
      y[j] = cmul(y[j], lo[jl]);
    } else if constexpr (jl == 0) {
      y[j] = cmul(y[j], hi[jh]);
    } else {
      y[j] = cmul(y[j], cmul(lo[jl], hi[jh]));
    }
  });
}

template <class C>
__device__ __forceinline__ void b_forward(int k1, float2 (&y)[C::N2]) {
  using PL = typename C::Plan;
  if constexpr (!PL::PFA) {
    if constexpr (C::N2 >= 32) {
      b_twiddle_split<C, false>(k1, y);
    } else {
      static_for<1, C::N2>([&](auto j) { y[j.value] = cmul(y[j.value], root_at<C::N>((unsigned)(k1 * j.value))); });
    }
  }
  Dft<C::N2, -1>::run(y);
}
// Inverse half of the B-step: inverse DFT over k2, then the conjugate
// twiddles, read from the mirrored entries N - k1*j (different addresses, so
// they are loaded where they are used instead of being kept live from the
// forward half).
template <class C>
__device__ __forceinline__ void b_inverse(int k1, float2 (&y)[C::N2]) {
  using PL = typename C::Plan;
  Dft<C::N2, 1>::run(y);
  if constexpr (!PL::PFA) {
    if constexpr (C::N2 >= 32) {
      b_twiddle_split<C, true>(k1, y);
    } else {
      static_for<1, C::N2>(
          [&](auto j) { y[j.value] = cmul(y[j.value], root_at<C::N>((unsigned)(C::N - k1 * j.value))); });
    }
  }
}

// The padding column of the shared tile (vector index T, pitch T+1) holds N
// spare entries: the per-frequency table of the pass lives there, B-item major
// (slot of entry i = i), so B-steps read it next to their data.
template <class C>
__device__ __forceinline__ void stage_table(float2* lds, const float2* __restrict__ tab) {
  for (int i = threadIdx.x; i < C::N; i += C::P) lds[i * C::TP + C::T] = tab[i];
}

// Stage a per-frequency table given in natural frequency order (entry f for
// frequency index f) in the plan's B-item order: entry i of the padding
// column is frequency freq(i / N2, i % N2).
template <class C>
__device__ __forceinline__ void stage_table_by_freq(float2* lds, const float2* __restrict__ tab) {
  using PL = typename C::Plan;
  for (int i = threadIdx.x; i < C::N; i += C::P) {
    const int k1 = i / C::N2;
    lds[i * C::TP + C::T] = tab[PL::freq(k1, i - k1 * C::N2)];
  }
}

// B-step "forward, multiply by the staged per-frequency table, inverse" used
// by every propagation; conj selects conj(table).  The items of a thread are
// unrolled so their shared-memory reads overlap.
// One B-item of the spectral B-step.  For long items (N2 >= 16) scheduling
// barriers keep each phase's loads (data, twiddles, table) next to their
// use: hoisted to the front, they kept 3*N2 complex values live at once.
template <class C>
__device__ __forceinline__ void b_spectral_item(const Tile<C>& t, int k1, bool conj_tab) {
  constexpr bool FENCE = C::N2 >= 16;
  auto fence = [] {
    if constexpr (FENCE) __builtin_amdgcn_sched_barrier(0);
  };
  float2 y[C::N2];
  read_b(t, k1, y);
  b_forward<C>(k1, y);
  fence();
  const float2* tk = t.lds + (C::N2 * k1) * C::TP + C::T;
  if (conj_tab) {
    static_for<0, C::N2>([&](auto k) { y[k.value] = cmulc(y[k.value], tk[k.value * C::TP]); });
  } else {
    static_for<0, C::N2>([&](auto k) { y[k.value] = cmul(y[k.value], tk[k.value * C::TP]); });
  }
  fence();
  b_inverse<C>(k1, y);
  fence();
  write_b(t, k1, y);
}
// The last round of B-items when it holds a quarter of a round: with
// N1 mod N2 = N2/4 and N2 = 4*Q, Q odd (N = 500: 25 items of 20 values over
// 20 slots, 5 left per vector), a plain last round keeps a quarter of the
// threads busy while the rest wait at the next barrier.  Instead every
// left-over item goes to a quad of consecutive lanes, which splits its
// length-N2 DFT by the Good-Thomas map 4 x Q: lane q takes the Q values
// n = (Q*q + 4*m) mod N2, m < Q (with their Cooley-Tukey twiddles), runs a
// length-Q DFT over m, and the length-4 DFTs over q run across the quad as
// two radix-2 stages on lane exchanges, leaving lane q with the frequencies
// k4 = bitrev2(q) of the 4-point step.  After the table the inverse runs the
// mirrored network.  All P threads take part, one item per quad.
template <class C>
struct QuadLast {
  static constexpr int R = C::N1 % C::N2;
  static constexpr int Q = C::N2 / 4;
  static constexpr bool ON = C::N2 % 4 == 0 && Q % 2 == 1 && Q > 1 && R * 4 == C::N2;
  // output element k2 of the length-N2 DFT for (k4, k5): k4*E1 + k5*E2 mod N2
  static constexpr int E1 = ON ? Q * inv_mod(Q % 4, 4) : 0;
  static constexpr int E2 = ON ? 4 * inv_mod(4 % Q, Q) : 0;
};

// Value of the lane whose index differs in bit D (1 or 2) within its quad.
template <int D>
__device__ __forceinline__ float2 quad_xor(float2 v) {
  constexpr int kCtrl = D == 1 ? 0xB1 : 0x4E;  // quad_perm [1,0,3,2] / [2,3,0,1]
  return c2(__int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v.x), kCtrl, 0xF, 0xF, false)),
            __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v.y), kCtrl, 0xF, 0xF, false)));
}

// Radix-2 butterfly across lanes differing in bit D: the lower lane keeps
// own + partner, the upper one partner - own (sg = -1 there).
template <int D, int Q>
__device__ __forceinline__ void quad_butterfly(float2 (&z)[Q], float sg) {
  static_for<0, Q>([&](auto m) {
    const float2 p = quad_xor<D>(z[m.value]);
    z[m.value] = c2(fmaf(sg, z[m.value].x, p.x), fmaf(sg, z[m.value].y, p.y));
  });
}

template <class C>
__device__ __forceinline__ void b_spectral_quad(float2* lds, bool conj_tab) {
  using QL = QuadLast<C>;
  using PL = typename C::Plan;
  constexpr int Q = QL::Q;
  // the lane index behind an empty asm statement: the addresses and roots
  // derived from it are formed at each call, not hoisted out of the
  // caller's loops and kept live across them
  int tid = (int)threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int q = tid & 3;
  const int item = tid >> 2;
  const int v = item % C::T;
  const int k1 = C::N2 * (C::IB - 1) + item / C::T;
  float2* const base = lds + (C::N2 * k1) * C::TP + v;
  const float2* const tab = lds + (C::N2 * k1) * C::TP + C::T;
  // element n(q, m) = (Q*q + 4*m) mod N2 of the item
  auto elem = [&](auto m) {
    const int e = Q * q + 4 * decltype(m)::value;
    return e >= C::N2 ? e - C::N2 : e;
  };
  const float s1 = (q & 1) ? -1.f : 1.f;
  const float s2 = (q & 2) ? -1.f : 1.f;
  const bool l3 = q == 3;
  float2 z[Q];
  static_for<0, Q>([&](auto m) {
    const int e = elem(m);
    z[m.value] = base[e * C::TP];
    if constexpr (!PL::PFA) z[m.value] = cmul(z[m.value], root_at<C::N>((unsigned)(k1 * e)));
  });
  Dft<Q, -1>::run(z);
  // 4-point DFT over the quad by decimation in frequency: (x_q + x_{q+2}),
  // (x_q - x_{q+2}) w4^q, then pairs; w4 = -i on lane 3
  quad_butterfly<2, Q>(z, s2);
  static_for<0, Q>([&](auto m) {
    const float2 u = z[m.value];
    z[m.value] = l3 ? c2(u.y, -u.x) : u;
  });
  quad_butterfly<1, Q>(z, s1);
  const int k4 = ((q & 1) << 1) | (q >> 1);
  static_for<0, Q>([&](auto m) {
    int f = QL::E1 * k4 + QL::E2 * decltype(m)::value;
    f %= C::N2;
    const float2 h = tab[f * C::TP];
    z[m.value] = conj_tab ? cmulc(z[m.value], h) : cmul(z[m.value], h);
  });
  // inverse: the mirrored network with w4 = +i, bit-reversed in, natural out
  quad_butterfly<1, Q>(z, s1);
  static_for<0, Q>([&](auto m) {
    const float2 u = z[m.value];
    z[m.value] = l3 ? c2(-u.y, u.x) : u;
  });
  quad_butterfly<2, Q>(z, s2);
  Dft<Q, 1>::run(z);
  static_for<0, Q>([&](auto m) {
    const int e = elem(m);
    float2 r = z[m.value];
    if constexpr (!PL::PFA) r = cmul(r, root_at<C::N>((unsigned)(C::N - k1 * e)));
    base[e * C::TP] = r;
  });
}

template <class C, bool SERIAL = false>
__device__ __forceinline__ void b_spectral(const Tile<C>& t, bool conj_tab) {
  // The B-item index behind an empty asm statement: twiddle offsets derived
  // from it are formed here, not hoisted out of the caller's loops.
  int s = t.s;
  asm volatile("" : "+v"(s));
  constexpr bool QUAD = QuadLast<C>::ON;
  constexpr int IBR = QUAD ? C::IB - 1 : C::IB;  // rounds of whole items
  if constexpr (C::N2 >= 16) {
    // long B-items: one at a time, so that their registers are not doubled
#pragma unroll 1
    for (int ic = 0; ic < IBR; ++ic) {
      const int k1 = s + C::S * ic;
      if (C::B_FULL || QUAD || k1 < C::N1) b_spectral_item(t, k1, conj_tab);
    }
  } else {
    static_for<0, IBR>([&](auto ic) {
      const int k1 = s + C::S * decltype(ic)::value;
      if (C::B_FULL || QUAD || k1 < C::N1) b_spectral_item(t, k1, conj_tab);
      // SERIAL: one item's registers at a time (for kernels that hold other
      // arrays across the B-step)
      if constexpr (SERIAL) __builtin_amdgcn_sched_barrier(0);
    });
  }
  if constexpr (QUAD) b_spectral_quad<C>(t.lds, conj_tab);
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
