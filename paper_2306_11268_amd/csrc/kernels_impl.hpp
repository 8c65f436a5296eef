// HIP kernel templates of the DONN physics path for gfx950 (instantiated per FFT size).
//
// Free-space propagation of one hop is the spectral product of §3.1.1,
// Eqs. (forward_diff)-(diffraction_freq): U -> IFFT2(H * FFT2(pad U)) then crop.
// For the Fresnel transfer function (Eq. (fresnel)) H factors into
// exp(jkz) * h(fy) * h(fx), so a hop is a 1-D propagation along x followed by
// one along y; consecutive 1-D propagations along the same axis, with the
// pointwise phase modulation of Eq. (phase_mod_matrix) between them, run in a
// single pass over the field.  The angular-spectrum transfer function does not
// factor; its hops use a row pass (FFT_x), a column pass (FFT_y, x H, IFFT_y)
// and a row pass (IFFT_x, modulation, next FFT_x).
#pragma once

#include <hip/hip_runtime.h>

#include "kernels.hpp"
#include "tile.hpp"

namespace lr {

// ---------------------------------------------------------------------------
// Natural-layout tile I/O.  The tile covers vectors vec0 .. vec0+nvalid-1 and
// layer positions q in [0, n); in shared memory position q lives in the
// slot of natural position q + off.  Element (v, q) is global (y, x) = (vec0+v, q) for a row
// pass and (q, vec0+v) for a column pass.  Iteration order keeps consecutive
// threads on consecutive x, so global accesses are coalesced.
// ---------------------------------------------------------------------------
template <class C, int AXIS, class F>
__device__ __forceinline__ void for_tile_elems(int n, int nvalid, F&& fn) {
  if constexpr (AXIS == kRow) {
    for (int v = 0; v < nvalid; ++v)
      for (int q = threadIdx.x; q < n; q += C::P) fn(v, q);
  } else {
    const int total = n * C::T;
    for (int e = threadIdx.x; e < total; e += C::P) {
      const int q = e / C::T;
      const int v = e - q * C::T;
      if (v < nvalid) fn(v, q);
    }
  }
}

template <int AXIS>
__device__ __forceinline__ size_t nat_index(int n, int vec, int q) {
  return AXIS == kRow ? (size_t)vec * n + q : (size_t)q * n + vec;
}

// Shared-memory slot of natural position p of vector v.
template <class C>
__device__ __forceinline__ int lds_index(int p, int v) {
  return C::Plan::slot_of_pos(p) * C::TP + v;
}

// Zero the padding positions [0, off) and [off+n, N) of every vector.
template <class C>
__device__ __forceinline__ void zero_padding(float2* lds, int n, int off) {
  if (off == 0 && n == C::N) return;
  const int npad = C::N - n;
  for (int e = threadIdx.x; e < npad * C::T; e += C::P) {
    const int r = e / C::T;
    const int v = e - r * C::T;
    const int p = r < off ? r : r + n;
    lds[lds_index<C>(p, v)] = c2(0.f, 0.f);
  }
}

__device__ __forceinline__ bool in_region(int y, int x, int y0, int x0, int s) {
  return (unsigned)(y - y0) < (unsigned)s && (unsigned)(x - x0) < (unsigned)s;
}

// ---------------------------------------------------------------------------
// Loading a tile in natural order (zero padding, optional adjoint seed).
// ---------------------------------------------------------------------------
template <class C, int AXIS, bool SEED>
__device__ __forceinline__ void load_tile(float2* lds, const PassArgs& a, int b, int vec0, int nvalid) {
  const int n = a.n;
  const int off = a.off;
  const size_t nn = (size_t)n * n;
  zero_padding<C>(lds, n, off);
  if constexpr (SEED) {
    // G_D = 2 * (dL/dI) * U_D with dL/dI a full map or region-constant from dL/dS
    const float2* __restrict__ ud = a.ud_in + (size_t)b * nn;
    const float* __restrict__ gint = a.grad_int ? a.grad_int + (size_t)b * nn : nullptr;
    const float* __restrict__ gsum = a.grad_sums ? a.grad_sums + (size_t)b * a.K : nullptr;
    const int2* __restrict__ regions = a.regions;
    const int K = a.K;
    const int dsz = a.det_size;
    for_tile_elems<C, AXIS>(n, nvalid, [&](int v, int q) {
      const int y = AXIS == kRow ? vec0 + v : q;
      const int x = AXIS == kRow ? q : vec0 + v;
      const size_t idx = (size_t)y * n + x;
      float g = 0.f;
      if (gint) {
        g = gint[idx];
      } else {
        for (int k = 0; k < K; ++k) {
          const int2 r = regions[k];
          if (in_region(y, x, r.x, r.y, dsz)) g += gsum[k];
        }
      }
      lds[lds_index<C>(q + off, v)] = g != 0.f ? cscale(ud[idx], 2.f * g) : c2(0.f, 0.f);
    });
  } else if (a.in_real) {
    const float* __restrict__ in = static_cast<const float*>(a.in) + (size_t)b * nn;
    for_tile_elems<C, AXIS>(n, nvalid, [&](int v, int q) {
      lds[lds_index<C>(q + off, v)] = c2(in[nat_index<AXIS>(n, vec0 + v, q)], 0.f);
    });
  } else {
    const float2* __restrict__ in = static_cast<const float2*>(a.in) + (size_t)b * nn;
    for_tile_elems<C, AXIS>(n, nvalid, [&](int v, int q) {
      lds[lds_index<C>(q + off, v)] = in[nat_index<AXIS>(n, vec0 + v, q)];
    });
  }
}

// Detector-plane outputs from a tile that holds U_D in natural order:
// |U|^2, U_D copies, and per-(sample, tile, region) partial sums.
template <class C, int AXIS>
__device__ __forceinline__ void tile_outputs(const float2* lds, float* red, const PassArgs& a, int b, int vec0,
                                             int nvalid) {
  const int n = a.n;
  const int off = a.off;
  const size_t nn = (size_t)n * n;
  float2* fo = a.field_out ? a.field_out + (size_t)b * nn : nullptr;
  float2* sv = a.saved_ud ? a.saved_ud + (size_t)b * nn : nullptr;
  float* io = a.intensity ? a.intensity + (size_t)b * nn : nullptr;
  if (fo || sv || io) {
    for_tile_elems<C, AXIS>(n, nvalid, [&](int v, int q) {
      const float2 u = lds[lds_index<C>(q + off, v)];
      const size_t idx = nat_index<AXIS>(n, vec0 + v, q);
      if (fo) fo[idx] = u;
      if (sv) sv[idx] = u;
      if (io) io[idx] = cabs2(u);
    });
  }
  if (a.sums_part) {
    const int K = a.K;
    const int s = a.det_size;
    for (int k = 0; k < K; ++k) {
      const int2 r = a.regions[k];                 // (y0, x0)
      const int vlo_g = AXIS == kRow ? r.x : r.y;  // region start along the vector index
      const int qlo = AXIS == kRow ? r.y : r.x;    // region start along positions
      const int v_lo = max(vlo_g - vec0, 0);
      const int v_hi = min(vlo_g + s - vec0, nvalid);
      float part = 0.f;
      if (v_hi > v_lo) {
        const int nv = v_hi - v_lo;
        float my = 0.f;
        for (int e = threadIdx.x; e < nv * s; e += C::P) {
          const int qq = e / nv;
          const int vv = e - qq * nv;
          my += cabs2(lds[lds_index<C>(qlo + qq + off, v_lo + vv)]);
        }
        part = block_sum<C::P>(my, red);
      }
      if (threadIdx.x == 0) a.sums_part[((size_t)b * a.ntiles + blockIdx.x) * K + k] = part;
    }
  }
}

// Forward A-step (DFT over the N1 elements of each A-item).
template <class C>
__device__ __forceinline__ void a_forward(const Tile<C>& t) {
  for_a_items<C>(t, [&](int j) {
    float2 x[C::N1];
    read_a(t, j, x);
    Dft<C::N1, -1>::run(x);
    write_a(t, j, x);
  });
}
// Inverse A-step.
template <class C>
__device__ __forceinline__ void a_inverse(const Tile<C>& t) {
  for_a_items<C>(t, [&](int j) {
    float2 x[C::N1];
    read_a(t, j, x);
    Dft<C::N1, 1>::run(x);
    write_a(t, j, x);
  });
}

// Inverse A-step, the layer operation at every cropped position, forward A-step.
// Forward: U_l = V * M_l (optionally stored).  Backward: dphi += Im(conj(U_l) G),
// G *= conj(M_l); with FWD_AFTER false (last backward pass) only the
// accumulation is done.  Oriented arrays are indexed [q][vec].
template <class C, bool BWD, bool FWD_AFTER, class ACC>
__device__ __forceinline__ void a_layer_op(const Tile<C>& t, const PassArgs& a, int b, int vec, bool vok, ACC& acc) {
  using PL = typename C::Plan;
  const int n = a.n;
  const int off = a.off;
  const size_t nn = (size_t)n * n;
  const float2* __restrict__ mod = a.mod;
  const float2* __restrict__ act_in = BWD ? a.act_in + (size_t)b * nn : nullptr;
  float2* __restrict__ act_out = (!BWD && a.act_out) ? a.act_out + (size_t)b * nn : nullptr;
  auto body = [&](auto ic, int j) {
    constexpr int ii = decltype(ic)::value;
    const int pb = PL::pos_base(j);
    float2 x[C::N1];
    read_a(t, j, x);
    Dft<C::N1, 1>::run(x);
    static_for<0, C::N1>([&](auto kc) {
      constexpr int k = decltype(kc)::value;
      const int q = PL::pos_at(pb, k) - off;
      const bool in = vok && (unsigned)q < (unsigned)n;
      float2 u = c2(0.f, 0.f);
      if (in) {
        const size_t oi = (size_t)q * n + vec;
        if constexpr (!BWD) {
          u = cmul(x[k], mod[oi]);
          if (act_out) act_out[oi] = u;
        } else {
          const float2 ul = act_in[oi];
          acc[ii][k] += ul.x * x[k].y - ul.y * x[k].x;  // Im(conj(U_l) * G)
          if constexpr (FWD_AFTER) u = cmulc(x[k], mod[oi]);
        }
      }
      x[k] = u;
    });
    if constexpr (FWD_AFTER) {
      Dft<C::N1, -1>::run(x);
      write_a(t, j, x);
    }
  };
  if constexpr (BWD) {
    for_a_items_static<C>(t, body);
  } else {
    for_a_items<C>(t, [&](int i2) { body(std::integral_constant<int, 0>{}, i2); });
  }
}

template <class C, class ACC>
__device__ __forceinline__ void write_dphi(const Tile<C>& t, const PassArgs& a, int vec, bool vok, ACC& acc) {
  using PL = typename C::Plan;
  const int n = a.n;
  const int off = a.off;
  float* __restrict__ dp = a.dphi_part + (size_t)blockIdx.y * n * n;
  for_a_items_static<C>(t, [&](auto ic, int j) {
    constexpr int ii = decltype(ic)::value;
    const int pb = PL::pos_base(j);
    static_for<0, C::N1>([&](auto kc) {
      constexpr int k = decltype(kc)::value;
      const int q = PL::pos_at(pb, k) - off;
      if (vok && (unsigned)q < (unsigned)n) dp[(size_t)q * n + vec] = acc[ii][k];
    });
  });
}

// ---------------------------------------------------------------------------
// Separable (Fresnel) pass.
// ---------------------------------------------------------------------------
template <class C, int KIND, int AXIS>
__global__ void __launch_bounds__(C::P, C::WAVES) fresnel_pass(PassArgs a) {
  __shared__ float2 lds[C::LDS_ELEMS];
  __shared__ float red[C::P / 64];
  constexpr bool ACC = (KIND == kBwdMid || KIND == kBwdLast);
  constexpr bool TWO = (KIND == kFwdMid || KIND == kBwdMid);
  const Tile<C> t{lds, (int)(threadIdx.x % C::T), (int)(threadIdx.x / C::T)};

  const int n = a.n;
  const int off = a.off;
  const int vec0 = blockIdx.x * C::T;
  const int vec = vec0 + t.v;
  const int nvalid = min(C::T, a.nvec - vec0);
  const bool vok = t.v < nvalid;
  const int b0 = blockIdx.y * a.spg;
  const int b1 = min(a.batch, b0 + a.spg);
  const bool conj_tab = a.conj_tab != 0;

  float acc[ACC ? C::IA : 1][ACC ? C::N1 : 1];
  if constexpr (ACC) {
    static_for<0, C::IA>([&](auto i) { static_for<0, C::N1>([&](auto k) { acc[i.value][k.value] = 0.f; }); });
  }

  for (int b = b0; b < b1; ++b) {
    __syncthreads();
    load_tile<C, AXIS, KIND == kBwdFirst>(lds, a, b, vec0, nvalid);
    __syncthreads();
    a_forward<C>(t);
    __syncthreads();
    b_spectral(t, a.tab, conj_tab);
    __syncthreads();
    if constexpr (TWO) {
      a_layer_op<C, ACC, true>(t, a, b, vec, vok, acc);
      __syncthreads();
      b_spectral(t, a.tab, conj_tab);
      __syncthreads();
    }
    if constexpr (KIND == kBwdLast) {
      a_layer_op<C, true, false>(t, a, b, vec, vok, acc);
      continue;
    }
    a_inverse<C>(t);
    __syncthreads();
    if constexpr (KIND == kFwdLast) {
      tile_outputs<C, AXIS>(lds, red, a, b, vec0, nvalid);
    } else {
      float2* __restrict__ out = a.out + (size_t)b * n * n;
      for_tile_elems<C, AXIS>(n, nvalid, [&](int v, int q) {
        out[nat_index<AXIS>(n, vec0 + v, q)] = lds[lds_index<C>(q + off, v)];
      });
    }
  }
  if constexpr (ACC) write_dphi(t, a, vec, vok, acc);
}

// ---------------------------------------------------------------------------
// Angular-spectrum passes.  Between passes a sample is stored as n rows of
// N x-spectrum values in the plan's slot order ([B][n][N]).
// ---------------------------------------------------------------------------
template <class C>
__device__ __forceinline__ void b_forward_all(const Tile<C>& t) {
#pragma unroll 1
  for (int ii = 0; ii < C::IB; ++ii) {
    const int k1 = t.s + C::S * ii;
    if (!C::B_FULL && k1 >= C::N1) break;
    float2 y[C::N2];
    read_b(t, k1, y);
    b_forward<C>(k1, y);
    write_b(t, k1, y);
  }
}
template <class C>
__device__ __forceinline__ void b_inverse_all(const Tile<C>& t) {
#pragma unroll 1
  for (int ii = 0; ii < C::IB; ++ii) {
    const int k1 = t.s + C::S * ii;
    if (!C::B_FULL && k1 >= C::N1) break;
    float2 y[C::N2];
    read_b(t, k1, y);
    b_inverse<C>(k1, y);
    write_b(t, k1, y);
  }
}

template <class C, int KIND>
__global__ void __launch_bounds__(C::P, C::WAVES) as_pass(PassArgs a) {
  __shared__ float2 lds[C::LDS_ELEMS];
  __shared__ float red[C::P / 64];
  using PL = typename C::Plan;
  constexpr int N = C::N;
  constexpr bool ACC = (KIND == kAsRowBwdMid || KIND == kAsRowBwdLast);
  constexpr bool SPECTRAL_IN = (KIND == kAsRowMid || KIND == kAsRowLast || KIND == kAsRowBwdMid ||
                                KIND == kAsRowBwdLast || KIND == kAsRowIfft);
  constexpr bool FWD_OUT = (KIND == kAsRowFirst || KIND == kAsRowMid || KIND == kAsRowBwdFirst ||
                            KIND == kAsRowBwdMid);
  const Tile<C> t{lds, (int)(threadIdx.x % C::T), (int)(threadIdx.x / C::T)};

  const int n = a.n;
  const int off = a.off;
  const int vec0 = blockIdx.x * C::T;
  const int vec = vec0 + t.v;
  const int nvalid = min(C::T, a.nvec - vec0);
  const bool vok = t.v < nvalid;
  const int b0 = blockIdx.y * a.spg;
  const int b1 = min(a.batch, b0 + a.spg);

  float acc[ACC ? C::IA : 1][ACC ? C::N1 : 1];
  if constexpr (ACC) {
    static_for<0, C::IA>([&](auto i) { static_for<0, C::N1>([&](auto k) { acc[i.value][k.value] = 0.f; }); });
  }

  for (int b = b0; b < b1; ++b) {
    __syncthreads();
    if constexpr (KIND == kAsCol) {
      // vectors: spectrum columns (slot order); positions: rows y of the padded grid
      zero_padding<C>(lds, n, off);
      const float2* __restrict__ in = static_cast<const float2*>(a.in) + (size_t)b * n * N;
      for (int e = threadIdx.x; e < n * C::T; e += C::P) {
        const int q = e / C::T;
        const int v = e - q * C::T;
        if (v < nvalid) lds[lds_index<C>(q + off, v)] = in[(size_t)q * N + vec0 + v];
      }
      __syncthreads();
      a_forward<C>(t);
      __syncthreads();
      // B-step with the 2-D table: element k2 of item k1 is ky = freq(k1, k2)
      const bool cj = a.conj_tab != 0;
#pragma unroll 1
      for (int ii = 0; ii < C::IB; ++ii) {
        const int k1 = t.s + C::S * ii;
        if (!C::B_FULL && k1 >= C::N1) break;
        float2 y[C::N2];
        read_b(t, k1, y);
        b_forward<C>(k1, y);
        if (vok) {
          static_for<0, C::N2>([&](auto kc) {
            constexpr int k2 = decltype(kc)::value;
            const float2 h = a.tab[(size_t)PL::freq(k1, k2) * N + vec];
            y[k2] = cj ? cmulc(y[k2], h) : cmul(y[k2], h);
          });
        }
        b_inverse<C>(k1, y);
        write_b(t, k1, y);
      }
      __syncthreads();
      a_inverse<C>(t);
      __syncthreads();
      float2* __restrict__ out = a.out + (size_t)b * n * N;
      for (int e = threadIdx.x; e < n * C::T; e += C::P) {
        const int q = e / C::T;
        const int v = e - q * C::T;
        if (v < nvalid) out[(size_t)q * N + vec0 + v] = lds[lds_index<C>(q + off, v)];
      }
      continue;
    }

    // ---- row passes: vectors are layer rows y = vec0 + v
    if constexpr (SPECTRAL_IN) {
      const float2* __restrict__ in = static_cast<const float2*>(a.in) + (size_t)b * n * N;
      for (int v = 0; v < nvalid; ++v)
        for (int c = threadIdx.x; c < N; c += C::P) lds[c * C::TP + v] = in[(size_t)(vec0 + v) * N + c];
      __syncthreads();
      b_inverse_all<C>(t);
      __syncthreads();
      if constexpr (KIND == kAsRowMid) {
        a_layer_op<C, false, true>(t, a, b, vec, vok, acc);
      } else if constexpr (KIND == kAsRowBwdMid) {
        a_layer_op<C, true, true>(t, a, b, vec, vok, acc);
      } else if constexpr (KIND == kAsRowBwdLast) {
        a_layer_op<C, true, false>(t, a, b, vec, vok, acc);
        continue;
      } else {
        a_inverse<C>(t);  // kAsRowLast, kAsRowIfft: back to positions (crop on output)
      }
    } else {
      load_tile<C, kRow, KIND == kAsRowBwdFirst>(lds, a, b, vec0, nvalid);
      __syncthreads();
      a_forward<C>(t);
    }
    __syncthreads();

    if constexpr (FWD_OUT) {
      if constexpr (SPECTRAL_IN) {
        // a_layer_op already ran the forward A-step
      }
      b_forward_all<C>(t);
      __syncthreads();
      float2* __restrict__ out = a.out + (size_t)b * n * N;
      for (int v = 0; v < nvalid; ++v)
        for (int c = threadIdx.x; c < N; c += C::P) out[(size_t)(vec0 + v) * N + c] = lds[c * C::TP + v];
    } else if constexpr (KIND == kAsRowIfft) {
      float2* __restrict__ out = a.out + (size_t)b * n * n;
      for_tile_elems<C, kRow>(n, nvalid, [&](int v, int q) {
        out[(size_t)(vec0 + v) * n + q] = lds[lds_index<C>(q + off, v)];
      });
    } else {  // kAsRowLast
      tile_outputs<C, kRow>(lds, red, a, b, vec0, nvalid);
    }
  }
  if constexpr (ACC) write_dphi(t, a, vec, vok, acc);
}

// ---------------------------------------------------------------------------
// Helper kernels
// ---------------------------------------------------------------------------

// Separable chirps from the 2-D Fresnel table: row (x) chirp H[0][k] and
// column (y) chirp H[k][0]*conj(H[0][0]) (so their product carries exp(jkz)
// once), with the 1/N of each inverse DFT folded in, stored B-item major.
template <class PL>
__global__ void prep_chirps_kernel(const float2* __restrict__ H, float2* __restrict__ cx, float2* __restrict__ cy) {
  constexpr int N = PL::N;
  const float2 h00c = cconj(H[0]);
  const float inv = 1.0f / (float)N;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < N; i += gridDim.x * blockDim.x) {
    const int k1 = i / PL::N2;
    const int k2 = i - k1 * PL::N2;
    const int f = PL::freq(k1, k2);
    cx[i] = cscale(H[f], inv);
    cy[i] = cscale(cmul(H[(size_t)f * N], h00c), inv);
  }
}

// Column-permuted 2-D table for the angular-spectrum column pass:
// Hp[ky][c] = H[ky][kx(c)] / N^2, c the slot of frequency kx.
template <class PL>
__global__ void prep_as_table_kernel(const float2* __restrict__ H, float2* __restrict__ Hp) {
  constexpr int N = PL::N;
  const float inv = 1.0f / ((float)N * (float)N);
  const size_t total = (size_t)N * N;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int ky = (int)(i / N);
    const int c = (int)(i - (size_t)ky * N);
    // slot c holds element k2 of B-item k1
    const int k1 = c / PL::N2;
    const int k2 = c - k1 * PL::N2;
    const int kx = PL::freq(k1, k2);
    Hp[i] = cscale(H[(size_t)ky * N + kx], inv);
  }
}

// ---------------------------------------------------------------------------
// Per-size launchers (explicitly instantiated in one translation unit per size)
// ---------------------------------------------------------------------------

template <int N> struct Shape;
// T vectors per workgroup, S slots per vector.
template <> struct Shape<64>   { static constexpr int T = 16, S = 8; };
template <> struct Shape<100>  { static constexpr int T = 16, S = 4; };
template <> struct Shape<128>  { static constexpr int T = 16, S = 8; };
template <> struct Shape<200>  { static constexpr int T = 16, S = 8; };
template <> struct Shape<256>  { static constexpr int T = 8, S = 16; };
template <> struct Shape<400>  { static constexpr int T = 8, S = 8; };
template <> struct Shape<500>  { static constexpr int T = 8, S = 8; };
template <> struct Shape<512>  { static constexpr int T = 4, S = 16; };
template <> struct Shape<1000> { static constexpr int T = 4, S = 16; };
template <> struct Shape<1024> { static constexpr int T = 4, S = 16; };

template <int N>
using CfgFor = Cfg<typename PlanFor<N>::type, Shape<N>::T, Shape<N>::S>;

template <int N, int KIND, int AXIS>
hipError_t launch_fr(const PassArgs& a, hipStream_t st) {
  using C = CfgFor<N>;
  const dim3 grid(a.ntiles, (a.batch + a.spg - 1) / a.spg);
  hipLaunchKernelGGL((fresnel_pass<C, KIND, AXIS>), grid, dim3(C::P), 0, st, a);
  return hipGetLastError();
}

template <int N, int KIND>
hipError_t launch_fr_axis(Axis axis, const PassArgs& a, hipStream_t st) {
  return axis == kRow ? launch_fr<N, KIND, kRow>(a, st) : launch_fr<N, KIND, kCol>(a, st);
}

template <int N>
hipError_t launch_fr_n(PassKind kind, Axis axis, const PassArgs& a, hipStream_t st) {
  switch (kind) {
    case kPropOnce: return launch_fr_axis<N, kPropOnce>(axis, a, st);
    case kFwdMid: return launch_fr_axis<N, kFwdMid>(axis, a, st);
    case kFwdLast: return launch_fr_axis<N, kFwdLast>(axis, a, st);
    case kBwdFirst: return launch_fr_axis<N, kBwdFirst>(axis, a, st);
    case kBwdMid: return launch_fr_axis<N, kBwdMid>(axis, a, st);
    case kBwdLast: return launch_fr_axis<N, kBwdLast>(axis, a, st);
  }
  return hipErrorInvalidValue;
}

template <int N, int KIND>
hipError_t launch_as(const PassArgs& a, hipStream_t st) {
  using C = CfgFor<N>;
  const dim3 grid(a.ntiles, (a.batch + a.spg - 1) / a.spg);
  hipLaunchKernelGGL((as_pass<C, KIND>), grid, dim3(C::P), 0, st, a);
  return hipGetLastError();
}

template <int N>
hipError_t launch_as_n(AsPassKind kind, const PassArgs& a, hipStream_t st) {
  switch (kind) {
    case kAsRowFirst: return launch_as<N, kAsRowFirst>(a, st);
    case kAsCol: return launch_as<N, kAsCol>(a, st);
    case kAsRowMid: return launch_as<N, kAsRowMid>(a, st);
    case kAsRowLast: return launch_as<N, kAsRowLast>(a, st);
    case kAsRowBwdFirst: return launch_as<N, kAsRowBwdFirst>(a, st);
    case kAsRowBwdMid: return launch_as<N, kAsRowBwdMid>(a, st);
    case kAsRowBwdLast: return launch_as<N, kAsRowBwdLast>(a, st);
    case kAsRowIfft: return launch_as<N, kAsRowIfft>(a, st);
  }
  return hipErrorInvalidValue;
}

template <int N>
hipError_t prep_chirps_n(const float2* H, float2* cx, float2* cy, hipStream_t st) {
  hipLaunchKernelGGL((prep_chirps_kernel<typename PlanFor<N>::type>), dim3((N + 255) / 256), dim3(256), 0, st, H, cx, cy);
  return hipGetLastError();
}

template <int N>
hipError_t prep_as_n(const float2* H, float2* Hp, hipStream_t st) {
  const int blocks = (int)(((size_t)N * N + 255) / 256);
  hipLaunchKernelGGL((prep_as_table_kernel<typename PlanFor<N>::type>), dim3(blocks < 4096 ? blocks : 4096), dim3(256), 0,
                     st, H, Hp);
  return hipGetLastError();
}

template <int N>
TileShape shape_n() { return TileShape{Shape<N>::T, Shape<N>::S}; }

}  // namespace lr
