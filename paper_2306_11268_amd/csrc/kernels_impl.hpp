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
//
// Every thread owns one A-item (j = its slot) of its vector, so the A-step
// data of a thread is a plain register array x[N1].  Global I/O of a tile is
// batched in chunks: a thread issues several loads before it uses them.
// Per-layer arrays (modulation, activations, dphi) are oriented [q][vec],
// q the position along the pass axis and vec the vector index.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "kernels.hpp"
#include "tile.hpp"

namespace lr {

// Global accesses at a uniform base plus a 32-bit unsigned element index: the
// byte offset is formed in 32 bits so the scalar-base addressing form is used.
template <class T>
__device__ __forceinline__ T ld(const T* base, unsigned idx) {
  return *reinterpret_cast<const T*>(reinterpret_cast<const char*>(base) + idx * (unsigned)sizeof(T));
}
template <class T>
__device__ __forceinline__ void st(T* base, unsigned idx, T v) {
  *reinterpret_cast<T*>(reinterpret_cast<char*>(base) + idx * (unsigned)sizeof(T)) = v;
}

// Streaming variants for data touched once per pass (saved activations):
// non-temporal hints keep them from displacing reused lines in the caches.
__device__ __forceinline__ float2 ld_stream(const float2* base, unsigned idx) {
  const unsigned long long u = __builtin_nontemporal_load(
      reinterpret_cast<const unsigned long long*>(reinterpret_cast<const char*>(base) + idx * 8u));
  return __builtin_bit_cast(float2, u);
}
__device__ __forceinline__ void st_stream(float2* base, unsigned idx, float2 v) {
  __builtin_nontemporal_store(__builtin_bit_cast(unsigned long long, v),
                              reinterpret_cast<unsigned long long*>(reinterpret_cast<char*>(base) + idx * 8u));
}

// Raw buffer access.  A buffer resource bounds every access to [0, bytes):
// a load at an out-of-range offset returns zero and a store there is
// dropped, so masked elements take the offset kOutOfRange instead of a
// branch, and runs of loads and stores stay in one basic block.  The base
// must be uniform over the wave.
constexpr unsigned kOutOfRange = 0x80000000u;
using Rsrc = __amdgpu_buffer_rsrc_t;
typedef int lr_v2i __attribute__((ext_vector_type(2)));
__device__ __forceinline__ Rsrc make_rsrc(const void* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
// Field loads carry the non-temporal hint (cache policy bit 1) by default:
// every field is read once per pass, and the hint keeps those lines from
// displacing the field the previous pass just wrote, which the large
// last-level cache can still hold when this pass reads it.  Tables shared by
// the batch load without it (bload_keep).  field_load_policy drops the hint
// at 400-512 points, whose fields of a few hundred samples (0.6-1 GB) are
// several times the 256 MB last-level cache: there the hinted row and column
// passes measured slower (5-layer training step, batch 500: 400 points 5.20
// against 4.90 ms, 500 points 11.61 against 11.43 ms), while at 200 points
// (160 MB) and 1000 points (batch 16, 128 MB) the hint saves 2-3%.
template <int N>
constexpr int field_load_policy() {
  return (N >= 400 && N <= 512) ? 0 : 2;
}
template <int POL = 2>
__device__ __forceinline__ float2 bload(Rsrc r, unsigned off) {
  return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, POL));
}
__device__ __forceinline__ float2 bload_keep(Rsrc r, unsigned off) {
  return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0));
}
__device__ __forceinline__ void bstore(Rsrc r, unsigned off, float2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(lr_v2i, v), r, (int)off, 0, 0);
}
__device__ __forceinline__ void bstore_f(Rsrc r, unsigned off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), r, (int)off, 0, 0);
}
// The same with a wave-uniform scalar offset added to the per-lane one.  A
// per-lane offset at or past kOutOfRange stays out of range with any scalar
// offset used here (at most a few MB), whether or not the hardware's range
// check includes the scalar part.
template <int POL = 2>
__device__ __forceinline__ float2 bload_so(Rsrc r, unsigned off, int soff) {
  return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, soff, POL));
}
__device__ __forceinline__ float2 bload_keep_so(Rsrc r, unsigned off, int soff) {
  return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, soff, 0));
}
__device__ __forceinline__ void bstore_so(Rsrc r, unsigned off, int soff, float2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(lr_v2i, v), r, (int)off, soff, 0);
}
__device__ __forceinline__ void bstore_f_so(Rsrc r, unsigned off, int soff, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), r, (int)off, soff, 0);
}

// threadIdx.x behind an empty asm statement: values derived from it are not
// hoisted out of the per-sample loop (which would keep dozens of index
// registers alive through the whole kernel); they are recomputed next to
// their use instead.
__device__ __forceinline__ int opaque_tid() {
  int t = (int)threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2).  The 1-D grid is remapped so that the workgroups one XCD runs at the
// same time take consecutive tiles of the same samples: neighbouring column
// tiles share cache lines, which then come from that XCD's L2 once.
struct WorkItem {
  int tile;
  int group;
  bool valid;
};
__device__ __forceinline__ WorkItem work_item(int ntiles, int ngroups) {
  const int total = ntiles * ngroups;
  const int per = (total + 7) / 8;
  const int l = (int)blockIdx.x;
  const int logical = (l & 7) * per + (l >> 3);
  return WorkItem{logical % ntiles, logical / ntiles, logical < total};
}
inline int work_grid(int ntiles, int ngroups) { return 8 * ((ntiles * ngroups + 7) / 8); }

// Persistent passes (workers = lanes * ntiles; rank r keeps tile r % ntiles
// and lane r / ntiles) with the XCD-contiguous index rx of the workgroup taken
// tile-major (tile rx / lanes, lane rx % lanes): the workgroups of one XCD
// hold every lane of a contiguous range of tiles.  An index past the workers
// is returned unchanged.
__device__ __forceinline__ int persistent_rank(int l, int G, int ntiles, int lanes) {
  const int rx = (l & 7) * (G >> 3) + (l >> 3);
  if (lanes < 1 || rx >= ntiles * lanes) return rx;
  return (rx % lanes) * ntiles + rx / lanes;
}

// Offsets inside one sample fit in 32 bits (n <= 1024).
template <int AXIS>
__device__ __forceinline__ int nat_index(int n, int vec, int q) {
  return AXIS == kRow ? vec * n + q : q * n + vec;
}

// Shared-memory index of natural position p of vector v.
template <class C>
__device__ __forceinline__ int lds_index(int p, int v) {
  return C::Plan::slot_of_pos(p) * C::TP + v;
}

__device__ __forceinline__ bool in_region(int y, int x, int y0, int x0, int s) {
  return (unsigned)(y - y0) < (unsigned)s && (unsigned)(x - x0) < (unsigned)s;
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

// ---------------------------------------------------------------------------
// Batched tile walks.  A tile has nvalid vectors of n elements (positions
// q < n; shared-memory position q + off).  The callbacks receive
// (i, v, q, li, ok): i the compile-time buffer index inside the current
// chunk, v the tile vector, q the position, li its shared-memory index and
// ok whether (v, q) is an element of the tile.
//
//   row tiles (whole rows per wave):  wave w moves rows v = w, w + NW, ... and
//     its lanes cover positions q = lane + 64*m, so every global access of a
//     wave is one contiguous run of a row and the shared-memory index of each
//     (lane, m) is a per-lane constant plus v.  Every (row, run) slot is
//     visited, without branches: for slots outside the tile ok is false, li
//     is the spare shared-memory row (position q >= n) or an unused vector of
//     the tile (v >= nvalid), and global accesses take kOutOfRange.  When the
//     T rows do not split evenly over the NW waves, the last round is partial
//     and the waves past row T - 1 skip it;
//   column tiles: only elements of the tile are visited (ok is true); column
//     thread tid handles elements e = tid + i*P, i < N1, with
//     (v, q) = (e mod T, e div T): every access of a wave covers T
//     consecutive columns of a few rows.
//
// With ST (a field stored in slot order, n = N, off = 0) position q of a
// vector is its slot: li = q*(T+1) + v, no Good-Thomas index map.
//
// The walk runs in chunks of at most W elements per thread: first() is
// called for the whole chunk (issue loads), then second() (consume them).
// Loads use one chunk (every load of the thread in flight before the first
// wait); stores, which do not wait, use small chunks.
// WalkShape<C, AXIS, W>::BUF is the buffer length a chunk needs.
// ---------------------------------------------------------------------------
template <class C>
struct RowLanes {
  static constexpr int NW = C::P / 64;                 // waves per workgroup
  static constexpr bool EVEN = C::T % NW == 0;         // rows split evenly over the waves
  static constexpr int RPW = (C::T + NW - 1) / NW;     // rows per wave (the last round may be partial)
  static constexpr int NCH = (C::N + 63) / 64;         // 64-position runs per row
};

constexpr int kAll = 1 << 20;

template <class C, int AXIS, int W>
struct WalkShape {
  static constexpr bool ROWS = AXIS == kRow;
  static constexpr int NCH = RowLanes<C>::NCH;
  static constexpr int RPW = RowLanes<C>::RPW;
  // rows: chunks of whole rows; columns: chunks of W elements
  static constexpr int RCH = ROWS ? (W / NCH < 1 ? 1 : (W / NCH > RPW ? RPW : W / NCH)) : 1;
  static constexpr int CH = ROWS ? RCH * NCH : (W < C::N1 ? W : C::N1);
  static constexpr int NCHUNK = ROWS ? (RPW + RCH - 1) / RCH : (C::N1 + CH - 1) / CH;
  static constexpr int BUF = CH;
};

template <class C, int AXIS, int W, bool ST, class F1, class F2>
__device__ __forceinline__ void tile_walk2(int n, int off, int nvalid, F1&& first, F2&& second) {
  using WS = WalkShape<C, AXIS, W>;
  if constexpr (WS::ROWS) {
    using RL = RowLanes<C>;
    const int tid = opaque_tid();
    const int lane = tid & 63;
    const int wv = tid >> 6;
    int lofs[RL::NCH];  // shared-memory index of position lane + 64*m in tile vector 0
    bool qok[RL::NCH];
    static_for<0, RL::NCH>([&](auto m) {
      const int q = lane + 64 * decltype(m)::value;
      qok[m.value] = q < n;
      lofs[m.value] = q < n ? (ST ? q * C::TP : lds_index<C>(q + off, 0)) : C::SPARE;
    });
    static_for<0, WS::NCHUNK>([&](auto c) {
      auto visit = [&](auto& f) {
        static_for<0, WS::RCH>([&](auto rr) {
          constexpr int r = decltype(c)::value * WS::RCH + decltype(rr)::value;
          if constexpr (r < RL::RPW) {
            const int v = wv + RL::NW * r;
            // rows that do not split evenly: in the last round the waves
            // past the tile's last row skip it (a wave-uniform branch)
            if (RL::EVEN || r + 1 < RL::RPW || v < C::T) {
              const bool vok = v < nvalid;
              static_for<0, RL::NCH>([&](auto m) {
                const int q = lane + 64 * decltype(m)::value;
                f(std::integral_constant<int, decltype(rr)::value * RL::NCH + decltype(m)::value>{}, v, q,
                  lofs[m.value] + v, vok && qok[m.value]);
              });
            }
          }
        });
      };
      visit(first);
      visit(second);
    });
  } else {
    static_for<0, WS::NCHUNK>([&](auto c) {
      auto visit = [&](auto& f) {
        const int tid = opaque_tid();
        static_for<0, WS::CH>([&](auto i) {
          constexpr int ii = decltype(c)::value * WS::CH + decltype(i)::value;
          if constexpr (ii < C::N1) {
            const int e = tid + ii * C::P;
            const int q = e / C::T;
            const int v = e - q * C::T;
            if (q < n && v < nvalid) f(i, v, q, ST ? q * C::TP + v : lds_index<C>(q + off, v), true);
          }
        });
      };
      visit(first);
      visit(second);
    });
  }
}

constexpr int kStoreChunk = 8;

// Byte offset of element (vector vf(v), position q) of an n x n field, or
// kOutOfRange outside the tile.
template <int AXIS, int BYTES>
__device__ __forceinline__ unsigned elem_off(bool ok, int n, int vec, int q) {
  return ok ? (unsigned)nat_index<AXIS>(n, vec, q) * (unsigned)BYTES : kOutOfRange;
}

// Load a tile of complex (or real) natural-layout rows/columns of an n x n
// field (src, wave-uniform) into shared memory.  Tile vector v is field
// row/column vf(v).
// (ST: src is stored in slot order; the real amplitudes are always natural)
template <class C, int AXIS, bool ST, class VF>
__device__ __forceinline__ void load_tile(float2* lds, const void* src, bool real, int n, int off, VF&& vf,
                                          int nvalid) {
  if constexpr (!ST) zero_padding<C>(lds, n, off);
  constexpr int BUF = WalkShape<C, AXIS, kAll>::BUF;
  if (real) {
    // (real input: loads masked per lane; 4-byte buffer loads over the whole
    // row runs measured slower here)
    const float* __restrict__ in = static_cast<const float*>(src);
    float buf[BUF];
    tile_walk2<C, AXIS, kAll, false>(n, off, nvalid,
        [&](auto i, int v, int q, int, bool ok) { buf[i.value] = ok ? ld(in, nat_index<AXIS>(n, vf(v), q)) : 0.f; },
        [&](auto i, int, int, int li, bool) { lds[li] = c2(buf[i.value], 0.f); });
  } else {
    const Rsrc r = make_rsrc(src, (unsigned)(n * n) * 8u);
    float2 buf[BUF];
    tile_walk2<C, AXIS, kAll, ST>(n, off, nvalid,
        [&](auto i, int v, int q, int, bool ok) { buf[i.value] = bload<field_load_policy<C::N>()>(r, elem_off<AXIS, 8>(ok, n, vf(v), q)); },
        [&](auto i, int, int, int li, bool) { lds[li] = buf[i.value]; });
  }
}

// Two-phase tile load for prefetching: issue the global loads of a tile into
// registers, later write them into shared memory (with the padding zeroed).
template <class C, int AXIS>
using TileBuf = float2[WalkShape<C, AXIS, kAll>::BUF];

template <class C, int AXIS, class VF>
__device__ __forceinline__ void tile_issue(TileBuf<C, AXIS>& buf, const void* src, bool real, int n, VF&& vf,
                                           int nvalid) {
  if (real) {
    const float* __restrict__ in = static_cast<const float*>(src);
    tile_walk2<C, AXIS, kAll, false>(n, 0, nvalid,
        [&](auto i, int v, int q, int, bool ok) { buf[i.value].x = ok ? ld(in, nat_index<AXIS>(n, vf(v), q)) : 0.f; },
        [](auto, int, int, int, bool) {});
  } else {
    const Rsrc r = make_rsrc(src, (unsigned)(n * n) * 8u);
    tile_walk2<C, AXIS, kAll, false>(n, 0, nvalid,
        [&](auto i, int v, int q, int, bool ok) { buf[i.value] = bload<field_load_policy<C::N>()>(r, elem_off<AXIS, 8>(ok, n, vf(v), q)); },
        [](auto, int, int, int, bool) {});
  }
}
template <class C, int AXIS, bool ST>
__device__ __forceinline__ void tile_commit(float2* lds, const TileBuf<C, AXIS>& buf, bool real, int n, int off,
                                            int nvalid) {
  if constexpr (!ST) zero_padding<C>(lds, n, off);
  if (real) {
    tile_walk2<C, AXIS, kAll, ST>(n, off, nvalid, [](auto, int, int, int, bool) {},
        [&](auto i, int, int, int li, bool) { lds[li] = c2(buf[i.value].x, 0.f); });
  } else {
    tile_walk2<C, AXIS, kAll, ST>(n, off, nvalid, [](auto, int, int, int, bool) {},
        [&](auto i, int, int, int li, bool) { lds[li] = buf[i.value]; });
  }
}

// Tile vector v is field vector vec0 + v.
struct Consecutive {
  int vec0;
  __device__ __forceinline__ int operator()(int v) const { return vec0 + v; }
};
// Tile vector v is field vector map[v] (shared memory, T entries).
struct Mapped {
  const int* map;
  __device__ __forceinline__ int operator()(int v) const { return map[v]; }
};

// Adjoint seed at the detector plane: G_D = 2 * (dL/dI) * U_D, with dL/dI a
// full map or constant over each detector region (from dL/dS).
template <class C, int AXIS>
__device__ __forceinline__ void load_seed(float2* lds, const PassArgs& a, int b, int vec0, int nvalid) {
  const int n = a.n;
  const int off = a.off;
  const size_t nn = (size_t)n * n;
  zero_padding<C>(lds, n, off);
  const float2* __restrict__ ud = a.ud_in + (size_t)b * nn;
  const float* __restrict__ gint = a.grad_int ? a.grad_int + (size_t)b * nn : nullptr;
  const float* __restrict__ gsum = a.grad_sums ? a.grad_sums + (size_t)b * a.K : nullptr;
  constexpr int BUF = WalkShape<C, AXIS, kAll>::BUF;
  float2 buf[BUF];
  float g[BUF];
  tile_walk2<C, AXIS, kAll, false>(n, off, nvalid,
      [&](auto i, int v, int q, int, bool ok) {
        float gv = 0.f;
        float2 u = c2(0.f, 0.f);
        if (ok) {
          const int y = AXIS == kRow ? vec0 + v : q;
          const int x = AXIS == kRow ? q : vec0 + v;
          if (gint) {
            gv = ld(gint, y * n + x);
          } else {
            // dL/dI is dL/dS_k on region k: sum over the regions covering (y, x)
            unsigned long long mask = ld(a.row_mask, y) & ld(a.col_mask, x);
            while (mask) {
              gv += gsum[__builtin_ctzll(mask)];
              mask &= mask - 1;
            }
          }
          if (gv != 0.f) u = ld(ud, y * n + x);
        }
        g[i.value] = gv;
        buf[i.value] = u;
      },
      [&](auto i, int, int, int li, bool) { lds[li] = cscale(buf[i.value], 2.f * g[i.value]); });
}

// Store a tile from shared memory into natural-layout rows/columns of an
// n x n field (out, wave-uniform).
template <class C, int AXIS, bool ST, class VF>
__device__ __forceinline__ void store_tile(const float2* lds, float2* __restrict__ out, int n, int off, VF&& vf,
                                           int nvalid) {
  const Rsrc r = make_rsrc(out, (unsigned)(n * n) * 8u);
  float2 buf[WalkShape<C, AXIS, kStoreChunk>::BUF];
  tile_walk2<C, AXIS, kStoreChunk, ST>(n, off, nvalid,
      [&](auto i, int, int, int li, bool) { buf[i.value] = lds[li]; },
      [&](auto i, int v, int q, int, bool ok) { bstore(r, elem_off<AXIS, 8>(ok, n, vf(v), q), buf[i.value]); });
}

// Zero vectors vf(0..nvalid) of a natural-layout n x n field.
template <class C, int AXIS, class VF>
__device__ __forceinline__ void zero_vectors(float2* __restrict__ out, int n, VF&& vf, int nvalid) {
  const Rsrc r = make_rsrc(out, (unsigned)(n * n) * 8u);
  tile_walk2<C, AXIS, kStoreChunk, false>(n, 0, nvalid, [&](auto, int, int, int, bool) {},
      [&](auto, int v, int q, int, bool ok) { bstore(r, elem_off<AXIS, 8>(ok, n, vf(v), q), c2(0.f, 0.f)); });
}

// Detector-plane outputs from a tile that holds U_D in natural order:
// |U|^2, U_D copies, and per-(sample, tile, region) partial sums.  The
// partial sums are formed in a fixed order: thread pairs (region k, tile
// vector v) sum their vector's run of |U|^2 inside the region into rsum
// ([K][T] floats of shared memory), then one thread per region adds the T
// runs.
template <class C, int AXIS, class VF>
__device__ __forceinline__ void tile_outputs(const float2* lds, float* rsum, const PassArgs& a, int b, VF&& vf,
                                             int nvalid, int tile) {
  using PL = typename C::Plan;
  const int n = a.n;
  const int off = a.off;
  const size_t nn = (size_t)n * n;
  float2* fo = a.field_out ? a.field_out + (size_t)b * nn : nullptr;
  float2* sv = a.saved_ud ? a.saved_ud + (size_t)b * nn : nullptr;
  float* io = a.intensity ? a.intensity + (size_t)b * nn : nullptr;
  if (fo || sv || io) {
    float2 buf[WalkShape<C, AXIS, kStoreChunk>::BUF];
    tile_walk2<C, AXIS, kStoreChunk, false>(n, off, nvalid,
        [&](auto i, int, int, int li, bool) { buf[i.value] = lds[li]; },
        [&](auto i, int v, int q, int, bool ok) {
          if (ok) {
            const int idx = nat_index<AXIS>(n, vf(v), q);
            if (fo) st(fo, idx, buf[i.value]);
            if (sv) st(sv, idx, buf[i.value]);
            if (io) st(io, idx, a.accumulate ? ld(io, idx) + cabs2(buf[i.value]) : cabs2(buf[i.value]));
          }
        });
  }
  if (a.sums_part) {
    const int K = a.K;
    const int s = a.det_size;
    for (int idx = threadIdx.x; idx < K * C::T; idx += C::P) {
      const int k = idx / C::T;
      const int v = idx - k * C::T;
      float run = 0.f;
      if (v < nvalid) {
        const int2 r = a.regions[k];                // (y0, x0)
        const int vlo = AXIS == kRow ? r.x : r.y;   // region start along the vector index
        const int qlo = AXIS == kRow ? r.y : r.x;   // region start along positions
        if ((unsigned)(vf(v) - vlo) < (unsigned)s) {
          auto w = PL::walk(qlo + off);
          for (int d = 0; d < s; ++d) {
            run += cabs2(lds[PL::walk_slot(w) * C::TP + v]);
            PL::walk_next(w);
          }
        }
      }
      rsum[idx] = run;
    }
    __syncthreads();
    for (int k = threadIdx.x; k < K; k += C::P) {
      float part = 0.f;
      for (int v = 0; v < C::T; ++v) part += rsum[k * C::T + v];
      a.sums_part[((size_t)b * a.ntiles + tile) * K + k] = part;
    }
  }
}

// ---------------------------------------------------------------------------
// Column tiles read and write their A-items straight from/to global memory:
// element x of A-item j is row pos(x, j) - off of column vec (pitch floats2).
// ---------------------------------------------------------------------------
// Walk the N1 elements of this thread's A-item along the pass axis:
// f(k, idx, valid) with idx = (pos(k, j) - off) * pitch + vec, computed
// incrementally (no multiplications per element).
template <class C, class F>
__device__ __forceinline__ void for_a_elems(int off, int n, int pitch, int vec, bool vok, F&& f) {
  using PL = typename C::Plan;
  const int j = opaque_tid() / C::T;
  int p = PL::pos_base(j);
  int idx = (p - off) * pitch + vec;
  static_for<0, C::N1>([&](auto k) {
    f(k, idx, vok && (unsigned)(p - off) < (unsigned)n);
    p += C::N2;
    idx += C::N2 * pitch;
    if constexpr (PL::PFA) {
      if (p >= C::N) {
        p -= C::N;
        idx -= C::N * pitch;
      }
    }
  });
}

// Add the skip field of sample b (natural layout) to this thread's A-item of
// detector-plane values along vector vec (a row for row passes, a column for
// column passes); positions outside the aperture are left as they are.
template <class C, int AXIS>
__device__ __forceinline__ void add_skip(const PassArgs& a, int b, int vec, bool vok, float2 (&x)[C::N1]) {
  if (!a.skip) return;
  const int n = a.n;
  const float2* __restrict__ sk = a.skip + (size_t)b * n * n;
  for_a_elems<C>(a.off, n, 1, 0, vok, [&](auto k, int q, bool in) {
    if (in) {
      const float2 s = ld(sk, AXIS == kRow ? vec * n + q : q * n + vec);
      x[k.value] = c2(x[k.value].x + s.x, x[k.value].y + s.y);
    }
  });
}

// Stored-order A-item access (ST: an N x N array whose axis positions are
// slots): element k of this thread's A-item j lies at stored index
// j + N2*k along the pass axis, a constant stride of N2*N elements, so every
// element is one per-lane base plus a compile-time scalar offset and costs
// no vector instructions.  Lanes outside the tile (vok false) take the
// out-of-range base.
template <class C, int ES>
__device__ __forceinline__ unsigned a_base_st(int vec, bool vok) {
  const int j = opaque_tid() / C::T;
  return vok ? (unsigned)(j * C::N + vec) * (unsigned)ES : kOutOfRange;
}
template <class C, int ES, int K>
constexpr int a_soff_st() { return K * C::N2 * C::N * ES; }

// (in / out: n rows of pitch elements, wave-uniform; with ST, n = pitch = N)
template <class C, bool ST = false>
__device__ __forceinline__ void load_a_direct(const float2* __restrict__ in, int pitch, int n, int off, int vec,
                                              bool vok, float2 (&x)[C::N1]) {
  const Rsrc r = make_rsrc(in, (unsigned)(n * pitch) * 8u);
  if constexpr (ST) {
    const unsigned base = a_base_st<C, 8>(vec, vok);
    static_for<0, C::N1>([&](auto k) { x[k.value] = bload_so<field_load_policy<C::N>()>(r, base, a_soff_st<C, 8, k.value>()); });
  } else {
    for_a_elems<C>(off, n, pitch, vec, vok, [&](auto k, int idx, bool valid) {
      x[k.value] = bload<field_load_policy<C::N>()>(r, valid ? (unsigned)idx * 8u : kOutOfRange);
    });
  }
}
template <class C, bool ST = false>
__device__ __forceinline__ void store_a_direct(float2* __restrict__ out, int pitch, int n, int off, int vec,
                                               bool vok, const float2 (&x)[C::N1]) {
  const Rsrc r = make_rsrc(out, (unsigned)(n * pitch) * 8u);
  if constexpr (ST) {
    const unsigned base = a_base_st<C, 8>(vec, vok);
    static_for<0, C::N1>([&](auto k) { bstore_so(r, base, a_soff_st<C, 8, k.value>(), x[k.value]); });
  } else {
    for_a_elems<C>(off, n, pitch, vec, vok, [&](auto k, int idx, bool valid) {
      bstore(r, valid ? (unsigned)idx * 8u : kOutOfRange, x[k.value]);
    });
  }
}
// As load_a_direct, reading only the elements k with bit k of mask set (the
// others are zero).
template <class C, bool ST = false>
__device__ __forceinline__ void load_a_direct_masked(const float2* __restrict__ in, int pitch, int n, int off,
                                                     int vec, bool vok, unsigned mask, float2 (&x)[C::N1]) {
  const Rsrc r = make_rsrc(in, (unsigned)(n * pitch) * 8u);
  if constexpr (ST) {
    const unsigned base = a_base_st<C, 8>(vec, vok);
    static_for<0, C::N1>([&](auto k) {
      x[k.value] = bload_so<field_load_policy<C::N>()>(r, ((mask >> k.value) & 1u) ? base : kOutOfRange,
                                                      a_soff_st<C, 8, k.value>());
    });
  } else {
    for_a_elems<C>(off, n, pitch, vec, vok, [&](auto k, int idx, bool valid) {
      x[k.value] = bload<field_load_policy<C::N>()>(r, valid && ((mask >> k.value) & 1u) ? (unsigned)idx * 8u : kOutOfRange);
    });
  }
}
// Per-layer [q][vec] table of n x n entries at this thread's A-item.
template <class C, bool ST = false>
__device__ __forceinline__ void load_a_table(const float2* __restrict__ tab, int n, int off, int vec, bool vok,
                                             float2 (&m)[C::N1]) {
  const Rsrc r = make_rsrc(tab, (unsigned)(n * n) * 8u);
  if constexpr (ST) {
    const unsigned base = a_base_st<C, 8>(vec, vok);
    static_for<0, C::N1>([&](auto k) { m[k.value] = bload_keep_so(r, base, a_soff_st<C, 8, k.value>()); });
  } else {
    for_a_elems<C>(off, n, n, vec, vok, [&](auto k, int idx, bool valid) {
      m[k.value] = bload_keep(r, valid ? (unsigned)idx * 8u : kOutOfRange);
    });
  }
}

// ---------------------------------------------------------------------------
// Separable (Fresnel) passes through the layers.
//
// What the forward pass keeps for the backward one is the field each of its
// passes writes: W_0 after the first half hop, and W_l after the pass of
// layer l (end of hop l, modulation, first-axis half of hop l+1).  The
// adjoint pass of layer l runs along the same axis as the forward pass that
// made W_l from W_{l-1}, so it recomputes the arriving field
// A_l = (half hop)(W_{l-1}) with one more 1-D propagation instead of reading
// a stored activation.  A forward layer pass therefore moves 16 bytes per
// pixel (one field read, one written) instead of 24, at the price of a third
// propagation in the adjoint pass.  The recomputation repeats the forward
// arithmetic, so it is exact with and without aperture padding.
//
// Schedule (PassArgs::workers / lanes): workgroup rank r takes the (tile,
// sample) items r, r + workers, ...  Forward kinds get one item per
// workgroup; accumulating kinds run persistently with workers = lanes *
// ntiles, so a workgroup keeps one tile and strides through the batch.  The
// ranks are XCD-contiguous: the workgroups of one XCD work on neighbouring
// items at the same time.
//
// FULL (the layer fills the FFT grid, n = N): the fields the passes hand to
// each other, the modulation tables and the dphi partials are stored in slot
// order along both axes (plan.hpp), so A-items are read and written at a
// constant stride with no index arithmetic; only the input amplitudes of the
// first pass are natural.  Otherwise everything is in natural order.
// ---------------------------------------------------------------------------
template <class C, int KIND, int AXIS, bool FULL>
__global__ void __launch_bounds__(C::P, C::WAVES_ACC)
    fresnel_pass(PassArgs a) {
  static_assert(KIND == kPropOnce || KIND == kFwdMid || KIND == kBwdMid || KIND == kBwdLast,
                "detector-plane kinds run in detector_pass");
  __shared__ float2 lds[C::LDS_ELEMS];
  constexpr int N1 = C::N1;
  constexpr bool ACC = (KIND == kBwdMid || KIND == kBwdLast);
  constexpr bool DIRECT = AXIS == kCol;  // column tiles address their A-items in global memory
  const Tile<C> t{lds, (int)(threadIdx.x % C::T), (int)(threadIdx.x / C::T)};
  const int j = t.s;

  const int G = (int)gridDim.x;
  const int l = (int)blockIdx.x;
  // XCD-contiguous ranks let neighbouring column tiles share cache lines in
  // one XCD's L2; row tiles read whole rows and stream faster in dispatch
  // order (a memory-only probe of the row pattern: 6.4 against 5.8 TB/s)
  // The 1000-point adjoint row passes take the tile-major persistent order
  // (one XCD keeps whole tiles: 245 -> 231 us, workload 5 1.505 -> 1.493 ms;
  // at 200-500 points it measured neutral or slower)
  constexpr bool TILE_MAJOR = ACC && AXIS == kRow && C::N == 1000;
  const int rank = TILE_MAJOR       ? persistent_rank(l, G, a.ntiles, a.lanes)
                   : AXIS == kCol ? (l & 7) * (G >> 3) + (l >> 3)
                                  : l;
  if (rank >= a.workers) return;
  const int n = a.n;
  const int off = a.off;
  const size_t nn = (size_t)n * n;
  const int total = a.ntiles * a.batch;
  const bool conj_tab = a.conj_tab != 0;
  const bool real = a.in_real != 0;

  // dphi accumulators, one per A-item element: registers, or (column kinds)
  // this thread's private shared-memory slots, which leaves the registers to
  // the two A-items, the modulation and the prefetch buffer that are live at
  // once in the adjoint passes
  constexpr bool ACC_LDS = ACC && DIRECT;
  __shared__ float acc_lds[ACC_LDS ? N1 * C::P : 1];
  float acc[ACC && !ACC_LDS ? N1 : 1];
  auto acc_add = [&](auto k, float v) {
    if constexpr (ACC_LDS) {
      acc_lds[k.value * C::P + threadIdx.x] += v;
    } else {
      acc[k.value] += v;
    }
  };
  auto acc_get = [&](auto k) {
    if constexpr (ACC_LDS) {
      return acc_lds[k.value * C::P + threadIdx.x];
    } else {
      return acc[k.value];
    }
  };
  if constexpr (ACC) {
    static_for<0, N1>([&](auto k) {
      if constexpr (ACC_LDS) {
        acc_lds[k.value * C::P + threadIdx.x] = 0.f;
      } else {
        acc[k.value] = 0.f;
      }
    });
  }
  stage_table_by_freq<C>(lds, a.tab);  // visible after the first barrier below

  // One 1-D propagation of the A-items in v, in place: A-step, B-step with
  // the staged table (conjugated when cj), inverse A-step.  mid() runs
  // between the shared-memory writes and the B-step (loads issued there
  // arrive during it).
  auto prop = [&](float2(&v)[N1], bool cj, auto&& mid) {
    Dft<N1, -1>::run(v);
    write_a(t, j, v);
    mid();
    __syncthreads();
    b_spectral<C, ACC>(t, cj);
    __syncthreads();
    read_a(t, j, v);
    Dft<N1, 1>::run(v);
  };
  auto nothing = [] {};

  // Adjoint column kinds load one input of their next item into pf as soon
  // as registers are free for it, so it arrives while the current item is
  // still being transformed: kBwdMid loads W_{l-1} during its last
  // propagation (after the dphi update), kBwdLast, which has no third
  // propagation, transforms G first and loads the next G while W_0
  // propagates.  After the last item the loads are still issued (which
  // keeps the live ranges simple), at out-of-range offsets: they move no
  // data.  (The forward kinds, one item per workgroup, rely on the other
  // resident workgroups instead: prefetching within chunks of items measured
  // slower for them.)
  // elements of this thread's A-item at which G can be nonzero (column passes)
  unsigned gmask = ~0u;
  if constexpr (ACC && DIRECT) {
    if (a.live) {
      gmask = 0u;
      for_a_elems<C>(off, n, 1, 0, true, [&](auto k, int q, bool in) {
        if (in && ld(a.live, q) != 0ull) gmask |= 1u << k.value;
      });
    }
  }
  // From N = 500 on (B-items of 16-40 values next to A-items of 25-32) the
  // prefetch buffer and a modulation loaded during the B-step no longer fit
  // next to the propagating item in 256 registers (they spilled 12-122
  // registers), so these sizes load each input when it is needed and rely
  // on the other resident waves (the forward layer pass likewise loads its
  // modulation after the B-step).
  constexpr bool BIG = C::N >= 500;
  constexpr bool PREFETCH = ACC && (DIRECT || KIND == kBwdMid) && !BIG;
  constexpr bool G_FIRST = DIRECT && KIND == kBwdLast;
  float2 pf[PREFETCH && DIRECT ? N1 : 1];
  TileBuf<C, AXIS> pft;  // row tiles
  auto issue_next = [&](int item, bool live) {
    if constexpr (PREFETCH) {
      const int v0 = (item % a.ntiles) * C::T;
      const int nv = live ? min(C::T, a.nvec - v0) : 0;
      const float2* src = G_FIRST ? static_cast<const float2*>(a.in) : a.act_in;
      if constexpr (DIRECT) {
        load_a_direct_masked<C, FULL>(src + (size_t)(item / a.ntiles) * nn, n, n, off, v0 + t.v, t.v < nv,
                                      G_FIRST ? gmask : ~0u, pf);
      } else {
        tile_issue<C, AXIS>(pft, src + (size_t)(item / a.ntiles) * nn, false, n, Consecutive{v0}, nv);
      }
    }
  };
  if (rank < total) issue_next(rank, true);

  for (int it = rank; it < total; it += a.workers) {
    const int tile = it % a.ntiles;
    const int b = it / a.ntiles;
    const int vec0 = tile * C::T;
    const int vec = vec0 + t.v;
    const int nvalid = min(C::T, a.nvec - vec0);
    const bool vok = t.v < nvalid;
    const float2* __restrict__ fin = static_cast<const float2*>(a.in) + (size_t)b * nn;
    auto prefetch = [&] {
      if constexpr (PREFETCH) {
        __builtin_amdgcn_sched_barrier(0);  // not hoisted above the last use of the registers it reuses
        const bool more = it + a.workers < total;
        issue_next(more ? it + a.workers : it, more);
      }
    };

    float2 x[N1];
    if constexpr (G_FIRST) {
      // G_1 = adjoint of the first-axis half of hop 2, while W_0 is in flight
      float2 ar[N1];
      if constexpr (PREFETCH) {
        static_for<0, N1>([&](auto k) { x[k.value] = pf[k.value]; });
      } else {
        load_a_direct_masked<C, FULL>(fin, n, n, off, vec, vok, gmask, x);
      }
      load_a_direct<C, FULL>(a.act_in + (size_t)b * nn, n, n, off, vec, vok, ar);
      float2 m[N1];
      if constexpr (BIG) {
        prop(x, true, nothing);
        load_a_table<C, FULL>(a.mod, n, off, vec, vok, m);
      } else {
        prop(x, true, [&] { load_a_table<C, FULL>(a.mod, n, off, vec, vok, m); });
      }
      static_for<0, N1>([&](auto k) { x[k.value] = cmulc(x[k.value], m[k.value]); });
      // A_1, then dphi_1 += Im(conj(A_1) conj(M_1) G_1)
      prop(ar, false, prefetch);
      static_for<0, N1>([&](auto k) { acc_add(k, ar[k.value].x * x[k.value].y - ar[k.value].y * x[k.value].x); });
    } else if constexpr (ACC) {
      // A_l from the saved input of the forward pass, while G (the gradient
      // with respect to W_l) is in flight
      float2 ar[N1];
      if constexpr (DIRECT) {
        if constexpr (PREFETCH) {
          static_for<0, N1>([&](auto k) { ar[k.value] = pf[k.value]; });
        } else {
          load_a_direct<C, FULL>(a.act_in + (size_t)b * nn, n, n, off, vec, vok, ar);
        }
        load_a_direct_masked<C, FULL>(fin, n, n, off, vec, vok, gmask, x);
        prop(ar, false, nothing);
      } else {
        __syncthreads();  // shared memory reuse across items
        if constexpr (PREFETCH) {
          tile_commit<C, AXIS, FULL>(lds, pft, false, n, off, nvalid);
        } else {
          load_tile<C, AXIS, FULL>(lds, a.act_in + (size_t)b * nn, false, n, off, Consecutive{vec0}, nvalid);
        }
        __syncthreads();
        read_a(t, j, ar);
        prop(ar, false, nothing);
        __syncthreads();
        load_tile<C, AXIS, FULL>(lds, fin, false, n, off, Consecutive{vec0}, nvalid);
        __syncthreads();
        read_a(t, j, x);
      }
      // G_l = adjoint of the first-axis half of hop l+1; the modulation is
      // loaded during its B-step (after it from N = 500 on)
      float2 m[N1];
      if constexpr (BIG) {
        prop(x, true, nothing);
        load_a_table<C, FULL>(a.mod, n, off, vec, vok, m);
      } else {
        prop(x, true, [&] { load_a_table<C, FULL>(a.mod, n, off, vec, vok, m); });
      }
      // conj(M_l) G_l (zero outside the aperture) and dphi_l += Im(conj(U_l) G_l) = Im(conj(A_l) conj(M_l) G_l)
      static_for<0, N1>([&](auto k) {
        const float2 h = cmulc(x[k.value], m[k.value]);
        acc_add(k, ar[k.value].x * h.y - ar[k.value].y * h.x);
        x[k.value] = h;
      });
      if constexpr (KIND == kBwdMid && DIRECT) {
        prop(x, true, prefetch);
      } else if constexpr (KIND == kBwdMid) {
        prop(x, true, nothing);
      } else {
        prefetch();
      }
    } else {
      if constexpr (DIRECT) {
        load_a_direct<C, FULL>(fin, n, n, off, vec, vok, x);
      } else {
        __syncthreads();  // shared memory reuse across items
        const void* src = static_cast<const char*>(a.in) + (size_t)b * nn * (real ? 4 : 8);
        if (FULL && real) {
          // natural amplitudes: stored row vec0 + v is natural row pos_of_slot(vec0 + v)
          load_tile<C, AXIS, false>(lds, src, true, n, off,
                                    [&](int v) { return C::Plan::pos_of_slot(vec0 + v); }, nvalid);
        } else {
          load_tile<C, AXIS, FULL>(lds, src, real, n, off, Consecutive{vec0}, nvalid);
        }
        __syncthreads();
        read_a(t, j, x);
      }
      if constexpr (KIND == kFwdMid) {
        float2 m[N1];
        if constexpr (BIG) {
          prop(x, conj_tab, nothing);
          load_a_table<C, FULL>(a.mod, n, off, vec, vok, m);
        } else {
          prop(x, conj_tab, [&] { load_a_table<C, FULL>(a.mod, n, off, vec, vok, m); });
        }
        // U_l = M_l A_l, zero outside the aperture (crop)
        static_for<0, N1>([&](auto k) { x[k.value] = cmul(x[k.value], m[k.value]); });
      }
      prop(x, conj_tab, prefetch);
    }

    if constexpr (KIND != kBwdLast) {
      if constexpr (DIRECT) {
        store_a_direct<C, FULL>(a.out + (size_t)b * nn, n, n, off, vec, vok, x);
      } else {
        write_a(t, j, x);
        __syncthreads();
        store_tile<C, AXIS, FULL>(lds, a.out + (size_t)b * nn, n, off, Consecutive{vec0}, nvalid);
        if constexpr (ACC) prefetch();
      }
    }
  }
  if constexpr (ACC) {
    // one partial per lane (the tile is fixed); a lane with no samples contributes zeros
    const int vec0 = (rank % a.ntiles) * C::T;
    const int vec = vec0 + t.v;
    const bool vok = t.v < min(C::T, a.nvec - vec0);
    const Rsrc dp = make_rsrc(a.dphi_part + (size_t)(rank / a.ntiles) * nn, (unsigned)nn * 4u);
    if constexpr (FULL) {
      const unsigned base = a_base_st<C, 4>(vec, vok);
      static_for<0, N1>([&](auto k) { bstore_f_so(dp, base, a_soff_st<C, 4, k.value>(), acc_get(k)); });
    } else {
      for_a_elems<C>(off, n, n, vec, vok, [&](auto k, int idx, bool in) {
        bstore_f(dp, in ? (unsigned)idx * 4u : kOutOfRange, acc_get(k));
      });
    }
  }
}

// ---------------------------------------------------------------------------
// Detector-plane passes of the separable path.  Their input W is the field
// after the first-axis half of the last hop (it is also what the forward pass
// keeps for the backward one).
//   kFwdLast:  W -> rest of the hop -> U_D -> |U_D|^2, U_D, region partial sums
//   kBwdFirst: W -> rest of the hop -> U_D -> G_D = 2 (dL/dI) U_D -> adjoint of
//              that half hop -> G
// A region loss depends on U_D only on the rows (row pass) or columns (column
// pass) the detector regions cover, and G_D vanishes on the others; with
// a.vperm only those vectors are transformed, and the seed pass writes zero
// vectors for the rest.
// ---------------------------------------------------------------------------
template <class C, int KIND, int AXIS, bool FULL>
__global__ void __launch_bounds__(C::P, C::WAVES) detector_pass(PassArgs a) {
  static_assert(KIND == kFwdLast || KIND == kBwdFirst, "detector-plane kinds only");
  __shared__ float2 lds[C::LDS_ELEMS];
  __shared__ float rsum[KIND == kFwdLast ? C::T * kMaxRegions : 1];
  __shared__ int vmap[C::T];  // natural index of tile vector v
  __shared__ int vst[C::T];   // its index in the stored (input / gradient) layout
  constexpr int N1 = C::N1;
  const Tile<C> t{lds, (int)(threadIdx.x % C::T), (int)(threadIdx.x / C::T)};
  const int j = t.s;

  const WorkItem wi = work_item(a.ntiles, (a.batch + a.spg - 1) / a.spg);
  if (!wi.valid) return;
  const int n = a.n;
  const int off = a.off;
  const size_t nn = (size_t)n * n;
  const int b0 = wi.group * a.spg;
  const int b1 = min(a.batch, b0 + a.spg);

  // tile vectors: a run of the covered-first permutation, or consecutive vectors
  int first;
  int nvalid;
  bool zero_tile = false;
  if (a.vperm) {
    if (wi.tile < a.ntiles_act) {
      first = wi.tile * C::T;
      nvalid = min(C::T, a.nact - first);
    } else {
      zero_tile = true;
      first = a.nact + (wi.tile - a.ntiles_act) * C::T;
      nvalid = min(C::T, n - first);
    }
  } else {
    first = wi.tile * C::T;
    nvalid = min(C::T, n - first);
  }
  // (with FULL, vperm lists stored indices)
  if ((int)threadIdx.x < C::T) {
    const int v = (int)threadIdx.x;
    const int sv = v < nvalid ? (a.vperm ? a.vperm[first + v] : first + v) : 0;
    vst[v] = sv;
    vmap[v] = FULL ? C::Plan::pos_of_slot(sv) : sv;
  }
  const Mapped vf{vmap};
  const Mapped vfs{vst};
  if (KIND == kBwdFirst && zero_tile) {
    __syncthreads();
    for (int b = b0; b < b1; ++b) zero_vectors<C, AXIS>(a.out + (size_t)b * nn, n, vfs, nvalid);
    return;
  }
  stage_table_by_freq<C>(lds, a.tab);
  __syncthreads();
  const bool vok = t.v < nvalid;
  const int vec = vmap[t.v];

  for (int b = b0; b < b1; ++b) {
    float2 x[N1];
    __syncthreads();
    load_tile<C, AXIS, FULL>(lds, static_cast<const float2*>(a.in) + (size_t)b * nn, false, n, off, vfs, nvalid);
    __syncthreads();
    read_a(t, j, x);
    // rest of the last hop: U_D
    Dft<N1, -1>::run(x);
    write_a(t, j, x);
    __syncthreads();
    b_spectral(t, false);
    __syncthreads();
    read_a(t, j, x);
    Dft<N1, 1>::run(x);
    add_skip<C, AXIS>(a, b, vec, vok, x);

    if constexpr (KIND == kFwdLast) {
      write_a(t, j, x);
      __syncthreads();
      tile_outputs<C, AXIS>(lds, rsum, a, b, vf, nvalid, wi.tile);
    } else {
      // seed G_D = 2 (dL/dI) U_D at this thread's positions (zero outside the aperture)
      if (a.grad_int) {
        float2 g[N1];
        __syncthreads();  // every read of U_D from shared memory is done
        load_tile<C, AXIS, false>(lds, a.grad_int + (size_t)b * nn, true, n, off, vf, nvalid);
        __syncthreads();
        read_a(t, j, g);
        static_for<0, N1>([&](auto k) { x[k.value] = cscale(x[k.value], 2.f * g[k.value].x); });
      } else {
        // dL/dI is dL/dS_k on region k: sum over the regions covering the pixel
        const float* __restrict__ gs = a.grad_sums + (size_t)b * a.K;
        const unsigned long long vmask = vok ? ld(AXIS == kRow ? a.row_mask : a.col_mask, vec) : 0ull;
        const unsigned long long* __restrict__ qmask = AXIS == kRow ? a.col_mask : a.row_mask;
        for_a_elems<C>(off, n, 1, 0, vok, [&](auto k, int q, bool in) {
          float gv = 0.f;
          if (in && vmask) {
            unsigned long long mk = vmask & ld(qmask, q);
            while (mk) {
              gv += gs[__builtin_ctzll(mk)];
              mk &= mk - 1;
            }
          }
          x[k.value] = cscale(x[k.value], 2.f * gv);
        });
      }
      // adjoint of the half hop
      Dft<N1, -1>::run(x);
      write_a(t, j, x);
      __syncthreads();
      b_spectral(t, true);
      __syncthreads();
      read_a(t, j, x);
      Dft<N1, 1>::run(x);
      if constexpr (AXIS == kCol) {
        store_a_direct<C, FULL>(a.out + (size_t)b * nn, n, n, off, vst[t.v], vok, x);
      } else {
        write_a(t, j, x);
        __syncthreads();
        store_tile<C, AXIS, FULL>(lds, a.out + (size_t)b * nn, n, off, vfs, nvalid);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Angular-spectrum passes.  Between passes a sample is stored as n rows of
// N x-spectrum values in the plan's slot order ([B][n][N]).
// ---------------------------------------------------------------------------
// (The B-item index goes behind an empty asm statement, as in b_spectral:
// twiddle offsets derived from it are formed at their use, not hoisted out
// of the per-sample loop.)
template <class C>
__device__ __forceinline__ void b_forward_all(const Tile<C>& t) {
  int s = t.s;
  asm volatile("" : "+v"(s));
#pragma unroll 1
  for (int ii = 0; ii < C::IB; ++ii) {
    const int k1 = s + C::S * ii;
    if (!C::B_FULL && k1 >= C::N1) break;
    float2 y[C::N2];
    read_b(t, k1, y);
    b_forward<C>(k1, y);
    write_b(t, k1, y);
  }
}
template <class C>
__device__ __forceinline__ void b_inverse_all(const Tile<C>& t) {
  int s = t.s;
  asm volatile("" : "+v"(s));
#pragma unroll 1
  for (int ii = 0; ii < C::IB; ++ii) {
    const int k1 = s + C::S * ii;
    if (!C::B_FULL && k1 >= C::N1) break;
    float2 y[C::N2];
    read_b(t, k1, y);
    b_inverse<C>(k1, y);
    write_b(t, k1, y);
  }
}

// Spectrum rows (pitch N, slot order) of a row tile <-> shared memory (the
// loads are non-temporal: each row is read once per pass).
template <class C>
__device__ __forceinline__ void load_spec_rows(float2* lds, const float2* __restrict__ in, int vec0, int nvalid) {
  float2 buf[C::N1];
  const int total = nvalid * C::N;
  const int tid = opaque_tid();
  static_for<0, C::N1>([&](auto i) {
    const int e = tid + i.value * C::P;
    if (e < total) buf[i.value] = ld_stream(in, vec0 * C::N + e);
  });
  static_for<0, C::N1>([&](auto i) {
    const int e = tid + i.value * C::P;
    const int v = e / C::N;
    if (e < total) lds[(e - v * C::N) * C::TP + v] = buf[i.value];
  });
}
// With centred, position p of a stored row holds frequency (p + N/2) mod N
// instead of slot p (N even).
template <class C>
__device__ __forceinline__ void store_spec_rows(const float2* lds, float2* __restrict__ out, int vec0, int nvalid,
                                                bool centred) {
  using PL = typename C::Plan;
  float2 buf[C::N1];
  const int total = nvalid * C::N;
  const int tid = opaque_tid();
  static_for<0, C::N1>([&](auto i) {
    const int e = tid + i.value * C::P;
    const int v = e / C::N;
    const int p = e - v * C::N;
    const int slot = centred ? PL::slot_of_freq(p + C::N / 2 < C::N ? p + C::N / 2 : p - C::N / 2) : p;
    if (e < total) buf[i.value] = lds[slot * C::TP + v];
  });
  static_for<0, C::N1>([&](auto i) {
    const int e = tid + i.value * C::P;
    if (e < total) st(out, vec0 * C::N + e, buf[i.value]);
  });
}

template <class C, int KIND>
__global__ void __launch_bounds__(C::P, (KIND == kAsRowBwdMid || KIND == kAsRowBwdLast || KIND == kAsRowMid)
                                            ? C::WAVES_ACC : C::WAVES)
    as_pass(PassArgs a) {
  __shared__ float2 lds[C::LDS_ELEMS];
  // region partial sums of the detector-plane outputs (row kinds that end in positions)
  __shared__ float rsum[(KIND == kAsRowLast || KIND == kAsRowBwdLast || KIND == kAsRowIfft)
                            ? C::T * kMaxRegions : 1];
  using PL = typename C::Plan;
  constexpr int N = C::N;
  constexpr int N1 = C::N1;
  constexpr bool ACC = (KIND == kAsRowBwdMid || KIND == kAsRowBwdLast);
  constexpr bool LAYER = (KIND == kAsRowMid || ACC);
  constexpr bool SPECTRAL_IN = (KIND == kAsRowMid || KIND == kAsRowLast || KIND == kAsRowBwdMid ||
                                KIND == kAsRowBwdLast || KIND == kAsRowIfft);
  constexpr bool FWD_OUT = (KIND == kAsRowFirst || KIND == kAsRowMid || KIND == kAsRowBwdFirst ||
                            KIND == kAsRowBwdMid);
  const Tile<C> t{lds, (int)(threadIdx.x % C::T), (int)(threadIdx.x / C::T)};
  const int j = t.s;

  const WorkItem wi = work_item(a.ntiles, (a.batch + a.spg - 1) / a.spg);
  if (!wi.valid) return;
  const int n = a.n;
  const int off = a.off;
  const size_t nn = (size_t)n * n;
  const int vec0 = wi.tile * C::T;
  const int vec = vec0 + t.v;
  const int nvalid = min(C::T, a.nvec - vec0);
  const bool vok = t.v < nvalid;
  const int b0 = wi.group * a.spg;
  const int b1 = min(a.batch, b0 + a.spg);

  float acc[ACC ? N1 : 1];
  if constexpr (ACC) {
    static_for<0, N1>([&](auto k) { acc[k.value] = 0.f; });
  }

  for (int b = b0; b < b1; ++b) {
    float2 x[N1];
    if constexpr (KIND == kAsCol) {
      // vectors: spectrum columns (slot order); positions: rows of the padded grid
      const float2* __restrict__ in = static_cast<const float2*>(a.in) + (size_t)b * n * N;
      __syncthreads();
      load_a_direct<C>(in, N, n, off, vec, vok, x);
      Dft<N1, -1>::run(x);
      write_a(t, j, x);
      __syncthreads();
      // B-step with the 2-D table: element k2 of item k1 is ky = freq(k1, k2);
      // scheduling barriers keep the twiddle and table loads next to their use.
      // An even table is read at min(ky, N - ky): half the rows, so half the
      // table traffic of a launch (each sample reads the whole table)
      const bool cj = a.conj_tab != 0;
      int s_op = t.s;
      asm volatile("" : "+v"(s_op));
#pragma unroll 1
      for (int ii = 0; ii < C::IB; ++ii) {
        const int k1 = s_op + C::S * ii;
        if (!C::B_FULL && k1 >= C::N1) break;
        float2 y[C::N2];
        read_b(t, k1, y);
        b_forward<C>(k1, y);
        __builtin_amdgcn_sched_barrier(0);
        if (vok) {
          static_for<0, C::N2>([&](auto kc) {
            constexpr int k2 = decltype(kc)::value;
            const int ky = PL::freq(k1, k2);
            const float2 h = ld(a.tab, (a.tab_sym && ky > N / 2 ? N - ky : ky) * N + vec);
            y[k2] = cj ? cmulc(y[k2], h) : cmul(y[k2], h);
          });
        }
        __builtin_amdgcn_sched_barrier(0);
        b_inverse<C>(k1, y);
        __builtin_amdgcn_sched_barrier(0);
        write_b(t, k1, y);
      }
      __syncthreads();
      read_a(t, j, x);
      Dft<N1, 1>::run(x);
      store_a_direct<C>(a.out + (size_t)b * n * N, N, n, off, vec, vok, x);
      continue;
    }
    if constexpr (KIND == kAsColFar) {
      // unnormalised DFT along y of x-spectrum column vec, stored by the row
      // pass in centred order (column vec holds kx = (vec + N/2) mod N);
      // frequency (ky, kx) goes to [(ky + N/2) mod N][vec] times the table
      // (in the same column order, carrying the far-field factors), so a
      // tile writes whole runs of consecutive output columns
      const float2* __restrict__ in = static_cast<const float2*>(a.in) + (size_t)b * n * N;
      __syncthreads();
      load_a_direct<C>(in, N, n, off, vec, vok, x);
      Dft<N1, -1>::run(x);
      write_a(t, j, x);
      __syncthreads();
      b_forward_all<C>(t);
      __syncthreads();
      if (vok) {
        const int ocol = vec;
        float2* __restrict__ out = a.out + (size_t)b * N * N;
#pragma unroll 4
        for (int ky = t.s; ky < N; ky += C::S) {
          const float2 v = t.lds[PL::slot_of_freq(ky) * C::TP + t.v];
          const int orow = ky + N / 2 < N ? ky + N / 2 : ky - N / 2;
          st(out, orow * N + ocol, cmul(v, ld(a.tab, ky * N + vec)));
        }
      }
      continue;
    }

    // ---- row passes: vectors are layer rows y = vec0 + v
    __syncthreads();
    if constexpr (SPECTRAL_IN) {
      load_spec_rows<C>(lds, static_cast<const float2*>(a.in) + (size_t)b * n * N, vec0, nvalid);
      __syncthreads();
      b_inverse_all<C>(t);
      __syncthreads();
      read_a(t, j, x);
      Dft<N1, 1>::run(x);
      if constexpr (LAYER) {
        const float2* __restrict__ ai = ACC ? a.act_in + (size_t)b * nn : nullptr;
        float2* __restrict__ ao = (KIND == kAsRowMid && a.act_out) ? a.act_out + (size_t)b * nn : nullptr;
        for_a_elems<C>(off, n, n, vec, vok, [&](auto k, int oi, bool in) {
          if constexpr (KIND == kAsRowMid) {
            const float2 u = in ? cmul(x[k.value], ld(a.mod, oi)) : c2(0.f, 0.f);
            if (ao && in) st(ao, oi, u);
            x[k.value] = u;
          } else {
            const float2 ul = in ? ld(ai, oi) : c2(0.f, 0.f);
            acc[k.value] += ul.x * x[k.value].y - ul.y * x[k.value].x;
            if constexpr (KIND == kAsRowBwdMid) x[k.value] = in ? cmulc(x[k.value], ld(a.mod, oi)) : c2(0.f, 0.f);
          }
        });
        if constexpr (KIND == kAsRowBwdLast) continue;
      }
    } else {
      if constexpr (KIND == kAsRowBwdFirst) {
        load_seed<C, kRow>(lds, a, b, vec0, nvalid);
      } else {
        const size_t es = a.in_real ? sizeof(float) : sizeof(float2);
        load_tile<C, kRow, false>(lds, static_cast<const char*>(a.in) + (size_t)b * nn * es, a.in_real != 0, n, off,
                           Consecutive{vec0}, nvalid);
      }
      __syncthreads();
      read_a(t, j, x);
    }

    if constexpr (FWD_OUT) {
      Dft<N1, -1>::run(x);
      write_a(t, j, x);
      __syncthreads();
      b_forward_all<C>(t);
      __syncthreads();
      store_spec_rows<C>(lds, a.out + (size_t)b * n * N, vec0, nvalid, a.spec_centred != 0);
    } else {
      if constexpr (KIND == kAsRowLast) add_skip<C, kRow>(a, b, vec, vok, x);
      write_a(t, j, x);  // positions, cropped on output
      __syncthreads();
      if constexpr (KIND == kAsRowIfft) {
        store_tile<C, kRow, false>(lds, a.out + (size_t)b * nn, n, off, Consecutive{vec0}, nvalid);
      } else {  // kAsRowLast
        tile_outputs<C, kRow>(lds, rsum, a, b, Consecutive{vec0}, nvalid, wi.tile);
      }
    }
  }
  if constexpr (ACC) {
    float* __restrict__ dp = a.dphi_part + (size_t)wi.group * nn;
    for_a_elems<C>(off, n, n, vec, vok, [&](auto k, int idx, bool in) {
      if (in) st(dp, idx, acc[k.value]);
    });
  }
}

// ---------------------------------------------------------------------------
// Wave-tile layer passes: the layer kinds of the separable path for a field
// stored in slot order (FULL) with a plan whose B-step has N2 = 8 points
// (N = 64, 128, 200).
//
// A workgroup is one wave and transforms 8 vectors.  Lane (v, j) holds A-item
// j of vector vec0 + v in registers: its N1 elements at the stored indices
// j + 8k, one per-lane base plus a compile-time offset each.  The B-step
// exchange stays inside the wave, 8 B-item indices at a time, through a
// private shared-memory buffer: the lanes write elements k1 = 8c .. 8c+7 of
// their A-items, lane (v, s) transforms B-item 8c + s of vector v, and the
// lanes read their elements back.  Against the workgroup tiles this needs no
// cross-wave barrier, has no partial tiles (N is a multiple of 8) and holds
// about 5 KB of shared memory per wave instead of the wave's share of a whole
// tile (13 KB at N = 200), so more waves stay resident to hide latency.
// Columns take lanes v-fastest (each load covers 64 contiguous bytes of 8
// rows), rows j-fastest (64 contiguous bytes of each of 8 rows).
// ---------------------------------------------------------------------------
template <class PL, int AXIS>
struct WaveTile {
  static constexpr int N = PL::N;
  static constexpr int N1 = PL::N1;
  static_assert(PL::N2 == 8, "wave tiles pair 8 A-items with 8 vectors");
  static constexpr int NC = (N1 + 7) / 8;  // exchange chunks
  // the last chunk holds one B-item per vector, whose values the 8 lanes of
  // a row hold one each (rows: lanes 8v .. 8v+7); Good-Thomas plans only
  // (no B-step twiddles)
  static constexpr bool LAST_ACROSS = AXIS == kRow && PL::PFA && N1 % 8 == 1 && NC > 1;
  static __device__ __forceinline__ int v_of(int lane) { return AXIS == kCol ? (lane & 7) : (lane >> 3); }
  static __device__ __forceinline__ int j_of(int lane) { return AXIS == kCol ? (lane >> 3) : (lane & 7); }
  // Exchange buffer index of (B-item offset s, A-item j, vector v), in
  // complex entries: s*PS + j*PJ + v*PV.  Each half wave's 32 lanes hit 32
  // distinct 8-byte bank slots on both sides of the exchange.
  static constexpr int PJ = AXIS == kCol ? 8 : 1;
  static constexpr int PV = AXIS == kCol ? 1 : 8;
  static constexpr int PS = AXIS == kCol ? 72 : 65;
  static constexpr int XCH = 7 * PS + 64;
};

// Exchange with the lane whose index differs in bit D (D = 1, 2, 4) inside
// each group of 8 lanes (a swizzle: no shared-memory access).
template <int D>
__device__ __forceinline__ float2 lane_xor(float2 v) {
  constexpr int kPattern = (D << 10) | 0x1F;  // bit mode: and 0x1F, or 0, xor D
  return c2(__int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v.x), kPattern)),
            __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v.y), kPattern)));
}

// The spectral B-step of one 8-value B-item held one value per lane by 8
// consecutive lanes (lane j: element j): forward DFT8 by decimation in
// frequency (lane j ends with frequency bitrev(j)), times the chirp entry of
// that frequency (tk: the item's 8 entries by frequency; conjugated when
// cj), then the inverse transform as the mirrored network with conjugate
// twiddles (bit-reversed in, natural out, unnormalised).
__device__ __forceinline__ float2 b_item_across_lanes(float2 u, int j, const float2* tk, bool cj) {
  constexpr float c = 0.70710678118654752440f;
  const bool u4 = (j & 4) != 0;
  const bool u2 = (j & 2) != 0;
  const bool u1 = (j & 1) != 0;
  const int m = j & 3;
  // exp(-2 pi i m / 8) for the pairs of the first stage, exp(-2 pi i (j&1) / 4) for the second
  const float2 w1 = c2(m == 0 ? 1.f : (m == 1 ? c : (m == 2 ? 0.f : -c)), m == 0 ? 0.f : (m == 2 ? -1.f : -c));
  const float2 w2 = u1 ? c2(0.f, -1.f) : c2(1.f, 0.f);
  {
    const float2 p = lane_xor<4>(u);
    const float2 d = u4 ? csub(p, u) : cadd(p, u);
    u = u4 ? cmul(d, w1) : d;
  }
  {
    const float2 p = lane_xor<2>(u);
    const float2 d = u2 ? csub(p, u) : cadd(p, u);
    u = u2 ? cmul(d, w2) : d;
  }
  {
    const float2 p = lane_xor<1>(u);
    u = u1 ? csub(p, u) : cadd(p, u);
  }
  const int br = ((j & 1) << 2) | (j & 2) | ((j >> 2) & 1);
  u = cj ? cmulc(u, tk[br]) : cmul(u, tk[br]);
  {
    const float2 p = lane_xor<1>(u);
    u = u1 ? csub(p, u) : cadd(u, p);
  }
  {
    const float2 p = lane_xor<2>(u);
    const float2 t = cmulc(u2 ? u : p, w2);
    u = u2 ? csub(p, t) : cadd(u, t);
  }
  {
    const float2 p = lane_xor<4>(u);
    const float2 t = cmulc(u4 ? u : p, w1);
    u = u4 ? csub(p, t) : cadd(u, t);
  }
  return u;
}

// Byte offset of element (stored index j, vector vec) of an N x N array
// oriented [q][vec] (tables, dphi partials, column fields) or [vec][q] (row
// fields); element k of the A-item adds wt_soff<...k>.
template <int N, int ES, bool QMAJOR>
__device__ __forceinline__ unsigned wt_base(int j, int vec, bool vok) {
  const unsigned e = QMAJOR ? (unsigned)(j * N + vec) : (unsigned)(vec * N + j);
  return vok ? e * (unsigned)ES : kOutOfRange;
}
template <int N, int ES, bool QMAJOR, int K>
constexpr int wt_soff() { return QMAJOR ? K * 8 * N * ES : K * 8 * ES; }

template <class PL, int KIND, int AXIS>
__global__ void __launch_bounds__(64, (KIND == kBwdMid || KIND == kBwdLast) ? 3 : 4) wave_pass(PassArgs a) {
  using WT = WaveTile<PL, AXIS>;
  constexpr int N = PL::N;
  constexpr int N1 = PL::N1;
  constexpr bool ACC = (KIND == kBwdMid || KIND == kBwdLast);
  constexpr bool FQ = AXIS == kCol;  // field arrays q-major along this pass
  static_assert(KIND == kFwdMid || ACC, "wave tiles run the layer kinds");
  // chirp entries of B-item k1 at 9*k1 + k2: the 8 B-items a wave reads at
  // once then start in 8 different bank pairs (a pitch of 8 put two of them
  // on each pair)
  __shared__ float2 tab[9 * N1];
  __shared__ float2 xch[WT::XCH];
  __shared__ float acc_lds[ACC ? N1 * 64 : 1];  // per-lane dphi accumulators

  const int G = (int)gridDim.x;
  const int l = (int)blockIdx.x;
  // XCD-contiguous ranks let neighbouring column tiles share cache lines in
  // one XCD's L2; row tiles read whole rows and stream faster in dispatch
  // order (a memory-only probe of the row pattern: 6.4 against 5.8 TB/s)
  const int rank = AXIS == kCol ? (l & 7) * (G >> 3) + (l >> 3) : l;
  if (rank >= a.workers) return;
  const int lane = (int)threadIdx.x;
  const int total = a.ntiles * a.batch;
  const size_t nn = (size_t)N * N;

  // chirp in B-item order: entry 9*k1 + k2 is frequency freq(k1, k2)
  for (int i = lane; i < N; i += 64) tab[i + (i >> 3)] = a.tab[PL::freq(i >> 3, i & 7)];
  if constexpr (ACC) {
    static_for<0, N1>([&](auto k) { acc_lds[k.value * 64 + lane] = 0.f; });
  }

  // One 1-D propagation of this lane's A-item: A-step DFT, B-step (DFT,
  // x chirp, inverse DFT) in chunks of 8 B-items through the exchange
  // buffer, inverse A-step DFT.  mid() runs once the first chunk is written
  // (loads issued there arrive during the B-step).
  auto prop = [&](float2(&x)[N1], bool cj, auto&& mid) {
    Dft<N1, -1>::run(x);
    int vv = WT::v_of(opaque_tid() & 63);
    int jj = WT::j_of(opaque_tid() & 63);
    const int wb = jj * WT::PJ + vv * WT::PV;  // A side: + s * PS
    const int bb = jj * WT::PS + vv * WT::PV;  // B side: + j' * PJ
    static_for<0, WT::NC>([&](auto cc) {
      constexpr int c = decltype(cc)::value;
      if constexpr (WT::LAST_ACROSS && c == WT::NC - 1) {
        // a last chunk of one B-item per vector (N1 = 8 (NC - 1) + 1): its 8
        // values sit one per lane in the 8 lanes of the vector, so the lanes
        // transform it together instead of 1 lane in 8 doing the whole item
        x[8 * c] = b_item_across_lanes(x[8 * c], jj, tab + 9 * (8 * c), cj);
        return;
      }
      static_for<0, 8>([&](auto sc) {
        constexpr int k1 = 8 * c + decltype(sc)::value;
        if constexpr (k1 < N1) xch[decltype(sc)::value * WT::PS + wb] = x[k1];
      });
      __syncthreads();
      if constexpr (c == 0) {
        // loads issued here arrive during the B-step; the scheduling
        // barriers keep them from being hoisted over the A-step
        __builtin_amdgcn_sched_barrier(0);
        mid();
        __builtin_amdgcn_sched_barrier(0);
      }
      const int k1 = 8 * c + jj;
      if (8 * c + 8 <= N1 || k1 < N1) {
        float2 y[8];
        static_for<0, 8>([&](auto jp) { y[jp.value] = xch[bb + jp.value * WT::PJ]; });
        if constexpr (!PL::PFA) {
          static_for<1, 8>([&](auto jp) { y[jp.value] = cmul(y[jp.value], root_at<N>((unsigned)(k1 * jp.value))); });
        }
        Dft<8, -1>::run(y);
        const float2* tk = tab + 9 * k1;
        if (cj) {
          static_for<0, 8>([&](auto k2) { y[k2.value] = cmulc(y[k2.value], tk[k2.value]); });
        } else {
          static_for<0, 8>([&](auto k2) { y[k2.value] = cmul(y[k2.value], tk[k2.value]); });
        }
        Dft<8, 1>::run(y);
        if constexpr (!PL::PFA) {
          static_for<1, 8>(
              [&](auto jp) { y[jp.value] = cmul(y[jp.value], root_at<N>((unsigned)(N - k1 * jp.value))); });
        }
        static_for<0, 8>([&](auto jp) { xch[bb + jp.value * WT::PJ] = y[jp.value]; });
      }
      __syncthreads();
      static_for<0, 8>([&](auto sc) {
        constexpr int k1r = 8 * c + decltype(sc)::value;
        if constexpr (k1r < N1) x[k1r] = xch[decltype(sc)::value * WT::PS + wb];
      });
    });
    Dft<N1, 1>::run(x);
  };
  auto nothing = [] {};

  // rows of G that can be nonzero (layer L of a region loss, column passes)
  unsigned gmask = ~0u;
  if constexpr (ACC && AXIS == kCol) {
    if (a.live) {
      gmask = 0u;
      const int j = WT::j_of(lane);
      static_for<0, N1>([&](auto k) {
        if (ld(a.live, PL::pos_of_slot(j + 8 * k.value)) != 0ull) gmask |= 1u << k.value;
      });
    }
  }

  for (int it = rank; it < total; it += a.workers) {
    const int tile = it % a.ntiles;
    const int b = it / a.ntiles;
    const int vec = tile * 8 + WT::v_of(opaque_tid() & 63);
    const int j = WT::j_of(opaque_tid() & 63);
    const bool vok = vec < a.nvec;
    const unsigned fb = wt_base<N, 8, FQ>(j, vec, vok);    // field arrays
    const unsigned tb = wt_base<N, 8, true>(j, vec, vok);  // [q][vec] tables
    const Rsrc rin = make_rsrc(static_cast<const float2*>(a.in) + (size_t)b * nn, (unsigned)nn * 8u);
    const Rsrc rmod = make_rsrc(a.mod, (unsigned)nn * 8u);
    auto load_field = [&](Rsrc r, unsigned mask, float2(&x)[N1]) {
      static_for<0, N1>([&](auto k) {
        x[k.value] = bload_so<field_load_policy<N>()>(r, ((mask >> k.value) & 1u) ? fb : kOutOfRange,
                                                      wt_soff<N, 8, FQ, k.value>());
      });
    };
    auto load_mod = [&](float2(&m)[N1]) {
      static_for<0, N1>([&](auto k) { m[k.value] = bload_keep_so(rmod, tb, wt_soff<N, 8, true, k.value>()); });
    };
    float2 x[N1];
    if constexpr (KIND == kFwdMid) {
      load_field(rin, ~0u, x);
      float2 m[N1];
      prop(x, a.conj_tab != 0, nothing);
      load_mod(m);
      static_for<0, N1>([&](auto k) { x[k.value] = cmul(x[k.value], m[k.value]); });
      prop(x, a.conj_tab != 0, nothing);
    } else {
      const Rsrc rw = make_rsrc(a.act_in + (size_t)b * nn, (unsigned)nn * 8u);
      float2 ar[N1];
      float2 m[N1];
      if constexpr (KIND == kBwdMid) {
        // A_l from the saved input of the forward pass, then the gradient
        load_field(rw, ~0u, ar);
        load_field(rin, gmask, x);
        prop(ar, false, nothing);
        prop(x, true, nothing);
      } else {
        load_field(rin, gmask, x);
        load_field(rw, ~0u, ar);
        prop(x, true, nothing);
        prop(ar, false, nothing);
      }
      load_mod(m);
      // h = conj(M_l) G_l and dphi_l += Im(conj(A_l) h)
      static_for<0, N1>([&](auto k) {
        const float2 h = cmulc(x[k.value], m[k.value]);
        acc_lds[k.value * 64 + lane] += ar[k.value].x * h.y - ar[k.value].y * h.x;
        x[k.value] = h;
      });
      if constexpr (KIND == kBwdMid) prop(x, true, nothing);
    }
    if constexpr (KIND != kBwdLast) {
      const Rsrc rout = make_rsrc(a.out + (size_t)b * nn, (unsigned)nn * 8u);
      static_for<0, N1>([&](auto k) { bstore_so(rout, fb, wt_soff<N, 8, FQ, k.value>(), x[k.value]); });
    }
  }
  if constexpr (ACC) {
    // one partial per lane for the tile this wave kept
    const int vec = (rank % a.ntiles) * 8 + WT::v_of(lane);
    const unsigned base = wt_base<N, 4, true>(WT::j_of(lane), vec, vec < a.nvec);
    const Rsrc dp = make_rsrc(a.dphi_part + (size_t)(rank / a.ntiles) * nn, (unsigned)nn * 4u);
    static_for<0, N1>(
        [&](auto k) { bstore_f_so(dp, base, wt_soff<N, 4, true, k.value>(), acc_lds[k.value * 64 + lane]); });
  }
}

// ---------------------------------------------------------------------------
// Row layer passes at N = 500 (25 x 20 Cooley-Tukey) on wave tiles.  The
// 16-vector workgroup tiles this plan needs are five waves of 68 KB, which
// run alone on their CU; here a workgroup is one wave of 17 KB and
// transforms 3 whole rows.  Lane (r, j), r = lane / 20, j = lane mod 20,
// holds A-item j of row r in registers (lanes 60..63 read row 0's items,
// write nothing and touch no global memory).  The exchange runs through a
// private buffer, slot s of row r at r * 525 + s + s / 20, so that the
// elements of the A-items and the 20 B-items a wave reads at once start in
// distinct bank pairs; B-items k1 < 20 go one per lane, the five left
// (k1 = 20..24) one per lane quad, split by Good-Thomas 4 x 5 as in
// b_spectral_quad.  Fields, this layer's modulation table and the dphi
// partials are [vec][q] (rows, slot order): consecutive lanes read
// consecutive slots of a row.  First pass (kPropOnce, real amplitudes in)
// and forward (kFwdMid): one item per workgroup; adjoint (kBwdMid):
// persistent, as fresnel_pass.
// ---------------------------------------------------------------------------
template <class PL>
struct WideRows {
  static constexpr int N = PL::N;
  static constexpr int N1 = PL::N1;
  static constexpr int N2 = PL::N2;
  static constexpr int R = 64 / N2;      // rows per wave
  static constexpr int P1 = N2 + 1;      // buffer stride of a B-item
  static constexpr int PR = P1 * N1;     // buffer pitch of a row
  static constexpr int Q = N2 / 4;       // the quad split's odd factor
  static constexpr int E1 = Q * inv_mod(Q % 4, 4);
  static constexpr int E2 = 4 * inv_mod(4 % Q, Q);
  static_assert(N == 500 && N1 == 25 && N2 == 20 && !PL::PFA, "wide row tiles are written for 25 x 20");
  static_assert(N1 - N2 == Q, "the last round is one item per quad");
};

template <class PL, int KIND>
__global__ void __launch_bounds__(64, KIND == kBwdMid ? 2 : 3) wide_row_pass(PassArgs a) {
  using W = WideRows<PL>;
  constexpr int N = W::N;
  constexpr int N1 = W::N1;
  constexpr int N2 = W::N2;
  constexpr int R = W::R;
  constexpr int P1 = W::P1;
  constexpr int PR = W::PR;
  constexpr int Q = W::Q;
  constexpr bool ACC = KIND == kBwdMid;
  static_assert(KIND == kPropOnce || KIND == kFwdMid || KIND == kBwdMid, "wide row tiles run the layer kinds");
  constexpr int POL = field_load_policy<N>();
  // The adjoint stages the chirp in shared memory (B-item k1, frequency k2
  // at P1 * k1 + k2; its registers allow 8 waves per CU either way); the
  // forward kinds read it from the (cached) table in global memory, which
  // leaves 12.6 KB of shared memory per wave: 12 waves per CU.
  constexpr bool TAB_LDS = ACC;
  __shared__ float2 tab[TAB_LDS ? PR : 1];
  __shared__ float2 xch[R * PR];  // R rows

  const int rank = (int)blockIdx.x;
  if (rank >= a.workers) return;
  const int lane = (int)threadIdx.x;
  const bool act = lane < R * N2;
  const int r = act ? lane / N2 : 0;
  const int j = act ? lane - r * N2 : lane - R * N2;
  const int total = a.ntiles * a.batch;
  const size_t nn = (size_t)N * N;
  const bool cj = a.conj_tab != 0;

  if constexpr (TAB_LDS) {
    for (int i = lane; i < N; i += 64) tab[P1 * (i / N2) + i % N2] = a.tab[PL::freq(i / N2, i % N2)];
  }
  // chirp entry of B-item k1, element k2 (frequency k1 + N1 * k2)
  const float2* __restrict__ gtab = a.tab;
  auto chirp = [&](int k1, int k2) -> float2 {
    if constexpr (TAB_LDS) {
      return tab[P1 * k1 + k2];
    } else {
      return gtab[k1 + N1 * k2];
    }
  };
  float acc[ACC ? N1 : 1];
  if constexpr (ACC) {
    static_for<0, N1>([&](auto k) { acc[k.value] = 0.f; });
  }

  // one 1-D propagation of this lane's A-item along its row.  The lane's
  // indices pass through an empty asm statement at every call, so the
  // twiddles and addresses derived from them are formed here and not kept
  // live across the item loop; scheduling barriers keep each phase's loads
  // (data, twiddles, table) next to their use, as in b_spectral_item.
  auto prop = [&](float2(&v)[N1], bool conj_t) {
    int jo = j;
    int ro = r;
    asm volatile("" : "+v"(jo), "+v"(ro));
    Dft<N1, -1>::run(v);
    float2* const xr = xch + ro * PR;
    if (act) {
      static_for<0, N1>([&](auto x) { xr[P1 * x.value + jo] = v[x.value]; });
    }
    __syncthreads();
    if (act) {
      // B-item k1 = j of row r
      float2* const yb = xr + P1 * jo;
      float2 y[N2];
      static_for<0, N2>([&](auto q) { y[q.value] = yb[q.value]; });
      static_for<1, N2>([&](auto q) { y[q.value] = cmul(y[q.value], root_at<N>((unsigned)(jo * q.value))); });
      Dft<N2, -1>::run(y);
      __builtin_amdgcn_sched_barrier(0);
      if (conj_t) {
        static_for<0, N2>([&](auto q) { y[q.value] = cmulc(y[q.value], chirp(jo, q.value)); });
      } else {
        static_for<0, N2>([&](auto q) { y[q.value] = cmul(y[q.value], chirp(jo, q.value)); });
      }
      __builtin_amdgcn_sched_barrier(0);
      Dft<N2, 1>::run(y);
      static_for<1, N2>(
          [&](auto q) { y[q.value] = cmul(y[q.value], root_at<N>((unsigned)(N - jo * q.value))); });
      static_for<0, N2>([&](auto q) { yb[q.value] = y[q.value]; });
      __builtin_amdgcn_sched_barrier(0);
    }
    if (lane < R * N2) {
      // B-items k1 = N2 .. N1-1: item qi = lane / 4 (row qi / Q, k1 = N2 + qi mod Q), one per quad
      // (the last quad, lanes 60..63, has none)
      int t = lane;
      asm volatile("" : "+v"(t));
      const int qi = t >> 2;
      const int qq = t & 3;
      const int qrow = qi / Q;
      const int k1 = N2 + qi - qrow * Q;
      float2* const base = xch + qrow * PR + P1 * k1;
      auto elem = [&](auto m) {
        const int e = Q * qq + 4 * decltype(m)::value;
        return e >= N2 ? e - N2 : e;
      };
      const float s1 = (qq & 1) ? -1.f : 1.f;
      const float s2 = (qq & 2) ? -1.f : 1.f;
      const bool l3 = qq == 3;
      float2 z[Q];
      static_for<0, Q>([&](auto m) {
        const int e = elem(m);
        z[m.value] = cmul(base[e], root_at<N>((unsigned)(k1 * e)));
      });
      Dft<Q, -1>::run(z);
      quad_butterfly<2, Q>(z, s2);
      static_for<0, Q>([&](auto m) {
        const float2 u = z[m.value];
        z[m.value] = l3 ? c2(u.y, -u.x) : u;
      });
      quad_butterfly<1, Q>(z, s1);
      const int k4 = ((qq & 1) << 1) | (qq >> 1);
      static_for<0, Q>([&](auto m) {
        const int f = (W::E1 * k4 + W::E2 * decltype(m)::value) % N2;
        const float2 h = chirp(k1, f);
        z[m.value] = conj_t ? cmulc(z[m.value], h) : cmul(z[m.value], h);
      });
      quad_butterfly<1, Q>(z, s1);
      static_for<0, Q>([&](auto m) {
        const float2 u = z[m.value];
        z[m.value] = l3 ? c2(-u.y, u.x) : u;
      });
      quad_butterfly<2, Q>(z, s2);
      Dft<Q, 1>::run(z);
      static_for<0, Q>([&](auto m) {
        const int e = elem(m);
        base[e] = cmul(z[m.value], root_at<N>((unsigned)(N - k1 * e)));
      });
    }
    __syncthreads();
    static_for<0, N1>([&](auto x) { v[x.value] = xr[P1 * x.value + jo]; });
    Dft<N1, 1>::run(v);
  };

  // element x of this lane's A-item: [vec][q] offset vec * N + j + N2 * x
  for (int it = rank; it < total; it += a.workers) {
    const int tile = it % a.ntiles;
    const int b = it / a.ntiles;
    const int vec = tile * R + r;
    const bool vok = act && vec < a.nvec;
    const unsigned base = vok ? (unsigned)(vec * N + j) * 8u : kOutOfRange;
    const Rsrc rin = make_rsrc(static_cast<const float2*>(a.in) + (size_t)b * nn, (unsigned)nn * 8u);
    const Rsrc rmod = make_rsrc(a.mod, (unsigned)nn * 8u);
    float2 x[N1];
    if constexpr (ACC) {
      // A_l from the saved input of the forward pass, then G's half hop
      float2 ar[N1];
      const Rsrc ract = make_rsrc(a.act_in + (size_t)b * nn, (unsigned)nn * 8u);
      static_for<0, N1>([&](auto k) { ar[k.value] = bload_so<POL>(ract, base, N2 * 8 * k.value); });
      prop(ar, false);
      static_for<0, N1>([&](auto k) { x[k.value] = bload_so<POL>(rin, base, N2 * 8 * k.value); });
      prop(x, true);
      // conj(M_l) G_l and dphi_l += Im(conj(A_l) conj(M_l) G_l)
      static_for<0, N1>([&](auto k) {
        const float2 h = cmulc(x[k.value], bload_keep_so(rmod, base, N2 * 8 * k.value));
        acc[k.value] += ar[k.value].x * h.y - ar[k.value].y * h.x;
        x[k.value] = h;
      });
      prop(x, true);
    } else if constexpr (KIND == kPropOnce) {
      // real amplitudes in; along a row slot order is natural order (Cooley-Tukey plan)
      const Rsrc ramp = make_rsrc(static_cast<const float*>(a.in) + (size_t)b * nn, (unsigned)nn * 4u);
      const unsigned base4 = vok ? (unsigned)(vec * N + j) * 4u : kOutOfRange;
      static_for<0, N1>([&](auto k) {
        x[k.value] = c2(__builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ramp, (int)base4, N2 * 4 * k.value, POL)), 0.f);
      });
      prop(x, cj);
    } else {
      static_for<0, N1>([&](auto k) { x[k.value] = bload_so<POL>(rin, base, N2 * 8 * k.value); });
      prop(x, cj);
      // U_l = M_l A_l
      static_for<0, N1>([&](auto k) { x[k.value] = cmul(x[k.value], bload_keep_so(rmod, base, N2 * 8 * k.value)); });
      prop(x, cj);
    }
    const Rsrc rout = make_rsrc(a.out + (size_t)b * nn, (unsigned)nn * 8u);
    static_for<0, N1>([&](auto k) { bstore_so(rout, base, N2 * 8 * k.value, x[k.value]); });
  }
  if constexpr (ACC) {
    // one partial per lane for the tile this wave kept
    const int vec = (rank % a.ntiles) * R + r;
    const bool vok = act && vec < a.nvec;
    const unsigned base = vok ? (unsigned)(vec * N + j) * 4u : kOutOfRange;
    const Rsrc dp = make_rsrc(a.dphi_part + (size_t)(rank / a.ntiles) * nn, (unsigned)nn * 4u);
    static_for<0, N1>([&](auto k) { bstore_f_so(dp, base, N2 * 4 * k.value, acc[k.value]); });
  }
}

// ---------------------------------------------------------------------------
// Whole-field forward for grids whose field fits in one CU's shared memory
// (N <= 128: 132 KB at N = 128).  One workgroup per sample reads the
// amplitude once, runs every hop and modulation of Eq. (forward_diff) and
// (phase_mod_matrix) on the resident field, and writes only the detector-
// plane outputs (region sums of §2.1, and the intensity map and field when
// asked for), so no field crosses HBM between layers.
//
// The field is held in slot order on both axes (plan.hpp), f[sy][sx] with
// pitch N + 1.  A hop is the separable 1-D propagation along x for every row,
// then along y for every column: thread (v, j) (v = tid mod N) owns A-item j
// of vector v, and the B-items k1 = j, j + N2, ... of that vector, as in the
// tile passes but with all N vectors of the field in one tile; along x the
// vector is a row (f[v][slot]), along y a column (f[slot][v]).  Consecutive
// lanes take consecutive vectors, so with the odd pitch every shared-memory
// access of a wave falls in distinct banks along both axes.
// ---------------------------------------------------------------------------
template <class PL>
struct WholeCfg {
  using Plan = PL;
  static constexpr int N = PL::N;
  static constexpr int N1 = PL::N1;
  static constexpr int N2 = PL::N2;
  static constexpr int P = N * N2;  // threads
  static constexpr int TP = N + 1;  // pitch of the field in shared memory
};

template <class PL>
__global__ void __launch_bounds__(PL::N * PL::N2) field_forward_kernel(FieldArgs a) {
  using C = WholeCfg<PL>;
  constexpr int N = C::N;
  constexpr int N1 = C::N1;
  constexpr int N2 = C::N2;
  constexpr int P = C::P;
  constexpr int TP = C::TP;
  // The field, and in its padding column (x = N) the x chirp; the y chirp
  // apart.  Both in B-item order: entry N2*k1 + k2 is frequency
  // freq(k1, k2).  (At N = 100 this keeps a workgroup within 80 KB, two
  // per CU.)
  __shared__ float2 f[N * TP];
  __shared__ float2 ty[N];

  const int b = (int)blockIdx.x;
  const int tid = (int)threadIdx.x;
  const int v = tid % N;
  const int j = tid / N;
  const size_t nn = (size_t)N * N;

  for (int i = tid; i < N; i += P) {
    const int fr = PL::freq(i / N2, i % N2);
    f[i * TP + N] = a.chirp_x[fr];
    ty[i] = a.chirp_y[fr];
  }
  // amplitudes (natural, zero phase) into slot order: stored (sy, sx) holds
  // natural pixel (pos_of_slot(sy), pos_of_slot(sx)); consecutive threads take
  // consecutive natural x
  {
    const float* __restrict__ amp = a.amp + (size_t)b * nn;
    for (int e = tid; e < N * N; e += P) {
      const int y = e / N;
      const int x = e - y * N;
      f[PL::slot_of_pos(y) * TP + PL::slot_of_pos(x)] = c2(amp[e], 0.f);
    }
  }
  __syncthreads();

  // 1-D propagation of every vector along one axis, in place
  auto prop = [&](auto axis_c, const float2* tab, int tstride) {
    constexpr bool ROWS = decltype(axis_c)::value == kRow;
    auto at = [&](int vec, int slot) -> float2& { return ROWS ? f[vec * TP + slot] : f[slot * TP + vec]; };
    float2 x[N1];
    static_for<0, N1>([&](auto k) { x[k.value] = at(v, j + N2 * k.value); });
    Dft<N1, -1>::run(x);
    static_for<0, N1>([&](auto k) { at(v, j + N2 * k.value) = x[k.value]; });
    __syncthreads();
    for (int k1 = j; k1 < N1; k1 += N2) {
      float2 y[N2];
      static_for<0, N2>([&](auto q) { y[q.value] = at(v, N2 * k1 + q.value); });
      b_forward<C>(k1, y);
      static_for<0, N2>([&](auto q) { y[q.value] = cmul(y[q.value], tab[(N2 * k1 + q.value) * tstride]); });
      b_inverse<C>(k1, y);
      static_for<0, N2>([&](auto q) { at(v, N2 * k1 + q.value) = y[q.value]; });
    }
    __syncthreads();
    static_for<0, N1>([&](auto k) { x[k.value] = at(v, j + N2 * k.value); });
    Dft<N1, 1>::run(x);
    static_for<0, N1>([&](auto k) { at(v, j + N2 * k.value) = x[k.value]; });
    __syncthreads();
  };

  for (int hop = 1; hop <= a.layers + 1; ++hop) {
    prop(std::integral_constant<int, kRow>{}, f + N, TP);
    prop(std::integral_constant<int, kCol>{}, ty, 1);
    if (hop <= a.layers) {
      // U_l = gamma exp(j phi_l) A_l; the table is in slot order, [y][x] or
      // [x][y]: consecutive threads take consecutive positions of its rows
      const float2* __restrict__ m = a.mod + (size_t)(hop - 1) * nn;
      const bool tr = (a.mod_t >> (hop - 1)) & 1ull;
      for (int e = tid; e < N * N; e += P) {
        const int r = e / N;
        const int c = e - r * N;
        float2& u = tr ? f[c * TP + r] : f[r * TP + c];
        u = cmul(u, m[e]);
      }
      __syncthreads();
    }
  }

  // S_k = sum of |U_D|^2 over region k: wave w sums regions w, w + waves, ...
  // over natural pixels in a fixed order (lane stride 64, then a fixed
  // butterfly), so the sums are reproducible
  constexpr int NW = P / 64;  // whole waves (at N = 100 the last wave is partial and sums nothing)
  const int wv = tid >> 6;
  const int lane = tid & 63;
  const int side = a.reg.s;
  for (int k = wv; wv < NW && k < a.reg.K; k += NW) {
    const int y0 = a.reg.y0[k];
    const int x0 = a.reg.x0[k];
    float acc = 0.f;
    for (int e = lane; e < side * side; e += 64) {
      const int dy = e / side;
      const int y = y0 + dy;
      const int x = x0 + (e - dy * side);
      const float2 u = f[PL::slot_of_pos(y) * TP + PL::slot_of_pos(x)];
      acc = fmaf(u.x, u.x, fmaf(u.y, u.y, acc));
    }
    for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (lane == 0) a.sums_part[(size_t)b * a.reg.K + k] = acc;
  }
  // full-map outputs in natural order (consecutive threads, consecutive x)
  if (a.intensity || a.field_out) {
    float* __restrict__ io = a.intensity ? a.intensity + (size_t)b * nn : nullptr;
    float2* __restrict__ fo = a.field_out ? a.field_out + (size_t)b * nn : nullptr;
    for (int e = tid; e < N * N; e += P) {
      const int y = e / N;
      const int x = e - y * N;
      const float2 u = f[PL::slot_of_pos(y) * TP + PL::slot_of_pos(x)];
      if (io) {
        const float in = fmaf(u.x, u.x, u.y * u.y);
        io[e] = a.accumulate ? io[e] + in : in;
      }
      if (fo) fo[e] = u;
    }
  }
}

// ---------------------------------------------------------------------------
// Whole-field forward at N = 200 (25 x 8 Good-Thomas): the 320 KB field is
// twice a CU's shared memory, so half of it lives there and half in
// registers.  Thread (v, j), v < 100, j < 8 (800 threads), holds in R[25]
// A-item j of vector 100 + v; shared memory holds vectors 0..99.  Along x
// ("row phase") the vectors are rows; along y ("column phase") columns.
//
// Shared layout: row r < 100 of the stored field (slot order on both axes)
// at rowaddr(r) = 200 r + r / 4 (the skew keeps the 32 rows a half wave
// touches at once in distinct bank pairs).  Quadrants by slot: Q1 (sy, sx
// < 100) stays at rowaddr(sy) + sx in both phases; Q2 (sy < 100 <= sx) is
// at rowaddr(sy) + sx in the row phase, in registers (by column) in the
// column phase; Q3 (sx < 100 <= sy) is in registers (by row) in the row
// phase and at rowaddr(sy - 100) + 100 + sx (Q2's place) in the column
// phase; Q4 is always in registers.  A phase change moves Q2, Q3 and Q4
// through shared memory in four steps (read the quadrant leaving shared
// memory into the new register layout, park Q4 in the freed region, read
// it back in the new layout, store the quadrant entering shared memory).
//
// A 1-D propagation of the whole field transforms the shared half (A-step
// from and to shared memory, B-step there, inverse A-step into registers x),
// then the register half through the same shared buffer, then writes x back.
// After the last hop the intensities of all 40000 pixels replace the field in
// shared memory (4 bytes each), and the region sums and intensity map read
// them there.
// ---------------------------------------------------------------------------
template <class PL>
struct SplitCfg {
  using Plan = PL;
  static constexpr int N = PL::N;
  static constexpr int N1 = PL::N1;
  static constexpr int N2 = PL::N2;
  static constexpr int H = N / 2;   // vectors in shared memory
  static constexpr int P = H * N2;  // threads
  static constexpr int LDS = H * N + H / 4;
  static_assert(N == 200 && N1 == 25 && N2 == 8 && PL::PFA, "the split whole-field layout is written for 25 x 8");
  static_assert(N * N * 4 <= LDS * 8, "the intensity map must fit where the field half was");
  __device__ static constexpr int rowaddr(int r) { return r * N + (r >> 2); }
  // rowaddr(j + 8x) = rowaddr(j) + XS * x for j < 8
  static constexpr int XS = 8 * N + 2;
  // rowaddr(s - H) + H = rowaddr(s) - SHIFT for s >= H
  static constexpr int SHIFT = H * N + H / 4 - H;
  // first A-item element with slot j + 8x >= H: x = 12 for j >= 4, 13 below
  static constexpr int XH = H / N2;  // 12
};

template <class PL>
__global__ void __launch_bounds__(SplitCfg<PL>::P) field_forward_split_kernel(FieldArgs a) {
  using C = SplitCfg<PL>;
  constexpr int N = C::N;
  constexpr int N1 = C::N1;
  constexpr int N2 = C::N2;
  constexpr int H = C::H;
  constexpr int P = C::P;
  constexpr int XS = C::XS;
  constexpr int SHIFT = C::SHIFT;
  constexpr int XH = C::XH;
  __shared__ float2 f[C::LDS];
  __shared__ float2 tabx[N];
  __shared__ float2 taby[N];

  const int b = (int)blockIdx.x;
  const int tid = (int)threadIdx.x;
  const int v = tid % H;
  const int j = tid / H;
  const size_t nn = (size_t)N * N;
  // element XH of the A-item lies in the upper half (slot >= H) for j >= N2 / 2
  const bool up12 = j + N2 * XH >= H;

  for (int i = tid; i < N; i += P) {
    const int fr = PL::freq(i / N2, i % N2);
    tabx[i] = a.chirp_x[fr];
    taby[i] = a.chirp_y[fr];
  }
  // amplitudes (natural, zero phase) into the row phase: shared rows sy < H,
  // registers rows H + v
  const float* __restrict__ amp = a.amp + (size_t)b * nn;
  for (int e = tid; e < H * N; e += P) {
    const int sy = e / N;
    const int sx = e - sy * N;
    f[C::rowaddr(sy) + sx] = c2(amp[(size_t)PL::pos_of_slot(sy) * N + PL::pos_of_slot(sx)], 0.f);
  }
  float2 R[N1];
  {
    const int y = PL::pos_of_slot(H + v);
    static_for<0, N1>([&](auto x) { R[x.value] = c2(amp[(size_t)y * N + PL::pos_of_slot(j + N2 * x.value)], 0.f); });
  }
  __syncthreads();

  // A-item j of shared vector v, element x: row phase rowaddr(v) + j + 8x;
  // column phase rowaddr(j + 8x) + v, less SHIFT in the upper half
  const int arow = C::rowaddr(v) + j;
  const int acol = C::rowaddr(j) + v;
  auto a_addr = [&](auto rows_c, auto x_c) -> int {
    constexpr int x = decltype(x_c)::value;
    if constexpr (decltype(rows_c)::value) {
      return arow + N2 * x;
    } else if constexpr (x < XH) {
      return acol + XS * x;
    } else if constexpr (x > XH) {
      return acol + XS * x - SHIFT;
    } else {
      return acol + XS * x - (up12 ? SHIFT : 0);
    }
  };
  auto a_load = [&](auto rows_c, float2(&x)[N1]) {
    static_for<0, N1>([&](auto k) { x[k.value] = f[a_addr(rows_c, k)]; });
  };
  auto a_store = [&](auto rows_c, const float2(&x)[N1]) {
    static_for<0, N1>([&](auto k) { f[a_addr(rows_c, k)] = x[k.value]; });
  };
  // spectral B-step of the shared half: B-items k1 = j, j + 8, ... of vector v
  auto b_step = [&](auto rows_c) {
    constexpr bool ROWS = decltype(rows_c)::value;
    const float2* tab = ROWS ? tabx : taby;
    for (int k1 = j; k1 < N1; k1 += N2) {
      int base;
      int off_lo = 0;
      int off_hi = 0;
      if constexpr (ROWS) {
        base = C::rowaddr(v) + N2 * k1;
      } else {
        // rowaddr(8 k1 + q) = XS k1 + N q + q / 4; slots >= H shift down
        base = XS * k1 + v;
        off_lo = N2 * k1 >= H ? -SHIFT : 0;           // elements q < 4
        off_hi = N2 * k1 + N2 / 2 >= H ? -SHIFT : 0;  // elements q >= 4
      }
      auto addr = [&](auto q_c) {
        constexpr int q = decltype(q_c)::value;
        if constexpr (ROWS) {
          return base + q;
        } else {
          return base + N * q + (q >> 2) + (q < N2 / 2 ? off_lo : off_hi);
        }
      };
      float2 y[N2];
      static_for<0, N2>([&](auto q) { y[q.value] = f[addr(q)]; });
      Dft<N2, -1>::run(y);
      static_for<0, N2>([&](auto q) { y[q.value] = cmul(y[q.value], tab[N2 * k1 + q.value]); });
      Dft<N2, 1>::run(y);
      static_for<0, N2>([&](auto q) { f[addr(q)] = y[q.value]; });
    }
  };
  // 1-D propagation of the whole field along the phase's axis
  auto prop = [&](auto rows_c) {
    float2 x[N1];
    a_load(rows_c, x);
    Dft<N1, -1>::run(x);
    a_store(rows_c, x);
    __syncthreads();
    b_step(rows_c);
    __syncthreads();
    a_load(rows_c, x);
    Dft<N1, 1>::run(x);
    __syncthreads();
    Dft<N1, -1>::run(R);
    a_store(rows_c, R);
    __syncthreads();
    b_step(rows_c);
    __syncthreads();
    a_load(rows_c, R);
    Dft<N1, 1>::run(R);
    __syncthreads();
    a_store(rows_c, x);
    __syncthreads();
  };
  // phase changes; T[x] holds the new register layout's element x
  auto to_cols = [&] {
    float2 T[N1];
    // Q2 (shared, row phase) -> registers by column: column H + v, slot j + 8x < H
    static_for<0, XH + 1>([&](auto x) {
      if (x.value < XH || !up12) T[x.value] = f[acol + XS * x.value + H];
    });
    __syncthreads();
    // Q4 (registers by row: row H + v, slot j + 8x >= H) parked at rowaddr(v) + j + 8x
    static_for<XH, N1>([&](auto x) {
      if (x.value > XH || up12) f[arow + N2 * x.value] = R[x.value];
    });
    __syncthreads();
    // Q4 by column: column H + v, slot sy = j + 8x >= H, parked at rowaddr(sy - H) + H + v
    static_for<XH, N1>([&](auto x) {
      if (x.value > XH || up12) T[x.value] = f[acol + XS * x.value - SHIFT];
    });
    __syncthreads();
    // Q3 (registers by row: row H + v, slot j + 8x < H) to rowaddr(v) + H + j + 8x
    static_for<0, XH + 1>([&](auto x) {
      if (x.value < XH || !up12) f[arow + N2 * x.value + H] = R[x.value];
    });
    static_for<0, N1>([&](auto x) { R[x.value] = T[x.value]; });
    __syncthreads();
  };
  auto to_rows = [&] {
    float2 T[N1];
    // Q3 (shared, column phase, at rowaddr(v) + H + sx) -> registers by row
    static_for<0, XH + 1>([&](auto x) {
      if (x.value < XH || !up12) T[x.value] = f[arow + N2 * x.value + H];
    });
    __syncthreads();
    // Q4 (registers by column: column H + v, slot sy = j + 8x >= H) parked at rowaddr(sy - H) + H + v
    static_for<XH, N1>([&](auto x) {
      if (x.value > XH || up12) f[acol + XS * x.value - SHIFT] = R[x.value];
    });
    __syncthreads();
    // Q4 by row: row H + v, slot sx = j + 8x >= H, parked at rowaddr(v) + sx
    static_for<XH, N1>([&](auto x) {
      if (x.value > XH || up12) T[x.value] = f[arow + N2 * x.value];
    });
    __syncthreads();
    // Q2 (registers by column: column H + v, slot sy = j + 8x < H) to rowaddr(sy) + H + v
    static_for<0, XH + 1>([&](auto x) {
      if (x.value < XH || !up12) f[acol + XS * x.value + H] = R[x.value];
    });
    static_for<0, N1>([&](auto x) { R[x.value] = T[x.value]; });
    __syncthreads();
  };

  for (int hop = 1; hop <= a.layers + 1; ++hop) {
    prop(std::true_type{});
    to_cols();
    prop(std::false_type{});
    if (hop <= a.layers) {
      // U_l = gamma exp(j phi_l) A_l on both halves; table [sy][sx] or [sx][sy] in slot order
      const float2* __restrict__ m = a.mod + (size_t)(hop - 1) * nn;
      const bool tr = (a.mod_t >> (hop - 1)) & 1ull;
      for (int e = tid; e < H * N; e += P) {
        const int sy = e / H;
        const int sx = e - sy * H;
        float2& u = f[sy < H ? C::rowaddr(sy) + sx : C::rowaddr(sy - H) + H + sx];
        u = cmul(u, m[tr ? (size_t)sx * N + sy : (size_t)sy * N + sx]);
      }
      static_for<0, N1>([&](auto x) {
        const int sy = j + N2 * x.value;
        const int sx = H + v;
        R[x.value] = cmul(R[x.value], m[tr ? (size_t)sx * N + sy : (size_t)sy * N + sx]);
      });
      __syncthreads();
      to_rows();
    }
  }

  // detector plane (column phase): the complex field out, then every
  // pixel's intensity into shared memory, slot order [sy][sx]
  float2* __restrict__ fo = a.field_out ? a.field_out + (size_t)b * nn : nullptr;
  float il[N1];
  float ir[N1];
  static_for<0, N1>([&](auto i) {
    const int e = tid + P * i.value;
    const int sy = e / H;
    const int sx = e - sy * H;
    const float2 u = f[sy < H ? C::rowaddr(sy) + sx : C::rowaddr(sy - H) + H + sx];
    il[i.value] = fmaf(u.x, u.x, u.y * u.y);
    if (fo) fo[(size_t)PL::pos_of_slot(sy) * N + PL::pos_of_slot(sx)] = u;
  });
  static_for<0, N1>([&](auto x) {
    const float2 u = R[x.value];
    ir[x.value] = fmaf(u.x, u.x, u.y * u.y);
    if (fo) fo[(size_t)PL::pos_of_slot(j + N2 * x.value) * N + PL::pos_of_slot(H + v)] = u;
  });
  __syncthreads();
  float* const inten = reinterpret_cast<float*>(f);
  static_for<0, N1>([&](auto i) {
    const int e = tid + P * i.value;
    const int sy = e / H;
    const int sx = e - sy * H;
    inten[sy * N + sx] = il[i.value];
  });
  static_for<0, N1>([&](auto x) { inten[(j + N2 * x.value) * N + H + v] = ir[x.value]; });
  __syncthreads();

  // S_k = sum of I over region k: wave w sums regions w, w + waves, ... over
  // natural pixels in a fixed order (lane stride 64, then a fixed butterfly)
  constexpr int NW = P / 64;  // whole waves (the last one has 32 lanes and sums nothing)
  const int wv = tid >> 6;
  const int lane = tid & 63;
  const int side = a.reg.s;
  for (int k = wv; wv < NW && k < a.reg.K; k += NW) {
    const int y0 = a.reg.y0[k];
    const int x0 = a.reg.x0[k];
    float acc = 0.f;
    for (int e = lane; e < side * side; e += 64) {
      const int dy = e / side;
      const int y = y0 + dy;
      const int x = x0 + (e - dy * side);
      acc += inten[PL::slot_of_pos(y) * N + PL::slot_of_pos(x)];
    }
    for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (lane == 0) a.sums_part[(size_t)b * a.reg.K + k] = acc;
  }
  if (a.intensity) {
    float* __restrict__ io = a.intensity + (size_t)b * nn;
    for (int e = tid; e < N * N; e += P) {
      const int y = e / N;
      const int x = e - y * N;
      const float in = inten[PL::slot_of_pos(y) * N + PL::slot_of_pos(x)];
      io[e] = a.accumulate ? io[e] + in : in;
    }
  }
}

template <int N>
constexpr bool whole_field_size() {
  return N == 64 || N == 100 || N == 128 || N == 200;
}

template <int N>
hipError_t launch_field_fwd_n(const FieldArgs& a, hipStream_t st) {
  if constexpr (whole_field_size<N>()) {
    using PL = typename PlanFor<N>::type;
    static_assert(std::is_same_v<PL, typename RowPlanFor<N>::type>, "one plan on both axes");
    if (a.batch < 1 || a.layers < 0 || a.layers > 64 || a.reg.K < 0 || a.reg.K > kMaxRegions ||
        (a.reg.K > 0 && !a.sums_part))
      return hipErrorInvalidValue;
    if constexpr (N == 200) {
      hipLaunchKernelGGL((field_forward_split_kernel<PL>), dim3(a.batch), dim3(SplitCfg<PL>::P), 0, st, a);
    } else {
      hipLaunchKernelGGL((field_forward_kernel<PL>), dim3(a.batch), dim3(PL::N * PL::N2), 0, st, a);
    }
    return hipGetLastError();
  } else {
    return hipErrorInvalidValue;
  }
}

// ---------------------------------------------------------------------------
// Helper kernels
// ---------------------------------------------------------------------------

// Column-permuted 2-D table for the angular-spectrum column pass:
// Hp[ky][c] = inv * H[ky][kx(c)] (inv = 1/N^2 for a propagation, 1 for the
// far-field table), c the slot of frequency kx in the row plan (the layout
// in which row passes store x-spectra).
template <class PL>
__global__ void prep_as_table_kernel(const float2* __restrict__ H, float2* __restrict__ Hp, float inv, int centred) {
  constexpr int N = PL::N;
  const size_t total = (size_t)N * N;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int ky = (int)(i / N);
    const int c = (int)(i - (size_t)ky * N);
    int kx;
    if (centred) {
      // column c holds frequency (c + N/2) mod N (the far field's centred order)
      kx = c + N / 2 < N ? c + N / 2 : c - N / 2;
    } else {
      // slot c holds element k2 of B-item k1
      const int k1 = c / PL::N2;
      const int k2 = c - k1 * PL::N2;
      kx = PL::freq(k1, k2);
    }
    Hp[i] = cscale(H[(size_t)ky * N + kx], inv);
  }
}

// ---------------------------------------------------------------------------
// Per-size launchers (explicitly instantiated in one translation unit per size)
// ---------------------------------------------------------------------------

// Vectors per workgroup by FFT length (the workgroup has T * N2 threads).
template <int N> struct TileT;
template <> struct TileT<64>   { static constexpr int T = 16; };
template <> struct TileT<100>  { static constexpr int T = 16; };
template <> struct TileT<128>  { static constexpr int T = 16; };
template <> struct TileT<200>  { static constexpr int T = 32; };  // detector-plane passes: 47.7 -> 45.7 and 30.6 -> 29.7 us against 16
template <> struct TileT<256>  { static constexpr int T = 8; };
template <> struct TileT<350>  { static constexpr int T = 32; };  // 14 slots: T * 14 threads must be whole waves
template <> struct TileT<400>  { static constexpr int T = 8; };
template <> struct TileT<500>  { static constexpr int T = 16; };  // 20 slots: T * 20 threads must be whole waves
template <> struct TileT<512>  { static constexpr int T = 8; };
template <> struct TileT<1000> { static constexpr int T = 8; };
template <> struct TileT<1024> { static constexpr int T = 8; };

template <int N>
using CfgFor = Cfg<typename PlanFor<N>::type, TileT<N>::T>;
template <int N>
using RowCfgFor = Cfg<typename RowPlanFor<N>::type, TileT<N>::T>;

// Vectors per workgroup of the separable layer passes, by kind and axis where
// a measured sweep preferred another width than the size default (fields and
// tables do not depend on it).
template <int N, int KIND, int AXIS>
struct LayerTile {
  static constexpr int T = TileT<N>::T;
};
template <> struct LayerTile<200, kFwdMid, kCol> { static constexpr int T = 32; };
template <> struct LayerTile<200, kPropOnce, kRow> { static constexpr int T = 32; };
template <> struct LayerTile<200, kBwdMid, kCol> { static constexpr int T = 16; };
template <> struct LayerTile<200, kFwdMid, kRow> { static constexpr int T = 8; };
template <> struct LayerTile<200, kBwdMid, kRow> { static constexpr int T = 8; };
template <> struct LayerTile<200, kBwdLast, kCol> { static constexpr int T = 32; };
// 400: the column layer passes at 16 vectors (pitch 17: the A-item and
// B-item reads of a 16-lane group fall in distinct bank pairs; at 8 vectors
// two B-items share each group's pairs), four-wave workgroups of 55 KB, 8
// waves per CU against 10; the row passes keep 8 (5-layer training step,
// batch 500: adjoint column passes 576 -> 485 us and 391 -> 337 us; rows at 16
// measured slower, 360 -> 380 us forward, and so did every pass at 512)
template <> struct LayerTile<400, kFwdMid, kCol> { static constexpr int T = 16; };
template <> struct LayerTile<400, kBwdMid, kCol> { static constexpr int T = 16; };
template <> struct LayerTile<400, kBwdLast, kCol> { static constexpr int T = 16; };
// 500: the forward passes in one ten-wave workgroup of 32 vectors per CU
// instead of one five-wave workgroup of 16 (a 68 KB five-wave workgroup
// leaves no room for a second one on a CU)
template <> struct LayerTile<500, kPropOnce, kRow> { static constexpr int T = 32; };
template <> struct LayerTile<500, kFwdMid, kRow> { static constexpr int T = 32; };
template <> struct LayerTile<500, kFwdMid, kCol> { static constexpr int T = 32; };
// 512: the first and the adjoint row passes at 16 vectors (5-layer training
// step, batch 500: 446 -> 429 and 1113 -> 1077 us, step 11.22 -> 11.11 ms)
template <> struct LayerTile<512, kPropOnce, kRow> { static constexpr int T = 16; };
template <> struct LayerTile<512, kBwdMid, kRow> { static constexpr int T = 16; };
template <> struct LayerTile<1000, kPropOnce, kRow> { static constexpr int T = 16; };
template <> struct LayerTile<1000, kFwdMid, kRow> { static constexpr int T = 16; };
template <> struct LayerTile<1000, kFwdMid, kCol> { static constexpr int T = 16; };
// (its detector-plane passes measured slower at 16: 185 -> 215 us for the seed
// pass of a 1000 x 1000 training step, batch 16)
// (the adjoint passes keep 16: at 32 their registers, capped at 168 for ten
// waves, spill, and the column pass measured slower; so do the detector-plane
// passes, which transform only the covered rows and measured slower at 32)

template <int N, int KIND, int AXIS>
using LayerCfg = Cfg<std::conditional_t<AXIS == kRow, typename RowPlanFor<N>::type, typename PlanFor<N>::type>,
                     LayerTile<N, KIND, AXIS>::T>;

// Layer kinds of a slot-ordered field run as wave tiles where the plan allows,
// along rows: there each wave's loads cover 8 whole 64-byte runs of its rows.
// Along columns a wave covers half of each 128-byte line and the other half
// is fetched again by the next tile (counters: 450 against 348 MB per
// forward layer pass at N = 200), so columns keep the workgroup tiles.
template <int N, int KIND, int AXIS>
constexpr bool wave_tile_kind() {
  using PL = typename PlanFor<N>::type;
  return AXIS == kRow && PL::N2 == 8 && std::is_same_v<PL, typename RowPlanFor<N>::type> &&
         (KIND == kFwdMid || KIND == kBwdMid || KIND == kBwdLast);
}

// Row layer kinds at 500 points run on the wide row tiles (wide_row_pass).
template <int N, int KIND, int AXIS>
constexpr bool wide_row_kind() {
  return N == 500 && AXIS == kRow && (KIND == kPropOnce || KIND == kFwdMid || KIND == kBwdMid);
}

template <int N, int KIND, int AXIS, bool FULL>
hipError_t launch_fr(const PassArgs& a, hipStream_t st) {
  if constexpr (FULL && wide_row_kind<N, KIND, AXIS>()) {
    if (a.workers < 1) return hipErrorInvalidValue;
    const dim3 grid(8 * ((a.workers + 7) / 8));
    hipLaunchKernelGGL((wide_row_pass<typename PlanFor<N>::type, KIND>), grid, dim3(64), 0, st, a);
  } else if constexpr (FULL && wave_tile_kind<N, KIND, AXIS>()) {
    if (a.workers < 1) return hipErrorInvalidValue;
    const dim3 grid(8 * ((a.workers + 7) / 8));
    hipLaunchKernelGGL((wave_pass<typename PlanFor<N>::type, KIND, AXIS>), grid, dim3(64), 0, st, a);
  } else if constexpr (KIND == kFwdLast || KIND == kBwdFirst) {
    using C = std::conditional_t<AXIS == kRow, RowCfgFor<N>, CfgFor<N>>;
    const dim3 grid(work_grid(a.ntiles, (a.batch + a.spg - 1) / a.spg));
    hipLaunchKernelGGL((detector_pass<C, KIND, AXIS, FULL>), grid, dim3(C::P), 0, st, a);
  } else {
    using C = LayerCfg<N, KIND, AXIS>;
    if (a.workers < 1) return hipErrorInvalidValue;
    const dim3 grid(8 * ((a.workers + 7) / 8));
    hipLaunchKernelGGL((fresnel_pass<C, KIND, AXIS, FULL>), grid, dim3(C::P), 0, st, a);
  }
  return hipGetLastError();
}

// Compute units of the current device (cached per device).
inline int device_cus() {
  static int cache[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cache[dev] == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cache[dev] = cus;
  }
  return cache[dev];
}

// Workgroups of a kernel resident per compute unit: the runtime's occupancy
// figure, capped by shared memory counted in its allocation granules (512
// bytes), which the occupancy query does not round to.
inline int resident_per_cu(const void* kernel, int block) {
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kernel, block, 0) != hipSuccess) return 0;
  hipFuncAttributes at;
  if (hipFuncGetAttributes(&at, kernel) != hipSuccess) return 0;
  int dev = 0;
  int lds_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) != hipSuccess)
    return 0;
  const size_t granule = 512;
  const size_t lds = (at.sharedSizeBytes + granule - 1) / granule * granule;
  if (lds > 0) nb = std::min(nb, static_cast<int>(static_cast<size_t>(lds_cu) / lds));
  return nb;
}

template <int N, int KIND, int AXIS, bool FULL>
int slots_fr() {
  static int per_cu = 0;
  if (per_cu == 0) {
    if constexpr (FULL && wide_row_kind<N, KIND, AXIS>()) {
      per_cu = resident_per_cu(reinterpret_cast<const void*>(&wide_row_pass<typename PlanFor<N>::type, KIND>), 64);
    } else if constexpr (FULL && wave_tile_kind<N, KIND, AXIS>()) {
      per_cu = resident_per_cu(reinterpret_cast<const void*>(&wave_pass<typename PlanFor<N>::type, KIND, AXIS>), 64);
    } else {
      using C = LayerCfg<N, KIND, AXIS>;
      per_cu = resident_per_cu(reinterpret_cast<const void*>(&fresnel_pass<C, KIND, AXIS, FULL>), C::P);
    }
  }
  return per_cu * device_cus();
}

template <int N, int KIND>
int slots_fr_axis(Axis axis, bool full) {
  if (full) return axis == kRow ? slots_fr<N, KIND, kRow, true>() : slots_fr<N, KIND, kCol, true>();
  return axis == kRow ? slots_fr<N, KIND, kRow, false>() : slots_fr<N, KIND, kCol, false>();
}

template <int N, int KIND>
int tile_fr_axis(Axis axis, bool full) {
  if constexpr (wide_row_kind<N, KIND, kRow>()) {
    if (axis == kRow && full) return WideRows<typename PlanFor<N>::type>::R;
  }
  if (axis == kRow) return full && wave_tile_kind<N, KIND, kRow>() ? 8 : LayerTile<N, KIND, kRow>::T;
  return full && wave_tile_kind<N, KIND, kCol>() ? 8 : LayerTile<N, KIND, kCol>::T;
}

// Vectors per workgroup of a separable pass.
template <int N>
int tile_fr_n(PassKind kind, Axis axis, bool full) {
  switch (kind) {
    case kPropOnce: return tile_fr_axis<N, kPropOnce>(axis, full);
    case kFwdMid: return tile_fr_axis<N, kFwdMid>(axis, full);
    case kBwdMid: return tile_fr_axis<N, kBwdMid>(axis, full);
    case kBwdLast: return tile_fr_axis<N, kBwdLast>(axis, full);
    default: return TileT<N>::T;  // detector-plane passes
  }
}

template <int N>
int slots_fr_n(PassKind kind, Axis axis, bool full) {
  switch (kind) {
    case kPropOnce: return slots_fr_axis<N, kPropOnce>(axis, full);
    case kFwdMid: return slots_fr_axis<N, kFwdMid>(axis, full);
    case kBwdMid: return slots_fr_axis<N, kBwdMid>(axis, full);
    case kBwdLast: return slots_fr_axis<N, kBwdLast>(axis, full);
    default: return 0;
  }
}

template <int N, int KIND>
hipError_t launch_fr_axis(Axis axis, const PassArgs& a, hipStream_t st) {
  if (a.full) return axis == kRow ? launch_fr<N, KIND, kRow, true>(a, st) : launch_fr<N, KIND, kCol, true>(a, st);
  return axis == kRow ? launch_fr<N, KIND, kRow, false>(a, st) : launch_fr<N, KIND, kCol, false>(a, st);
}

template <int N>
hipError_t launch_fr_n(PassKind kind, Axis axis, const PassArgs& a, hipStream_t st) {
  if (a.full && a.n != N) return hipErrorInvalidValue;
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
  using C = std::conditional_t<KIND == kAsCol || KIND == kAsColFar, CfgFor<N>, RowCfgFor<N>>;
  const dim3 grid(work_grid(a.ntiles, (a.batch + a.spg - 1) / a.spg));
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
    case kAsColFar: return launch_as<N, kAsColFar>(a, st);
  }
  return hipErrorInvalidValue;
}

template <int N>
hipError_t prep_as_n(const float2* H, float2* Hp, float scale, int centred, hipStream_t st) {
  if (centred && (N & 1)) return hipErrorInvalidValue;
  const int blocks = (int)(((size_t)N * N + 255) / 256);
  hipLaunchKernelGGL((prep_as_table_kernel<typename RowPlanFor<N>::type>), dim3(blocks < 4096 ? blocks : 4096), dim3(256),
                     0, st, H, Hp, scale, centred);
  return hipGetLastError();
}

template <int N>
TileShape shape_n() { return TileShape{CfgFor<N>::T, CfgFor<N>::S}; }

// The slot order of the separable passes' stored fields: rows and columns
// use the same plan, so one map serves both axes.
template <int N>
SlotMap slot_map_n() {
  using PL = typename PlanFor<N>::type;
  static_assert(std::is_same_v<PL, typename RowPlanFor<N>::type>, "stored slot order needs one plan for both axes");
  return SlotMap{PL::N1, PL::N2, PL::PFA ? 1 : 0};
}

}  // namespace lr
