// Helper kernels and the size dispatch of the pass kernels.
#include <hip/hip_runtime.h>

#include "kernels.hpp"
#include "tile.hpp"

namespace lr {

// Per-size entry points, defined in kern_size.hip (one object per size).
template <int N> hipError_t launch_fr_n(PassKind, Axis, const PassArgs&, hipStream_t);
template <int N> int slots_fr_n(PassKind, Axis, bool);
template <int N> int tile_fr_n(PassKind, Axis, bool);
template <int N> hipError_t launch_as_n(AsPassKind, const PassArgs&, hipStream_t);
template <int N> hipError_t prep_as_n(const float2*, float2*, float, int, hipStream_t);
template <int N> TileShape shape_n();
template <int N> SlotMap slot_map_n();
template <int N> hipError_t launch_field_fwd_n(const FieldArgs&, hipStream_t);

// ---------------------------------------------------------------------------
// Helper kernels
// ---------------------------------------------------------------------------

struct OrientArg { int o[64]; };

// mod[l][sq][sv] = gamma * exp(j*phi_l[y][x]) with (q, vec) = (sm.pos(sq),
// sm.pos(sv)) and (y, x) = (q, vec), or (vec, q) when transposed.
__device__ __forceinline__ void prep_mod_body(const float* __restrict__ phi, int layers, int n, float gamma,
                                              const OrientArg& orient, SlotMap sm, float2* __restrict__ mod) {
  const size_t nn = (size_t)n * n;
  const size_t total = nn * layers;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int l = (int)(i / nn);
    const size_t r = i - (size_t)l * nn;
    const int sq = (int)(r / n);
    const int q = sm.pos(sq);
    const int vec = sm.pos((int)(r - (size_t)sq * n));
    const bool tr = orient.o[l < 64 ? l : 63] != 0;
    const int y = tr ? vec : q;
    const int x = tr ? q : vec;
    float s, c;
    sincosf(phi[(size_t)l * nn + (size_t)y * n + x], &s, &c);
    mod[i] = c2(gamma * c, gamma * s);
  }
}

__global__ void finish_sums_kernel(const float* __restrict__ part, int batch, int ntiles, int K, float* __restrict__ sums,
                                   int accumulate) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= batch * K) return;
  const int b = i / K;
  const int k = i - b * K;
  float s = 0.f;
  for (int tl = 0; tl < ntiles; ++tl) s += part[((size_t)b * ntiles + tl) * K + k];
  sums[i] = accumulate ? sums[i] + s : s;
}

// Loss of the detector sums, averaged over the batch, and its gradient
// dL/dS.  kind 0: softmax cross-entropy, -log p_t.  kind 1: the paper's
// ||softmax(S) - onehot(t)||^2, whose gradient goes through the softmax
// Jacobian: dL/dS_j = p_j (d_j - sum_i d_i p_i), d = 2 (p - t) / B.
// One workgroup; sample b is handled by thread b % 1024 and the per-thread
// losses are summed in a fixed order.  An out-of-range label makes the loss NaN.
__global__ void __launch_bounds__(1024) loss_kernel(int kind, const float* __restrict__ sums,
                                                    const int32_t* __restrict__ labels, int batch, int K,
                                                    float* __restrict__ grad, float* __restrict__ loss) {
  __shared__ float red[16];
  float my = 0.f;
  const float invb = 1.0f / (float)batch;
  for (int b = threadIdx.x; b < batch; b += 1024) {
    const float* s = sums + (size_t)b * K;
    float mx = s[0];
    for (int k = 1; k < K; ++k) mx = fmaxf(mx, s[k]);
    float z = 0.f;
    for (int k = 0; k < K; ++k) z += expf(s[k] - mx);
    const float lz = logf(z);
    const int tl = labels[b];
    const bool valid = (unsigned)tl < (unsigned)K;
    float lb;
    if (kind == 0) {
      lb = lz + mx - (valid ? s[tl] : 0.f);
      if (grad) {
        for (int k = 0; k < K; ++k) grad[(size_t)b * K + k] = (expf(s[k] - mx - lz) - (k == tl ? 1.f : 0.f)) * invb;
      }
    } else {
      lb = 0.f;
      float c = 0.f;  // sum_i d_i p_i
      for (int k = 0; k < K; ++k) {
        const float p = expf(s[k] - mx - lz);
        const float r = p - (k == tl ? 1.f : 0.f);
        lb += r * r;
        c += 2.f * r * invb * p;
      }
      if (grad) {
        for (int k = 0; k < K; ++k) {
          const float p = expf(s[k] - mx - lz);
          const float d = 2.f * (p - (k == tl ? 1.f : 0.f)) * invb;
          grad[(size_t)b * K + k] = p * (d - c);
        }
      }
    }
    my += valid ? lb : __builtin_nanf("");
  }
  const float tot = block_sum<1024>(my, red);
  if (threadIdx.x == 0 && loss) *loss = tot * invb;
}

// One Adam step on every element: m = b1 m + (1-b1) g, v = b2 v + (1-b2) g^2,
// phi -= lr * (m / bc1) / (sqrt(v / bc2) + eps), bc = 1 - beta^t.
// Codesign layer (§3.2): per pixel, w = softmax((logits + noise) / tau) over
// the K device levels; the phase is sum_k w_k levels_k, or (hard) the level
// of the largest logits + noise, the first on ties.  One wave per pixel; lane
// l handles levels l, l + 64, ...; the scores are read coalesced.
constexpr int kCodesignMaxLevels = 1024;

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ int wave_min_int(int x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = min(x, __shfl_xor(x, o, 64));
  return x;
}

// Per-pixel softmax statistics: max of y = (logits + noise) / tau, the first
// level index reaching the largest logits + noise, and sum_k exp(y_k - max).
// The scores of a pixel are read once into registers: lane l holds
// s[i] = logits + noise of level l + 64 i, i < NI = ceil(K / 64) (-inf past K).
struct CodesignStats {
  float ymax;
  int kbest;
  float esum;
};
template <int NI>
__device__ __forceinline__ void codesign_load(const float* __restrict__ lg, const float* __restrict__ nz, int K,
                                              int lane, float (&sc)[NI]) {
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int k = lane + 64 * i;
    sc[i] = k < K ? lg[k] + nz[k] : -INFINITY;
  }
}
template <int NI>
__device__ __forceinline__ CodesignStats codesign_stats(const float (&sc)[NI], int K, float inv_tau, int lane) {
  float smax = -INFINITY;
#pragma unroll
  for (int i = 0; i < NI; ++i) smax = fmaxf(smax, sc[i]);
  smax = wave_max(smax);
  int kb = K;
#pragma unroll
  for (int i = NI - 1; i >= 0; --i) {
    const int k = lane + 64 * i;
    if (k < K && sc[i] == smax) kb = k;  // the lowest level of this lane reaching the maximum
  }
  kb = wave_min_int(kb);
  const float ymax = smax * inv_tau;
  float es = 0.f;
#pragma unroll
  for (int i = 0; i < NI; ++i)
    if (lane + 64 * i < K) es += expf(sc[i] * inv_tau - ymax);
  return CodesignStats{ymax, kb, wave_sum(es)};
}

template <int NI>
__global__ void __launch_bounds__(256) codesign_kernel(const float* __restrict__ logits, const float* __restrict__ noise,
                                                       const float* __restrict__ levels, int K, long long count,
                                                       float inv_tau, int hard, float* __restrict__ phi) {
  const int lane = threadIdx.x & 63;
  const long long waves = (long long)gridDim.x * (blockDim.x >> 6);
  for (long long p = (long long)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); p < count; p += waves) {
    float sc[NI];
    codesign_load<NI>(logits + p * K, noise + p * K, K, lane, sc);
    const CodesignStats cs = codesign_stats<NI>(sc, K, inv_tau, lane);
    float out;
    if (hard) {
      out = levels[cs.kbest < K ? cs.kbest : 0];  // (no index reaches the maximum only for NaN scores)
    } else {
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int k = lane + 64 * i;
        if (k < K) acc += expf(sc[i] * inv_tau - cs.ymax) * levels[k];
      }
      out = wave_sum(acc) / cs.esum;
    }
    if (lane == 0) phi[p] = out;
  }
}

// dL/dlogit_j = w_j (levels_j - sum_k w_k levels_k) dL/dphi / tau (the soft
// Jacobian, also the straight-through gradient of the hard layer).
template <int NI>
__global__ void __launch_bounds__(256) codesign_bwd_kernel(const float* __restrict__ logits,
                                                           const float* __restrict__ noise,
                                                           const float* __restrict__ levels, int K, long long count,
                                                           float inv_tau, const float* __restrict__ grad_phi,
                                                           float* __restrict__ grad_logits) {
  const int lane = threadIdx.x & 63;
  const long long waves = (long long)gridDim.x * (blockDim.x >> 6);
  for (long long p = (long long)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); p < count; p += waves) {
    float sc[NI];
    codesign_load<NI>(logits + p * K, noise + p * K, K, lane, sc);
    const CodesignStats cs = codesign_stats<NI>(sc, K, inv_tau, lane);
    const float inv_s = 1.f / cs.esum;
    float acc = 0.f;
    float lv[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int k = lane + 64 * i;
      lv[i] = k < K ? levels[k] : 0.f;
      if (k < K) acc += expf(sc[i] * inv_tau - cs.ymax) * lv[i];
    }
    const float mean = wave_sum(acc) * inv_s;
    const float gs = grad_phi[p] * inv_tau;
    float* gl = grad_logits + p * K;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int k = lane + 64 * i;
      if (k < K) {
        const float w = expf(sc[i] * inv_tau - cs.ymax) * inv_s;
        gl[k] = w * (lv[i] - mean) * gs;
      }
    }
  }
}

template <int NI>
static void launch_codesign_ni(const float* logits, const float* noise, const float* levels, int K, long long count,
                               float tau, int hard, const float* grad_phi, float* phi_or_grad, unsigned blocks,
                               hipStream_t st) {
  if (grad_phi) {
    hipLaunchKernelGGL(codesign_bwd_kernel<NI>, dim3(blocks), dim3(256), 0, st, logits, noise, levels, K, count,
                       1.f / tau, grad_phi, phi_or_grad);
  } else {
    hipLaunchKernelGGL(codesign_kernel<NI>, dim3(blocks), dim3(256), 0, st, logits, noise, levels, K, count, 1.f / tau,
                       hard, phi_or_grad);
  }
}

__global__ void adam_kernel(float* __restrict__ phi, const float* __restrict__ g, float* __restrict__ m,
                            float* __restrict__ v, long long count, float lr, float b1, float b2, float eps,
                            float bc1, float bc2) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < count;
       i += (long long)gridDim.x * blockDim.x) {
    const float gi = g[i];
    const float mi = b1 * m[i] + (1.f - b1) * gi;
    const float vi = b2 * v[i] + (1.f - b2) * gi * gi;
    m[i] = mi;
    v[i] = vi;
    phi[i] -= lr * (mi / bc1) / (sqrtf(vi / bc2) + eps);
  }
}

// dphi_l[y][x] = sum over groups of part_l[g][sq][sv], oriented (transposed:
// q = x) and in the slot order sm ((q, vec) = (sm.pos(sq), sm.pos(sv))), for
// every layer l = blockIdx.y in one launch; part_l starts at
// part + l * layer_stride.  A workgroup covers 64 consecutive elements with 4
// slices of 64 threads; slice s sums groups s, s+4, s+8, ... in order and the
// four partial sums are added in slice order, so the result does not depend
// on scheduling.  A layer with no groups gets zeros.
struct ReduceArg {
  int groups[64];
  int transposed[64];
};
__global__ void __launch_bounds__(256) reduce_dphi_kernel(const float* __restrict__ part, size_t layer_stride,
                                                          ReduceArg arg, int n, SlotMap sm, float* __restrict__ out) {
  __shared__ float red[4][64];
  const int l = blockIdx.y;
  const int groups = arg.groups[l];
  const float* __restrict__ pl = part + (size_t)l * layer_stride;
  const size_t nn = (size_t)n * n;
  const int lane = threadIdx.x & 63;
  const int slice = threadIdx.x >> 6;
  const size_t i = (size_t)blockIdx.x * 64 + lane;
  float s = 0.f;
  if (i < nn) {
    int g = slice;
    for (; g + 12 < groups; g += 16) {
      const float a0 = pl[(size_t)g * nn + i];
      const float a1 = pl[(size_t)(g + 4) * nn + i];
      const float a2 = pl[(size_t)(g + 8) * nn + i];
      const float a3 = pl[(size_t)(g + 12) * nn + i];
      s += a0;
      s += a1;
      s += a2;
      s += a3;
    }
    for (; g < groups; g += 4) s += pl[(size_t)g * nn + i];
  }
  red[slice][lane] = s;
  __syncthreads();
  if (slice == 0 && i < nn) {
    const float r = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
    const int sq = (int)(i / n);
    const int q = sm.pos(sq);
    const int v = sm.pos((int)(i - (size_t)sq * n));
    out[(size_t)l * nn + (arg.transposed[l] ? (size_t)v * n + q : (size_t)q * n + v)] = r;
  }
}

// Region corners, per-row / per-column coverage masks (natural indices) and
// the covered-first permutations of the stored rows and columns (slot order
// sm): stored indices whose natural row / column a region covers, in
// ascending order, then the others.  Run by one workgroup of 1024 threads,
// thread i handles row i and column i (n <= 1024).
__device__ void set_regions_body(const Regions& reg, int n, SlotMap sm, int2* dst, unsigned long long* row_mask,
                                 unsigned long long* col_mask, int* row_perm, int* col_perm, int (*wave_count)[16]) {
  const int i = threadIdx.x;
  if (i < reg.K) dst[i] = make_int2(reg.y0[i], reg.x0[i]);
  auto masks = [&](int p, unsigned long long& rm, unsigned long long& cm) {
    rm = 0;
    cm = 0;
    for (int k = 0; k < reg.K; ++k) {
      if ((unsigned)(p - reg.y0[k]) < (unsigned)reg.s) rm |= 1ull << k;
      if ((unsigned)(p - reg.x0[k]) < (unsigned)reg.s) cm |= 1ull << k;
    }
  };
  unsigned long long rm = 0, cm = 0;
  if (i < n) {
    masks(i, rm, cm);
    row_mask[i] = rm;
    col_mask[i] = cm;
    masks(sm.pos(i), rm, cm);  // coverage of stored index i
  }
  const bool rc = i < n && rm != 0;
  const bool cc = i < n && cm != 0;
  const int lane = i & 63;
  const int wave = i >> 6;
  const unsigned long long rb = __ballot(rc);
  const unsigned long long cb = __ballot(cc);
  const unsigned long long below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  if (lane == 0) {
    wave_count[0][wave] = __popcll(rb);
    wave_count[1][wave] = __popcll(cb);
  }
  __syncthreads();
  int r_rank = __popcll(rb & below), c_rank = __popcll(cb & below), r_total = 0, c_total = 0;
  for (int w = 0; w < 16; ++w) {
    if (w < wave) {
      r_rank += wave_count[0][w];
      c_rank += wave_count[1][w];
    }
    r_total += wave_count[0][w];
    c_total += wave_count[1][w];
  }
  if (i < n) {
    // r_rank = covered rows before i, so i - r_rank uncovered rows precede it
    row_perm[rc ? r_rank : r_total + (i - r_rank)] = i;
    col_perm[cc ? c_rank : c_total + (i - c_rank)] = i;
  }
}

// Separable Fresnel chirps in natural frequency order from the 2-D table H
// (N x N): x chirp H[0][f], y chirp H[f][0] * conj(H[0][0]) (so the two
// carry exp(jkz) once), each with the 1/N of the inverse DFT folded in.
__device__ __forceinline__ void prep_chirps_body(const float2* __restrict__ H, int N, float2* __restrict__ cx,
                                                 float2* __restrict__ cy) {
  const float inv = 1.0f / (float)N;
  const float2 h00c = c2(H[0].x, -H[0].y);
  for (int f = blockIdx.x * blockDim.x + threadIdx.x; f < N; f += gridDim.x * blockDim.x) {
    cx[f] = cscale(H[f], inv);
    cy[f] = cscale(cmul(H[(size_t)f * N], h00c), inv);
  }
}

// Per-call tables in one launch: the modulation of every layer (all
// workgroups), the separable chirps when H is given, and, when the call reads
// detector regions, the region tables (workgroup 0).  Workgroups of 1024
// threads.
__global__ void __launch_bounds__(1024) prep_layers_kernel(const float* __restrict__ phi, int layers, int n, float gamma,
                                                           OrientArg orient, SlotMap sm, float2* __restrict__ mod,
                                                           Regions reg,
                                                           int2* dst, unsigned long long* row_mask,
                                                           unsigned long long* col_mask, int* row_perm, int* col_perm,
                                                           const float2* __restrict__ H, int nfft,
                                                           float2* __restrict__ cx, float2* __restrict__ cy) {
  __shared__ int wave_count[2][16];
  if (blockIdx.x == 0 && dst) set_regions_body(reg, n, sm, dst, row_mask, col_mask, row_perm, col_perm, wave_count);
  if (H) prep_chirps_body(H, nfft, cx, cy);
  if (phi) prep_mod_body(phi, layers, n, gamma, orient, sm, mod);
}

// Detector readout from a field: one workgroup per (sample, region).
__global__ void __launch_bounds__(256) readout_kernel(const float2* __restrict__ field, int n, Regions reg,
                                                      float* __restrict__ sums) {
  __shared__ float red[4];
  const int b = blockIdx.y;
  const int k = blockIdx.x;
  const int K = reg.K;
  const int s = reg.s;
  const float2* f = field + (size_t)b * n * n;
  const int ry = reg.y0[k];
  const int rx = reg.x0[k];
  float my = 0.f;
  for (int e = threadIdx.x; e < s * s; e += 256) {
    const int dy = e / s;
    const int dx = e - dy * s;
    my += cabs2(f[(size_t)(ry + dy) * n + rx + dx]);
  }
  const float tot = block_sum<256>(my, red);
  if (threadIdx.x == 0) sums[(size_t)b * K + k] = tot;
}

// ---------------------------------------------------------------------------
// Dispatch
// ---------------------------------------------------------------------------

bool fft_size_supported(int N) {
  switch (N) {
    case 64:
    case 100:
    case 128:
    case 200:
    case 256:
    case 350:
    case 400:
    case 500:
    case 512:
    case 1000:
    case 1024:
      return true;
    default:
      return false;
  }
}

TileShape tile_shape(int N, int) {
  switch (N) {
    case 64: return shape_n<64>();
    case 100: return shape_n<100>();
    case 128: return shape_n<128>();
    case 200: return shape_n<200>();
    case 256: return shape_n<256>();
    case 350: return shape_n<350>();
    case 400: return shape_n<400>();
    case 500: return shape_n<500>();
    case 512: return shape_n<512>();
    case 1000: return shape_n<1000>();
    case 1024: return shape_n<1024>();
    default: return TileShape{0, 0};
  }
}

SlotMap slot_map(int N) {
  switch (N) {
    case 64: return slot_map_n<64>();
    case 100: return slot_map_n<100>();
    case 128: return slot_map_n<128>();
    case 200: return slot_map_n<200>();
    case 256: return slot_map_n<256>();
    case 350: return slot_map_n<350>();
    case 400: return slot_map_n<400>();
    case 500: return slot_map_n<500>();
    case 512: return slot_map_n<512>();
    case 1000: return slot_map_n<1000>();
    case 1024: return slot_map_n<1024>();
    default: return SlotMap{0, 0, 0};
  }
}

bool wide_row_tiles(int N) { return N == 500; }

bool field_forward_supported(int N) { return N == 64 || N == 100 || N == 128 || N == 200; }

bool field_forward_preferred(int N, int batch) {
  if (!field_forward_supported(N) || N == 200) return false;
  if (N == 64) return true;
  int dev = 0;
  int cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    return false;
  return batch >= cus;
}

hipError_t launch_field_forward(int N, const FieldArgs& a, hipStream_t st) {
  switch (N) {
    case 64: return launch_field_fwd_n<64>(a, st);
    case 100: return launch_field_fwd_n<100>(a, st);
    case 128: return launch_field_fwd_n<128>(a, st);
    case 200: return launch_field_fwd_n<200>(a, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_fresnel_pass(int N, PassKind kind, Axis axis, const PassArgs& a, hipStream_t st) {
  switch (N) {
    case 64: return launch_fr_n<64>(kind, axis, a, st);
    case 100: return launch_fr_n<100>(kind, axis, a, st);
    case 128: return launch_fr_n<128>(kind, axis, a, st);
    case 200: return launch_fr_n<200>(kind, axis, a, st);
    case 256: return launch_fr_n<256>(kind, axis, a, st);
    case 350: return launch_fr_n<350>(kind, axis, a, st);
    case 400: return launch_fr_n<400>(kind, axis, a, st);
    case 500: return launch_fr_n<500>(kind, axis, a, st);
    case 512: return launch_fr_n<512>(kind, axis, a, st);
    case 1000: return launch_fr_n<1000>(kind, axis, a, st);
    case 1024: return launch_fr_n<1024>(kind, axis, a, st);
    default: return hipErrorInvalidValue;
  }
}

int fresnel_pass_tile(int N, PassKind kind, Axis axis, bool full) {
  switch (N) {
    case 64: return tile_fr_n<64>(kind, axis, full);
    case 100: return tile_fr_n<100>(kind, axis, full);
    case 128: return tile_fr_n<128>(kind, axis, full);
    case 200: return tile_fr_n<200>(kind, axis, full);
    case 256: return tile_fr_n<256>(kind, axis, full);
    case 350: return tile_fr_n<350>(kind, axis, full);
    case 400: return tile_fr_n<400>(kind, axis, full);
    case 500: return tile_fr_n<500>(kind, axis, full);
    case 512: return tile_fr_n<512>(kind, axis, full);
    case 1000: return tile_fr_n<1000>(kind, axis, full);
    case 1024: return tile_fr_n<1024>(kind, axis, full);
    default: return 0;
  }
}

int fresnel_pass_slots(int N, PassKind kind, Axis axis, bool full) {
  switch (N) {
    case 64: return slots_fr_n<64>(kind, axis, full);
    case 100: return slots_fr_n<100>(kind, axis, full);
    case 128: return slots_fr_n<128>(kind, axis, full);
    case 200: return slots_fr_n<200>(kind, axis, full);
    case 256: return slots_fr_n<256>(kind, axis, full);
    case 350: return slots_fr_n<350>(kind, axis, full);
    case 400: return slots_fr_n<400>(kind, axis, full);
    case 500: return slots_fr_n<500>(kind, axis, full);
    case 512: return slots_fr_n<512>(kind, axis, full);
    case 1000: return slots_fr_n<1000>(kind, axis, full);
    case 1024: return slots_fr_n<1024>(kind, axis, full);
    default: return 0;
  }
}

hipError_t launch_as_pass(int N, AsPassKind kind, const PassArgs& a, hipStream_t st) {
  switch (N) {
    case 64: return launch_as_n<64>(kind, a, st);
    case 100: return launch_as_n<100>(kind, a, st);
    case 128: return launch_as_n<128>(kind, a, st);
    case 200: return launch_as_n<200>(kind, a, st);
    case 256: return launch_as_n<256>(kind, a, st);
    case 350: return launch_as_n<350>(kind, a, st);
    case 400: return launch_as_n<400>(kind, a, st);
    case 500: return launch_as_n<500>(kind, a, st);
    case 512: return launch_as_n<512>(kind, a, st);
    case 1000: return launch_as_n<1000>(kind, a, st);
    case 1024: return launch_as_n<1024>(kind, a, st);
    default: return hipErrorInvalidValue;
  }
}


hipError_t launch_prep_as_table(int N, const float2* H, float2* Hp, float scale, int centred, hipStream_t st) {
  switch (N) {
    case 64: return prep_as_n<64>(H, Hp, scale, centred, st);
    case 100: return prep_as_n<100>(H, Hp, scale, centred, st);
    case 128: return prep_as_n<128>(H, Hp, scale, centred, st);
    case 200: return prep_as_n<200>(H, Hp, scale, centred, st);
    case 256: return prep_as_n<256>(H, Hp, scale, centred, st);
    case 350: return prep_as_n<350>(H, Hp, scale, centred, st);
    case 400: return prep_as_n<400>(H, Hp, scale, centred, st);
    case 500: return prep_as_n<500>(H, Hp, scale, centred, st);
    case 512: return prep_as_n<512>(H, Hp, scale, centred, st);
    case 1000: return prep_as_n<1000>(H, Hp, scale, centred, st);
    case 1024: return prep_as_n<1024>(H, Hp, scale, centred, st);
    default: return hipErrorInvalidValue;
  }
}

// ---------------------------------------------------------------------------
// Layer normalisation of intensity maps (per sample, over count values).
// Chunk c of sample b covers values [c * kLnChunk, min(count, (c+1) * kLnChunk)).
// ---------------------------------------------------------------------------
constexpr int kLnThreads = 256;

// g == nullptr: part = (chunk mean, sum of squared deviations from it);
// otherwise part = (sum of g, sum of g * y) with y = x the normalised map.
__global__ void __launch_bounds__(kLnThreads) ln_partial_kernel(const float* __restrict__ x,
                                                                const float* __restrict__ g, long long count,
                                                                int nchunks, float2* __restrict__ part) {
  __shared__ float red[kLnThreads / 64];
  const int c = blockIdx.x;
  const int b = blockIdx.y;
  const size_t base = (size_t)b * (size_t)count;
  const long long lo = (long long)c * kLnChunk;
  const long long hi = min(count, lo + kLnChunk);
  float s1 = 0.f;
  float s2 = 0.f;
  if (g == nullptr) {
    for (long long i = lo + threadIdx.x; i < hi; i += kLnThreads) s1 += x[base + i];
    const float mean = block_sum<kLnThreads>(s1, red) / (float)(hi - lo);
    for (long long i = lo + threadIdx.x; i < hi; i += kLnThreads) {
      const float d = x[base + i] - mean;
      s2 += d * d;
    }
    const float m2 = block_sum<kLnThreads>(s2, red);
    if (threadIdx.x == 0) part[(size_t)b * nchunks + c] = c2(mean, m2);
  } else {
    for (long long i = lo + threadIdx.x; i < hi; i += kLnThreads) {
      const float gv = g[base + i];
      s1 += gv;
      s2 += gv * x[base + i];
    }
    const float a = block_sum<kLnThreads>(s1, red);
    const float bsum = block_sum<kLnThreads>(s2, red);
    if (threadIdx.x == 0) part[(size_t)b * nchunks + c] = c2(a, bsum);
  }
}

// One thread per sample combines its chunks in order.  Forward: the chunk
// means and squared-deviation sums merge by the pairwise update of Chan et
// al.; stats = (mean, 1/sqrt(M2 / count + eps)).  Backward: stats2 =
// (mean of g, mean of g * y).
__global__ void ln_combine_kernel(const float2* __restrict__ part, int batch, long long count, int nchunks,
                                  float eps, int backward, float2* __restrict__ out) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= batch) return;
  const float2* p = part + (size_t)b * nchunks;
  if (backward) {
    float a = 0.f;
    float m = 0.f;
    for (int c = 0; c < nchunks; ++c) {
      a += p[c].x;
      m += p[c].y;
    }
    out[b] = c2(a / (float)count, m / (float)count);
    return;
  }
  float n_a = 0.f;
  float mean = 0.f;
  float m2 = 0.f;
  for (int c = 0; c < nchunks; ++c) {
    const long long lo = (long long)c * kLnChunk;
    const float n_b = (float)(min(count, lo + kLnChunk) - lo);
    const float n = n_a + n_b;
    const float delta = p[c].x - mean;
    mean += delta * (n_b / n);
    m2 += p[c].y + delta * delta * (n_a * n_b / n);
    n_a = n;
  }
  out[b] = c2(mean, 1.f / sqrtf(m2 / (float)count + eps));
}

// Forward: y = (x - mean) * rstd.  Backward (g != nullptr, x = y the
// normalised map): dx = rstd * (g - mean(g) - y * mean(g * y)).
__global__ void ln_apply_kernel(const float* __restrict__ x, const float* __restrict__ g,
                                const float2* __restrict__ stats, const float2* __restrict__ stats2, int batch,
                                long long count, float* __restrict__ out) {
  const size_t total = (size_t)batch * (size_t)count;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const size_t b = i / (size_t)count;
    const float2 s = stats[b];
    if (g == nullptr) {
      out[i] = (x[i] - s.x) * s.y;
    } else {
      const float2 s2 = stats2[b];
      out[i] = s.y * (g[i] - s2.x - x[i] * s2.y);
    }
  }
}

static int ln_apply_blocks(size_t total) {
  size_t blocks = (total + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  return blocks < 1 ? 1 : (int)blocks;
}

hipError_t launch_layer_norm(const float* x, int batch, long long count, float eps, float* y, float2* stats,
                             float2* part, hipStream_t st) {
  if (batch < 1 || batch > 65535 || count < 1 || ln_chunks(count) > (1 << 30)) return hipErrorInvalidValue;
  const int nchunks = (int)ln_chunks(count);
  hipLaunchKernelGGL(ln_partial_kernel, dim3(nchunks, batch), dim3(kLnThreads), 0, st, x, nullptr, count, nchunks,
                     part);
  hipLaunchKernelGGL(ln_combine_kernel, dim3((batch + 63) / 64), dim3(64), 0, st, part, batch, count, nchunks, eps, 0,
                     stats);
  hipLaunchKernelGGL(ln_apply_kernel, dim3(ln_apply_blocks((size_t)batch * count)), dim3(256), 0, st, x, nullptr,
                     stats, nullptr, batch, count, y);
  return hipGetLastError();
}

hipError_t launch_layer_norm_backward(const float* g, const float* y, const float2* stats, int batch,
                                      long long count, float* dx, float2* part, float2* stats2, hipStream_t st) {
  if (batch < 1 || batch > 65535 || count < 1 || ln_chunks(count) > (1 << 30)) return hipErrorInvalidValue;
  const int nchunks = (int)ln_chunks(count);
  hipLaunchKernelGGL(ln_partial_kernel, dim3(nchunks, batch), dim3(kLnThreads), 0, st, y, g, count, nchunks, part);
  hipLaunchKernelGGL(ln_combine_kernel, dim3((batch + 63) / 64), dim3(64), 0, st, part, batch, count, nchunks, 0.f, 1,
                     stats2);
  hipLaunchKernelGGL(ln_apply_kernel, dim3(ln_apply_blocks((size_t)batch * count)), dim3(256), 0, st, y, g, stats,
                     stats2, batch, count, dx);
  return hipGetLastError();
}

hipError_t launch_prep_layers(const float* phi, int layers, int n, float gamma, const int* orient_host, SlotMap sm,
                              float2* mod, const Regions* regions, int2* dst, unsigned long long* row_mask,
                              unsigned long long* col_mask, int* row_perm, int* col_perm, const float2* H, int nfft,
                              float2* chirp_x, float2* chirp_y, hipStream_t st) {
  if (n < 1 || n > 1024 || layers < 0 || layers > 64 || (H && (nfft < n || !chirp_x || !chirp_y)))
    return hipErrorInvalidValue;
  if (sm.N1 != 0 && sm.N1 * sm.N2 != n) return hipErrorInvalidValue;
  if (regions && (regions->K < 1 || regions->K > kMaxRegions)) return hipErrorInvalidValue;
  OrientArg o{};
  for (int l = 0; l < layers; ++l) o.o[l] = orient_host[l];
  Regions r{};
  if (regions) r = *regions;
  const size_t total = (size_t)n * n * layers;
  int blocks = (int)((total + 1023) / 1024);
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(prep_layers_kernel, dim3(blocks), dim3(1024), 0, st, layers > 0 ? phi : nullptr, layers, n,
                     gamma, o, sm, mod, r, regions ? dst : nullptr, row_mask, col_mask, row_perm, col_perm, H, nfft,
                     chirp_x, chirp_y);
  return hipGetLastError();
}

hipError_t launch_finish_sums(const float* part, int batch, int ntiles, int K, float* sums, int accumulate,
                              hipStream_t st) {
  const int total = batch * K;
  hipLaunchKernelGGL(finish_sums_kernel, dim3((total + 255) / 256), dim3(256), 0, st, part, batch, ntiles, K, sums,
                     accumulate);
  return hipGetLastError();
}

hipError_t launch_loss(int kind, const float* sums, const int32_t* labels, int batch, int K, float* grad, float* loss,
                       hipStream_t st) {
  hipLaunchKernelGGL(loss_kernel, dim3(1), dim3(1024), 0, st, kind, sums, labels, batch, K, grad, loss);
  return hipGetLastError();
}

hipError_t launch_codesign(const float* logits, const float* noise, const float* levels, int K, long long count,
                           float tau, int hard, const float* grad_phi, float* phi_or_grad, hipStream_t st) {
  if (K < 1 || K > kCodesignMaxLevels) return hipErrorInvalidValue;
  if (count <= 0) return hipSuccess;
  long long blocks = (count + 3) / 4;  // four pixels (waves) per workgroup
  if (blocks > 65536) blocks = 65536;
  const unsigned nb = (unsigned)blocks;
  // registers per lane for the scores: ceil(K / 64) (K <= 1024)
  switch ((K + 63) / 64) {
    case 1: launch_codesign_ni<1>(logits, noise, levels, K, count, tau, hard, grad_phi, phi_or_grad, nb, st); break;
    case 2: launch_codesign_ni<2>(logits, noise, levels, K, count, tau, hard, grad_phi, phi_or_grad, nb, st); break;
    case 3:
    case 4: launch_codesign_ni<4>(logits, noise, levels, K, count, tau, hard, grad_phi, phi_or_grad, nb, st); break;
    case 5:
    case 6:
    case 7:
    case 8: launch_codesign_ni<8>(logits, noise, levels, K, count, tau, hard, grad_phi, phi_or_grad, nb, st); break;
    default: launch_codesign_ni<16>(logits, noise, levels, K, count, tau, hard, grad_phi, phi_or_grad, nb, st); break;
  }
  return hipGetLastError();
}

hipError_t launch_adam(float* phi, const float* g, float* m, float* v, long long count, float lr, float b1, float b2,
                       float eps, float bc1, float bc2, hipStream_t st) {
  if (count <= 0) return hipSuccess;
  long long blocks = (count + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(adam_kernel, dim3((unsigned)blocks), dim3(256), 0, st, phi, g, m, v, count, lr, b1, b2, eps, bc1,
                     bc2);
  return hipGetLastError();
}

hipError_t launch_reduce_dphi(const float* part, size_t layer_stride, const int* groups, const int* transposed,
                              int layers, int n, SlotMap sm, float* out, hipStream_t st) {
  if (layers < 1 || layers > 64) return hipErrorInvalidValue;
  if (sm.N1 != 0 && sm.N1 * sm.N2 != n) return hipErrorInvalidValue;
  ReduceArg arg{};
  for (int l = 0; l < layers; ++l) {
    arg.groups[l] = groups[l];
    arg.transposed[l] = transposed[l];
  }
  const size_t nn = (size_t)n * n;
  const int blocks = (int)((nn + 63) / 64);
  hipLaunchKernelGGL(reduce_dphi_kernel, dim3(blocks, layers), dim3(256), 0, st, part, layer_stride, arg, n, sm, out);
  return hipGetLastError();
}


hipError_t launch_readout(const float2* field, int batch, int n, const Regions& r, float* sums, hipStream_t st) {
  hipLaunchKernelGGL(readout_kernel, dim3(r.K, batch), dim3(256), 0, st, field, n, r, sums);
  return hipGetLastError();
}

}  // namespace lr
