// C ABI of the DONN physics kernel: argument validation, workspace layout,
// the float64 transfer-function build and the sequence of passes for each
// entry point.  Every compute step runs in the HIP kernels of kernels.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <complex>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <initializer_list>
#include <string>
#include <vector>

#include "../../include/lr.h"
#include "kernels.hpp"

using lr::Axis;
using lr::PassArgs;

#define LR_TRY(x)                  \
  do {                             \
    const int _r = (x);            \
    if (_r != LR_OK) return _r;    \
  } while (0)

namespace {

constexpr double kTwoPi = 6.283185307179586476925286766559;
constexpr double kPiD = 3.141592653589793238462643383280;

// ---------------------------------------------------------------------------
// Kernel timing (measurement mode)
// ---------------------------------------------------------------------------
struct TimingRecord {
  std::string name;
  hipEvent_t start;
  hipEvent_t stop;
};

struct TimingState {
  std::mutex mu;
  bool on = false;
  std::vector<TimingRecord> recs;
  std::vector<hipEvent_t> pool;
};

TimingState& timing() {
  static TimingState s;
  return s;
}

hipEvent_t take_event(TimingState& s) {
  if (!s.pool.empty()) {
    hipEvent_t e = s.pool.back();
    s.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Calls that must not allocate (lr_propagate_noalloc) launch untimed: the
// timing records create HIP events.
thread_local bool g_untimed = false;

template <class F>
int run_timed(const std::string& name, hipStream_t st, F&& launch) {
  TimingState& s = timing();
  bool on;
  {
    std::lock_guard<std::mutex> g(s.mu);
    on = s.on && !g_untimed;
  }
  if (!on) return launch() == hipSuccess ? LR_OK : LR_E_HIP;
  hipEvent_t a, b;
  {
    std::lock_guard<std::mutex> g(s.mu);
    a = take_event(s);
    b = take_event(s);
  }
  if (!a || !b) return LR_E_HIP;
  if (hipEventRecord(a, st) != hipSuccess) return LR_E_HIP;
  const hipError_t e = launch();
  if (hipEventRecord(b, st) != hipSuccess) return LR_E_HIP;
  {
    std::lock_guard<std::mutex> g(s.mu);
    s.recs.push_back(TimingRecord{name, a, b});
  }
  return e == hipSuccess ? LR_OK : LR_E_HIP;
}

// ---------------------------------------------------------------------------
// Validation
// ---------------------------------------------------------------------------
bool finite_pos(double v) { return std::isfinite(v) && v > 0.0; }

// Byte ranges [p, p + bytes) of two buffers overlap (empty or null ranges never do).
bool overlaps(const void* p, size_t bytes, const void* q, size_t qbytes) {
  if (!p || !q || bytes == 0 || qbytes == 0) return false;
  const char* a = static_cast<const char*>(p);
  const char* b = static_cast<const char*>(q);
  return a < b + qbytes && b < a + bytes;
}
struct Span {
  const void* p;
  size_t bytes;
};
// Some output range overlaps another buffer of the call (an input or another output).
bool outputs_alias(std::initializer_list<Span> outputs, std::initializer_list<Span> inputs) {
  for (auto o = outputs.begin(); o != outputs.end(); ++o) {
    for (const Span& i : inputs)
      if (overlaps(o->p, o->bytes, i.p, i.bytes)) return true;
    for (auto q = o + 1; q != outputs.end(); ++q)
      if (overlaps(o->p, o->bytes, q->p, q->bytes)) return true;
  }
  return false;
}

int validate_detector(const lr_detector& d, int n) {
  if (d.num < 0 || d.num > LR_MAX_REGIONS) return LR_E_ARG;
  if (d.num == 0) return LR_OK;
  if (!d.y0 || !d.x0) return LR_E_NULL;
  if (d.size < 1 || d.size > n) return LR_E_ARG;
  // (size <= n, so n - size does not overflow; y0 + size could)
  for (int k = 0; k < d.num; ++k) {
    if (d.y0[k] < 0 || d.x0[k] < 0 || d.y0[k] > n - d.size || d.x0[k] > n - d.size) return LR_E_ARG;
  }
  return LR_OK;
}

int validate_net(const lr_donn* net, bool need_layers) {
  if (!net) return LR_E_NULL;
  if (net->flags & ~(LR_ACCUMULATE | LR_LAYER_PASSES | LR_WHOLE_FIELD)) return LR_E_ARG;
  if ((net->flags & LR_LAYER_PASSES) && (net->flags & LR_WHOLE_FIELD)) return LR_E_ARG;
  if (!finite_pos(net->wavelength) || !finite_pos(net->pixel_pitch) || !std::isfinite(net->distance))
    return LR_E_ARG;
  if (net->approx < LR_FRESNEL || net->approx > LR_FRAUNHOFER) return LR_E_APPROX;
  // the far field changes the sample pitch and does not chain layers
  if (need_layers && net->approx == LR_FRAUNHOFER) return LR_E_APPROX;
  if (net->approx == LR_FRAUNHOFER && (net->n_fft % 2)) return LR_E_SIZE;
  if (!lr::fft_size_supported(net->n_fft)) return LR_E_SIZE;
  if (net->n < 1 || net->n > net->n_fft || ((net->n_fft - net->n) & 1)) return LR_E_SIZE;
  if (need_layers) {
    if (net->num_layers < 1 || net->num_layers > LR_MAX_LAYERS) return LR_E_SIZE;
    if (!std::isfinite(net->gamma)) return LR_E_ARG;
    const int dr = validate_detector(net->det, net->n);
    if (dr != LR_OK) return dr;
  }
  if (!net->d_H) return LR_E_NULL;
  return LR_OK;
}

// ---------------------------------------------------------------------------
// Workspace layout
// ---------------------------------------------------------------------------
size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

struct Layout {
  size_t chirp_x = 0, chirp_y = 0, hp = 0, mod = 0, w0 = 0, w1 = 0;
  size_t sums_part = 0, grad_sums = 0, dphi_part = 0, regions = 0, row_mask = 0, col_mask = 0, row_perm = 0,
         col_perm = 0, total = 0;
  int ntiles_vec = 0;   // tiles over n vectors
  int ntiles_spec = 0;  // tiles over n_fft spectrum columns (angular spectrum)
  int groups = 1;
  int spg = 1;
};

int ceil_div(int a, int b) { return (a + b - 1) / b; }

Layout make_layout(const lr_donn* net, int batch, int op) {
  Layout L;
  const int n = net->n;
  const int N = net->n_fft;
  const bool as = net->approx != LR_FRESNEL;  // the non-separable passes
  const lr::TileShape sh = lr::tile_shape(N, 0);
  L.ntiles_vec = ceil_div(n, sh.T);
  L.ntiles_spec = ceil_div(N, sh.T);
  const size_t c64 = 8;
  const size_t nn = static_cast<size_t>(n) * n;
  const size_t field = static_cast<size_t>(batch) * (as ? static_cast<size_t>(n) * N : nn) * c64;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align256(bytes);
    return at;
  };
  if (!as) {
    L.chirp_x = take(N * c64);
    L.chirp_y = take(N * c64);
  } else {
    L.hp = take(static_cast<size_t>(N) * N * c64);
  }
  if (op != LR_OP_PROPAGATE) L.mod = take(static_cast<size_t>(net->num_layers) * nn * c64);
  L.w0 = take(field);
  L.w1 = take(field);
  const int K = net->det.num;
  if (op != LR_OP_PROPAGATE && K > 0) {
    L.regions = take(static_cast<size_t>(K) * 8);
    L.row_mask = take(static_cast<size_t>(n) * 8);
    L.col_mask = take(static_cast<size_t>(n) * 8);
    L.row_perm = take(static_cast<size_t>(n) * 4);
    L.col_perm = take(static_cast<size_t>(n) * 4);
  }
  if (op == LR_OP_FORWARD && K > 0) L.sums_part = take(static_cast<size_t>(batch) * L.ntiles_vec * K * 4);
  if (op == LR_OP_BACKWARD) {
    if (K > 0) L.grad_sums = take(static_cast<size_t>(batch) * K * 4);
    const int work_tiles = L.ntiles_vec;
    int spg = ceil_div(batch * work_tiles, 2048);
    if (spg < 1) spg = 1;
    if (spg > batch) spg = batch > 0 ? batch : 1;
    L.spg = spg;
    L.groups = batch > 0 ? ceil_div(batch, spg) : 1;
    // one set of partials per layer, reduced in a single launch at the end
    L.dphi_part = take(static_cast<size_t>(net->num_layers) * L.groups * nn * 4);
  }
  L.total = off;
  return L;
}

// Bytes of the saved state (L + 1 complex64 fields of [batch][n][n]).
size_t saved_bytes(const lr_donn* net, int batch) {
  return static_cast<size_t>(net->num_layers + 1) * static_cast<size_t>(batch) * net->n * net->n * 8;
}

template <class T>
T* at(void* base, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}

// The separable path alternates axes: pass p (1-based) runs along rows for odd p.
Axis pass_axis(int p) { return (p & 1) ? lr::kRow : lr::kCol; }
// Layer l (1-based) is modulated in pass l+1: transposed storage when that pass is a row pass,
// except on the wide row tiles of the 500-point plan (full aperture), which read rows.
int layer_transposed(const lr_donn* net, int l) {
  if (net->approx != LR_FRESNEL) return 1;
  if (pass_axis(l + 1) != lr::kRow) return 0;
  return lr::wide_row_tiles(net->n_fft) && net->n == net->n_fft ? 0 : 1;
}

const char* kind_name(int k) {
  static const char* names[] = {"prop", "fwd_mid", "fwd_last", "bwd_first", "bwd_mid", "bwd_last"};
  return names[k];
}
const char* as_kind_name(int k) {
  static const char* names[] = {"row_first", "col", "row_mid", "row_last", "row_bwd_first", "row_bwd_mid",
                                "row_bwd_last", "row_ifft", "col_far"};
  return names[k];
}

std::string fr_name(int N, int kind, Axis ax) {
  char b[96];
  std::snprintf(b, sizeof b, "fresnel_pass_%s_%s_N%d", kind_name(kind), ax == lr::kRow ? "row" : "col", N);
  return b;
}
std::string as_name(int N, int kind) {
  char b[96];
  std::snprintf(b, sizeof b, "as_pass_%s_N%d", as_kind_name(kind), N);
  return b;
}

// Schedule of a separable layer pass (PassArgs::workers / lanes).
// Accumulating passes run persistently, as many workgroups as fit on the
// device at once: each keeps one tile and takes a share of the batch for one
// of `lanes` partial sums (lanes <= max_lanes, the partials the workspace
// holds).  The other passes take one (tile, sample) item per workgroup: the
// hardware dispatcher then balances them, which measured faster than a
// persistent schedule with prefetching for them.
int schedule_layer_pass(int N, lr::PassKind kind, Axis ax, int max_lanes, PassArgs& a) {
  const int slots = lr::fresnel_pass_slots(N, kind, ax, a.full != 0);
  const int tile_t = lr::fresnel_pass_tile(N, kind, ax, a.full != 0);
  if (slots <= 0 || tile_t <= 0) return LR_E_HIP;
  a.ntiles = ceil_div(a.nvec, tile_t);
  if (kind == lr::kBwdMid || kind == lr::kBwdLast) {
    int lanes = std::max(1, slots / std::max(1, a.ntiles));
    lanes = std::min(lanes, std::max(1, std::min(max_lanes, a.batch)));
    // Column passes: the same number of samples for every lane (the last
    // round of a persistent pass is as long as its longest lane).  Row
    // passes keep every resident lane instead: their workgroups are single
    // waves, and the extra residency outweighs the short last round of the
    // lanes with one sample more (200x200, batch 500: 122 lanes with 4 or 5
    // samples against 100 with 5, adjoint row pass 135.6 -> 128.3 us,
    // step -1%; the same on column passes cost 0.7%).
    if (ax == lr::kCol) {
      const int per = ceil_div(a.batch, lanes);
      lanes = ceil_div(a.batch, per);
    }
    a.lanes = lanes;
    a.workers = lanes * a.ntiles;
  } else {
    a.lanes = 0;
    a.workers = a.ntiles * a.batch;
  }
  return LR_OK;
}

// Launch a separable pass; layer passes without accumulation are scheduled here,
// accumulating ones by the caller (which needs the number of partials).
int fr_pass(int N, lr::PassKind kind, Axis ax, const PassArgs& a, hipStream_t st) {
  PassArgs s = a;
  if (kind == lr::kPropOnce || kind == lr::kFwdMid) LR_TRY(schedule_layer_pass(N, kind, ax, 0, s));
  return run_timed(fr_name(N, kind, ax), st, [&] { return lr::launch_fresnel_pass(N, kind, ax, s, st); });
}
int as_pass(int N, lr::AsPassKind kind, const PassArgs& a, hipStream_t st) {
  return run_timed(as_name(N, kind), st, [&] { return lr::launch_as_pass(N, kind, a, st); });
}

PassArgs base_args(const lr_donn* net, int batch) {
  PassArgs a;
  std::memset(&a, 0, sizeof a);
  a.n = net->n;
  a.off = (net->n_fft - net->n) / 2;
  a.batch = batch;
  a.spg = 1;
  a.tab_sym = net->approx == LR_ANGULAR_SPECTRUM ? 1 : 0;
  return a;
}

lr::Regions host_regions(const lr_detector& d) {
  lr::Regions r;
  std::memset(&r, 0, sizeof r);
  r.K = d.num;
  r.s = d.size;
  for (int k = 0; k < d.num && k < lr::kMaxRegions; ++k) {
    r.y0[k] = d.y0[k];
    r.x0[k] = d.x0[k];
  }
  return r;
}

// Number of rows (axis = row) or columns covered by at least one detector
// region: the same test the region kernel applies when it orders them first.
int covered_vectors(const lr_detector& d, int n, Axis ax) {
  int c = 0;
  for (int i = 0; i < n; ++i) {
    bool hit = false;
    for (int k = 0; k < d.num && !hit; ++k) {
      const int lo = ax == lr::kRow ? d.y0[k] : d.x0[k];
      hit = static_cast<unsigned>(i - lo) < static_cast<unsigned>(d.size);
    }
    c += hit ? 1 : 0;
  }
  return c;
}

// Restrict a detector-plane pass along `ax` to the vectors the regions
// cover; with zero_rest, tiles after those write zero vectors over the rest.
void restrict_to_regions(PassArgs& a, const lr_detector& d, const Layout& L, void* w, Axis ax, int tile_t,
                         bool zero_rest) {
  const int n = a.n;
  a.vperm = at<int>(w, ax == lr::kRow ? L.row_perm : L.col_perm);
  a.nact = covered_vectors(d, n, ax);
  a.ntiles_act = ceil_div(a.nact, tile_t);
  a.ntiles = a.ntiles_act + (zero_rest ? ceil_div(n - a.nact, tile_t) : 0);
}

void set_detector(PassArgs& a, const lr_detector& d, const Layout& L, void* w) {
  a.K = d.num;
  a.det_size = d.size;
  a.regions = at<int2>(w, L.regions);
  a.row_mask = at<unsigned long long>(w, L.row_mask);
  a.col_mask = at<unsigned long long>(w, L.col_mask);
}

int check_work(const lr_donn* net, int batch, int op, void* d_work, size_t work_bytes, Layout* out) {
  *out = make_layout(net, batch, op);
  if (!d_work) return LR_E_NULL;
  if (work_bytes < out->total) return LR_E_WORKSPACE;
  return LR_OK;
}

// Scale of the column-permuted 2-D table: 1/N^2 (the inverse transform's
// normalisation) for a propagation, 1 for the far-field table.
float as_table_scale(const lr_donn* net) {
  const double N = static_cast<double>(net->n_fft);
  return net->approx == LR_FRAUNHOFER ? 1.0f : static_cast<float>(1.0 / (N * N));
}

// The separable passes of a network whose layer fills the FFT grid keep
// their fields, modulation tables and dphi partials in the plan's slot order
// (no index arithmetic in the passes); padded layers use natural order.
bool slot_ordered(const lr_donn* net) { return net->approx == LR_FRESNEL && net->n == net->n_fft; }
lr::SlotMap slot_map_of(const lr_donn* net) {
  return slot_ordered(net) ? lr::slot_map(net->n_fft) : lr::SlotMap{0, 0, 0};
}

// Transfer-function tables of the passes: the separable Fresnel chirps (in
// natural frequency order; each pass stages them in its own plan order) or the
// column-permuted copy of H the angular-spectrum passes read.
int prep_tables(const lr_donn* net, const Layout& L, void* w, hipStream_t st) {
  const float2* H = reinterpret_cast<const float2*>(net->d_H);
  if (net->approx == LR_FRESNEL) {
    return run_timed("prep_layers", st, [&] {
      return lr::launch_prep_layers(nullptr, 0, net->n, 1.0f, nullptr, lr::SlotMap{0, 0, 0}, nullptr, nullptr,
                                    nullptr, nullptr, nullptr, nullptr, nullptr, H, net->n_fft, at<float2>(w, L.chirp_x),
                                    at<float2>(w, L.chirp_y), st);
    });
  }
  return run_timed("prep_as_table", st, [&] {
    return lr::launch_prep_as_table(net->n_fft, H, at<float2>(w, L.hp), as_table_scale(net),
                                    net->approx == LR_FRAUNHOFER ? 1 : 0, st);
  });
}

// Per-call tables of a forward or backward pass in one launch: the modulation
// of every layer, the Fresnel chirps, and (when the call reads detector
// regions) the region tables; the angular-spectrum table takes its own launch.
int prep_layers(const lr_donn* net, const float* d_phi, bool regions, const Layout& L, void* w, hipStream_t st) {
  int orient[LR_MAX_LAYERS];
  for (int l = 0; l < net->num_layers; ++l) orient[l] = layer_transposed(net, l + 1);
  const bool with_regions = regions && net->det.num > 0;
  const lr::Regions r = host_regions(net->det);
  const bool fresnel = net->approx == LR_FRESNEL;
  const float2* H = reinterpret_cast<const float2*>(net->d_H);
  if (!fresnel) {
    LR_TRY(run_timed("prep_as_table", st, [&] {
      return lr::launch_prep_as_table(net->n_fft, H, at<float2>(w, L.hp), as_table_scale(net),
                                    net->approx == LR_FRAUNHOFER ? 1 : 0, st);
    }));
  }
  return run_timed("prep_layers", st, [&] {
    return lr::launch_prep_layers(d_phi, net->num_layers, net->n, net->gamma, orient, slot_map_of(net),
                                  at<float2>(w, L.mod),
                                  with_regions ? &r : nullptr, at<int2>(w, L.regions),
                                  at<unsigned long long>(w, L.row_mask), at<unsigned long long>(w, L.col_mask),
                                  at<int>(w, L.row_perm), at<int>(w, L.col_perm), fresnel ? H : nullptr,
                                  net->n_fft, at<float2>(w, L.chirp_x), at<float2>(w, L.chirp_y), st);
  });
}

// ---------------------------------------------------------------------------
// Host-side float64 tables of lr_tf_build
// ---------------------------------------------------------------------------
using cd = std::complex<double>;

// Unnormalised forward DFT (exp(-2*pi*i*jk/m)) of the m samples x[0], x[s],
// x[2s], ... into X[0..m), by recursive decimation in time over the
// smallest prime factor (2, 3 or 5; lengths with other factors are rejected
// by the caller).  w holds exp(-2*pi*i*e/M) for e < M, M a multiple of m:
// exp(-2*pi*i*e/m) = w[(e mod m) * (M/m)].
void dft_rec(const cd* x, cd* X, int m, int s, const std::vector<cd>& w, std::vector<cd>& tmp) {
  if (m == 1) {
    X[0] = x[0];
    return;
  }
  const int M = static_cast<int>(w.size());
  const int p = m % 2 == 0 ? 2 : (m % 3 == 0 ? 3 : 5);
  const int q = m / p;
  for (int r = 0; r < p; ++r)
    dft_rec(x + static_cast<size_t>(r) * s, X + static_cast<size_t>(r) * q, q, s * p, w, tmp);
  // X[k + q*t] = sum_r exp(-2*pi*i*r*(k + q*t)/m) Y_r[k]
  tmp.assign(m, cd(0.0, 0.0));
  const long long stride = M / m;
  for (int k = 0; k < q; ++k)
    for (int t = 0; t < p; ++t) {
      cd acc(0.0, 0.0);
      for (int r = 0; r < p; ++r) {
        const long long e = (static_cast<long long>(r) * (k + q * t)) % m;
        acc += w[static_cast<size_t>(e * stride)] * X[r * q + k];
      }
      tmp[k + q * t] = acc;
    }
  for (int i = 0; i < m; ++i) X[i] = tmp[i];
}

bool smooth_235(int m) {
  for (int p : {2, 3, 5})
    while (m % p == 0) m /= p;
  return m == 1;
}

// In-place 2-D forward DFT of an m x m row-major array.
void dft2_host(std::vector<cd>& a, int m) {
  std::vector<cd> w(m);
  for (int e = 0; e < m; ++e) {
    const double ang = -kTwoPi * static_cast<double>(e) / static_cast<double>(m);
    w[e] = cd(std::cos(ang), std::sin(ang));
  }
  std::vector<cd> in(m), out(m), tmp;
  for (int y = 0; y < m; ++y) {
    for (int x = 0; x < m; ++x) in[x] = a[static_cast<size_t>(y) * m + x];
    dft_rec(in.data(), out.data(), m, 1, w, tmp);
    for (int x = 0; x < m; ++x) a[static_cast<size_t>(y) * m + x] = out[x];
  }
  for (int x = 0; x < m; ++x) {
    for (int y = 0; y < m; ++y) in[y] = a[static_cast<size_t>(y) * m + x];
    dft_rec(in.data(), out.data(), m, 1, w, tmp);
    for (int y = 0; y < m; ++y) a[static_cast<size_t>(y) * m + x] = out[y];
  }
}

// Wrapped index i -> i' (i' = i for i < (m+1)/2, else i - m).
int wrapped(int i, int m) { return i < (m + 1) / 2 ? i : i - m; }

// Sampled-kernel transfer function (Eq. (forward_diff) with the kernel of
// Eq. (fresnel) or of Eqs. (sommerfeld), (r01)): H = dx^2 DFT2(h), h at the
// displacements (y', x') * dx of the wrapped grid.  exp(jkz) is carried
// separately and k(r - z) = k*rho^2/(r + z), so no large phase is formed.
void impulse_response_tf(int approx, double lam, double dx, double z, int M, std::vector<cd>& H) {
  const double k = kTwoPi / lam;
  const cd ekz = std::polar(1.0, kTwoPi * std::fmod(z / lam, 1.0));
  const cd j(0.0, 1.0);
  H.assign(static_cast<size_t>(M) * M, cd(0.0, 0.0));
  for (int y = 0; y < M; ++y) {
    const double dy = wrapped(y, M) * dx;
    for (int x = 0; x < M; ++x) {
      const double dxx = wrapped(x, M) * dx;
      const double rho2 = dy * dy + dxx * dxx;
      cd h;
      if (approx == LR_FRESNEL_IR) {
        h = ekz / (j * lam * z) * std::polar(1.0, k * rho2 / (2.0 * z));
      } else {
        const double r = std::sqrt(z * z + rho2);
        h = z / (j * lam) * ekz * std::polar(1.0, k * rho2 / (r + z)) / (r * r);
      }
      H[static_cast<size_t>(y) * M + x] = h;
    }
  }
  dft2_host(H, M);
  for (auto& v : H) v *= dx * dx;
}

// Far-field table of Eq. (fraunhofer) in DFT-index order: with the input
// centred in the M x M grid (sample i at xi = (i - M/2) dx) and the output
// centred (sample k at x = (k - M/2) lambda z/(M dx)), output k holds
// (-1)^d DFT[d], d = (k + M/2) mod M, per axis.  Entry (dy, dx) is
// (-1)^(dy+dx) dx^2 exp(jkz) exp(jk(x^2+y^2)/(2z)) / (j lambda z) at the
// output coordinates (x, y) = (dx', dy') * lambda z/(M dx), d' the wrapped
// index.
void fraunhofer_table(double lam, double pitch, double z, int M, std::vector<cd>& Q) {
  const double k = kTwoPi / lam;
  const double po = lam * z / (static_cast<double>(M) * pitch);
  const cd pre = std::polar(1.0, kTwoPi * std::fmod(z / lam, 1.0)) / (cd(0.0, 1.0) * lam * z) * (pitch * pitch);
  Q.assign(static_cast<size_t>(M) * M, cd(0.0, 0.0));
  for (int y = 0; y < M; ++y) {
    const double yo = wrapped(y, M) * po;
    for (int x = 0; x < M; ++x) {
      const double xo = wrapped(x, M) * po;
      const double sgn = ((x + y) & 1) ? -1.0 : 1.0;
      Q[static_cast<size_t>(y) * M + x] = sgn * pre * std::polar(1.0, k * (xo * xo + yo * yo) / (2.0 * z));
    }
  }
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

int32_t lr_version(void) { return 1; }

const char* lr_status_string(int status) {
  switch (status) {
    case LR_OK: return "ok";
    case LR_E_NULL: return "required pointer is NULL";
    case LR_E_SIZE: return "unsupported size";
    case LR_E_ARG: return "invalid argument";
    case LR_E_APPROX: return "unknown diffraction approximation";
    case LR_E_HIP: return "HIP runtime error";
    case LR_E_WORKSPACE: return "workspace too small";
    case LR_E_ALIAS: return "output aliases an input";
    default: return "unknown status";
  }
}

int lr_tf_build(double wavelength, double pixel_pitch, double distance, int32_t approx, int32_t n_fft,
                lr_c64* d_H, void* stream) {
  if (!d_H) return LR_E_NULL;
  if (!finite_pos(wavelength) || !finite_pos(pixel_pitch) || !std::isfinite(distance)) return LR_E_ARG;
  if (approx < LR_FRESNEL || approx > LR_FRAUNHOFER) return LR_E_APPROX;
  if (n_fft < 1 || n_fft > 4096) return LR_E_SIZE;
  const int M = n_fft;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (approx == LR_FRESNEL_IR || approx == LR_RS_IR || approx == LR_FRAUNHOFER) {
    if (!(distance > 0.0)) return LR_E_ARG;
    std::vector<cd> t;
    if (approx == LR_FRAUNHOFER) {
      if (M % 2) return LR_E_SIZE;
      fraunhofer_table(wavelength, pixel_pitch, distance, M, t);
    } else {
      if (!smooth_235(M)) return LR_E_SIZE;
      impulse_response_tf(approx, wavelength, pixel_pitch, distance, M, t);
    }
    std::vector<lr_c64> hc(t.size());
    for (size_t i = 0; i < t.size(); ++i)
      hc[i] = lr_c64{static_cast<float>(t[i].real()), static_cast<float>(t[i].imag())};
    if (hipMemcpyAsync(d_H, hc.data(), hc.size() * sizeof(lr_c64), hipMemcpyHostToDevice, st) != hipSuccess)
      return LR_E_HIP;
    if (hipStreamSynchronize(st) != hipSuccess) return LR_E_HIP;
    return LR_OK;
  }
  const double lam = wavelength;
  const double z = distance;
  const double kz = kTwoPi * z / lam;
  // exp(jkz) with kz reduced modulo 2*pi through the exact fractional wave count z/lambda
  const double base = kTwoPi * std::fmod(z / lam, 1.0);
  const double fscale = 1.0 / (static_cast<double>(M) * pixel_pitch);
  std::vector<double> f(M);
  for (int k = 0; k < M; ++k) f[k] = static_cast<double>(k < (M + 1) / 2 ? k : k - M) * fscale;
  std::vector<lr_c64> h(static_cast<size_t>(M) * M);
  for (int ky = 0; ky < M; ++ky) {
    for (int kx = 0; kx < M; ++kx) {
      const double f2 = f[ky] * f[ky] + f[kx] * f[kx];
      double re, im;
      if (approx == LR_FRESNEL) {
        const double ph = base - kPiD * lam * z * f2;
        re = std::cos(ph);
        im = std::sin(ph);
      } else {
        const double s = lam * lam * f2;
        if (s <= 1.0) {
          // kz*sqrt(1-s) = kz - kz*s/(1+sqrt(1-s)), the first term reduced exactly
          const double ph = base - kz * s / (1.0 + std::sqrt(1.0 - s));
          re = std::cos(ph);
          im = std::sin(ph);
        } else {
          re = std::exp(-kz * std::sqrt(s - 1.0));
          im = 0.0;
        }
      }
      h[static_cast<size_t>(ky) * M + kx] = lr_c64{static_cast<float>(re), static_cast<float>(im)};
    }
  }
  if (hipMemcpyAsync(d_H, h.data(), h.size() * sizeof(lr_c64), hipMemcpyHostToDevice, st) != hipSuccess)
    return LR_E_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return LR_E_HIP;
  return LR_OK;
}

int64_t lr_workspace_size(const lr_donn* net, int32_t batch, int32_t op) {
  if (op != LR_OP_PROPAGATE && op != LR_OP_FORWARD && op != LR_OP_BACKWARD) return -LR_E_ARG;
  const int r = validate_net(net, op != LR_OP_PROPAGATE);
  if (r != LR_OK) return -r;
  if (batch < 0) return -LR_E_SIZE;
  return static_cast<int64_t>(make_layout(net, batch, op).total);
}

int64_t lr_saved_size(const lr_donn* net, int32_t batch) {
  const int r = validate_net(net, true);
  if (r != LR_OK) return -r;
  if (batch < 0) return -LR_E_SIZE;
  return static_cast<int64_t>(saved_bytes(net, batch));
}

int lr_propagate(const lr_donn* net, int32_t batch, const lr_c64* d_in, lr_c64* d_out, int32_t adjoint,
                 void* d_work, size_t work_bytes, void* stream) {
  LR_TRY(validate_net(net, false));
  if (batch < 0) return LR_E_SIZE;
  if (batch == 0) return LR_OK;
  if (!d_in || !d_out) return LR_E_NULL;
  if (net->approx == LR_FRAUNHOFER && adjoint) return LR_E_ARG;
  Layout L;
  LR_TRY(check_work(net, batch, LR_OP_PROPAGATE, d_work, work_bytes, &L));
  {
    const size_t m = static_cast<size_t>(net->approx == LR_FRAUNHOFER ? net->n_fft : net->n);
    const size_t in_bytes = static_cast<size_t>(batch) * net->n * net->n * 8;
    if (outputs_alias({{d_out, static_cast<size_t>(batch) * m * m * 8}, {d_work, L.total}}, {{d_in, in_bytes}}))
      return LR_E_ALIAS;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int N = net->n_fft;
  LR_TRY(prep_tables(net, L, d_work, st));
  PassArgs a = base_args(net, batch);
  a.conj_tab = adjoint ? 1 : 0;
  if (net->approx == LR_FRESNEL) {
    a.nvec = net->n;
    a.ntiles = L.ntiles_vec;
    a.in = d_in;
    a.out = at<float2>(d_work, L.w0);
    a.tab = at<float2>(d_work, L.chirp_x);
    LR_TRY(fr_pass(N, lr::kPropOnce, lr::kRow, a, st));
    a.in = at<float2>(d_work, L.w0);
    a.out = reinterpret_cast<float2*>(d_out);
    a.tab = at<float2>(d_work, L.chirp_y);
    return fr_pass(N, lr::kPropOnce, lr::kCol, a, st);
  }
  a.in = d_in;
  a.nvec = net->n;
  a.ntiles = L.ntiles_vec;
  a.out = at<float2>(d_work, L.w0);
  a.spec_centred = net->approx == LR_FRAUNHOFER ? 1 : 0;
  LR_TRY(as_pass(N, lr::kAsRowFirst, a, st));
  a.spec_centred = 0;
  if (net->approx == LR_FRAUNHOFER) {
    // far field: the column DFT with the output factors, straight into d_out ([batch][N][N])
    a.in = at<float2>(d_work, L.w0);
    a.out = reinterpret_cast<float2*>(d_out);
    a.nvec = N;
    a.ntiles = L.ntiles_spec;
    a.tab = at<float2>(d_work, L.hp);
    return as_pass(N, lr::kAsColFar, a, st);
  }
  a.in = at<float2>(d_work, L.w0);
  a.out = at<float2>(d_work, L.w1);
  a.nvec = N;
  a.ntiles = L.ntiles_spec;
  a.tab = at<float2>(d_work, L.hp);
  LR_TRY(as_pass(N, lr::kAsCol, a, st));
  a.in = at<float2>(d_work, L.w1);
  a.out = reinterpret_cast<float2*>(d_out);
  a.nvec = net->n;
  a.ntiles = L.ntiles_vec;
  return as_pass(N, lr::kAsRowIfft, a, st);
}

// ---------------------------------------------------------------------------
// lr_propagate without a caller workspace: the workspace is a fixed array in
// device memory, one per GPU (each device holds its own copy of the array
// while the library is loaded).  In host code the array's name is not a
// device address; its address on the current device comes from
// hipGetSymbolAddress, taken once per device and kept.
// ---------------------------------------------------------------------------
namespace {
constexpr size_t kScratchBytes = static_cast<size_t>(LR_NOALLOC_SCRATCH_BYTES);
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_on_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return LR_E_HIP;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return LR_E_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return LR_OK;
}

struct UntimedScope {
  bool prev;
  UntimedScope() : prev(g_untimed) { g_untimed = true; }
  ~UntimedScope() { g_untimed = prev; }
};
}  // namespace

int64_t lr_propagate_noalloc_limit(void) { return static_cast<int64_t>(kScratchBytes); }

int lr_propagate_noalloc(const lr_donn* net, int32_t batch, const lr_c64* d_in, lr_c64* d_out, int32_t adjoint,
                         void* stream) {
  LR_TRY(validate_net(net, false));
  if (batch < 0) return LR_E_SIZE;
  if (batch == 0) return LR_OK;
  // the same checks as lr_propagate, before the scratch size
  if (!d_in || !d_out) return LR_E_NULL;
  const Layout L = make_layout(net, batch, LR_OP_PROPAGATE);
  if (L.total > kScratchBytes) return LR_E_WORKSPACE;
  void* work = nullptr;
  LR_TRY(scratch_on_current_device(&work));
  UntimedScope untimed;
  // every part of the workspace a propagation uses is written before it is
  // read, so nothing left by an earlier call needs clearing
  return lr_propagate(net, batch, d_in, d_out, adjoint, work, kScratchBytes, stream);
}

int lr_detector_readout(const lr_c64* d_field, int32_t batch, int32_t n, const lr_detector* det, float* d_sums,
                        void* stream) {
  if (!det) return LR_E_NULL;
  if (batch < 0 || n < 1) return LR_E_SIZE;
  LR_TRY(validate_detector(*det, n));
  if (batch == 0 || det->num == 0) return LR_OK;
  if (!d_field || !d_sums) return LR_E_NULL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const lr::Regions reg = host_regions(*det);
  return run_timed("readout", st, [&] {
    return lr::launch_readout(reinterpret_cast<const float2*>(d_field), batch, n, reg, d_sums, st);
  });
}

int lr_donn_forward(const lr_donn* net, int32_t batch, const float* d_amp, const float* d_phi, void* d_saved,
                    float* d_sums, float* d_intensity, lr_c64* d_field_out, void* d_work, size_t work_bytes,
                    void* stream) {
  LR_TRY(validate_net(net, true));
  if (batch < 0) return LR_E_SIZE;
  if (batch == 0) return LR_OK;
  if (!d_amp || !d_phi) return LR_E_NULL;
  if (d_sums && net->det.num == 0) return LR_E_ARG;
  const bool accumulate = (net->flags & LR_ACCUMULATE) != 0;
  if (accumulate && d_field_out) return LR_E_ARG;  // fields of separate channels do not add
  Layout L;
  LR_TRY(check_work(net, batch, LR_OP_FORWARD, d_work, work_bytes, &L));
  {
    const size_t nn4 = static_cast<size_t>(batch) * net->n * net->n * 4;
    if (outputs_alias({{d_saved, saved_bytes(net, batch)},
                       {d_sums, static_cast<size_t>(batch) * net->det.num * 4},
                       {d_intensity, nn4},
                       {d_field_out, 2 * nn4},
                       {d_work, L.total}},
                      {{d_amp, nn4},
                       {d_phi, static_cast<size_t>(net->num_layers) * net->n * net->n * 4},
                       {net->d_skip, 2 * nn4}}))
      return LR_E_ALIAS;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int N = net->n_fft;
  const int n = net->n;
  const int Lyr = net->num_layers;
  const size_t nn = static_cast<size_t>(n) * n;
  float2* saved = static_cast<float2*>(d_saved);
  float2* ws_mod = at<float2>(d_work, L.mod);
  float2* w[2] = {at<float2>(d_work, L.w0), at<float2>(d_work, L.w1)};

  LR_TRY(prep_layers(net, d_phi, d_sums != nullptr, L, d_work, st));

  PassArgs a = base_args(net, batch);
  a.accumulate = accumulate ? 1 : 0;
  a.full = slot_ordered(net) ? 1 : 0;
  const int tile_t = lr::tile_shape(N, 0).T;
  int sum_tiles = L.ntiles_vec;  // tiles that wrote partial detector sums
  const bool whole_field = net->approx == LR_FRESNEL && n == N && lr::field_forward_supported(N) &&
                           ((net->flags & LR_WHOLE_FIELD) || lr::field_forward_preferred(N, batch)) && !saved &&
                           (d_sums || d_intensity || d_field_out) && !net->d_skip &&
                           !(net->flags & LR_LAYER_PASSES);
  if (whole_field) {
    // every hop of a sample in one workgroup, the field in shared memory
    lr::FieldArgs fa;
    std::memset(&fa, 0, sizeof fa);
    fa.amp = d_amp;
    fa.mod = ws_mod;
    for (int l = 1; l <= Lyr; ++l)
      if (layer_transposed(net, l)) fa.mod_t |= 1ull << (l - 1);
    fa.layers = Lyr;
    fa.chirp_x = at<float2>(d_work, L.chirp_x);
    fa.chirp_y = at<float2>(d_work, L.chirp_y);
    if (d_sums) {
      fa.reg = host_regions(net->det);
      fa.sums_part = at<float>(d_work, L.sums_part);
    }
    fa.intensity = d_intensity;
    fa.field_out = reinterpret_cast<float2*>(d_field_out);
    fa.accumulate = accumulate ? 1 : 0;
    fa.batch = batch;
    char name[48];
    std::snprintf(name, sizeof name, "field_forward_N%d", N);
    LR_TRY(run_timed(name, st, [&] { return lr::launch_field_forward(N, fa, st); }));
    sum_tiles = 1;
  } else if (net->approx == LR_FRESNEL) {
    a.nvec = n;
    a.ntiles = L.ntiles_vec;
    auto chirp = [&](Axis ax) { return at<float2>(d_work, ax == lr::kRow ? L.chirp_x : L.chirp_y); };
    // Pass p writes W_p: slot p of the saved state when there is one (the
    // backward pass reads W_0 .. W_L there), else the two work fields in turn.
    auto w_out = [&](int p) { return saved ? saved + static_cast<size_t>(p) * batch * nn : w[p & 1]; };
    // pass 0: first sweep of hop 1 along x
    a.in = d_amp;
    a.in_real = 1;
    a.out = w_out(0);
    a.tab = chirp(lr::kRow);
    LR_TRY(fr_pass(N, lr::kPropOnce, lr::kRow, a, st));
    a.in_real = 0;
    // passes 1..L: end of hop l, modulation of layer l, start of hop l+1
    for (int l = 1; l <= Lyr; ++l) {
      const Axis ax = pass_axis(l + 1);
      a.in = a.out;
      a.out = w_out(l);
      a.tab = chirp(ax);
      a.mod = ws_mod + static_cast<size_t>(l - 1) * nn;
      LR_TRY(fr_pass(N, lr::kFwdMid, ax, a, st));
    }
    // pass L+1: rest of hop L+1, detector plane
    if (d_sums || d_intensity || d_field_out) {
      const Axis ax = pass_axis(Lyr + 2);
      PassArgs d = a;
      d.in = a.out;
      d.out = nullptr;
      d.tab = chirp(ax);
      d.mod = nullptr;
      d.intensity = d_intensity;
      d.field_out = reinterpret_cast<float2*>(d_field_out);
      d.skip = reinterpret_cast<const float2*>(net->d_skip);
      if (d_sums) {
        set_detector(d, net->det, L, d_work);
        d.sums_part = at<float>(d_work, L.sums_part);
        // sums only: transform just the rows / columns the regions cover
        if (!d_intensity && !d_field_out) restrict_to_regions(d, net->det, L, d_work, ax, tile_t, false);
      }
      sum_tiles = d.ntiles;
      LR_TRY(fr_pass(N, lr::kFwdLast, ax, d, st));
    }
  } else {
    a.nvec = n;
    a.ntiles = L.ntiles_vec;
    a.in = d_amp;
    a.in_real = 1;
    a.out = w[0];
    LR_TRY(as_pass(N, lr::kAsRowFirst, a, st));
    a.in_real = 0;
    int cur = 0;
    for (int hop = 1; hop <= Lyr + 1; ++hop) {
      PassArgs c = a;
      c.in = w[cur];
      c.out = w[cur ^ 1];
      c.nvec = N;
      c.ntiles = L.ntiles_spec;
      c.tab = at<float2>(d_work, L.hp);
      LR_TRY(as_pass(N, lr::kAsCol, c, st));
      cur ^= 1;
      if (hop <= Lyr) {
        PassArgs r = a;
        r.in = w[cur];
        r.out = w[cur ^ 1];
        r.mod = ws_mod + static_cast<size_t>(hop - 1) * nn;
        r.act_out = saved ? saved + static_cast<size_t>(hop - 1) * batch * nn : nullptr;
        LR_TRY(as_pass(N, lr::kAsRowMid, r, st));
        cur ^= 1;
      } else {
        PassArgs r = a;
        r.in = w[cur];
        r.skip = reinterpret_cast<const float2*>(net->d_skip);
        r.intensity = d_intensity;
        r.field_out = reinterpret_cast<float2*>(d_field_out);
        r.saved_ud = saved ? saved + static_cast<size_t>(Lyr) * batch * nn : nullptr;
        if (d_sums) {
          set_detector(r, net->det, L, d_work);
          r.sums_part = at<float>(d_work, L.sums_part);
        }
        LR_TRY(as_pass(N, lr::kAsRowLast, r, st));
      }
    }
  }
  if (d_sums) {
    LR_TRY(run_timed("finish_sums", st, [&] {
      return lr::launch_finish_sums(at<float>(d_work, L.sums_part), batch, sum_tiles, net->det.num, d_sums,
                                    accumulate ? 1 : 0, st);
    }));
  }
  return LR_OK;
}

int lr_donn_backward(const lr_donn* net, int32_t batch, const float* d_phi, const void* d_saved, const float* d_sums,
                     const int32_t* d_labels, const float* d_grad_sums, const float* d_grad_intensity, float* d_loss,
                     float* d_grad_phi, void* d_work, size_t work_bytes, void* stream) {
  LR_TRY(validate_net(net, true));
  if (batch < 0) return LR_E_SIZE;
  if (!d_grad_phi) return LR_E_NULL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int N = net->n_fft;
  const int n = net->n;
  const int Lyr = net->num_layers;
  const size_t nn = static_cast<size_t>(n) * n;
  if (batch > 0) {
    if (!d_phi || !d_saved) return LR_E_NULL;
    const int nseeds = (d_labels ? 1 : 0) + (d_grad_sums ? 1 : 0) + (d_grad_intensity ? 1 : 0);
    if (nseeds != 1) return LR_E_ARG;
    if ((d_labels || d_grad_sums) && net->det.num == 0) return LR_E_ARG;
    if (d_labels && !d_sums) return LR_E_NULL;
  }
  Layout L;
  LR_TRY(check_work(net, batch, LR_OP_BACKWARD, d_work, work_bytes, &L));
  {
    const size_t nn4 = static_cast<size_t>(std::max(batch, 0)) * net->n * net->n * 4;
    const size_t bk4 = static_cast<size_t>(std::max(batch, 0)) * net->det.num * 4;
    if (outputs_alias({{d_grad_phi, static_cast<size_t>(net->num_layers) * net->n * net->n * 4},
                       {d_loss, 4},
                       {d_work, L.total}},
                      {{d_phi, static_cast<size_t>(net->num_layers) * net->n * net->n * 4},
                       {d_saved, batch > 0 ? saved_bytes(net, batch) : 0},
                       {d_sums, bk4},
                       {d_labels, static_cast<size_t>(std::max(batch, 0)) * 4},
                       {d_grad_sums, bk4},
                       {d_grad_intensity, nn4},
                       {net->d_skip, 2 * nn4}}))
      return LR_E_ALIAS;
  }
  if (batch == 0) {
    // an empty batch has a zero gradient: a fixed-order sum over no groups
    int none[LR_MAX_LAYERS] = {};
    return run_timed("reduce_dphi", st,
                     [&] {
                       return lr::launch_reduce_dphi(nullptr, 0, none, none, Lyr, n, lr::SlotMap{0, 0, 0}, d_grad_phi,
                                                     st);
                     });
  }
  const float2* saved = static_cast<const float2*>(d_saved);
  float2* ws_mod = at<float2>(d_work, L.mod);
  float2* w[2] = {at<float2>(d_work, L.w0), at<float2>(d_work, L.w1)};
  float* part = at<float>(d_work, L.dphi_part);

  LR_TRY(prep_layers(net, d_phi, d_labels || d_grad_sums, L, d_work, st));
  const float* gsum = d_grad_sums;
  if (d_labels) {
    float* g = at<float>(d_work, L.grad_sums);
    LR_TRY(run_timed("ce_loss", st,
                     [&] { return lr::launch_loss(0, d_sums, d_labels, batch, net->det.num, g, d_loss, st); }));
    gsum = g;
  }

  PassArgs a = base_args(net, batch);
  a.conj_tab = 1;
  a.conj_mod = 1;
  a.full = slot_ordered(net) ? 1 : 0;
  a.nvec = n;
  a.ntiles = L.ntiles_vec;
  // layer l accumulates into its own partials; one launch reduces all layers at the end
  const size_t layer_stride = static_cast<size_t>(L.groups) * nn;
  auto part_of = [&](int l) { return part + static_cast<size_t>(l - 1) * layer_stride; };
  int groups_of[LR_MAX_LAYERS] = {};
  int orient_of[LR_MAX_LAYERS] = {};
  for (int l = 1; l <= Lyr; ++l) orient_of[l - 1] = layer_transposed(net, l);
  auto reduce_all = [&]() {
    return run_timed("reduce_dphi", st, [&] {
      return lr::launch_reduce_dphi(part, layer_stride, groups_of, orient_of, Lyr, n, slot_map_of(net), d_grad_phi,
                                    st);
    });
  };

  if (net->approx == LR_FRESNEL) {
    auto chirp = [&](Axis ax) { return at<float2>(d_work, ax == lr::kRow ? L.chirp_x : L.chirp_y); };
    const unsigned long long* live_rows = nullptr;  // rows of the seed's output the first layer pass reads
    // rest of hop L+1 from the saved W_L, seed at the detector plane, adjoint of that half hop
    {
      PassArgs s = a;
      const Axis ax = pass_axis(Lyr + 2);
      s.tab = chirp(ax);
      s.in = saved + static_cast<size_t>(Lyr) * batch * nn;
      s.grad_int = d_grad_intensity;
      s.grad_sums = gsum;
      s.skip = reinterpret_cast<const float2*>(net->d_skip);
      if (gsum) {
        set_detector(s, net->det, L, d_work);
        // The seed vanishes off the covered rows (columns).  A row seed pass
        // leaves the other rows unwritten, and the next (column) pass skips
        // them; a column seed pass writes zero columns for the row pass after it.
        restrict_to_regions(s, net->det, L, d_work, ax, lr::tile_shape(N, 0).T, ax == lr::kCol);
        if (ax == lr::kRow) live_rows = at<unsigned long long>(d_work, L.row_mask);
      }
      s.out = w[0];
      LR_TRY(fr_pass(N, lr::kBwdFirst, ax, s, st));
    }
    int cur = 0;
    for (int l = Lyr; l >= 1; --l) {
      const Axis ax = pass_axis(l + 1);
      PassArgs m = a;
      m.spg = L.spg;
      m.in = w[cur];
      m.tab = chirp(ax);
      m.mod = ws_mod + static_cast<size_t>(l - 1) * nn;
      m.act_in = saved + static_cast<size_t>(l - 1) * batch * nn;  // W_{l-1}, input of layer l's forward pass
      m.dphi_part = part_of(l);
      m.live = l == Lyr ? live_rows : nullptr;
      const lr::PassKind kind = l > 1 ? lr::kBwdMid : lr::kBwdLast;
      LR_TRY(schedule_layer_pass(N, kind, ax, L.groups, m));
      if (l > 1) m.out = w[cur ^ 1];
      LR_TRY(fr_pass(N, kind, ax, m, st));
      if (l > 1) cur ^= 1;
      groups_of[l - 1] = m.lanes;
    }
    return reduce_all();
  }

  // angular spectrum
  {
    PassArgs s = a;
    s.ud_in = saved + static_cast<size_t>(Lyr) * batch * nn;
    s.grad_int = d_grad_intensity;
    s.grad_sums = gsum;
    if (gsum) set_detector(s, net->det, L, d_work);
    s.out = w[0];
    LR_TRY(as_pass(N, lr::kAsRowBwdFirst, s, st));
  }
  int cur = 0;
  for (int l = Lyr; l >= 1; --l) {
    PassArgs c = a;
    c.in = w[cur];
    c.out = w[cur ^ 1];
    c.nvec = N;
    c.ntiles = L.ntiles_spec;
    c.tab = at<float2>(d_work, L.hp);
    LR_TRY(as_pass(N, lr::kAsCol, c, st));
    cur ^= 1;
    PassArgs r = a;
    r.spg = L.spg;
    r.in = w[cur];
    r.mod = ws_mod + static_cast<size_t>(l - 1) * nn;
    r.act_in = saved + static_cast<size_t>(l - 1) * batch * nn;
    r.dphi_part = part_of(l);
    if (l > 1) {
      r.out = w[cur ^ 1];
      LR_TRY(as_pass(N, lr::kAsRowBwdMid, r, st));
      cur ^= 1;
    } else {
      LR_TRY(as_pass(N, lr::kAsRowBwdLast, r, st));
    }
    groups_of[l - 1] = L.groups;
  }
  return reduce_all();
}

int lr_loss(int32_t kind, const float* d_sums, const int32_t* d_labels, int32_t batch, int32_t classes,
            float* d_loss, float* d_grad_sums, void* stream) {
  if (kind != LR_LOSS_SOFTMAX_CE && kind != LR_LOSS_SOFTMAX_MSE) return LR_E_ARG;
  if (batch < 0 || classes < 1 || classes > LR_MAX_REGIONS) return LR_E_SIZE;
  if (!d_loss && !d_grad_sums) return LR_E_NULL;
  if (batch == 0) return LR_OK;
  if (!d_sums || !d_labels) return LR_E_NULL;
  {
    const size_t bk4 = static_cast<size_t>(batch) * classes * 4;
    if (outputs_alias({{d_grad_sums, bk4}, {d_loss, 4}}, {{d_sums, bk4}, {d_labels, static_cast<size_t>(batch) * 4}}))
      return LR_E_ALIAS;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  return run_timed(kind == LR_LOSS_SOFTMAX_CE ? "ce_loss" : "mse_loss", st, [&] {
    return lr::launch_loss(kind, d_sums, d_labels, batch, classes, d_grad_sums, d_loss, st);
  });
}

int lr_codesign_phase(const float* d_logits, const float* d_noise, const float* d_levels, int32_t levels,
                      int64_t count, float tau, int32_t hard, float* d_phi, void* stream) {
  if (levels < 1 || levels > LR_MAX_LEVELS || count < 0) return LR_E_SIZE;
  if (!(tau > 0.f) || !std::isfinite(tau)) return LR_E_ARG;
  if (count == 0) return LR_OK;
  if (!d_logits || !d_noise || !d_levels || !d_phi) return LR_E_NULL;
  {
    const size_t sc = static_cast<size_t>(count) * levels * 4;
    if (outputs_alias({{d_phi, static_cast<size_t>(count) * 4}},
                      {{d_logits, sc}, {d_noise, sc}, {d_levels, static_cast<size_t>(levels) * 4}}))
      return LR_E_ALIAS;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  return run_timed("codesign", st, [&] {
    return lr::launch_codesign(d_logits, d_noise, d_levels, levels, static_cast<long long>(count), tau, hard ? 1 : 0,
                               nullptr, d_phi, st);
  });
}

int lr_codesign_backward(const float* d_logits, const float* d_noise, const float* d_levels, int32_t levels,
                         int64_t count, float tau, const float* d_grad_phi, float* d_grad_logits, void* stream) {
  if (levels < 1 || levels > LR_MAX_LEVELS || count < 0) return LR_E_SIZE;
  if (!(tau > 0.f) || !std::isfinite(tau)) return LR_E_ARG;
  if (count == 0) return LR_OK;
  if (!d_logits || !d_noise || !d_levels || !d_grad_phi || !d_grad_logits) return LR_E_NULL;
  {
    const size_t sc = static_cast<size_t>(count) * levels * 4;
    if (outputs_alias({{d_grad_logits, sc}}, {{d_logits, sc},
                                              {d_noise, sc},
                                              {d_levels, static_cast<size_t>(levels) * 4},
                                              {d_grad_phi, static_cast<size_t>(count) * 4}}))
      return LR_E_ALIAS;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  return run_timed("codesign_bwd", st, [&] {
    return lr::launch_codesign(d_logits, d_noise, d_levels, levels, static_cast<long long>(count), tau, 0,
                               d_grad_phi, d_grad_logits, st);
  });
}

namespace {
constexpr int64_t kLnMaxCount = int64_t(1) << 28;

int ln_check(int32_t batch, int64_t count) {
  if (batch < 0 || batch > 65535 || count < 1 || count > kLnMaxCount) return LR_E_SIZE;
  return LR_OK;
}

size_t ln_work_bytes(int32_t batch, int64_t count) {
  return static_cast<size_t>(batch) * static_cast<size_t>(lr::ln_chunks(count) + 1) * sizeof(float2);
}

// [p, p + bytes) and [q, q + qbytes) overlap
}  // namespace

int64_t lr_layer_norm_workspace_size(int32_t batch, int64_t count) {
  const int e = ln_check(batch, count);
  if (e != LR_OK) return -static_cast<int64_t>(e);
  return static_cast<int64_t>(ln_work_bytes(batch, count));
}

int lr_layer_norm(const float* d_x, int32_t batch, int64_t count, float eps, float* d_y, float* d_stats,
                  void* d_work, size_t work_bytes, void* stream) {
  LR_TRY(ln_check(batch, count));
  if (!std::isfinite(eps) || eps < 0.f) return LR_E_ARG;
  if (batch == 0) return LR_OK;
  if (!d_x || !d_y || !d_stats || !d_work) return LR_E_NULL;
  if (work_bytes < ln_work_bytes(batch, count)) return LR_E_WORKSPACE;
  const size_t map_bytes = static_cast<size_t>(batch) * static_cast<size_t>(count) * sizeof(float);
  const size_t stat_bytes = static_cast<size_t>(batch) * 2 * sizeof(float);
  if (d_y != d_x && overlaps(d_y, map_bytes, d_x, map_bytes)) return LR_E_ALIAS;
  if (overlaps(d_stats, stat_bytes, d_x, map_bytes) || overlaps(d_stats, stat_bytes, d_y, map_bytes) ||
      overlaps(d_work, work_bytes, d_x, map_bytes) || overlaps(d_work, work_bytes, d_y, map_bytes) ||
      overlaps(d_work, work_bytes, d_stats, stat_bytes))
    return LR_E_ALIAS;
  hipStream_t st = static_cast<hipStream_t>(stream);
  float2* part = static_cast<float2*>(d_work);
  return run_timed("layer_norm", st, [&] {
    return lr::launch_layer_norm(d_x, batch, static_cast<long long>(count), eps, d_y,
                                 reinterpret_cast<float2*>(d_stats), part, st);
  });
}

int lr_layer_norm_backward(const float* d_grad_y, const float* d_y, const float* d_stats, int32_t batch,
                           int64_t count, float* d_grad_x, void* d_work, size_t work_bytes, void* stream) {
  LR_TRY(ln_check(batch, count));
  if (batch == 0) return LR_OK;
  if (!d_grad_y || !d_y || !d_stats || !d_grad_x || !d_work) return LR_E_NULL;
  if (work_bytes < ln_work_bytes(batch, count)) return LR_E_WORKSPACE;
  const size_t map_bytes = static_cast<size_t>(batch) * static_cast<size_t>(count) * sizeof(float);
  const size_t stat_bytes = static_cast<size_t>(batch) * 2 * sizeof(float);
  // dx may replace g (elementwise), not the normalised maps the partial sums read
  if (d_grad_x != d_grad_y && overlaps(d_grad_x, map_bytes, d_grad_y, map_bytes)) return LR_E_ALIAS;
  if (overlaps(d_grad_x, map_bytes, d_y, map_bytes) || overlaps(d_grad_x, map_bytes, d_stats, stat_bytes) ||
      overlaps(d_work, work_bytes, d_grad_x, map_bytes) || overlaps(d_work, work_bytes, d_grad_y, map_bytes) ||
      overlaps(d_work, work_bytes, d_y, map_bytes) || overlaps(d_work, work_bytes, d_stats, stat_bytes))
    return LR_E_ALIAS;
  hipStream_t st = static_cast<hipStream_t>(stream);
  float2* part = static_cast<float2*>(d_work);
  float2* stats2 = part + static_cast<size_t>(batch) * lr::ln_chunks(count);
  return run_timed("layer_norm_bwd", st, [&] {
    return lr::launch_layer_norm_backward(d_grad_y, d_y, reinterpret_cast<const float2*>(d_stats), batch,
                                          static_cast<long long>(count), d_grad_x, part, stats2, st);
  });
}

int lr_adam_update(float* d_phi, const float* d_grad, float* d_m, float* d_v, int64_t count, int32_t step, float lr,
                   float beta1, float beta2, float eps, void* stream) {
  if (count < 0 || step < 1) return LR_E_SIZE;
  if (!std::isfinite(lr) || !(beta1 >= 0.f && beta1 < 1.f) || !(beta2 >= 0.f && beta2 < 1.f) ||
      !(eps >= 0.f) || !std::isfinite(eps))
    return LR_E_ARG;
  if (count == 0) return LR_OK;
  if (!d_phi || !d_grad || !d_m || !d_v) return LR_E_NULL;
  {
    const size_t b4 = static_cast<size_t>(count) * 4;
    if (outputs_alias({{d_phi, b4}, {d_m, b4}, {d_v, b4}}, {{d_grad, b4}})) return LR_E_ALIAS;
  }
  const double bc1 = 1.0 - std::pow(static_cast<double>(beta1), step);
  const double bc2 = 1.0 - std::pow(static_cast<double>(beta2), step);
  if (!(bc1 > 0.0) || !(bc2 > 0.0)) return LR_E_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  return run_timed("adam", st, [&] {
    return lr::launch_adam(d_phi, d_grad, d_m, d_v, static_cast<long long>(count), lr, beta1, beta2, eps,
                           static_cast<float>(bc1), static_cast<float>(bc2), st);
  });
}

int lr_kernel_timing(int32_t enable) {
  TimingState& s = timing();
  std::lock_guard<std::mutex> g(s.mu);
  if (enable) {
    for (auto& r : s.recs) {
      s.pool.push_back(r.start);
      s.pool.push_back(r.stop);
    }
    s.recs.clear();
  }
  s.on = enable != 0;
  return LR_OK;
}

int lr_kernel_timing_report(char* buf, size_t len) {
  TimingState& s = timing();
  std::lock_guard<std::mutex> g(s.mu);
  std::map<std::string, std::pair<long, double>> agg;
  for (auto& r : s.recs) {
    if (hipEventSynchronize(r.stop) != hipSuccess) return -LR_E_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) return -LR_E_HIP;
    auto& e = agg[r.name];
    e.first += 1;
    e.second += ms;
  }
  std::string out = "{";
  bool first = true;
  for (auto& kv : agg) {
    char b[256];
    std::snprintf(b, sizeof b, "%s\"%s\": {\"count\": %ld, \"ms\": %.6f}", first ? "" : ", ", kv.first.c_str(),
                  kv.second.first, kv.second.second);
    out += b;
    first = false;
  }
  out += "}";
  if (buf && len > 0) {
    const size_t m = out.size() < len - 1 ? out.size() : len - 1;
    std::memcpy(buf, out.data(), m);
    buf[m] = '\0';
  }
  return static_cast<int>(out.size());
}

}  // extern "C"
