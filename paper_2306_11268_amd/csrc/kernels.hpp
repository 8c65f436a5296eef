// Internal launch interface between the C ABI (api.hip) and the kernels (kernels.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace lr {

constexpr int kMaxRegions = 64;

enum Axis : int { kRow = 0, kCol = 1 };

// What one pass of the separable (Fresnel) path does along its axis.
enum PassKind : int {
  kPropOnce = 0,   // load -> one 1-D propagation -> store
  kFwdMid = 1,     // load W_{l-1} -> prop -> x M_l -> prop -> store W_l
  kFwdLast = 2,    // load -> prop -> detector-plane outputs
  kBwdFirst = 3,   // load -> prop (U_D) -> seed 2*(dL/dI)*U_D -> adjoint prop -> store
  kBwdMid = 4,     // load W_{l-1} -> prop (A_l); load G -> adj prop -> dphi_l -> x conj(M_l) -> adj prop -> store
  kBwdLast = 5,    // load W_0 -> prop (A_1); load G -> adj prop -> dphi_1
};

// Passes of the non-separable (angular-spectrum) path.  Fields between
// passes hold rows of x-spectra: [B][n rows][N columns], columns in the
// plan's location order.
enum AsPassKind : int {
  kAsRowFirst = 0,   // rows: pad -> FFT_x (input amplitude or field)
  kAsCol = 1,        // columns: pad -> FFT_y -> x H -> IFFT_y -> crop
  kAsRowMid = 2,     // rows: IFFT_x -> crop -> x M_l (store U_l) -> pad -> FFT_x
  kAsRowLast = 3,    // rows: IFFT_x -> crop -> detector-plane outputs
  kAsRowBwdFirst = 4,// rows: seed -> pad -> FFT_x
  kAsRowBwdMid = 5,  // rows: IFFT_x -> crop -> dphi_l -> x conj(M_l) -> pad -> FFT_x
  kAsRowBwdLast = 6, // rows: IFFT_x -> crop -> dphi_1
  kAsRowIfft = 7,    // rows: IFFT_x -> crop -> store field (plain propagation)
  kAsColFar = 8,     // columns: pad -> FFT_y -> x table -> store [N][N], both indices shifted by N/2
};

struct PassArgs {
  int full;       // n == N: fields and per-layer tables in slot order (see SlotMap)
  int n;          // layer (aperture) size
  int off;        // (N - n) / 2
  int batch;
  int nvec;       // vectors along the tile axis
  int spg;        // samples per workgroup (group size of the batch reduction)
  int ntiles;     // tiles along the vector axis
  // Persistent schedule of the separable layer passes (fresnel_pass): the
  // first `workers` workgroup ranks work.  Without dphi accumulation, rank r
  // takes the (tile, sample) items r, r + workers, ... (item i = tile
  // i % ntiles of sample i / ntiles).  With it, rank r keeps tile r % ntiles
  // and takes samples r / ntiles + k * lanes, accumulating dphi over them
  // into partial r / ntiles (workers = lanes * ntiles).
  int workers;
  int lanes;
  // main field
  const void* in;
  int in_real;    // input is a real float amplitude
  float2* out;
  // spectral table: B-item-ordered 1-D chirp (separable path) or the
  // column-permuted 2-D transfer function (angular-spectrum path)
  const float2* tab;
  int conj_tab;
  // modulation gamma*exp(j*phi_l), oriented [q][vec]
  const float2* mod;
  int conj_mod;
  float2* act_out;      // angular-spectrum path: U_l, oriented [B][n][n]
  const float2* act_in; // angular-spectrum path: U_l, oriented; separable path: W_{l-1}, natural [B][n][n]
  // Adjoint column passes: when not NULL, the input field (G) is zero on the
  // rows y with live[y] == 0 (rows that no detector region covers, which the
  // detector-plane seed pass does not write); those rows are not read.
  const unsigned long long* live;
  float* dphi_part;     // oriented [groups][n][n]
  // detector-plane outputs (natural [B][n][n] layouts)
  float* intensity;
  float2* field_out;
  float2* saved_ud;     // angular-spectrum path only
  float* sums_part;     // [B][ntiles][K]
  // far field: row passes store each x-spectrum in centred natural order
  // (position p holds frequency (p + N/2) mod N), so that the column pass
  // reads and writes whole output columns
  int spec_centred;
  // angular-spectrum column pass: the table is even in ky (H[N - ky] =
  // H[ky], exact for the analytic angular-spectrum transfer function), so
  // only its rows ky <= N/2 are read
  int tab_sym;
  // field added to the detector-plane field before any output or seed is
  // formed (natural [B][n][n]; nullable): an optical skip connection
  const float2* skip;
  // backward seed
  const float* grad_sums;  // [B][K]
  const float* grad_int;   // [B][n][n]
  const float2* ud_in;     // [B][n][n] (angular-spectrum path)
  // Detector-plane passes restricted to the vectors the detector regions
  // cover: vperm lists those nact vectors first (ascending), then the others.
  // Tiles [0, ntiles_act) transform the covered vectors; a backward seed pass
  // writes zero vectors over the rest with tiles [ntiles_act, ntiles).
  const int* vperm;
  int nact;
  int ntiles_act;
  // detector regions: K squares of side det_size, corners regions[k] = (y0, x0);
  // row_mask[y] / col_mask[x] have bit k set when region k covers row y / column x
  int K;
  int det_size;
  int accumulate;  // detector-plane intensity is added to the output instead of stored
  const int2* regions;
  const unsigned long long* row_mask;
  const unsigned long long* col_mask;
};

struct TileShape { int T; int S; };

// Slot order of an FFT plan N = N1 * N2 (plan.hpp): stored index s along an
// axis holds natural position pos(s) = (N2 * (s / N2) + N1 * (s % N2)) mod N
// for a Good-Thomas plan (pfa != 0) and s otherwise.  The separable passes
// store the fields they hand to each other, the modulation tables and the
// dphi partials in this order along both axes when the layer fills the grid.
// N1 = 0 is the identity (natural order).
struct SlotMap {
  int N1;
  int N2;
  int pfa;
  __host__ __device__ int pos(int s) const {
    if (N1 == 0 || !pfa) return s;
    const int x = s / N2;
    const int j = s - x * N2;
    return (N2 * x + N1 * j) % (N1 * N2);
  }
};
SlotMap slot_map(int N);

// Detector regions passed by value: K squares of side s with corners (y0, x0).
struct Regions {
  int K;
  int s;
  int y0[kMaxRegions];
  int x0[kMaxRegions];
};


// Whole-field forward (field_forward_kernel): one workgroup per sample holds
// the N x N field on chip through every layer, for the grids whose field
// fits there (N = 64, 100, 128 in shared memory; N = 200 half in shared
// memory and half in registers, field_forward_split_kernel), full aperture,
// Fresnel path.  Outputs:
// region-sum partials [B][K] (for launch_finish_sums with one tile), the
// intensity map and the detector-plane field.
struct FieldArgs {
  const float* amp;            // [B][N][N] natural amplitudes
  const float2* mod;           // [L][N][N] gamma*exp(j*phi_l), slot order on both axes
  unsigned long long mod_t;    // bit l-1 set: layer l's table is stored [x][y]
  int layers;
  const float2* chirp_x;       // separable chirps, natural frequency order, 1/N folded in
  const float2* chirp_y;
  Regions reg;                 // region corners (natural coordinates); K = 0: no sums
  float* sums_part;            // [B][K]
  float* intensity;            // [B][N][N] natural, or NULL
  float2* field_out;           // [B][N][N] natural, or NULL
  int accumulate;              // intensity is added to the output
  int batch;
};
// Whether the row layer passes of this FFT length run on the wide row tiles
// (wide_row_pass, N = 500, full aperture), whose modulation tables and dphi
// partials are [row][col] instead of the row passes' [col][row].
bool wide_row_tiles(int N);
bool field_forward_supported(int N);
// Whether a forward call of this size and batch should take the whole-field
// kernel: it runs one sample per workgroup, so below one sample per CU it
// leaves CUs idle and the layer passes are faster, except at N = 64 where
// the passes are launch-bound (5-layer forward, batch 64: 42 against 44 us
// at N = 64, 103 against 88 us at N = 100, 107 against 84 us at N = 128).
// Never at N = 200, where the layer passes measured faster.
bool field_forward_preferred(int N, int batch);
hipError_t launch_field_forward(int N, const FieldArgs& a, hipStream_t st);

bool fft_size_supported(int N);
TileShape tile_shape(int N, int axis);

hipError_t launch_fresnel_pass(int N, PassKind kind, Axis axis, const PassArgs& a, hipStream_t st);
// Workgroups of a separable pass kernel that fit on the current device at
// once, and the vectors each of its workgroups transforms.
int fresnel_pass_slots(int N, PassKind kind, Axis axis, bool full);
int fresnel_pass_tile(int N, PassKind kind, Axis axis, bool full);
hipError_t launch_as_pass(int N, AsPassKind kind, const PassArgs& a, hipStream_t st);

// Small helper kernels.
// Hp[ky][c] = scale * H[ky][kx(c)] (columns in the row plan's slot order).
hipError_t launch_prep_as_table(int N, const float2* H, float2* Hp, float scale, int centred, hipStream_t st);
// sums[b][k] = (accumulate ? sums[b][k] : 0) + the per-tile partial sums, in tile order.
hipError_t launch_finish_sums(const float* part, int batch, int ntiles, int K, float* sums, int accumulate,
                              hipStream_t st);
// Loss of the detector sums (kind 0: softmax cross-entropy, 1: squared norm
// of softmax minus one-hot), mean over the batch, and dL/dS; grad and loss
// are nullable.
hipError_t launch_loss(int kind, const float* sums, const int32_t* labels, int batch, int K, float* grad_sums,
                       float* loss, hipStream_t st);
// Codesign layer: with grad_phi NULL, phi_or_grad[p] = the phase of pixel p
// (soft sum or, with hard, the chosen level); otherwise phi_or_grad
// [count][K] = dL/dlogits.  logits, noise [count][K]; levels [K]; K <= 1024.
hipError_t launch_codesign(const float* logits, const float* noise, const float* levels, int K, long long count,
                           float tau, int hard, const float* grad_phi, float* phi_or_grad, hipStream_t st);
// One Adam step over count elements (bc1, bc2: bias corrections 1 - beta^t).
hipError_t launch_adam(float* phi, const float* g, float* m, float* v, long long count, float lr, float b1, float b2,
                       float eps, float bc1, float bc2, hipStream_t st);
// dphi of `layers` layers in one launch: layer l sums groups[l] partials
// (oriented [q][vec], transposed[l] != 0: q = x, both indices in the slot
// order sm) starting at part + l * layer_stride floats into out + l * n * n
// (natural order).
hipError_t launch_reduce_dphi(const float* part, size_t layer_stride, const int* groups, const int* transposed,
                              int layers, int n, SlotMap sm, float* out, hipStream_t st);
// Per-call tables in one launch: mod[l] = gamma * exp(j*phi_l) oriented per
// layer (orient_host[l] != 0: transposed; none when layers = 0) in the slot
// order sm along both axes; when regions is not NULL, the region corners
// (int2 [K]), per-row / per-column coverage masks (uint64 [n], natural
// indices) and covered-first permutations of the stored rows and columns
// (int [n], slot order sm); when H is not NULL, the separable Fresnel chirps of the nfft grid
// in natural frequency order (chirp_x[f] = H[0][f] / nfft, chirp_y[f] =
// H[f][0] * conj(H[0][0]) / nfft).  n <= 1024.
hipError_t launch_prep_layers(const float* phi, int layers, int n, float gamma, const int* orient_host, SlotMap sm,
                              float2* mod, const Regions* regions, int2* dst, unsigned long long* row_mask,
                              unsigned long long* col_mask, int* row_perm, int* col_perm, const float2* H, int nfft,
                              float2* chirp_x, float2* chirp_y, hipStream_t st);
hipError_t launch_readout(const float2* field, int batch, int n, const Regions& r, float* sums, hipStream_t st);
// Layer normalisation of batch maps of count values over fixed chunks of
// kLnChunk values: part holds batch * ln_chunks(count) float2 partials and
// stats2 batch float2.  Forward: stats[b] = (mean, 1/sqrt(var + eps)),
// y = (x - mean) * rstd.  Backward (y the normalised maps, g = dL/dy):
// dx = rstd * (g - mean(g) - y * mean(g * y)).
constexpr int kLnChunk = 4096;
inline long long ln_chunks(long long count) { return (count + kLnChunk - 1) / kLnChunk; }
hipError_t launch_layer_norm(const float* x, int batch, long long count, float eps, float* y, float2* stats,
                             float2* part, hipStream_t st);
hipError_t launch_layer_norm_backward(const float* g, const float* y, const float2* stats, int batch,
                                      long long count, float* dx, float2* part, float2* stats2, hipStream_t st);

}  // namespace lr
