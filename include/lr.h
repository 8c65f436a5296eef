/*
 * lr.h -- C ABI of the MI355X (gfx950) DONN physics kernel.
 *
 * A diffractive optical neural network (DONN) in the sense of LightRidge
 * (arXiv 2306.11268) is emulated as a chain of free-space hops and phase
 * masks:
 *
 *   U_0 = A (amplitude, zero phase)                            -- §3.1
 *   U_l = gamma * P_z(U_{l-1}) * exp(j*phi_l),  l = 1..L        -- §3.1.1-§3.2,
 *                                                                Eqs. (forward_diff),
 *                                                                (diffraction_freq),
 *                                                                (phase_mod_matrix)
 *   U_D = P_z(U_L),  I = |U_D|^2,  S_k = sum of I over region k -- §2.1
 *
 * with P_z(U) = crop(IFFT2(H * FFT2(pad(U)))) and H the Fresnel
 * (Eq. (fresnel)) or Rayleigh-Sommerfeld angular-spectrum
 * (Eqs. (sommerfeld), (r01)) transfer function.  Training differentiates
 * a loss of I (or S) with respect to every phase mask phi_l (§2.1).
 *
 * Conventions shared by every entry point:
 *   - All sizes are in pixels, all lengths in metres.
 *   - Fields are complex64 (lr_c64, interleaved re/im, the layout of
 *     torch.complex64), real arrays are float32, all row-major.
 *   - Pointers named d_* are device (HIP) memory owned by the caller;
 *     the library allocates nothing on these paths.  Descriptor structs and
 *     detector coordinate arrays are host memory, read during the call only.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls validate
 *     their arguments on the host, enqueue their kernels on `stream` and return;
 *     an argument error returns a non-zero lr_status and enqueues nothing.
 *     Device-side faults surface at the caller's next synchronisation.
 *   - No C++ exception crosses the ABI.  Calls on distinct streams are
 *     thread safe; calls that share a workspace must be ordered by the caller.
 *   - Supported FFT grid sizes n_fft: 64, 100, 128, 200, 256, 350, 400,
 *     500, 512, 1000, 1024 (350 is the segmentation DONN's grid of §5.6.2).  The layer size n satisfies 1 <= n <= n_fft with n_fft - n
 *     even; the layer sits centred in the n_fft grid and is cropped back
 *     after every hop.
 */
#ifndef LR_H_
#define LR_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lr_c64 {
  float re;
  float im;
} lr_c64;

/* Diffraction approximations (§3.1.1).  The first two are the analytic
 * transfer functions; the next two take H as the DFT of the diffraction
 * kernel h of Eq. (forward_diff) sampled on the n_fft grid of displacements
 * (the discrete linear convolution of the field with h, exact on the
 * aperture when n_fft >= 2n - 1); the last is the far field of
 * Eq. (fraunhofer), a single scaled Fourier transform that changes the
 * sample pitch and is available through lr_propagate only. */
enum lr_approx {
  LR_FRESNEL = 0,           /* Eq. (fresnel): H = exp(jkz) exp(-j pi lambda z (fx^2+fy^2)) */
  LR_ANGULAR_SPECTRUM = 1,  /* Eqs. (sommerfeld),(r01): H = exp(jkz sqrt(1 - lambda^2 f^2)) */
  LR_FRESNEL_IR = 2,        /* Eq. (fresnel) kernel exp(jkz)/(j lambda z) exp(jk(dx^2+dy^2)/(2z)), H = dx^2 DFT2(h) */
  LR_RS_IR = 3,             /* Eqs. (sommerfeld),(r01) kernel z/(j lambda) exp(jkr)/r^2, H = dx^2 DFT2(h) */
  LR_FRAUNHOFER = 4         /* Eq. (fraunhofer): far field on the centred pitch lambda z/(n_fft dx) grid */
};

enum lr_status {
  LR_OK = 0,
  LR_E_NULL = 1,       /* a required pointer is NULL */
  LR_E_SIZE = 2,       /* unsupported n_fft, n > n_fft, odd n_fft - n, batch < 0, ... */
  LR_E_ARG = 3,        /* non-finite / non-positive physical parameter, bad detector, ... */
  LR_E_APPROX = 4,     /* unknown approximation */
  LR_E_HIP = 5,        /* a HIP runtime call failed (launch or copy) */
  LR_E_WORKSPACE = 6,  /* work_bytes smaller than lr_workspace_size() */
  LR_E_ALIAS = 7       /* an output buffer aliases an input it must not */
};

/* Ops for lr_workspace_size(). */
enum lr_op {
  LR_OP_PROPAGATE = 0,
  LR_OP_FORWARD = 1,
  LR_OP_BACKWARD = 2
};

#define LR_MAX_REGIONS 64
#define LR_MAX_LAYERS 64

/* Detector (§2.1; x_loc / y_loc / det_size of the paper's detector layer):
 * `num` square regions of side `size`, region k covering rows
 * [y0[k], y0[k]+size) and columns [x0[k], x0[k]+size) of the n x n plane.
 * num = 0 means no region readout.  y0/x0 are host arrays of length num. */
typedef struct lr_detector {
  int32_t num;
  int32_t size;
  const int32_t* y0;
  const int32_t* x0;
} lr_detector;

/* One DONN: the paper's system parameters (wavelength, pixel size,
 * diffraction distance, approximation, system size, layer count, detector)
 * plus the regularisation factor gamma of §3.2 and the transfer function. */
typedef struct lr_donn {
  double wavelength;    /* metres, finite and > 0 */
  double pixel_pitch;   /* metres, finite and > 0 */
  double distance;      /* metres per hop, finite (0 = identity, < 0 = back-propagation) */
  int32_t approx;       /* enum lr_approx */
  int32_t n;            /* layer size (system size) */
  int32_t n_fft;        /* FFT grid, n <= n_fft, n_fft - n even */
  int32_t num_layers;   /* L, 1 .. LR_MAX_LAYERS; the network makes L+1 hops */
  float gamma;          /* amplitude factor applied at every modulation, finite */
  lr_detector det;
  const lr_c64* d_H;    /* device [n_fft][n_fft], written by lr_tf_build for the same
                           wavelength / pixel_pitch / distance / approx / n_fft.
                           The Fresnel path relies on its separability. */
  int32_t flags;        /* 0, or LR_ACCUMULATE and / or one of LR_LAYER_PASSES, LR_WHOLE_FIELD */
  const lr_c64* d_skip; /* NULL, or device [batch][n][n]: a field added to the
                           detector-plane field before the intensity, the sums,
                           the field output or the backward seed are formed.
                           This is the optical skip connection of the
                           segmentation DONN (§5.6.2); under the residual
                           reading (the stack of layers as F in F(x) + x) it is
                           the input field itself, relayed to the detector.
                           lr_donn_forward and lr_donn_backward must see the
                           same field; it must not alias d_field_out. */
} lr_donn;

/* lr_donn.flags: lr_donn_forward adds its detector sums and intensity map
 * into d_sums / d_intensity instead of overwriting them (d_field_out must
 * then be NULL).  This is the detector of the multi-channel DONN of §5.6.1:
 * several optical channels (each an lr_donn with its own masks and input)
 * project onto one detector, where their intensities add.  A training step
 * of such a system runs lr_donn_forward per channel (the first without,
 * the others with LR_ACCUMULATE, or all with it on zeroed outputs),
 * lr_loss on the merged sums, and lr_donn_backward per channel with the
 * same d_grad_sums: the merged sums are the sum of the channels' sums, so
 * every channel receives the whole dL/dS. */
#define LR_ACCUMULATE 1

/* lr_donn.flags: lr_donn_forward runs one pass per layer even where it would
 * otherwise keep the whole field of a sample on chip.  Without it, a forward
 * call on the Fresnel path with n == n_fft in {64, 100, 128} (the field fits
 * in one compute unit's shared memory), no saved state and no skip field
 * (and, at 100 and 128, at least one sample per compute unit of the
 * device) runs every hop and modulation of a sample in one workgroup and
 * moves only
 * the amplitudes and the requested outputs (sums, intensity map, detector
 * field) through memory.  Both paths compute the same outputs (to
 * rounding); the flag exists to compare them. */
#define LR_LAYER_PASSES 2

/* lr_donn.flags: lr_donn_forward keeps the whole field of a sample on chip
 * also where one pass per layer is the default: Fresnel path, n == n_fft in
 * {64, 100, 128, 200}, no saved state, no skip field.  At 200 the field
 * (320 KB) is held half in shared memory and half in registers; the layer
 * passes measured faster there, so only this flag selects it.  Not together
 * with LR_LAYER_PASSES (LR_E_ARG). */
#define LR_WHOLE_FIELD 4

/* Transfer function of one hop (§3.1.1, Eqs. (fresnel), (sommerfeld), (r01),
 * (forward_diff), (fraunhofer)).
 * Writes d_H[ky][kx], ky, kx in [0, n_fft), at the unshifted DFT frequencies
 * f = k'/(n_fft*pixel_pitch), k' = k for k < (n_fft+1)/2 else k - n_fft.
 * Evaluated in float64 on the host (the phase kz is reduced modulo 2*pi
 * before the rest is added) and rounded once to complex64.
 *   LR_FRESNEL, LR_ANGULAR_SPECTRUM: the analytic transfer functions; the
 *     angular spectrum decays as exp(-kz sqrt(lambda^2 f^2 - 1)) on
 *     evanescent frequencies.
 *   LR_FRESNEL_IR, LR_RS_IR: pixel_pitch^2 times the 2-D DFT (float64,
 *     mixed radix) of the kernel sampled at the displacements
 *     (y', x') * pixel_pitch, y' and x' wrapped like k'.  n_fft must have no
 *     prime factor above 5; distance > 0.
 *   LR_FRAUNHOFER: not a transfer function but the far-field output table
 *     used by lr_propagate: entry (dy, dx) is
 *     (-1)^(dy+dx) pixel_pitch^2 exp(jkz) exp(jk(x^2+y^2)/(2z)) / (j lambda z)
 *     at x = dx' lambda z/(n_fft pixel_pitch), y likewise.  n_fft even;
 *     distance > 0.
 * Blocking: returns after the upload has completed.
 * Errors: LR_E_NULL (d_H), LR_E_ARG (non-finite or non-positive lambda / pitch,
 * non-finite z, z <= 0 for the last three), LR_E_APPROX, LR_E_SIZE (n_fft < 1
 * or > 4096, or not as required above), LR_E_HIP. */
int lr_tf_build(double wavelength, double pixel_pitch, double distance, int32_t approx,
                int32_t n_fft, lr_c64* d_H, void* stream);

/* Bytes of caller-provided workspace needed by `op` for this network and
 * batch; returns a negative lr_status on invalid arguments. */
int64_t lr_workspace_size(const lr_donn* net, int32_t batch, int32_t op);

/* Bytes of the saved-state buffer that lr_donn_forward fills for
 * lr_donn_backward: L+1 complex64 fields of [batch][n][n].  Their content is
 * internal state of the two calls, valid only for the same network, batch
 * and phase masks.  (The Fresnel path keeps the field each of its separable
 * passes wrote, from which the backward pass recomputes the activations
 * U_l; the angular-spectrum path keeps U_1..U_L and U_D.)  Negative
 * lr_status on invalid arguments. */
int64_t lr_saved_size(const lr_donn* net, int32_t batch);

/* One hop of `batch` fields (§3.1.1): d_out = P_z(d_in), or its Hilbert
 * adjoint P_z^H (the same pad/crop with conj(H), i.e. back-propagation) when
 * adjoint != 0.  Uses net->wavelength..net->d_H; net->num_layers, gamma and
 * det are ignored.  d_in, d_out: complex64 [batch][n][n]; they must not alias.
 * d_work: >= lr_workspace_size(net, batch, LR_OP_PROPAGATE) bytes.
 * With net->approx == LR_FRAUNHOFER (d_H the far-field table of lr_tf_build)
 * d_out is the far field of Eq. (fraunhofer), complex64 [batch][n_fft][n_fft]
 * on the centred output grid: sample (ky, kx) at
 * ((ky - n_fft/2), (kx - n_fft/2)) * lambda z/(n_fft pixel_pitch), the input
 * sitting centred in the n_fft grid (sample i at (i - n_fft/2) pixel_pitch);
 * adjoint must be 0.  lr_donn_forward / lr_donn_backward reject
 * LR_FRAUNHOFER (LR_E_APPROX): the far field does not chain layers. */
int lr_propagate(const lr_donn* net, int32_t batch, const lr_c64* d_in, lr_c64* d_out,
                 int32_t adjoint, void* d_work, size_t work_bytes, void* stream);

/* lr_propagate for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same hop, with the workspace taken from a fixed array of
 * LR_NOALLOC_SCRATCH_BYTES bytes that the library keeps in device memory on
 * every GPU it runs on until the process ends.  The call itself allocates
 * nothing (no hipMalloc, no events: kernel timing skips it).  Arguments,
 * results and errors as lr_propagate; additionally LR_E_WORKSPACE when
 * lr_workspace_size(net, batch, LR_OP_PROPAGATE) exceeds the array
 * (lr_propagate_noalloc_limit() returns its size), checked before anything
 * is enqueued.  All calls on one GPU share that GPU's array: calls that can
 * overlap on one GPU (different streams or host threads without ordering)
 * race, and the caller must order them. */
#define LR_NOALLOC_SCRATCH_BYTES (32u << 20)
int lr_propagate_noalloc(const lr_donn* net, int32_t batch, const lr_c64* d_in, lr_c64* d_out, int32_t adjoint,
                         void* stream);
int64_t lr_propagate_noalloc_limit(void);

/* Detector readout (§2.1): d_sums[b][k] = sum over region k of |d_field[b]|^2.
 * d_field: complex64 [batch][n][n]; d_sums: float32 [batch][det->num].
 * Regions must lie inside the n x n plane. */
int lr_detector_readout(const lr_c64* d_field, int32_t batch, int32_t n, const lr_detector* det,
                        float* d_sums, void* stream);

/* Forward pass of the network (§3.1, §2.1) on a batch.
 *   d_amp       float32 [batch][n][n] input amplitudes (the encoded image)
 *   d_phi       float32 [L][n][n] phase masks, radians
 *   d_saved     nullable; lr_saved_size() bytes; filled for lr_donn_backward
 *   d_sums      nullable; float32 [batch][det.num] detector sums (needs det.num > 0)
 *   d_intensity nullable; float32 [batch][n][n] detector-plane |U_D|^2
 *   d_field_out nullable; complex64 [batch][n][n] detector-plane field U_D
 *   d_work      >= lr_workspace_size(net, batch, LR_OP_FORWARD) bytes */
int lr_donn_forward(const lr_donn* net, int32_t batch, const float* d_amp, const float* d_phi,
                    void* d_saved, float* d_sums, float* d_intensity, lr_c64* d_field_out,
                    void* d_work, size_t work_bytes, void* stream);

/* Gradient of the loss with respect to every phase mask (§2.1), summed over
 * the batch, using the state saved by lr_donn_forward.  Exactly one seed:
 *   d_labels (int32 [batch], with d_sums from the forward pass): softmax
 *       cross-entropy over the detector sums, mean over the batch; the loss
 *       value is written to d_loss (nullable float32 scalar);
 *   d_grad_sums (float32 [batch][det.num]): upstream dL/dS;
 *   d_grad_intensity (float32 [batch][n][n]): upstream dL/dI.
 * Gradients follow the Wirtinger convention dL/dRe + j dL/dIm, so
 * d_grad_phi[l] = sum_b Im(conj(U_l) * G_l), G_l the gradient with respect to
 * the modulated field of layer l.  d_grad_phi: float32 [L][n][n], overwritten.
 * The batch reduction runs in a fixed order (bitwise reproducible).
 * d_work: >= lr_workspace_size(net, batch, LR_OP_BACKWARD) bytes. */
int lr_donn_backward(const lr_donn* net, int32_t batch, const float* d_phi, const void* d_saved,
                     const float* d_sums, const int32_t* d_labels, const float* d_grad_sums,
                     const float* d_grad_intensity, float* d_loss, float* d_grad_phi,
                     void* d_work, size_t work_bytes, void* stream);

/* Losses of the detector sums (§2.1: the class whose region collects the most
 * light is the prediction; §5.1: the prototypes are trained with an MSE loss
 * on one-hot labels). */
enum lr_loss_kind {
  LR_LOSS_SOFTMAX_CE = 0,   /* -log softmax(S)_t */
  LR_LOSS_SOFTMAX_MSE = 1   /* ||softmax(S) - onehot(t)||^2, summed over classes */
};

/* Loss of a batch of detector sums, averaged over the batch, and its
 * gradient dL/dS for lr_donn_backward's d_grad_sums.
 *   d_sums       float32 [batch][classes] (the region sums of lr_donn_forward)
 *   d_labels     int32 [batch], class indices in [0, classes); a label out of
 *                range makes the loss NaN
 *   d_loss       nullable float32 scalar
 *   d_grad_sums  nullable float32 [batch][classes], must not alias d_sums
 * At least one of d_loss, d_grad_sums.  The batch mean is summed in a fixed
 * order.  Errors: LR_E_ARG (unknown kind), LR_E_SIZE (batch < 0, classes not
 * in 1..LR_MAX_REGIONS), LR_E_NULL, LR_E_ALIAS. */
int lr_loss(int32_t kind, const float* d_sums, const int32_t* d_labels, int32_t batch, int32_t classes,
            float* d_loss, float* d_grad_sums, void* stream);

/* Layer normalisation before the detector of the segmentation DONN (§5.6.2,
 * used in training only): each of the batch maps of count values (an
 * intensity map, count = n*n) is normalised to zero mean and unit variance,
 *   y = (x - mean) / sqrt(var + eps),  var the biased variance,
 * without a learnable gain or bias.  lr_layer_norm_backward returns
 *   dL/dx = rstd * (g - mean(g) - y * mean(g * y)),  g = dL/dy, rstd = 1/sqrt(var + eps).
 *   d_x, d_y        float32 [batch][count]; d_y may be d_x
 *   d_stats         float32 [batch][2]: (mean, rstd) of each map, written by
 *                   lr_layer_norm and read by lr_layer_norm_backward
 *   d_grad_y, d_grad_x  float32 [batch][count]; d_grad_x may be d_grad_y
 *   d_work          lr_layer_norm_workspace_size(batch, count) bytes
 * The statistics are merged over fixed chunks of 4096 values in a fixed
 * order (results are reproducible).  Errors: LR_E_SIZE (batch < 0 or
 * > 65535, count < 1 or > 2^28), LR_E_ARG (eps not finite or < 0),
 * LR_E_NULL, LR_E_WORKSPACE, LR_E_ALIAS (maps overlapping other than in the
 * two in-place forms above, or d_stats or the workspace overlapping a map),
 * LR_E_HIP.  batch = 0 does nothing. */
int64_t lr_layer_norm_workspace_size(int32_t batch, int64_t count);
int lr_layer_norm(const float* d_x, int32_t batch, int64_t count, float eps, float* d_y, float* d_stats,
                  void* d_work, size_t work_bytes, void* stream);
int lr_layer_norm_backward(const float* d_grad_y, const float* d_y, const float* d_stats, int32_t batch,
                           int64_t count, float* d_grad_x, void* d_work, size_t work_bytes, void* stream);

/* Codesign layer (§3.2): trainable scores over the discrete, measured
 * optical responses of the hardware, relaxed with Gumbel-Softmax so that the
 * masks train directly on the available device levels.
 *   d_logits, d_noise: float32 [count][levels], the scores of each pixel's
 *     levels and Gumbel(0, 1) draws (-log(-log U)), supplied by the caller;
 *   d_levels: float32 [levels], the device's phase responses in radians;
 *   w = softmax((logits + noise) / tau) over the levels of a pixel.
 * lr_codesign_phase writes d_phi[p] = sum_k w_k levels_k, or with hard != 0
 * the level with the largest float32 logits + noise (the first on ties):
 * the phase masks (count = L n n) that lr_donn_forward then takes.
 * lr_codesign_backward writes dL/dlogits [count][levels] =
 * w_j (levels_j - sum_k w_k levels_k) dL/dphi / tau from dL/dphi [count]
 * (lr_donn_backward's output); for the hard layer this is the
 * straight-through gradient.  1 <= levels <= LR_MAX_LEVELS; tau finite > 0.
 * Errors: LR_E_SIZE, LR_E_ARG, LR_E_NULL, LR_E_ALIAS (output aliases an
 * input). */
#define LR_MAX_LEVELS 1024
int lr_codesign_phase(const float* d_logits, const float* d_noise, const float* d_levels, int32_t levels,
                      int64_t count, float tau, int32_t hard, float* d_phi, void* stream);
int lr_codesign_backward(const float* d_logits, const float* d_noise, const float* d_levels, int32_t levels,
                         int64_t count, float tau, const float* d_grad_phi, float* d_grad_logits, void* stream);

/* One Adam step on the phase masks (§5.1 trains them with Adam, learning
 * rate 0.5), element-wise over count floats, in place:
 *   m = beta1 m + (1 - beta1) g,  v = beta2 v + (1 - beta2) g^2,
 *   phi -= lr * (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps).
 * d_phi, d_m, d_v are updated; d_m and d_v start at zero before step 1.
 * step counts from 1.  No two pointers may be equal.  Errors: LR_E_SIZE
 * (count < 0, step < 1), LR_E_ARG (lr or eps not finite, eps < 0, beta not in
 * [0, 1)), LR_E_NULL, LR_E_ALIAS. */
int lr_adam_update(float* d_phi, const float* d_grad, float* d_m, float* d_v, int64_t count, int32_t step,
                   float lr, float beta1, float beta2, float eps, void* stream);

/* Human-readable name of an lr_status. */
const char* lr_status_string(int status);

/* Kernel timing for measurement: while enabled, every kernel the library
 * launches is bracketed by HIP events on its stream.  lr_kernel_timing_report
 * waits for the recorded events and writes a JSON object
 * {"<kernel>": {"count": c, "ms": total}, ...} into buf (NUL terminated,
 * truncated to len); it returns the number of characters needed, or a
 * negative lr_status.  lr_kernel_timing(1) clears earlier records. */
int lr_kernel_timing(int32_t enable);
int lr_kernel_timing_report(char* buf, size_t len);

int32_t lr_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LR_H_ */
