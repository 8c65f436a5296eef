"""Float64 reference of the DONN emulation and training step (test infrastructure only).

This module is the plain, slow, obviously-correct statement of what the
hot path computes, written from the LightRidge paper (arXiv 2306.11268):

* input encoding (§3.1, physics-kernel overview: the pixel value is the
  amplitude, the phase starts at zero);
* free-space diffraction as a spectral product (§3.1.1, Eqs. (forward_diff)
  and (diffraction_freq)) with the Fresnel transfer function (Eq. (fresnel))
  or the Rayleigh-Sommerfeld one in angular-spectrum form (Eqs. (sommerfeld),
  (r01)), or with H the sampled impulse response's DFT (the Fresnel or the
  Rayleigh-Sommerfeld kernel on the grid of displacements);
* the Fraunhofer far field (Eq. (fraunhofer)) as one scaled Fourier sum;
* phase modulation by exp(j*phi) with the amplitude scale gamma
  (§3.1.2, Eqs. (phase_euler), (phase_mod_matrix); §3.2);
* the detector: intensity |U|^2 summed over rectangular regions (§2.1);
* a loss on the detector sums and the gradient with respect to every phase
  mask (§2.1: the system is differentiable from detector to source).

Readings taken where the paper is silent or ambiguous:

* transfer functions are the analytic ones, sampled on the unshifted DFT
  frequency grid f_k = k'/(M*dx), k' = k for k < (M+1)//2 else k - M; the
  impulse-response variants sample the kernel h at the displacements
  d_i = i'*dx on the same wrapped index grid and take H = dx^2 * DFT2(h),
  which makes the spectral product the discrete linear convolution
  sum_xi U(xi) h(x - xi) dx^2 of Eq. (forward_diff) on the padded grid;
* the Fraunhofer input and output grids are centred: input sample i sits at
  xi = (i - M/2)*dx, output sample k at x = (k - M/2)*lambda*z/(M*dx);
* forward DFT uses exp(-2*pi*i*jk/M) and is unnormalised, the inverse uses
  exp(+2*pi*i*jk/M) / M (per axis);
* an L-layer network performs L+1 hops of the same distance z: source to
  layer 1, layer to layer, and layer L to the detector;
* with an FFT grid M larger than the layer size n the layer sits centred at
  offset (M-n)/2 in a zero field; after every hop the field is cropped back
  to the n x n aperture;
* gamma multiplies the modulated field of every layer;
* the loss of the training step is softmax cross-entropy over the raw
  detector sums, averaged over the batch; a full-map upstream gradient
  dL/dI may be given instead;
* gradients follow the Wirtinger convention g = dL/dRe(U) + j dL/dIm(U), so
  dL/dI contributes 2*(dL/dI)*U and dL/dphi_l = Im(conj(U_l) * g_l), with
  g_l the gradient with respect to the modulated field of layer l;
* the segmentation DONN (§5.6.2), whose topology the paper gives only in a
  figure: its optical skip connection is read as the residual form
  y = F(x) + x with the whole diffractive stack as F, i.e. the input field
  is relayed unchanged to the detector plane and added to the field the
  last hop delivers, U_D = P(U_L) + U_0 (``skip``: any field added there);
  its layer normalisation (training only, before the detector) normalises
  each sample's intensity map over its n x n pixels to zero mean and unit
  variance, (I - mean) / sqrt(var + eps) with the biased variance, without
  a learnable gain or bias.
"""

from __future__ import annotations

import dataclasses
from typing import Optional, Sequence

import numpy as np

FRESNEL = 0
ANGULAR_SPECTRUM = 1
FRESNEL_IR = 2   # H = dx^2 DFT2 of the sampled Fresnel kernel (Eq. (fresnel))
RS_IR = 3        # H = dx^2 DFT2 of the sampled Rayleigh-Sommerfeld kernel (Eqs. (sommerfeld), (r01))


# ---------------------------------------------------------------------------
# Discrete Fourier transforms by definition (§3.1.1: the convolution of
# Eq. (forward_diff) is evaluated spectrally, Eq. (diffraction_freq)).
# ---------------------------------------------------------------------------

def dft_matrix(m: int, inverse: bool = False) -> np.ndarray:
    """W[j, k] = exp(-/+ 2*pi*i * ((j*k) mod m) / m), complex128 [m, m].

    The exponent is reduced modulo m in integer arithmetic before it is
    scaled, so every entry is a correctly evaluated root of unity.  The
    inverse matrix carries no 1/m factor (see idft2).
    """
    j = np.arange(m, dtype=np.int64)
    e = np.outer(j, j) % m
    sign = 1.0 if inverse else -1.0
    return np.exp(sign * 2j * np.pi * e.astype(np.float64) / m)


def dft2(x: np.ndarray) -> np.ndarray:
    """Unnormalised 2-D DFT over the last two axes: F = W_rows @ X @ W_cols^T."""
    m0, m1 = x.shape[-2:]
    return dft_matrix(m0) @ x @ dft_matrix(m1).T


def idft2(y: np.ndarray) -> np.ndarray:
    """Inverse 2-D DFT over the last two axes, normalised by 1/(m0*m1)."""
    m0, m1 = y.shape[-2:]
    return (dft_matrix(m0, True) @ y @ dft_matrix(m1, True).T) / (m0 * m1)


# ---------------------------------------------------------------------------
# Transfer functions (§3.1.1).
# ---------------------------------------------------------------------------

def frequencies(m: int, pixel_pitch: float) -> np.ndarray:
    """Spatial frequencies of the unshifted DFT grid, in cycles per metre."""
    k = np.arange(m, dtype=np.int64)
    ks = np.where(k < (m + 1) // 2, k, k - m)
    return ks.astype(np.float64) / (m * pixel_pitch)


def displacements(m: int, pixel_pitch: float) -> np.ndarray:
    """Displacements d_i = i' * dx of the wrapped index grid (i' = i for
    i < (m+1)//2 else i - m), in metres: index i of a circular convolution
    kernel holds the kernel at d_i."""
    i = np.arange(m, dtype=np.int64)
    ii = np.where(i < (m + 1) // 2, i, i - m)
    return ii.astype(np.float64) * pixel_pitch


def impulse_response(wavelength: float, pixel_pitch: float, distance: float,
                     approx: int, m: int) -> np.ndarray:
    """The diffraction kernel h(x - xi, y - eta, z) of Eq. (forward_diff) at the
    m x m displacements of the wrapped grid, complex128.

    FRESNEL_IR (Eq. (fresnel)): h = exp(jkz)/(j*lambda*z) * exp(jk(dx^2+dy^2)/(2z)).
    RS_IR (Eqs. (sommerfeld), (r01)): h = z/(j*lambda) * exp(jkr)/r^2 with
    r = sqrt(z^2 + dx^2 + dy^2).
    The phase kz is carried as exp(jkz) and the rest of the phase added
    separately (k(r - z) = k(dx^2 + dy^2)/(r + z)), so that no large argument
    loses precision.
    """
    d = displacements(m, pixel_pitch)
    rho2 = d[:, None] ** 2 + d[None, :] ** 2
    k = 2.0 * np.pi / wavelength
    z = distance
    ekz = np.exp(1j * 2.0 * np.pi * np.fmod(z / wavelength, 1.0))
    if approx == FRESNEL_IR:
        return ekz / (1j * wavelength * z) * np.exp(1j * k * rho2 / (2.0 * z))
    if approx == RS_IR:
        r = np.sqrt(z * z + rho2)
        return z / (1j * wavelength) * ekz * np.exp(1j * k * rho2 / (r + z)) / (r * r)
    raise ValueError(f"no impulse response for approximation {approx}")


def transfer_function(wavelength: float, pixel_pitch: float, distance: float,
                      approx: int, m: int) -> np.ndarray:
    """H[ky, kx] for one hop of length ``distance`` on an m x m grid, complex128.

    FRESNEL (Eq. (fresnel)): the Fourier transform of the paraxial kernel
        exp(jkz)/(j*lambda*z) * exp(jk((x-xi)^2+(y-eta)^2)/(2z)),
    i.e. H = exp(jkz) * exp(-j*pi*lambda*z*(fx^2 + fy^2)).

    ANGULAR_SPECTRUM (Eqs. (sommerfeld), (r01)): the Fourier transform of the
    Rayleigh-Sommerfeld kernel, H = exp(jkz*sqrt(1 - lambda^2 (fx^2 + fy^2)))
    on propagating frequencies and exp(-kz*sqrt(lambda^2 f^2 - 1)) on
    evanescent ones.

    FRESNEL_IR, RS_IR: dx^2 times the DFT of the sampled kernel
    (impulse_response), the discrete form of Eq. (forward_diff).
    """
    if approx in (FRESNEL_IR, RS_IR):
        return pixel_pitch ** 2 * dft2(impulse_response(wavelength, pixel_pitch, distance, approx, m))
    f = frequencies(m, pixel_pitch)
    f2 = f[:, None] ** 2 + f[None, :] ** 2
    k = 2.0 * np.pi / wavelength
    if approx == FRESNEL:
        return np.exp(1j * k * distance) * np.exp(-1j * np.pi * wavelength * distance * f2)
    if approx == ANGULAR_SPECTRUM:
        arg = 1.0 - (wavelength ** 2) * f2
        prop = arg >= 0.0
        h = np.empty((m, m), dtype=np.complex128)
        h[prop] = np.exp(1j * k * distance * np.sqrt(arg[prop]))
        h[~prop] = np.exp(-k * distance * np.sqrt(-arg[~prop]))
        return h
    raise ValueError(f"unsupported approximation {approx}")


# ---------------------------------------------------------------------------
# One hop: pad -> DFT2 -> x H -> IDFT2 -> crop (§3.1.1).
# ---------------------------------------------------------------------------

def propagate(u: np.ndarray, h: np.ndarray, adjoint: bool = False) -> np.ndarray:
    """Propagate fields u [..., n, n] by one hop with transfer function h [m, m].

    The n x n field sits centred in an m x m zero grid (offset (m-n)/2); the
    result is cropped back to the same n x n window.  ``adjoint`` applies the
    Hilbert adjoint of that linear map, which is the same pad/crop with conj(h).
    """
    m = h.shape[0]
    n = u.shape[-1]
    if u.shape[-2] != n or h.shape != (m, m) or n > m or (m - n) % 2:
        raise ValueError("field must be n x n with n <= m and m - n even")
    o = (m - n) // 2
    x = np.zeros(u.shape[:-2] + (m, m), dtype=np.complex128)
    x[..., o:o + n, o:o + n] = u
    spec = dft2(x) * (np.conj(h) if adjoint else h)
    return idft2(spec)[..., o:o + n, o:o + n]


# ---------------------------------------------------------------------------
# Fraunhofer far field (§3.1.1, Eq. (fraunhofer)).
# ---------------------------------------------------------------------------

def fraunhofer(u: np.ndarray, wavelength: float, pixel_pitch: float, distance: float, m: int) -> np.ndarray:
    """Far field of fields u [..., n, n] on the centred m x m output grid.

    U(x, y) = exp(jkz) exp(jk(x^2+y^2)/(2z)) / (j*lambda*z)
              * sum_{xi, eta} U(xi, eta) exp(-j*2*pi*(x*xi + y*eta)/(lambda*z)) dx^2,
    the input sitting centred in the m x m grid (sample i at xi = (i - m/2) dx)
    and the output at x = (k - m/2) * lambda*z/(m*dx), k < m (pitch
    fraunhofer_pitch).  With those grids the exponent is
    -2*pi*i*(k - m/2)*(i - m/2)/m, evaluated with the product reduced modulo m
    in integers.  m must be even.
    """
    n = u.shape[-1]
    if u.shape[-2] != n or n > m or (m - n) % 2 or m % 2:
        raise ValueError("field must be n x n with n <= m, m - n even and m even")
    o = (m - n) // 2
    x = np.zeros(u.shape[:-2] + (m, m), dtype=np.complex128)
    x[..., o:o + n, o:o + n] = u
    c = np.arange(m, dtype=np.int64) - m // 2
    e = np.outer(c, c) % m
    w = np.exp(-2j * np.pi * e.astype(np.float64) / m)
    s = w @ x @ w.T * pixel_pitch ** 2
    k = 2.0 * np.pi / wavelength
    xo = c.astype(np.float64) * fraunhofer_pitch(wavelength, pixel_pitch, distance, m)
    r2 = xo[:, None] ** 2 + xo[None, :] ** 2
    ekz = np.exp(1j * 2.0 * np.pi * np.fmod(distance / wavelength, 1.0))
    return ekz * np.exp(1j * k * r2 / (2.0 * distance)) / (1j * wavelength * distance) * s


def fraunhofer_pitch(wavelength: float, pixel_pitch: float, distance: float, m: int) -> float:
    """Sample pitch of the Fraunhofer output plane, lambda*z/(m*dx)."""
    return wavelength * distance / (m * pixel_pitch)


# ---------------------------------------------------------------------------
# Encoding, modulation, detection (§3.1, §3.1.2, §3.2, §2.1).
# ---------------------------------------------------------------------------

def encode_amplitude(amp: np.ndarray) -> np.ndarray:
    """U0 = A * exp(j*0): the pixel value is the amplitude (§3.1)."""
    return np.asarray(amp, dtype=np.float64).astype(np.complex128)


def modulate(v: np.ndarray, phi: np.ndarray, gamma: float = 1.0) -> np.ndarray:
    """U = gamma * V * exp(j*phi) (Eq. (phase_mod_matrix), gamma from §3.2)."""
    return gamma * v * np.exp(1j * np.asarray(phi, dtype=np.float64))


def intensity(u: np.ndarray) -> np.ndarray:
    """I = |U|^2."""
    return u.real ** 2 + u.imag ** 2


@dataclasses.dataclass(frozen=True)
class Detector:
    """K square regions of side ``size`` with top-left corners (y0[k], x0[k])."""
    size: int
    y0: Sequence[int]
    x0: Sequence[int]

    @property
    def num(self) -> int:
        return len(self.y0)


def detector_readout(i_map: np.ndarray, det: Detector) -> np.ndarray:
    """S[b, k] = sum of I over region k (§2.1: one region per class)."""
    s = det.size
    out = np.zeros(i_map.shape[:-2] + (det.num,), dtype=np.float64)
    for k, (y, x) in enumerate(zip(det.y0, det.x0)):
        out[..., k] = i_map[..., y:y + s, x:x + s].sum(axis=(-2, -1))
    return out


def region_scatter(grad_sums: np.ndarray, det: Detector, n: int) -> np.ndarray:
    """dL/dI [B, n, n] from dL/dS [B, K]: the adjoint of detector_readout."""
    s = det.size
    g = np.zeros(grad_sums.shape[:-1] + (n, n), dtype=np.float64)
    for k, (y, x) in enumerate(zip(det.y0, det.x0)):
        g[..., y:y + s, x:x + s] += grad_sums[..., k, None, None]
    return g


# ---------------------------------------------------------------------------
# The network (§3.1: diffraction and modulation alternate layer by layer,
# then one more hop to the detector plane).
# ---------------------------------------------------------------------------

def donn_forward(amp: np.ndarray, phi: np.ndarray, h: np.ndarray, gamma: float = 1.0,
                 det: Optional[Detector] = None, skip: Optional[np.ndarray] = None) -> dict:
    """Forward pass of an L-layer DONN on a batch.

    amp [B, n, n] amplitudes, phi [L, n, n] phase masks, h [m, m].
    Returns acts [L, B, n, n] (modulated field of each layer), field (the
    detector-plane field U_D), intensity |U_D|^2 and, with a detector, sums.
    skip [B, n, n] (complex), when given, is added to the detector-plane
    field (the segmentation DONN's optical skip connection, §5.6.2: the
    input field itself under the residual reading).
    """
    u = encode_amplitude(amp)
    phi = np.asarray(phi, dtype=np.float64)
    acts = []
    for layer in range(phi.shape[0]):
        u = modulate(propagate(u, h), phi[layer], gamma)
        acts.append(u)
    ud = propagate(u, h)
    if skip is not None:
        ud = ud + np.asarray(skip, dtype=np.complex128)
    i_map = intensity(ud)
    return {
        "acts": np.stack(acts) if acts else np.zeros((0,) + u.shape, np.complex128),
        "field": ud,
        "intensity": i_map,
        "sums": detector_readout(i_map, det) if det is not None else None,
    }


def softmax_cross_entropy(sums: np.ndarray, labels: np.ndarray):
    """Mean softmax cross-entropy over the batch and its gradient dL/dS.

    The detector sums are the logits; the paper trains on Softmax(I)
    against one-hot labels (§2.1) and this is the cross-entropy form of it.
    """
    s = np.asarray(sums, dtype=np.float64)
    b = s.shape[0]
    shift = s - s.max(axis=1, keepdims=True)
    lse = np.log(np.exp(shift).sum(axis=1))
    t = np.asarray(labels, dtype=np.int64)
    loss = float(np.mean(lse - shift[np.arange(b), t]))
    p = np.exp(shift - lse[:, None])
    grad = p.copy()
    grad[np.arange(b), t] -= 1.0
    return loss, grad / b


def mse_softmax_loss(sums: np.ndarray, labels: np.ndarray):
    """The paper's loss form ||Softmax(I) - t||^2 (§2.1), mean over the batch.

    Reading: the squared norm summed over classes, averaged over samples.
    Returns (loss, dL/dS).
    """
    s = np.asarray(sums, dtype=np.float64)
    b, k = s.shape
    shift = s - s.max(axis=1, keepdims=True)
    e = np.exp(shift)
    p = e / e.sum(axis=1, keepdims=True)
    t = np.zeros_like(p)
    t[np.arange(b), np.asarray(labels, dtype=np.int64)] = 1.0
    r = p - t
    loss = float(np.mean((r ** 2).sum(axis=1)))
    dp = 2.0 * r / b
    # softmax Jacobian: dS_j = p_j * (dp_j - sum_i dp_i p_i)
    grad = p * (dp - (dp * p).sum(axis=1, keepdims=True))
    return loss, grad


def donn_backward(fwd: dict, phi: np.ndarray, h: np.ndarray, gamma: float = 1.0,
                  det: Optional[Detector] = None, grad_sums: Optional[np.ndarray] = None,
                  grad_intensity: Optional[np.ndarray] = None) -> np.ndarray:
    """dL/dphi [L, n, n], summed over the batch.

    Either grad_sums (dL/dS, needs det) or grad_intensity (dL/dI) seeds the
    adjoint.  The adjoint of each hop is the same pad/crop propagation with
    conj(H); the adjoint of the modulation multiplies by gamma*exp(-j*phi).
    """
    ud = fwd["field"]
    acts = fwd["acts"]
    n = ud.shape[-1]
    if (grad_sums is None) == (grad_intensity is None):
        raise ValueError("give exactly one of grad_sums / grad_intensity")
    if grad_sums is not None:
        g_i = region_scatter(np.asarray(grad_sums, dtype=np.float64), det, n)
    else:
        g_i = np.asarray(grad_intensity, dtype=np.float64)
    phi = np.asarray(phi, dtype=np.float64)
    n_layers = phi.shape[0]
    g = propagate(2.0 * g_i * ud, h, adjoint=True)
    dphi = np.zeros((n_layers, n, n), dtype=np.float64)
    for layer in range(n_layers - 1, -1, -1):
        dphi[layer] = np.imag(np.conj(acts[layer]) * g).sum(axis=0)
        g = gamma * np.exp(-1j * phi[layer]) * g
        if layer > 0:
            g = propagate(g, h, adjoint=True)
    return dphi


# ---------------------------------------------------------------------------
# Layer normalisation before the detector of the segmentation DONN (§5.6.2,
# training only), per sample over the intensity map.
# ---------------------------------------------------------------------------

def layer_norm(i_map: np.ndarray, eps: float = 1e-5):
    """(I - mean) / sqrt(var + eps) over the last two axes of each sample
    (biased variance).  Returns (normalised map, mean [B], 1/sqrt(var+eps) [B])."""
    x = np.asarray(i_map, dtype=np.float64)
    mean = x.mean(axis=(-2, -1))
    var = ((x - mean[:, None, None]) ** 2).mean(axis=(-2, -1))
    rstd = 1.0 / np.sqrt(var + eps)
    return (x - mean[:, None, None]) * rstd[:, None, None], mean, rstd


def layer_norm_backward(grad_out: np.ndarray, normed: np.ndarray, rstd: np.ndarray) -> np.ndarray:
    """dL/dI from dL/d(normalised map): with y = (x - mean) * rstd over M
    pixels, dL/dx = rstd * (g - mean(g) - y * mean(g * y))."""
    g = np.asarray(grad_out, dtype=np.float64)
    y = np.asarray(normed, dtype=np.float64)
    mg = g.mean(axis=(-2, -1))[:, None, None]
    mgy = (g * y).mean(axis=(-2, -1))[:, None, None]
    return np.asarray(rstd, dtype=np.float64)[:, None, None] * (g - mg - y * mgy)


# ---------------------------------------------------------------------------
# Optimiser of the training step (§5.1: the prototypes' phase masks are
# trained with Adam, learning rate 0.5, batch 500).
# ---------------------------------------------------------------------------

def multichannel_forward(amps: Sequence[np.ndarray], phis: Sequence[np.ndarray], h: np.ndarray, gamma: float,
                         det: Detector):
    """Multi-channel DONN (§5.6.1): channel c is a DONN with its own masks
    phis[c] on its own input amps[c]; the channels project onto one detector,
    where their intensities add, so the merged region sums are the sum of the
    channels' sums.  Returns (per-channel forward dicts, merged sums)."""
    fwds = [donn_forward(a, p, h, gamma, det) for a, p in zip(amps, phis)]
    merged = fwds[0]["sums"].copy()
    for f in fwds[1:]:
        merged = merged + f["sums"]
    return fwds, merged


def multichannel_backward(fwds, phis: Sequence[np.ndarray], h: np.ndarray, gamma: float, det: Detector,
                          grad_sums: np.ndarray):
    """dL/dphi of every channel for an upstream dL/dS of the merged sums: the
    merged sums depend on each channel's sums with unit weight, so every
    channel's backward pass receives the same dL/dS."""
    return [donn_backward(f, p, h, gamma, det, grad_sums=grad_sums) for f, p in zip(fwds, phis)]


def codesign_phase(logits: np.ndarray, noise: np.ndarray, levels: np.ndarray, tau: float, hard: bool = False):
    """Hardware-level phase of the codesign layer (§3.2: the measured,
    discrete device responses mapped with Gumbel-Softmax).

    logits, noise [..., K]: per-pixel scores of the K device levels and the
    Gumbel(0, 1) draws; levels [K]: the device's phase values (radians).
    w = softmax((logits + noise) / tau) over K; the phase is sum_k w_k
    levels_k, or with ``hard`` the level of the largest logits + noise (the
    straight-through estimator keeps the soft w for the gradient).  The hard
    choice is an integer decision and is taken on float32 logits + noise, the
    precision of the device path.
    Returns (phi [...], w [..., K])."""
    y = (np.asarray(logits, np.float64) + np.asarray(noise, np.float64)) / tau
    y = y - y.max(axis=-1, keepdims=True)
    e = np.exp(y)
    w = e / e.sum(axis=-1, keepdims=True)
    lv = np.asarray(levels, np.float64)
    if hard:
        # an integer decision: taken on the float32 sums the device forms (first index on ties)
        score = np.asarray(logits, np.float32) + np.asarray(noise, np.float32)
        phi = lv[np.argmax(score, axis=-1)]
    else:
        phi = w @ lv
    return phi, w


def codesign_backward(w: np.ndarray, levels: np.ndarray, tau: float, grad_phi: np.ndarray) -> np.ndarray:
    """dL/dlogits of the codesign layer from dL/dphi through the softmax
    Jacobian of the soft phase sum_k w_k levels_k (also the straight-through
    gradient of the hard layer):
    dL/dlogit_j = w_j (levels_j - sum_k w_k levels_k) dL/dphi / tau."""
    lv = np.asarray(levels, np.float64)
    mean = w @ lv
    return w * (lv - mean[..., None]) * (np.asarray(grad_phi, np.float64)[..., None] / tau)


def adam_update(phi: np.ndarray, grad: np.ndarray, m: np.ndarray, v: np.ndarray, step: int,
                lr: float = 0.5, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8):
    """One Adam step (Kingma and Ba, 2014, Algorithm 1) on the phase masks.

    step is the 1-based step count t.  Returns (phi', m', v'), float64:
      m' = beta1 m + (1 - beta1) g,  v' = beta2 v + (1 - beta2) g^2,
      phi' = phi - lr * (m' / (1 - beta1^t)) / (sqrt(v' / (1 - beta2^t)) + eps).
    """
    if step < 1:
        raise ValueError("step counts from 1")
    g = np.asarray(grad, dtype=np.float64)
    m1 = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * g
    v1 = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * g * g
    mhat = m1 / (1.0 - beta1 ** step)
    vhat = v1 / (1.0 - beta2 ** step)
    return np.asarray(phi, dtype=np.float64) - lr * mhat / (np.sqrt(vhat) + eps), m1, v1
