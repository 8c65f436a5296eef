"""Plant plausible mistakes in the oracle (on the CPU) and show the pins catch each one.

Every mutant replaces one function of ``oracle.donn`` for the duration of a
test.  The test passes when at least one of the named pins reports an error
far above its tolerance.
"""

import numpy as np
import pytest

import oracle.donn as od
import oracle_checks as c

_orig = {name: getattr(od, name) for name in (
    "dft_matrix", "idft2", "transfer_function", "frequencies", "propagate",
    "modulate", "detector_readout", "region_scatter", "softmax_cross_entropy",
    "mse_softmax_loss", "donn_forward", "donn_backward", "adam_update",
    "impulse_response", "displacements", "fraunhofer", "fraunhofer_pitch",
    "multichannel_forward", "multichannel_backward", "codesign_phase", "codesign_backward",
    "layer_norm", "layer_norm_backward")}


def _dft_sign_flipped(m, inverse=False):
    return _orig["dft_matrix"](m, not inverse)


def _idft_unnormalised(y):
    m0, m1 = y.shape[-2:]
    return _orig["idft2"](y) * (m0 * m1)


def _fresnel_no_global_phase(lam, dx, z, approx, m):
    h = _orig["transfer_function"](lam, dx, z, approx, m)
    if approx == od.FRESNEL:
        h = h * np.exp(-1j * 2 * np.pi / lam * z)
    return h


def _fresnel_chirp_conjugated(lam, dx, z, approx, m):
    h = _orig["transfer_function"](lam, dx, z, approx, m)
    if approx == od.FRESNEL:
        g = np.exp(1j * 2 * np.pi / lam * z)
        h = g * np.conj(h / g)
    return h


def _frequencies_unwrapped(m, dx):
    return np.arange(m, dtype=np.float64) / (m * dx)


def _as_paraxial(lam, dx, z, approx, m):
    if approx == od.ANGULAR_SPECTRUM:
        return _orig["transfer_function"](lam, dx, z, od.FRESNEL, m)
    return _orig["transfer_function"](lam, dx, z, approx, m)


def _adjoint_without_conj(u, h, adjoint=False):
    return _orig["propagate"](u, h, adjoint=False)


def _modulate_without_gamma(v, phi, gamma=1.0):
    return _orig["modulate"](v, phi, 1.0)


def _readout_off_by_one(i_map, det):
    return _orig["detector_readout"](i_map, od.Detector(det.size + 1, det.y0, det.x0))


def _scatter_transposed(grad_sums, det, n):
    return _orig["region_scatter"](grad_sums, od.Detector(det.size, det.x0, det.y0), n)


def _ce_grad_not_averaged(sums, labels):
    loss, grad = _orig["softmax_cross_entropy"](sums, labels)
    return loss, grad * np.asarray(sums).shape[0]


def _forward_missing_last_hop(amp, phi, h, gamma=1.0, det=None):
    out = _orig["donn_forward"](amp, phi, h, gamma, det)
    ud = out["acts"][-1] if len(out["acts"]) else od.encode_amplitude(amp)
    out["field"] = ud
    out["intensity"] = od.intensity(ud)
    return out


def _make_backward(variant):
    def bwd(fwd, phi, h, gamma=1.0, det=None, grad_sums=None, grad_intensity=None):
        ud, acts = fwd["field"], fwd["acts"]
        n = ud.shape[-1]
        g_i = (od.region_scatter(grad_sums, det, n) if grad_sums is not None
               else np.asarray(grad_intensity, dtype=np.float64))
        two = 1.0 if variant == "no_factor_two" else 2.0
        g = od.propagate(two * g_i * ud, h, adjoint=True)
        dphi = np.zeros((phi.shape[0], n, n))
        for layer in range(phi.shape[0] - 1, -1, -1):
            if variant == "sign":
                dphi[layer] = np.imag(acts[layer] * np.conj(g)).sum(axis=0)
            else:
                dphi[layer] = np.imag(np.conj(acts[layer]) * g).sum(axis=0)
            rot = np.exp(1j * phi[layer]) if variant == "mask_not_conj" else np.exp(-1j * phi[layer])
            g = (1.0 if variant == "no_gamma" else gamma) * rot * g
            if layer > 0:
                g = od.propagate(g, h, adjoint=True)
        return dphi
    return bwd


def _mse_no_softmax_jacobian(sums, labels):
    # gradient taken with respect to p instead of S
    s = np.asarray(sums, dtype=np.float64)
    loss, _ = _orig["mse_softmax_loss"](s, labels)
    e = np.exp(s - s.max(axis=1, keepdims=True))
    p = e / e.sum(axis=1, keepdims=True)
    t = np.zeros_like(p)
    t[np.arange(s.shape[0]), np.asarray(labels)] = 1.0
    return loss, 2.0 * (p - t) / s.shape[0]


def _mse_not_squared(sums, labels):
    s = np.asarray(sums, dtype=np.float64)
    e = np.exp(s - s.max(axis=1, keepdims=True))
    p = e / e.sum(axis=1, keepdims=True)
    t = np.zeros_like(p)
    t[np.arange(s.shape[0]), np.asarray(labels)] = 1.0
    _, grad = _orig["mse_softmax_loss"](s, labels)
    return float(np.mean(np.sqrt(((p - t) ** 2).sum(axis=1)))), grad


def _adam_no_bias_correction(phi, grad, m, v, step, lr=0.5, beta1=0.9, beta2=0.999, eps=1e-8):
    g = np.asarray(grad, dtype=np.float64)
    m1 = beta1 * m + (1 - beta1) * g
    v1 = beta2 * v + (1 - beta2) * g * g
    return phi - lr * m1 / (np.sqrt(v1) + eps), m1, v1


def _adam_eps_inside_sqrt(phi, grad, m, v, step, lr=0.5, beta1=0.9, beta2=0.999, eps=1e-8):
    g = np.asarray(grad, dtype=np.float64)
    m1 = beta1 * m + (1 - beta1) * g
    v1 = beta2 * v + (1 - beta2) * g * g
    return phi - lr * (m1 / (1 - beta1 ** step)) / np.sqrt(v1 / (1 - beta2 ** step) + 1e-4), m1, v1


def _adam_betas_swapped(phi, grad, m, v, step, lr=0.5, beta1=0.9, beta2=0.999, eps=1e-8):
    return _orig["adam_update"](phi, grad, m, v, step, lr, beta2, beta1, eps)


def _fails_grad(**kw):
    return c.grad_fd(**kw)[0] > 1e-3


def _ir_no_area_element(lam, dx, z, approx, m):
    h = _orig["transfer_function"](lam, dx, z, approx, m)
    return h / (dx * dx) if approx in (od.FRESNEL_IR, od.RS_IR) else h


def _displacements_unwrapped(m, dx):
    return np.arange(m, dtype=np.float64) * dx


def _rs_one_over_r(lam, dx, z, approx, m):
    h = _orig["impulse_response"](lam, dx, z, approx, m)
    if approx == od.RS_IR:
        d = _orig["displacements"](m, dx)
        r = np.sqrt(z * z + d[:, None] ** 2 + d[None, :] ** 2)
        h = h * r
    return h


def _rs_kernel_conjugated(lam, dx, z, approx, m):
    h = _orig["impulse_response"](lam, dx, z, approx, m)
    return np.conj(h) if approx == od.RS_IR else h


def _fraunhofer_output_uncentred(u, lam, dx, z, m):
    return np.roll(_orig["fraunhofer"](u, lam, dx, z, m), (m // 2, m // 2), axis=(-2, -1))


def _fraunhofer_no_output_chirp(u, lam, dx, z, m):
    out = _orig["fraunhofer"](u, lam, dx, z, m)
    c = (np.arange(m) - m // 2) * _orig["fraunhofer_pitch"](lam, dx, z, m)
    k = 2.0 * np.pi / lam
    return out * np.exp(-1j * k * (c[:, None] ** 2 + c[None, :] ** 2) / (2.0 * z))


def _fraunhofer_pitch_no_m(lam, dx, z, m):
    return lam * z / dx


def _multichannel_sums_averaged(amps, phis, h, gamma, det):
    fwds, merged = _orig["multichannel_forward"](amps, phis, h, gamma, det)
    return fwds, merged / len(fwds)


def _multichannel_grad_split(fwds, phis, h, gamma, det, grad_sums):
    return _orig["multichannel_backward"](fwds, phis, h, gamma, det, grad_sums / len(fwds))


def _codesign_no_temperature(logits, noise, levels, tau, hard=False):
    return _orig["codesign_phase"](logits, noise, levels, 1.0, hard)


def _codesign_hard_in_float64(logits, noise, levels, tau, hard=False):
    phi, w = _orig["codesign_phase"](logits, noise, levels, tau, False)
    if hard:
        s = np.asarray(logits, np.float64) + np.asarray(noise, np.float64)
        phi = np.asarray(levels, np.float64)[np.argmax(s, axis=-1)]
    return phi, w


def _codesign_hard_last_on_ties(logits, noise, levels, tau, hard=False):
    phi, w = _orig["codesign_phase"](logits, noise, levels, tau, False)
    if hard:
        s = (np.asarray(logits, np.float32) + np.asarray(noise, np.float32))[..., ::-1]
        k = s.shape[-1] - 1 - np.argmax(s, axis=-1)
        phi = np.asarray(levels, np.float64)[k]
    return phi, w


def _codesign_backward_no_centering(w, levels, tau, grad_phi):
    lv = np.asarray(levels, np.float64)
    return w * lv * (np.asarray(grad_phi, np.float64)[..., None] / tau)


def _forward_skip_before_last_hop(amp, phi, h, gamma=1.0, det=None, skip=None):
    if skip is None:
        return _orig["donn_forward"](amp, phi, h, gamma, det)
    # the skip field joins the last layer's output instead of the detector-plane field
    out = _orig["donn_forward"](amp, phi, h, gamma, det)
    ud = od.propagate(out["acts"][-1] + skip, h)
    out["field"] = ud
    out["intensity"] = od.intensity(ud)
    out["sums"] = od.detector_readout(out["intensity"], det) if det is not None else None
    return out


def _forward_skip_not_in_field(amp, phi, h, gamma=1.0, det=None, skip=None):
    # the intensity sees the skip, the stored detector field (the adjoint's seed) does not
    out = _orig["donn_forward"](amp, phi, h, gamma, det, skip=skip)
    if skip is not None:
        out["field"] = out["field"] - skip
    return out


def _layer_norm_unbiased(i_map, eps=1e-5):
    x = np.asarray(i_map, dtype=np.float64)
    mean = x.mean(axis=(-2, -1))
    var = x.var(axis=(-2, -1), ddof=1)
    rstd = 1.0 / np.sqrt(var + eps)
    return (x - mean[:, None, None]) * rstd[:, None, None], mean, rstd


def _layer_norm_backward_no_projection(grad_out, normed, rstd):
    g = np.asarray(grad_out, dtype=np.float64)
    return np.asarray(rstd)[:, None, None] * (g - g.mean(axis=(-2, -1))[:, None, None])


MUTANTS = [
    ("dft_sign", "dft_matrix", _dft_sign_flipped, lambda: c.dft_vs_numpy() > 1e-3),
    ("idft_norm", "idft2", _idft_unnormalised, lambda: c.dft_delta_parseval() > 1e-3),
    ("fresnel_no_exp_jkz", "transfer_function", _fresnel_no_global_phase, lambda: c.fresnel_gaussian() > 1e-3),
    ("fresnel_chirp_sign", "transfer_function", _fresnel_chirp_conjugated, lambda: c.fresnel_gaussian() > 1e-3),
    ("freq_unwrapped", "frequencies", _frequencies_unwrapped, lambda: c.fresnel_gaussian() > 1e-3),
    ("as_is_paraxial", "transfer_function", _as_paraxial, lambda: c.rs_bruteforce(True, True) > 1e-7),
    ("adjoint_no_conj", "propagate", _adjoint_without_conj, lambda: c.adjoint_dot() > 1e-3),
    ("no_gamma_forward", "modulate", _modulate_without_gamma, lambda: c.donn_energy()[0] > 1e-3),
    ("readout_off_by_one", "detector_readout", _readout_off_by_one, lambda: c.readout_tiling() > 1e-3),
    ("scatter_transposed", "region_scatter", _scatter_transposed, lambda: _fails_grad(mode="ce")),
    ("ce_grad_sum_not_mean", "softmax_cross_entropy", _ce_grad_not_averaged,
     lambda: c.loss_fd(od.softmax_cross_entropy) > 1e-3),
    ("mse_no_softmax_jacobian", "mse_softmax_loss", _mse_no_softmax_jacobian,
     lambda: c.loss_fd(od.mse_softmax_loss) > 1e-3),
    ("mse_norm_not_squared", "mse_softmax_loss", _mse_not_squared, lambda: c.mse_known_values() > 1e-3),
    ("ir_no_dx2", "transfer_function", _ir_no_area_element, lambda: c.ir_linear_convolution(od.FRESNEL_IR) > 1e-3),
    ("ir_unwrapped", "displacements", _displacements_unwrapped, lambda: c.ir_linear_convolution(od.RS_IR) > 1e-3),
    ("rs_one_over_r", "impulse_response", _rs_one_over_r, lambda: c.rs_ir_paraxial_bound()[0] > 10.0),
    ("rs_conjugated", "impulse_response", _rs_kernel_conjugated, lambda: c.rs_ir_paraxial_bound()[0] > 10.0),
    ("fraunhofer_uncentred", "fraunhofer", _fraunhofer_output_uncentred, lambda: c.fraunhofer_rectangle() > 1e-3),
    ("fraunhofer_no_chirp", "fraunhofer", _fraunhofer_no_output_chirp, lambda: c.fraunhofer_vs_fresnel_sum() > 1e-3),
    ("fraunhofer_pitch", "fraunhofer_pitch", _fraunhofer_pitch_no_m, lambda: c.fraunhofer_vs_fresnel_sum() > 1e-3),
    ("multichannel_sums_averaged", "multichannel_forward", _multichannel_sums_averaged,
     lambda: c.multichannel_sums_add() > 1e-3),
    ("multichannel_grad_split", "multichannel_backward", _multichannel_grad_split,
     lambda: c.multichannel_grad_fd() > 1e-3),
    ("codesign_no_temperature", "codesign_phase", _codesign_no_temperature, lambda: c.codesign_limits() > 1e-3),
    ("codesign_hard_float64", "codesign_phase", _codesign_hard_in_float64, lambda: c.codesign_hard_near_ties() > 0),
    ("codesign_hard_last_on_ties", "codesign_phase", _codesign_hard_last_on_ties,
     lambda: c.codesign_hard_near_ties() > 0),
    ("codesign_grad_not_centred", "codesign_backward", _codesign_backward_no_centering,
     lambda: c.codesign_grad_fd() > 1e-3),
    ("adam_no_bias_correction", "adam_update", _adam_no_bias_correction, lambda: c.adam_first_step() > 1e-3),
    ("adam_eps_inside_sqrt", "adam_update", _adam_eps_inside_sqrt, lambda: c.adam_constant_gradient() > 1e-3),
    ("adam_betas_swapped", "adam_update", _adam_betas_swapped, lambda: c.adam_vs_torch() > 1e-3),
    ("missing_last_hop", "donn_forward", _forward_missing_last_hop, lambda: c.donn_zero_phase_gaussian() > 1e-3),
    ("bwd_no_factor_two", "donn_backward", _make_backward("no_factor_two"), lambda: _fails_grad(mode="map")),
    ("bwd_sign", "donn_backward", _make_backward("sign"), lambda: _fails_grad(mode="ce")),
    ("bwd_mask_not_conj", "donn_backward", _make_backward("mask_not_conj"), lambda: _fails_grad(mode="map")),
    ("bwd_no_gamma", "donn_backward", _make_backward("no_gamma"), lambda: _fails_grad(mode="map", gamma=0.7)),
    ("skip_before_last_hop", "donn_forward", _forward_skip_before_last_hop,
     lambda: c.skip_adds_at_detector() > 1e-3),
    ("skip_not_in_seed", "donn_forward", _forward_skip_not_in_field, lambda: c.segmentation_grad_fd() > 1e-3),
    ("layer_norm_unbiased_var", "layer_norm", _layer_norm_unbiased, lambda: c.layer_norm_moments() > 1e-3),
    ("layer_norm_grad_no_projection", "layer_norm_backward", _layer_norm_backward_no_projection,
     lambda: c.layer_norm_grad_fd() > 1e-3),
]


@pytest.mark.parametrize("name,attr,fn,caught", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(monkeypatch, name, attr, fn, caught):
    monkeypatch.setattr(od, attr, fn)
    assert caught(), f"mutant {name} was not caught"
