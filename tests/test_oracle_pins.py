"""The float64 oracle pinned to what the paper and the mathematics fix (CPU only).

Tolerances are float64 rounding levels except where a physical
approximation sets the floor (the brute-force Rayleigh-Sommerfeld sum and the
paraxial bound); each is stated next to its check.
"""

import numpy as np
import pytest

import oracle.donn as od
import oracle_checks as c


def test_dft_is_numpy_fft():
    assert c.dft_vs_numpy() < 1e-12


def test_dft_delta_roundtrip_parseval():
    assert c.dft_delta_parseval() < 1e-12


def test_frequency_grid_is_fftfreq():
    assert c.frequencies_vs_numpy() < 1e-14


def test_zero_distance_is_identity():
    assert c.z0_identity() < 1e-14


def test_energy_conservation_unpadded():
    assert c.parseval_unpadded() < 1e-13


def test_composition_z1_plus_z2():
    # limited by float64 rounding of kz ~ 3.5e6 rad
    assert c.composition() < 1e-9


def test_reciprocity_and_adjoint_is_back_propagation():
    assert c.reciprocity() < 1e-13


def test_fresnel_gaussian_beam_closed_form():
    assert c.fresnel_gaussian() < 1e-12


def test_fresnel_gaussian_beam_padded_aperture():
    assert c.fresnel_gaussian_padded() < 1e-12


def test_fresnel_is_separable():
    assert c.fresnel_separable() < 1e-12


@pytest.mark.parametrize("exact,smooth,tol", [
    (True, True, 1e-7),    # exact RS-I kernel: agreement to ~1.4e-8
    (False, True, 3e-5),   # the r >> lambda kernel of Eq. (sommerfeld): O(1/(kz)) gap
    (True, False, 0.1),    # non-smooth source: band-edge truncation, still catches O(1) errors
])
def test_angular_spectrum_vs_bruteforce_rayleigh_sommerfeld(exact, smooth, tol):
    assert c.rs_bruteforce(exact, smooth) < tol


def test_fresnel_angular_spectrum_paraxial_bound():
    lhs, bound = c.fresnel_as_bound()
    assert lhs <= bound


def test_donn_zero_phase_is_one_long_hop():
    assert c.donn_zero_phase_gaussian() < 1e-9


def test_donn_energy_with_gamma_and_padding():
    e, padded_ok = c.donn_energy()
    assert e < 1e-12 and padded_ok


def test_detector_readout():
    assert c.readout_tiling() < 1e-14


def test_cross_entropy_known_values():
    assert c.ce_known_values() < 1e-14


def test_mse_loss_known_values():
    assert c.mse_known_values() < 1e-14


def test_adam_first_step_closed_form():
    assert c.adam_first_step() < 1e-14


def test_adam_constant_gradient_constant_step():
    assert c.adam_constant_gradient() < 1e-12


def test_adam_matches_torch_optimizer():
    pytest.importorskip("torch")
    assert c.adam_vs_torch() < 1e-12


@pytest.mark.parametrize("fn", [od.softmax_cross_entropy, od.mse_softmax_loss])
def test_loss_gradients_by_finite_differences(fn):
    assert c.loss_fd(fn) < 1e-7


def test_adjoint_dot_product():
    assert c.adjoint_dot() < 1e-12


@pytest.mark.parametrize("kw", [
    dict(mode="ce"), dict(mode="map"), dict(mode="ce", n=10, m=16),
    dict(mode="map", gamma=0.7), dict(mode="ce", approx=od.ANGULAR_SPECTRUM),
])
def test_phase_gradient_by_finite_differences(kw):
    err, _ = c.grad_fd(**kw)
    assert err < 1e-6


def test_phase_gradient_global_phase_invariance():
    assert c.global_phase_invariance() < 1e-12


def test_transfer_function_rejects_unknown_approximation():
    with pytest.raises(ValueError):
        od.transfer_function(532e-9, 36e-6, 0.3, 7, 8)


@pytest.mark.parametrize("approx", [od.FRESNEL_IR, od.RS_IR])
def test_sampled_kernel_hop_is_linear_convolution(approx):
    # the padded spectral hop against the direct sum of Eq. (forward_diff)
    assert c.ir_linear_convolution(approx) < 1e-12


def test_sampled_fresnel_kernel_gaussian_beam():
    # Riemann-sum error of the discrete convolution of a 6-px Gaussian (~1e-10 measured)
    assert c.fresnel_ir_gaussian() < 1e-7


def test_sampled_rayleigh_sommerfeld_within_paraxial_bound():
    ratio, diff = c.rs_ir_paraxial_bound()
    assert ratio <= 1.0 and diff > 1e-8


def test_sampled_fresnel_kernel_is_separable():
    assert c.fresnel_ir_separable() < 1e-12


def test_fraunhofer_is_the_expanded_fresnel_sum():
    assert c.fraunhofer_vs_fresnel_sum() < 1e-12


def test_fraunhofer_rectangle_dirichlet_kernel():
    assert c.fraunhofer_rectangle() < 1e-12


def test_fraunhofer_output_pitch():
    assert abs(od.fraunhofer_pitch(532e-9, 36e-6, 1.0, 100) - 532e-9 / (100 * 36e-6)) < 1e-20


def test_multichannel_sums_add():
    assert c.multichannel_sums_add() < 1e-13


def test_multichannel_gradients_by_finite_differences():
    # central differences with step 1e-6 in float64: ~1e-8 truncation and rounding
    assert c.multichannel_grad_fd() < 1e-6


def test_codesign_limits_and_shift_invariance():
    assert c.codesign_limits() < 1e-9


def test_codesign_hard_choice_on_float32_near_ties():
    assert c.codesign_hard_near_ties() == 0


def test_codesign_gradient_by_finite_differences():
    assert c.codesign_grad_fd() < 1e-8


def test_segmentation_skip_adds_at_the_detector():
    assert c.skip_adds_at_detector() < 1e-13


def test_layer_norm_moments_and_constant_map():
    assert c.layer_norm_moments() < 1e-12


def test_layer_norm_affine_invariance():
    assert c.layer_norm_affine_invariance() < 1e-12


def test_layer_norm_gradient_by_finite_differences():
    assert c.layer_norm_grad_fd() < 1e-7


def test_segmentation_chain_gradient_by_finite_differences():
    # skip + layer norm + DONN, central differences with step 1e-6 in float64
    assert c.segmentation_grad_fd() < 1e-6
