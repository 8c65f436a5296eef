"""Segmentation DONN (§5.6.2) against the oracle: the optical skip connection
(a field added at the detector plane; under the residual reading the input
field itself) in the forward and backward passes of both propagation paths,
the per-sample layer normalisation of the intensity map and its backward, and
the whole training chain detector -> layer norm -> upstream gradient.

Tolerances as in the other parity tests: relative L2 1e-4 for fields, maps
and sums, 1e-3 for phase gradients.
"""

import numpy as np
import pytest

import oracle.donn as od
from paper_2306_11268_amd import workloads as wl

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

TOL_FIELD = 1e-4
TOL_GRAD = 1e-3


def rel(a, b):
    a = np.asarray(a)
    b = np.asarray(b)
    r = float(np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(b.ravel()), 1e-300))
    print(f"  rel-L2 {r:.3e} over {b.size} values")
    return r


@pytest.fixture(scope="module")
def lrb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2306_11268_amd import binding
    binding.load()
    return binding


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def host(t):
    return t.detach().cpu().numpy()


def network(lrb, w, layers=None, det=True):
    d = w.detector if det else None
    detector = lrb.Detector(d.size, d.y0, d.x0) if d is not None else None
    return lrb.Network(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n, w.n_fft,
                       w.layers if layers is None else layers, 1.0, detector)


def oracle_det(d):
    return od.Detector(d.size, tuple(d.y0), tuple(d.x0))


def input_skip(amp):
    """The residual reading's skip field: the input field itself."""
    return np.asarray(amp, dtype=np.float32).astype(np.complex64)


@pytest.mark.parametrize("layers", [5, 2])
def test_skip_forward_fresnel(lrb, layers):
    w = wl.WORKLOADS[3]
    b = 4
    net = network(lrb, w, layers)
    amp = wl.amplitudes(w, b)
    phi = wl.phases(w)[:layers]
    skip = input_skip(amp)
    out = lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=True, intensity=True, field=True, skip=dev(skip))
    h = od.transfer_function(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n_fft)
    ref = od.donn_forward(amp, phi, h, 1.0, oracle_det(w.detector), skip=skip)
    assert rel(host(out["field"]), ref["field"]) < TOL_FIELD
    assert rel(host(out["intensity"]), ref["intensity"]) < TOL_FIELD
    assert rel(host(out["sums"]), ref["sums"]) < TOL_FIELD
    # sums-only (only the covered rows are transformed)
    s_only = lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=True, skip=dev(skip))
    assert rel(host(s_only["sums"]), ref["sums"]) < TOL_FIELD


@pytest.mark.parametrize("layers,mode", [(5, "ce"), (4, "ce"), (3, "map")])
def test_skip_backward_fresnel(lrb, layers, mode):
    w = wl.WORKLOADS[3]
    b = 4
    net = network(lrb, w, layers)
    amp = wl.amplitudes(w, b)
    phi = wl.phases(w)[:layers]
    skip = input_skip(amp)
    saved = net.new_saved(b)
    out = lrb.lr_donn_forward(net, dev(amp), dev(phi), saved=saved, sums=True, skip=dev(skip))
    h = od.transfer_function(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n_fft)
    det = oracle_det(w.detector)
    ref = od.donn_forward(amp, phi, h, 1.0, det, skip=skip)
    if mode == "ce":
        labels = wl.labels(w, b)
        grad, loss = lrb.lr_donn_backward(net, dev(phi), saved, sums=out["sums"], labels=dev(labels), skip=dev(skip))
        ref_loss, gs = od.softmax_cross_entropy(ref["sums"], labels)
        ref_grad = od.donn_backward(ref, phi, h, 1.0, det, grad_sums=gs)
        assert abs(float(loss) - ref_loss) / abs(ref_loss) < TOL_FIELD
    else:
        gi = np.random.default_rng(71).standard_normal((b, w.n, w.n)).astype(np.float32)
        grad, _ = lrb.lr_donn_backward(net, dev(phi), saved, grad_intensity=dev(gi), skip=dev(skip))
        ref_grad = od.donn_backward(ref, phi, h, 1.0, grad_intensity=gi)
    assert rel(host(grad), ref_grad) < TOL_GRAD


def test_skip_angular_spectrum_padded(lrb):
    # 512 x 512 aperture centred in a 1024-point grid, angular spectrum
    w = wl.WORKLOADS[4]
    b, layers = 2, 2
    net = network(lrb, w, layers, det=False)
    amp = wl.amplitudes(w, b)
    phi = wl.phases(w)[:layers]
    skip = input_skip(amp)
    saved = net.new_saved(b)
    out = lrb.lr_donn_forward(net, dev(amp), dev(phi), saved=saved, sums=False, intensity=True, field=True,
                              skip=dev(skip))
    h = od.transfer_function(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n_fft)
    ref = od.donn_forward(amp, phi, h, 1.0, None, skip=skip)
    assert rel(host(out["field"]), ref["field"]) < TOL_FIELD
    assert rel(host(out["intensity"]), ref["intensity"]) < TOL_FIELD
    gi = np.random.default_rng(72).standard_normal((b, w.n, w.n)).astype(np.float32)
    grad, _ = lrb.lr_donn_backward(net, dev(phi), saved, grad_intensity=dev(gi), skip=dev(skip))
    ref_grad = od.donn_backward(ref, phi, h, 1.0, grad_intensity=gi)
    assert rel(host(grad), ref_grad) < TOL_GRAD


@pytest.mark.parametrize("shape", [(3, 200, 200), (2, 1000, 1000), (5, 7, 9)])
def test_layer_norm_forward_backward(lrb, shape):
    g = np.random.default_rng(73)
    x = (g.uniform(0, 2, shape) ** 2 + 0.5).astype(np.float32)
    gy = g.standard_normal(shape).astype(np.float32)
    y, stats = lrb.lr_layer_norm(dev(x), eps=1e-5)
    ry, rmean, rrstd = od.layer_norm(x, 1e-5)
    assert rel(host(y), ry) < TOL_FIELD
    assert rel(host(stats)[:, 0], rmean) < 1e-5 and rel(host(stats)[:, 1], rrstd) < 1e-5
    dx = lrb.lr_layer_norm_backward(dev(gy), y, stats)
    rdx = od.layer_norm_backward(gy, ry, rrstd)
    assert rel(host(dx), rdx) < TOL_FIELD
    # in place, and reproducible bit for bit
    xt = dev(x)
    y2, stats2 = lrb.lr_layer_norm(xt, eps=1e-5, out=xt)
    assert torch.equal(y2, y) and torch.equal(stats2, stats)
    gt = dev(gy)
    dx2 = lrb.lr_layer_norm_backward(gt, y, stats, out=gt)
    assert torch.equal(dx2, dx)


def test_segmentation_training_step(lrb):
    # 5 layers, 200 x 200 (the paper's segmentation network is 5 layers); the
    # loss is the linear functional sum G * LN(I) of an upstream gradient G
    w = wl.WORKLOADS[3]
    b = 3
    net = network(lrb, w, det=False)
    amp = wl.amplitudes(w, b)
    phi = wl.phases(w)
    skip = input_skip(amp)
    G = np.random.default_rng(74).standard_normal((b, w.n, w.n)).astype(np.float32)
    saved = net.new_saved(b)
    out = lrb.lr_donn_forward(net, dev(amp), dev(phi), saved=saved, sums=False, intensity=True, skip=dev(skip))
    y, stats = lrb.lr_layer_norm(out["intensity"], eps=1e-5)
    gi = lrb.lr_layer_norm_backward(dev(G), y, stats)
    grad, _ = lrb.lr_donn_backward(net, dev(phi), saved, grad_intensity=gi, skip=dev(skip))

    h = od.transfer_function(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n_fft)
    ref = od.donn_forward(amp, phi, h, 1.0, None, skip=skip)
    ry, _, rrstd = od.layer_norm(ref["intensity"], 1e-5)
    assert rel(host(y), ry) < TOL_FIELD
    rgi = od.layer_norm_backward(G, ry, rrstd)
    ref_grad = od.donn_backward(ref, phi, h, 1.0, grad_intensity=rgi)
    assert rel(host(grad), ref_grad) < TOL_GRAD


def test_segmentation_training_step_at_the_papers_grid(lrb):
    # the paper's segmentation system: 5 layers on a 350 x 350 grid (§5.6.2),
    # the optics of the validation setup
    w = wl.scaled(wl.WORKLOADS[3], n=350)
    b = 2
    net = network(lrb, w, det=False)
    amp = wl.amplitudes(w, b)
    phi = wl.phases(w)
    skip = input_skip(amp)
    G = np.random.default_rng(75).standard_normal((b, w.n, w.n)).astype(np.float32)
    saved = net.new_saved(b)
    out = lrb.lr_donn_forward(net, dev(amp), dev(phi), saved=saved, sums=False, intensity=True, skip=dev(skip))
    y, stats = lrb.lr_layer_norm(out["intensity"], eps=1e-5)
    gi = lrb.lr_layer_norm_backward(dev(G), y, stats)
    grad, _ = lrb.lr_donn_backward(net, dev(phi), saved, grad_intensity=gi, skip=dev(skip))

    h = od.transfer_function(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n_fft)
    ref = od.donn_forward(amp, phi, h, 1.0, None, skip=skip)
    assert rel(host(out["intensity"]), ref["intensity"]) < TOL_FIELD
    ry, _, rrstd = od.layer_norm(ref["intensity"], 1e-5)
    assert rel(host(y), ry) < TOL_FIELD
    ref_grad = od.donn_backward(ref, phi, h, 1.0, grad_intensity=od.layer_norm_backward(G, ry, rrstd))
    assert rel(host(grad), ref_grad) < TOL_GRAD
