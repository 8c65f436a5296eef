"""Training-step paths of the separable (Fresnel) network against the oracle.

The forward pass here asks for the detector sums only, as a training step
does: the detector-plane pass then transforms just the rows (or columns)
covered by detector regions, and the backward seed pass finishes the last
hop itself from the saved half-hop field.  Tolerances as in
test_gpu_parity.py: relative L2 1e-4 on sums and loss, 1e-3 on dL/dphi.
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
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
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


def odet(d):
    return od.Detector(d.size, tuple(d.y0), tuple(d.x0))


def sums_only_forward(lrb, w, batch, layers, det, gamma=1.0):
    net = lrb.Network(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n, w.n_fft, layers, gamma,
                      lrb.Detector(det.size, det.y0, det.x0))
    amp = wl.amplitudes(w, batch)
    phi = wl.phases(w)[:layers]
    saved = net.new_saved(batch)
    out = lrb.lr_donn_forward(net, dev(amp), dev(phi), saved=saved, sums=True)
    h = od.transfer_function(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n_fft)
    ref = od.donn_forward(amp, phi, h, gamma, odet(det))
    return net, phi, saved, out, ref, h


# L odd: the detector-plane pass is a row pass; L even: a column pass
@pytest.mark.parametrize("layers", [5, 2, 1])
def test_cross_entropy_step_sums_only(lrb, layers):
    w = wl.WORKLOADS[3]
    b = 7
    net, phi, saved, out, ref, h = sums_only_forward(lrb, w, b, layers, w.detector)
    assert out.get("intensity") is None and out.get("field") is None
    assert rel(host(out["sums"]), ref["sums"]) < TOL_FIELD
    labels = wl.labels(w, b)
    grad, loss = lrb.lr_donn_backward(net, dev(phi), saved, sums=out["sums"], labels=dev(labels))
    ref_loss, gs = od.softmax_cross_entropy(ref["sums"], labels)
    ref_grad = od.donn_backward(ref, phi, h, 1.0, odet(w.detector), grad_sums=gs)
    assert abs(float(loss) - ref_loss) / abs(ref_loss) < TOL_FIELD
    assert rel(host(grad), ref_grad) < TOL_GRAD


@pytest.mark.parametrize("layers", [1, 2])
def test_full_map_backward_after_sums_only_forward(lrb, layers):
    # the saved half-hop field serves any seed, also a full dL/dI map
    w = wl.WORKLOADS[3]
    b = 3
    net, phi, saved, out, ref, h = sums_only_forward(lrb, w, b, layers, w.detector)
    gi = np.random.default_rng(17).standard_normal((b, w.n, w.n)).astype(np.float32)
    grad, _ = lrb.lr_donn_backward(net, dev(phi), saved, grad_intensity=dev(gi))
    ref_grad = od.donn_backward(ref, phi, h, 1.0, grad_intensity=gi)
    assert rel(host(grad), ref_grad) < TOL_GRAD


@pytest.mark.parametrize("layers", [1, 2, 3])
def test_overlapping_regions_at_the_edges(lrb, layers):
    # overlapping regions, regions touching the plane border, one region inside another
    w = wl.WORKLOADS[3]
    det = wl.DetectorLayout(size=30, y0=(0, 15, 170, 100, 105), x0=(0, 20, 170, 0, 5))
    b = 3
    net, phi, saved, out, ref, h = sums_only_forward(lrb, w, b, layers, det, gamma=0.9)
    assert rel(host(out["sums"]), ref["sums"]) < TOL_FIELD
    gs = np.random.default_rng(3).standard_normal((b, det.num)).astype(np.float32)
    grad, _ = lrb.lr_donn_backward(net, dev(phi), saved, grad_sums=dev(gs))
    ref_grad = od.donn_backward(ref, phi, h, 0.9, odet(det), grad_sums=gs)
    assert rel(host(grad), ref_grad) < TOL_GRAD


@pytest.mark.parametrize("layers", [2, 3])
def test_padded_grid_sums_only(lrb, layers):
    # n = 100 centred in a 128 grid: the pruned passes crop and pad as well
    w = wl.Workload(91, "test", 532e-9, 36e-6, 0.2, od.FRESNEL, 100, 128, 3, 3, "train",
                    wl.layout_grid(100, 4, 12), "sums", "uniform")
    b = 3
    net, phi, saved, out, ref, h = sums_only_forward(lrb, w, b, layers, w.detector)
    assert rel(host(out["sums"]), ref["sums"]) < TOL_FIELD
    gs = np.random.default_rng(4).standard_normal((b, w.detector.num)).astype(np.float32)
    grad, _ = lrb.lr_donn_backward(net, dev(phi), saved, grad_sums=dev(gs))
    ref_grad = od.donn_backward(ref, phi, h, 1.0, odet(w.detector), grad_sums=gs)
    assert rel(host(grad), ref_grad) < TOL_GRAD


def test_single_region_single_row(lrb):
    # a 1 x 1 region: one covered row and one covered column
    w = wl.WORKLOADS[3]
    det = wl.DetectorLayout(size=1, y0=(123,), x0=(45,))
    for layers in (1, 2):
        net, phi, saved, out, ref, h = sums_only_forward(lrb, w, 2, layers, det)
        assert rel(host(out["sums"]), ref["sums"]) < TOL_FIELD
        gs = np.array([[1.0], [-0.5]], dtype=np.float32)
        grad, _ = lrb.lr_donn_backward(net, dev(phi), saved, grad_sums=dev(gs))
        ref_grad = od.donn_backward(ref, phi, h, 1.0, odet(det), grad_sums=gs)
        assert rel(host(grad), ref_grad) < TOL_GRAD


def test_training_step_at_full_size(lrb):
    """The benchmarked step itself: 5 layers, 200 x 200, batch 500, sums-only
    forward, cross-entropy, backward, in the benchmark's launch configuration,
    compared with the oracle on the whole batch."""
    w = wl.WORKLOADS[3]
    b = w.batch
    net, phi, saved, out, ref, h = sums_only_forward(lrb, w, b, w.layers, w.detector)
    assert rel(host(out["sums"]), ref["sums"]) < TOL_FIELD
    labels = wl.labels(w, b)
    grad, loss = lrb.lr_donn_backward(net, dev(phi), saved, sums=out["sums"], labels=dev(labels))
    g1 = host(grad).copy()
    ref_loss, gs = od.softmax_cross_entropy(ref["sums"], labels)
    assert abs(float(loss) - ref_loss) / abs(ref_loss) < TOL_FIELD
    ref_grad = od.donn_backward(ref, phi, h, 1.0, odet(w.detector), grad_sums=gs)
    assert rel(g1, ref_grad) < TOL_GRAD
    # bitwise repeatable, and invariant to a global phase of each mask
    grad2, _ = lrb.lr_donn_backward(net, dev(phi), saved, sums=out["sums"], labels=dev(labels))
    assert np.array_equal(g1, host(grad2))
    s = g1.sum(axis=(1, 2))
    assert np.all(np.abs(s) <= 1e-4 * np.abs(g1).sum(axis=(1, 2)))


# ---------------------------------------------------------------------------
# losses and the optimiser step (§2.1, §5.1)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("kind,fn", [(0, od.softmax_cross_entropy), (1, od.mse_softmax_loss)])
def test_loss_modes(lrb, kind, fn):
    g = np.random.default_rng(31)
    sums = g.normal(0.0, 3.0, (500, 10)).astype(np.float32)
    labels = g.integers(0, 10, 500).astype(np.int32)
    loss, grad = lrb.lr_loss(dev(sums), dev(labels), kind=kind)
    ref_loss, ref_grad = fn(sums, labels)
    assert abs(float(loss) - ref_loss) / abs(ref_loss) < 1e-5
    assert rel(host(grad), ref_grad) < 1e-5


def test_mse_training_step(lrb):
    # the prototypes' loss (§5.1): squared norm of softmax(S) - onehot(t)
    w = wl.WORKLOADS[3]
    b = 6
    net, phi, saved, out, ref, h = sums_only_forward(lrb, w, b, w.layers, w.detector)
    labels = wl.labels(w, b)
    loss, gs = lrb.lr_loss(out["sums"], dev(labels), kind=lrb.LR_LOSS_SOFTMAX_MSE)
    grad, _ = lrb.lr_donn_backward(net, dev(phi), saved, grad_sums=gs)
    ref_loss, ref_gs = od.mse_softmax_loss(ref["sums"], labels)
    ref_grad = od.donn_backward(ref, phi, h, 1.0, odet(w.detector), grad_sums=ref_gs)
    assert abs(float(loss) - ref_loss) / abs(ref_loss) < TOL_FIELD
    assert rel(host(grad), ref_grad) < TOL_GRAD


# the library receives its hyper-parameters as float32; the oracle gets the same values
ADAM_F32 = dict(lr=float(np.float32(0.5)), beta1=float(np.float32(0.9)), beta2=float(np.float32(0.999)),
                eps=float(np.float32(1e-8)))


def test_adam_steps(lrb):
    g = np.random.default_rng(32)
    phi0 = g.uniform(0.0, 2 * np.pi, (5, 200, 200)).astype(np.float32)
    grads = [g.normal(0.0, 1e-3, (5, 200, 200)).astype(np.float32) for _ in range(4)]
    phi = dev(phi0.copy())
    m = torch.zeros_like(phi)
    v = torch.zeros_like(phi)
    ref = (phi0.astype(np.float64), np.zeros(phi0.shape), np.zeros(phi0.shape))
    for t, gr in enumerate(grads, start=1):
        lrb.lr_adam_update(phi, dev(gr), m, v, t, **ADAM_F32)
        ref = od.adam_update(ref[0], gr, ref[1], ref[2], t, **ADAM_F32)
    assert rel(host(phi), ref[0]) < 1e-6
    assert rel(host(m), ref[1]) < 1e-5
    assert rel(host(v), ref[2]) < 1e-5


def test_training_iteration_at_full_size(lrb):
    """One iteration of the prototypes' training (§5.1) on the benchmark
    workload: sums-only forward, MSE loss, backward, Adam with learning rate
    0.5.  The gradient is checked against the oracle's, and the step against
    the oracle's Adam applied to the same float32 gradient."""
    w = wl.WORKLOADS[3]
    b = w.batch
    net, phi, saved, out, ref, h = sums_only_forward(lrb, w, b, w.layers, w.detector)
    labels = wl.labels(w, b)
    _, gs = lrb.lr_loss(out["sums"], dev(labels), kind=lrb.LR_LOSS_SOFTMAX_MSE, want_loss=False)
    grad, _ = lrb.lr_donn_backward(net, dev(phi), saved, grad_sums=gs)
    _, ref_gs = od.mse_softmax_loss(ref["sums"], labels)
    assert rel(host(grad), od.donn_backward(ref, phi, h, 1.0, odet(w.detector), grad_sums=ref_gs)) < TOL_GRAD
    g32 = host(grad)
    phi_dev = dev(phi.copy())
    m = torch.zeros_like(phi_dev)
    v = torch.zeros_like(phi_dev)
    lrb.lr_adam_update(phi_dev, grad, m, v, 1, **ADAM_F32)
    ref_phi, _, _ = od.adam_update(phi, g32, np.zeros(phi.shape), np.zeros(phi.shape), 1, **ADAM_F32)
    assert rel(host(phi_dev), ref_phi) < 1e-6


# Depth and grid variants of the benchmark workload (the paper's runtime
# study, §5.3): deep networks accumulate rounding over many hops, and N=500
# runs the 25 x 20 Cooley-Tukey plan with its twiddled 20-point B-step.
@pytest.mark.parametrize("n,layers,b", [(100, 30, 2), (200, 10, 3), (500, 3, 2)])
def test_cross_entropy_step_depth_and_grid_variants(lrb, n, layers, b):
    w = wl.scaled(wl.WORKLOADS[3], n=n, layers=layers)
    net, phi, saved, out, ref, h = sums_only_forward(lrb, w, b, layers, w.detector)
    assert rel(host(out["sums"]), ref["sums"]) < TOL_FIELD
    labels = wl.labels(w, b)
    grad, loss = lrb.lr_donn_backward(net, dev(phi), saved, sums=out["sums"], labels=dev(labels))
    ref_loss, gs = od.softmax_cross_entropy(ref["sums"], labels)
    ref_grad = od.donn_backward(ref, phi, h, 1.0, odet(w.detector), grad_sums=gs)
    assert abs(float(loss) - ref_loss) / abs(ref_loss) < TOL_FIELD
    assert rel(host(grad), ref_grad) < TOL_GRAD


# The multi-channel DONN of §5.6.1: three channels (own masks, own inputs)
# whose intensities add at one detector, trained on the shared loss.
def test_multichannel_training_step(lrb):
    w = wl.WORKLOADS[3]
    b, layers, channels = 4, 5, 3
    det = w.detector
    g = np.random.default_rng(7)
    amps = [wl.amplitudes(w, b)] + [g.uniform(0, 1, (b, w.n, w.n)).astype(np.float32) for _ in range(channels - 1)]
    phis = [wl.phases(w)] + [g.uniform(0, 2 * np.pi, (layers, w.n, w.n)).astype(np.float32)
                             for _ in range(channels - 1)]
    nets = [lrb.Network(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n, w.n_fft, layers, 1.0,
                        lrb.Detector(det.size, det.y0, det.x0)) for _ in range(channels)]
    saveds = [net.new_saved(b) for net in nets]
    labels = wl.labels(w, b)
    loss, merged, grads = lrb.multichannel_train_step(nets, [dev(a) for a in amps], [dev(p) for p in phis], saveds,
                                                      dev(labels))
    h = od.transfer_function(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n_fft)
    fwds, ref_merged = od.multichannel_forward(amps, phis, h, 1.0, odet(det))
    ref_loss, gs = od.softmax_cross_entropy(ref_merged, labels)
    ref_grads = od.multichannel_backward(fwds, phis, h, 1.0, odet(det), gs)
    assert rel(host(merged), ref_merged) < TOL_FIELD
    assert abs(float(loss) - ref_loss) / abs(ref_loss) < TOL_FIELD
    for gr, rg in zip(grads, ref_grads):
        assert rel(host(gr), rg) < TOL_GRAD


def test_accumulated_intensity_maps(lrb):
    w = wl.WORKLOADS[2]
    b = 3
    g = np.random.default_rng(8)
    amps = [wl.amplitudes(w, b), g.uniform(0, 1, (b, w.n, w.n)).astype(np.float32)]
    phis = [wl.phases(w), g.uniform(0, 2 * np.pi, (w.layers, w.n, w.n)).astype(np.float32)]
    net = lrb.Network(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n, w.n_fft, w.layers)
    out = lrb.lr_donn_forward(net, dev(amps[0]), dev(phis[0]), sums=False, intensity=True)
    lrb.lr_donn_forward(net, dev(amps[1]), dev(phis[1]), sums=False, intensity=True,
                        out_intensity=out["intensity"], accumulate=True)
    h = od.transfer_function(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n_fft)
    ref = sum(od.donn_forward(a, p, h, 1.0)["intensity"] for a, p in zip(amps, phis))
    assert rel(host(out["intensity"]), ref) < TOL_FIELD
