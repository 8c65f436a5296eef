"""The codesign layer (§3.2) on the GPU against the oracle.

Phases from scores over a device's levels (soft Gumbel-Softmax and the hard
choice), the gradient back to the scores, and a training step that runs
scores -> phases -> DONN forward -> cross-entropy -> DONN backward -> scores.
Tolerances: relative L2 1e-4 on phases and sums, 1e-3 on gradients; the hard
choice is compared exactly (both sides decide on float32 scores).
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


@pytest.mark.parametrize("K,shape,tau", [(256, (2, 40, 40), 1.0), (16, (3, 7, 9), 0.3), (1000, (50,), 2.0),
                                         (1, (10,), 1.0)])
def test_codesign_phase_and_gradient(lrb, K, shape, tau):
    lv = wl.device_levels(3, K)
    lg = wl.codesign_scores(3, shape, K)
    nz = wl.gumbel_draws(3, shape, K)
    gphi = np.random.default_rng(K).standard_normal(shape).astype(np.float32)
    for hard in (False, True):
        phi = host(lrb.lr_codesign_phase(dev(lg), dev(nz), dev(lv), tau, hard=hard))
        ref, w = od.codesign_phase(lg, nz, lv, tau, hard=hard)
        if hard:
            assert np.array_equal(phi, ref.astype(np.float32))
        else:
            assert rel(phi, ref) < TOL_FIELD
    gl = host(lrb.lr_codesign_backward(dev(lg), dev(nz), dev(lv), tau, dev(gphi)))
    ref_gl = od.codesign_backward(w, lv, tau, gphi)
    if K == 1:
        assert np.all(gl == 0.0) and np.all(ref_gl == 0.0)
    else:
        assert rel(gl, ref_gl) < TOL_GRAD


@pytest.mark.parametrize("hard", [False, True])
def test_codesign_training_step(lrb, hard):
    w = wl.scaled(wl.WORKLOADS[3], n=64, layers=2)
    b, K, tau = 3, 32, 0.5
    det = wl.ten_class_layout(64)
    lv = wl.device_levels(w.wid, K)
    lg = wl.codesign_scores(w.wid, (w.layers, w.n, w.n), K)
    nz = wl.gumbel_draws(w.wid, (w.layers, w.n, w.n), K)
    amp = wl.amplitudes(w, b)
    labels = wl.labels(w, b)
    net = lrb.Network(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n, w.n_fft, w.layers, 1.0,
                      lrb.Detector(det.size, det.y0, det.x0))
    phi = lrb.lr_codesign_phase(dev(lg), dev(nz), dev(lv), tau, hard=hard)
    saved = net.new_saved(b)
    out = lrb.lr_donn_forward(net, dev(amp), phi, saved=saved, sums=True)
    gphi, loss = lrb.lr_donn_backward(net, phi, saved, sums=out["sums"], labels=dev(labels))
    glog = lrb.lr_codesign_backward(dev(lg), dev(nz), dev(lv), tau, gphi)

    rphi, rw = od.codesign_phase(lg, nz, lv, tau, hard=hard)
    h = od.transfer_function(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n_fft)
    odet = od.Detector(det.size, tuple(det.y0), tuple(det.x0))
    ref = od.donn_forward(amp, rphi, h, 1.0, odet)
    ref_loss, gs = od.softmax_cross_entropy(ref["sums"], labels)
    rg = od.donn_backward(ref, rphi, h, 1.0, odet, grad_sums=gs)
    assert rel(host(out["sums"]), ref["sums"]) < TOL_FIELD
    assert abs(float(loss) - ref_loss) / abs(ref_loss) < TOL_FIELD
    assert rel(host(glog), od.codesign_backward(rw, lv, tau, rg)) < TOL_GRAD
