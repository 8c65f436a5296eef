"""The sampled-kernel transfer functions and the Fraunhofer far field on the GPU.

lr_tf_build's float64 host tables against the oracle's (rounding to
complex64: relative L2 1e-6), one hop with the sampled Fresnel and
Rayleigh-Sommerfeld kernels, a training step with the Rayleigh-Sommerfeld
kernel, and the far field of Eq. (fraunhofer), padded and unpadded, against
the oracle (relative L2 1e-4 on fields and sums, 1e-3 on dL/dphi).
"""

import numpy as np
import pytest

import oracle.donn as od
from paper_2306_11268_amd import workloads as wl

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

TOL_TABLE = 1e-6
TOL_FIELD = 1e-4
TOL_GRAD = 1e-3


def rel(a, b):
    a = np.asarray(a, dtype=np.complex128)
    b = np.asarray(b, dtype=np.complex128)
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


def crand(seed, shape):
    g = np.random.default_rng(seed)
    return (g.standard_normal(shape) + 1j * g.standard_normal(shape)).astype(np.complex64)


@pytest.mark.parametrize("approx", [od.FRESNEL_IR, od.RS_IR])
@pytest.mark.parametrize("m", [64, 100, 200, 500, 1024])
def test_sampled_kernel_table(lrb, approx, m):
    lam, dx, z = (532e-9, 36e-6, 0.3) if approx == od.FRESNEL_IR else (1550e-9, 8e-6, 0.05)
    h = host(lrb.lr_tf_build(lam, dx, z, approx, m))
    assert rel(h, od.transfer_function(lam, dx, z, approx, m)) < TOL_TABLE


@pytest.mark.parametrize("approx", [od.FRESNEL_IR, od.RS_IR])
@pytest.mark.parametrize("n,m", [(64, 128), (100, 200), (200, 200)])
def test_sampled_kernel_hop(lrb, approx, n, m):
    lam, dx, z = (532e-9, 36e-6, 0.3) if approx == od.FRESNEL_IR else (1550e-9, 8e-6, 0.05)
    u = crand(n + m + approx, (2, n, n))
    net = lrb.Network(lam, dx, z, approx, n, m, 1)
    h = od.transfer_function(lam, dx, z, approx, m)
    for adjoint in (False, True):
        out = host(lrb.lr_propagate(net, dev(u), adjoint=adjoint))
        assert rel(out, od.propagate(u.astype(np.complex128), h, adjoint=adjoint)) < TOL_FIELD


@pytest.mark.parametrize("layers", [1, 2])
def test_rayleigh_sommerfeld_kernel_training_step(lrb, layers):
    w = wl.WORKLOADS[3]
    n, m, b = 128, 256, 3   # blobs of sigma up to 40 px need n > 80
    lam, dx, z = 1550e-9, 8e-6, 0.05
    det = wl.layout_grid(n, 4, 16)
    net = lrb.Network(lam, dx, z, od.RS_IR, n, m, layers, 0.9, lrb.Detector(det.size, det.y0, det.x0))
    amp = wl.blobs_batch(w.wid, b, n)
    phi = wl.phases(wl.scaled(w, n=n, layers=layers))
    saved = net.new_saved(b)
    out = lrb.lr_donn_forward(net, dev(amp), dev(phi), saved=saved, sums=True)
    h = od.transfer_function(lam, dx, z, od.RS_IR, m)
    odet = od.Detector(det.size, tuple(det.y0), tuple(det.x0))
    ref = od.donn_forward(amp, phi, h, 0.9, odet)
    assert rel(host(out["sums"]), ref["sums"]) < TOL_FIELD
    labels = wl.labels(w, b, classes=det.num)
    grad, loss = lrb.lr_donn_backward(net, dev(phi), saved, sums=out["sums"], labels=dev(labels))
    ref_loss, gs = od.softmax_cross_entropy(ref["sums"], labels)
    assert abs(float(loss) - ref_loss) / abs(ref_loss) < TOL_FIELD
    assert rel(host(grad), od.donn_backward(ref, phi, h, 0.9, odet, grad_sums=gs)) < TOL_GRAD


@pytest.mark.parametrize("n,m,z", [(64, 128, 5.0), (200, 200, 2.0), (100, 200, 0.8), (512, 1024, 20.0)])
def test_fraunhofer_far_field(lrb, n, m, z):
    lam, dx = 532e-9, 36e-6
    b = 2 if m <= 512 else 1
    u = crand(n * 7 + m, (b, n, n))
    net = lrb.Network(lam, dx, z, lrb.LR_FRAUNHOFER, n, m, 1)
    out = host(lrb.lr_propagate(net, dev(u)))
    assert out.shape == (b, m, m)
    assert rel(out, od.fraunhofer(u.astype(np.complex128), lam, dx, z, m)) < TOL_FIELD
