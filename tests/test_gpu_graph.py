"""A training step recorded as a HIP graph and replayed (as bench.py times it).

The step's launches are kernels only, so the recorded graph must reproduce the
eager step exactly (every reduction runs in a fixed order): each of several
replays, with eager work and synchronisation between them, is compared bit for
bit with the eager result.
"""

import numpy as np
import pytest

from paper_2306_11268_amd import workloads as wl

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lrb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2306_11268_amd import binding
    binding.load()
    return binding


def test_training_step_graph_replays_match_eager(lrb):
    w = wl.WORKLOADS[3]
    b = 64
    det = w.detector
    net = lrb.Network(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n, w.n_fft, w.layers, 1.0,
                      lrb.Detector(det.size, det.y0, det.x0))
    amp = torch.from_numpy(wl.amplitudes(w, b)).cuda()
    phi = torch.from_numpy(wl.phases(w)).cuda()
    labels = torch.from_numpy(wl.labels(w, b)).cuda()
    saved = net.new_saved(b)
    sums = torch.empty((b, det.num), dtype=torch.float32, device="cuda")
    grad = torch.empty_like(phi)

    def step():
        lrb.lr_donn_forward(net, amp, phi, saved=saved, sums=True, out_sums=sums)
        return lrb.lr_donn_backward(net, phi, saved, sums=sums, labels=labels, out_grad_phi=grad)[1]

    loss = step()
    torch.cuda.synchronize()
    ref_grad, ref_sums, ref_loss = grad.clone(), sums.clone(), float(loss)

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        loss_g = step()
    torch.cuda.synchronize()
    for r in range(3):
        grad.fill_(float("nan"))
        sums.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(sums, ref_sums), f"replay {r}: sums"
        assert torch.equal(grad, ref_grad), f"replay {r}: dphi"
        assert float(loss_g) == ref_loss, f"replay {r}: loss"
        assert np.isfinite(grad.cpu().numpy()).all()
