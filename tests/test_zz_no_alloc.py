"""The no-allocation entry point lr_propagate_noalloc against lr_propagate.

Both run the same kernels on the same inputs, the first with the library's
fixed device scratch array as its workspace, the second with a caller
workspace, so the outputs must agree bit for bit.  Two calls in a row, the
second on a smaller input, check that what the first leaves in the shared
array does not leak into the second.  A third case compares one hop with
the float64 oracle at the tolerance of the other parity tests.
"""

import numpy as np
import pytest

import oracle.donn as od

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lrb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2306_11268_amd import binding
    binding.load()
    return binding


def field(seed, b, n):
    g = np.random.default_rng([230611268, 90, seed])
    x = (g.standard_normal((b, n, n)) + 1j * g.standard_normal((b, n, n))).astype(np.complex64)
    return torch.from_numpy(x).cuda()


# (approx, n, n_fft, distance, batch of the first call, batch of the second)
CASES = [
    (0, 64, 64, 0.3, 4, 2),        # Fresnel, one hop at 64 x 64 (the single-layer workload's grid)
    (0, 200, 200, 0.3, 24, 3),     # Fresnel, the 200 x 200 grid in slot order
    (1, 100, 200, 0.05, 8, 1),     # angular spectrum, 100 in a 200 grid (2-D table and two work fields)
]


@pytest.mark.parametrize("approx,n,nfft,z,b1,b2", CASES)
@pytest.mark.parametrize("adjoint", [False, True])
def test_noalloc_matches_lr_propagate_twice(lrb, approx, n, nfft, z, b1, b2, adjoint):
    net = lrb.Network(532e-9, 36e-6, z, approx, n, nfft)
    assert net.workspace_size(b1, lrb.LR_OP_PROPAGATE) <= lrb.lr_propagate_noalloc_limit()
    for seed, b in ((1, b1), (2, b2)):
        x = field(seed, b, n)
        ref = lrb.lr_propagate(net, x, adjoint=adjoint)
        got = lrb.lr_propagate_noalloc(net, x, adjoint=adjoint)
        torch.cuda.synchronize()
        print(f"  approx {approx} n {n} n_fft {nfft} batch {b} adjoint {adjoint}")
        assert torch.equal(got, ref)


def test_noalloc_hop_against_the_oracle(lrb):
    n = 64
    net = lrb.Network(532e-9, 36e-6, 0.3, 0, n, n)
    x = field(3, 2, n)
    got = lrb.lr_propagate_noalloc(net, x).cpu().numpy()
    h = od.transfer_function(532e-9, 36e-6, 0.3, 0, n)
    ref = od.propagate(x.cpu().numpy().astype(np.complex128), h)
    r = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    print(f"  rel-L2 {r:.3e}")
    assert r <= 1e-4


def test_noalloc_rejects_batches_over_the_limit(lrb):
    n = 200
    net = lrb.Network(532e-9, 36e-6, 0.3, 0, n, n)
    limit = lrb.lr_propagate_noalloc_limit()
    b = limit // (n * n * 8) + 1
    assert net.workspace_size(b, lrb.LR_OP_PROPAGATE) > limit
    x = torch.zeros((b, n, n), dtype=torch.complex64, device="cuda")
    with pytest.raises(lrb.LrError) as e:
        lrb.lr_propagate_noalloc(net, x)
    assert e.value.status == 6
