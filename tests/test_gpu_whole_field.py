"""Whole-field forward (one workgroup per sample, the field in shared memory
through every layer) against the float64 oracle and against the one-pass-per-
layer path on the same inputs.

It runs for forward calls on the Fresnel path with n == n_fft in
{64, 100, 128}, no saved state, no skip field, and at 100 and 128 at least
one sample per CU (256 on MI355X; smaller batches take the layer passes);
LR_LAYER_PASSES forces the layer passes.  At n == n_fft == 200 the field is
held half in shared memory and half in registers, and only LR_WHOLE_FIELD
selects it.  Every case checks, from the library's own launch record, which
path ran.  Tolerance: relative L2 1e-4
(the stated bound for fields and intensities).
"""

import numpy as np
import pytest

import oracle.donn as od
from paper_2306_11268_amd import workloads as wl

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

TOL = 1e-4


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


def ran_whole_field(lrb, fn):
    """Run fn with the library's launch timing on; True if the whole-field kernel ran."""
    lrb.kernel_timing(True)
    try:
        fn()
        torch.cuda.synchronize()
        names = set(lrb.kernel_timing_report())
    finally:
        lrb.kernel_timing(False)
    return any(k.startswith("field_forward") for k in names)


def setup(lrb, m, b, layers=5, gamma=0.9):
    det = wl.layout_grid(m, 4, max(2, m // 10))
    w = wl.Workload(94, "test", 532e-9, 36e-6, 0.3, od.FRESNEL, m, m, layers, b, "forward", det, "sums", "uniform")
    net = lrb.Network(w.wavelength, w.pixel_pitch, w.distance, w.approx, m, m, layers, gamma,
                      lrb.Detector(det.size, det.y0, det.x0))
    amp = wl.amplitudes(w, b)
    phi = wl.phases(w)
    h = od.transfer_function(w.wavelength, w.pixel_pitch, w.distance, w.approx, m)
    ref = od.donn_forward(amp, phi, h, gamma, od.Detector(det.size, tuple(det.y0), tuple(det.x0)))
    return net, amp, phi, ref


@pytest.mark.parametrize("m", [64, 100, 128])
@pytest.mark.parametrize("b", [256, 259, 3])
def test_whole_field_forward_matches_oracle_and_layer_passes(lrb, m, b):
    net, amp, phi, ref = setup(lrb, m, b)
    out = {}
    took = ran_whole_field(lrb, lambda: out.update(lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=True)))
    assert took == (m == 64 or b >= 256)
    whole = host(out["sums"])
    passes = host(lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=True, layer_passes=True)["sums"])
    assert rel(whole, ref["sums"]) < TOL
    assert rel(passes, ref["sums"]) < TOL
    assert rel(whole, passes) < TOL
    # reproducible: fixed-order sums
    again = host(lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=True)["sums"])
    assert np.array_equal(whole, again)


def test_whole_field_forward_accumulates_and_covers_one_layer(lrb):
    # LR_ACCUMULATE adds into the given sums; one layer (two hops) and gamma != 1
    net, amp, phi, ref = setup(lrb, 128, 256, layers=1, gamma=1.3)
    base = np.full(ref["sums"].shape, 2.5, dtype=np.float32)
    out = dev(base)
    lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=True, out_sums=out, accumulate=True)
    assert rel(host(out) - base, ref["sums"]) < TOL


@pytest.mark.parametrize("m,layers,b", [(64, 1, 4), (100, 3, 256), (128, 2, 257)])
def test_whole_field_forward_full_map_outputs(lrb, m, layers, b):
    # intensity map and detector-plane field (workload 1's outputs at 64 x 64),
    # with and without the sums, against the oracle and the layer passes
    net, amp, phi, ref = setup(lrb, m, b, layers=layers, gamma=1.0)
    for sums in (False, True):
        out = {}
        assert ran_whole_field(lrb, lambda: out.update(
            lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=sums, intensity=True, field=True)))
        lp = lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=sums, intensity=True, field=True, layer_passes=True)
        assert rel(host(out["intensity"]), ref["intensity"]) < TOL
        assert rel(host(out["field"]), ref["field"]) < TOL
        assert rel(host(out["intensity"]), host(lp["intensity"])) < TOL
        if sums:
            assert rel(host(out["sums"]), ref["sums"]) < TOL
    # accumulated intensity
    base = np.full((b, m, m), 0.75, dtype=np.float32)
    acc = dev(base)
    lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=False, intensity=True, out_intensity=acc, accumulate=True)
    assert rel(host(acc) - base, ref["intensity"]) < TOL


@pytest.mark.parametrize("b", [256, 3])
def test_whole_field_forward_200_split_field(lrb, b):
    # the 200 x 200 field half in shared memory, half in registers
    net, amp, phi, ref = setup(lrb, 200, b)
    assert not ran_whole_field(lrb, lambda: lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=True))
    out = {}
    assert ran_whole_field(lrb, lambda: out.update(
        lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=True, whole_field=True)))
    whole = host(out["sums"])
    passes = host(lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=True)["sums"])
    assert rel(whole, ref["sums"]) < TOL
    assert rel(whole, passes) < TOL
    again = host(lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=True, whole_field=True)["sums"])
    assert np.array_equal(whole, again)


@pytest.mark.parametrize("layers,b", [(1, 2), (2, 3), (4, 5)])
def test_whole_field_forward_200_full_map_outputs(lrb, layers, b):
    # every pixel of both halves: intensity map and detector-plane field against
    # the oracle, with and without the sums, and the accumulated intensity
    net, amp, phi, ref = setup(lrb, 200, b, layers=layers, gamma=1.1)
    for sums in (False, True):
        out = {}
        assert ran_whole_field(lrb, lambda: out.update(
            lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=sums, intensity=True, field=True, whole_field=True)))
        assert rel(host(out["intensity"]), ref["intensity"]) < TOL
        assert rel(host(out["field"]), ref["field"]) < TOL
        if sums:
            assert rel(host(out["sums"]), ref["sums"]) < TOL
    base = np.full((b, 200, 200), 0.5, dtype=np.float32)
    acc = dev(base)
    lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=False, intensity=True, out_intensity=acc, accumulate=True,
                        whole_field=True)
    assert rel(host(acc) - base, ref["intensity"]) < TOL


@pytest.mark.parametrize("m", [100, 128])
def test_whole_field_flag_below_one_sample_per_cu(lrb, m):
    # LR_WHOLE_FIELD takes the whole-field kernel where the default would not
    # (a batch below the CU count at 100 and 128 points)
    net, amp, phi, ref = setup(lrb, m, 3)
    out = {}
    assert ran_whole_field(lrb, lambda: out.update(
        lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=True, whole_field=True)))
    assert rel(host(out["sums"]), ref["sums"]) < TOL


def test_whole_field_flags_exclude_each_other(lrb):
    net, amp, phi, _ = setup(lrb, 64, 2, layers=1)
    with pytest.raises(ValueError):
        lrb.lr_donn_forward(net, dev(amp), dev(phi), sums=True, layer_passes=True, whole_field=True)
