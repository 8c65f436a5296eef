"""The C-ABI library loads, exports every declared symbol and rejects bad
arguments on the host, without a GPU (no compute call is made here)."""

import ctypes
import os
import re

import pytest

from paper_2306_11268_amd import binding as lb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lr.h")

needs_lib = pytest.mark.skipif(not os.path.exists(lb.LIB_PATH), reason="liblr.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lr_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_entry_points():
    fns = declared_functions()
    for f in ("lr_tf_build", "lr_propagate", "lr_donn_forward", "lr_donn_backward", "lr_detector_readout"):
        assert f in fns


@needs_lib
def test_library_exports_every_declared_symbol():
    lib = lb.load()
    for f in declared_functions():
        assert hasattr(lib, f), f
    assert set(declared_functions()) == set(lb.EXPORTS)


def _net(**kw):
    d = dict(wavelength=532e-9, pixel_pitch=36e-6, distance=0.3, approx=0, n=200, n_fft=200, num_layers=5,
             gamma=1.0, det=lb.LrDetector(0, 1, None, None), d_H=ctypes.c_void_p(0x1000))
    d.update(kw)
    return lb.LrDonn(d["wavelength"], d["pixel_pitch"], d["distance"], d["approx"], d["n"], d["n_fft"],
                     d["num_layers"], d["gamma"], d["det"], d["d_H"])


def _ws(net, batch=4, op=1):
    return lb.load().lr_workspace_size(ctypes.byref(net), batch, op)


@needs_lib
def test_status_strings_and_version():
    lib = lb.load()
    assert lib.lr_version() >= 1
    for s in range(0, 8):
        assert isinstance(lib.lr_status_string(s), bytes)


@needs_lib
@pytest.mark.parametrize("kw,status", [
    (dict(wavelength=float("nan")), 3), (dict(wavelength=-1.0), 3), (dict(pixel_pitch=0.0), 3),
    (dict(distance=float("inf")), 3), (dict(approx=5), 4), (dict(approx=-1), 4), (dict(approx=4), 4),
    (dict(n_fft=201, n=201), 2),
    (dict(n=202), 2), (dict(n=199), 2), (dict(n=0), 2), (dict(num_layers=0), 2), (dict(num_layers=65), 2),
    (dict(gamma=float("nan")), 3), (dict(d_H=ctypes.c_void_p(0)), 1),
])
def test_descriptor_validation(kw, status):
    assert _ws(_net(**kw)) == -status


@needs_lib
def test_detector_validation():
    ys = (ctypes.c_int32 * 2)(0, 190)
    xs = (ctypes.c_int32 * 2)(0, 0)
    P = ctypes.POINTER(ctypes.c_int32)
    bad = lb.LrDetector(2, 20, ctypes.cast(ys, P), ctypes.cast(xs, P))  # second region leaves the plane
    assert _ws(_net(det=bad)) == -3
    null = lb.LrDetector(2, 20, None, None)
    assert _ws(_net(det=null)) == -1
    many = lb.LrDetector(65, 1, ctypes.cast(ys, P), ctypes.cast(xs, P))
    assert _ws(_net(det=many)) == -3
    ok = lb.LrDetector(1, 20, ctypes.cast(ys, P), ctypes.cast(xs, P))
    assert _ws(_net(det=ok)) > 0


@needs_lib
def test_workspace_size_grows_with_batch_and_op():
    net = _net()
    assert _ws(net, 8, 1) > _ws(net, 4, 1) > 0
    assert _ws(net, 4, 2) > _ws(net, 4, 0) > 0
    assert _ws(net, -1, 1) == -2
    assert _ws(net, 4, 9) == -3


@needs_lib
def test_entry_points_reject_bad_arguments_without_touching_the_gpu():
    lib = lb.load()
    net = _net()
    ref = ctypes.byref(net)
    P = ctypes.c_void_p
    dummy = P(0x2000)
    # transfer function
    assert lib.lr_tf_build(532e-9, 36e-6, 0.3, 0, 64, None, None) == 1
    assert lib.lr_tf_build(0.0, 36e-6, 0.3, 0, 64, dummy, None) == 3
    assert lib.lr_tf_build(532e-9, 36e-6, 0.3, 5, 64, dummy, None) == 4
    assert lib.lr_tf_build(532e-9, 36e-6, 0.3, 0, 0, dummy, None) == 2
    # sampled kernels: lengths with a prime factor above 5, non-positive distance; far field: odd grid
    assert lib.lr_tf_build(532e-9, 36e-6, 0.3, 2, 14, dummy, None) == 2
    assert lib.lr_tf_build(532e-9, 36e-6, 0.0, 3, 64, dummy, None) == 3
    assert lib.lr_tf_build(532e-9, 36e-6, 0.3, 4, 63, dummy, None) == 2
    assert lib.lr_tf_build(532e-9, 36e-6, -1.0, 4, 64, dummy, None) == 3
    # the far field propagates only, forwards only
    far = _net(approx=4)
    assert _ws(far, 4, 0) > 0
    assert _ws(far, 4, 1) == -4 and _ws(far, 4, 2) == -4
    assert lib.lr_propagate(ctypes.byref(far), 2, dummy, P(0x3000), 1, dummy, 1 << 30, None) == 3
    assert _ws(_net(approx=5), 4, 0) == -4
    # flags: unknown bits, both path flags at once; accumulating outputs cannot include the field
    bad = _net()
    bad.flags = 8
    assert _ws(bad, 4, 1) == -3
    bad.flags = 6  # LR_LAYER_PASSES | LR_WHOLE_FIELD
    assert _ws(bad, 4, 1) == -3
    ok = _net()
    ok.flags = 3  # LR_ACCUMULATE | LR_LAYER_PASSES
    assert _ws(ok, 4, 1) > 0
    ok.flags = 5  # LR_ACCUMULATE | LR_WHOLE_FIELD
    assert _ws(ok, 4, 1) > 0
    acc = _net(det=lb.LrDetector(0, 1, None, None))
    acc.flags = 1
    assert lib.lr_donn_forward(ctypes.byref(acc), 2, dummy, dummy, None, None, None, P(0x3000), dummy, 1 << 30,
                               None) == 3
    # propagate: null fields, aliasing, missing / short workspace
    assert lib.lr_propagate(ref, 2, None, dummy, 0, dummy, 1 << 30, None) == 1
    assert lib.lr_propagate(ref, 2, dummy, dummy, 0, dummy, 1 << 30, None) == 7
    assert lib.lr_propagate(ref, 2, dummy, P(0x3000), 0, None, 1 << 30, None) == 1
    assert lib.lr_propagate(ref, 2, dummy, P(0x3000), 0, dummy, 16, None) == 6
    assert lib.lr_propagate(ref, -1, dummy, P(0x3000), 0, dummy, 1 << 30, None) == 2
    # forward: sums without a detector, null inputs
    assert lib.lr_donn_forward(ref, 2, dummy, dummy, None, dummy, None, None, dummy, 1 << 30, None) == 3
    assert lib.lr_donn_forward(ref, 2, None, dummy, None, None, None, None, dummy, 1 << 30, None) == 1
    # backward: exactly one seed, labels need sums and a detector
    assert lib.lr_donn_backward(ref, 2, dummy, dummy, None, None, None, None, None, dummy, dummy, 1 << 30,
                                None) == 3
    assert lib.lr_donn_backward(ref, 2, dummy, dummy, None, None, dummy, dummy, None, dummy, dummy, 1 << 30,
                                None) == 3
    assert lib.lr_donn_backward(ref, 2, dummy, None, None, None, None, dummy, None, dummy, dummy, 1 << 30,
                                None) == 1
    # loss: kind, sizes, outputs, aliasing
    assert lib.lr_loss(2, dummy, dummy, 4, 10, dummy, P(0x3000), None) == 3
    assert lib.lr_loss(0, dummy, dummy, -1, 10, dummy, P(0x3000), None) == 2
    assert lib.lr_loss(1, dummy, dummy, 4, 65, dummy, P(0x3000), None) == 2
    assert lib.lr_loss(0, dummy, dummy, 4, 10, None, None, None) == 1
    assert lib.lr_loss(0, None, dummy, 4, 10, dummy, None, None) == 1
    assert lib.lr_loss(0, dummy, P(0x3000), 4, 10, None, dummy, None) == 7
    assert lib.lr_loss(0, None, None, 0, 10, dummy, None, None) == 0
    # Adam: step, hyper-parameters, pointers, aliasing
    f = ctypes.c_float
    assert lib.lr_adam_update(dummy, P(0x3000), P(0x4000), P(0x5000), 8, 0, f(0.5), f(0.9), f(0.999), f(1e-8),
                              None) == 2
    assert lib.lr_adam_update(dummy, P(0x3000), P(0x4000), P(0x5000), -1, 1, f(0.5), f(0.9), f(0.999), f(1e-8),
                              None) == 2
    assert lib.lr_adam_update(dummy, P(0x3000), P(0x4000), P(0x5000), 8, 1, f(0.5), f(1.0), f(0.999), f(1e-8),
                              None) == 3
    assert lib.lr_adam_update(dummy, P(0x3000), P(0x4000), P(0x5000), 8, 1, f(float("nan")), f(0.9), f(0.999),
                              f(1e-8), None) == 3
    assert lib.lr_adam_update(dummy, P(0x3000), P(0x4000), P(0x5000), 8, 1, f(0.5), f(0.9), f(0.999), f(-1.0),
                              None) == 3
    assert lib.lr_adam_update(None, P(0x3000), P(0x4000), P(0x5000), 8, 1, f(0.5), f(0.9), f(0.999), f(1e-8),
                              None) == 1
    assert lib.lr_adam_update(dummy, P(0x3000), dummy, P(0x5000), 8, 1, f(0.5), f(0.9), f(0.999), f(1e-8),
                              None) == 7
    assert lib.lr_adam_update(None, None, None, None, 0, 1, f(0.5), f(0.9), f(0.999), f(1e-8), None) == 0
    # detector readout
    det = lb.LrDetector(1, 300, None, None)
    assert lib.lr_detector_readout(dummy, 2, 200, ctypes.byref(det), dummy, None) in (1, 3)
    assert lib.lr_detector_readout(dummy, 2, 200, None, dummy, None) == 1


@needs_lib
def test_kernel_timing_toggle_without_launches():
    lb.kernel_timing(True)
    assert lb.kernel_timing_report() == {}
    lb.kernel_timing(False)


@needs_lib
def test_codesign_rejects_bad_arguments_without_touching_the_gpu():
    lib = lb.load()
    P = ctypes.c_void_p
    a, b, c, d = P(0x1000), P(0x2000), P(0x3000), P(0x4000)
    assert lib.lr_codesign_phase(a, b, c, 0, 10, 1.0, 0, d, None) == 2
    assert lib.lr_codesign_phase(a, b, c, 1025, 10, 1.0, 0, d, None) == 2
    assert lib.lr_codesign_phase(a, b, c, 16, -1, 1.0, 0, d, None) == 2
    assert lib.lr_codesign_phase(a, b, c, 16, 10, 0.0, 0, d, None) == 3
    assert lib.lr_codesign_phase(a, b, c, 16, 10, float("nan"), 0, d, None) == 3
    assert lib.lr_codesign_phase(None, b, c, 16, 10, 1.0, 0, d, None) == 1
    assert lib.lr_codesign_phase(a, b, c, 16, 10, 1.0, 0, a, None) == 7
    assert lib.lr_codesign_phase(None, None, None, 16, 0, 1.0, 0, None, None) == 0
    assert lib.lr_codesign_backward(a, b, c, 16, 10, 1.0, d, None, None) == 1
    assert lib.lr_codesign_backward(a, b, c, 16, 10, 1.0, d, d, None) == 7
    assert lib.lr_codesign_backward(a, b, c, 16, 10, -2.0, d, P(0x5000), None) == 3


@needs_lib
def test_layer_norm_rejects_bad_arguments_without_touching_the_gpu():
    lib = lb.load()
    P = ctypes.c_void_p
    count = 200 * 200
    ws = lib.lr_layer_norm_workspace_size(4, count)
    assert ws == 4 * (((count + 4095) // 4096) + 1) * 8
    assert lib.lr_layer_norm_workspace_size(-1, count) == -2
    assert lib.lr_layer_norm_workspace_size(4, 0) == -2
    assert lib.lr_layer_norm_workspace_size(4, (1 << 28) + 1) == -2
    x, y, st, w = P(0x10000000), P(0x20000000), P(0x30000000), P(0x40000000)
    assert lib.lr_layer_norm(x, -1, count, 1e-5, y, st, w, ws, None) == 2
    assert lib.lr_layer_norm(x, 4, 0, 1e-5, y, st, w, ws, None) == 2
    assert lib.lr_layer_norm(x, 4, count, float("nan"), y, st, w, ws, None) == 3
    assert lib.lr_layer_norm(x, 4, count, -1.0, y, st, w, ws, None) == 3
    assert lib.lr_layer_norm(None, 4, count, 1e-5, y, st, w, ws, None) == 1
    assert lib.lr_layer_norm(x, 4, count, 1e-5, y, st, w, ws - 1, None) == 6
    assert lib.lr_layer_norm(x, 4, count, 1e-5, y, P(0x10000000 + 64), w, ws, None) == 7    # stats inside x
    assert lib.lr_layer_norm(x, 4, count, 1e-5, P(0x10000000 + 8), st, w, ws, None) == 7    # y overlaps x
    assert lib.lr_layer_norm(None, 0, count, 1e-5, None, None, None, 0, None) == 0
    g = P(0x50000000)
    assert lib.lr_layer_norm_backward(g, y, st, 4, count, None, w, ws, None) == 1
    assert lib.lr_layer_norm_backward(g, y, st, 4, count, x, w, ws - 8, None) == 6
    assert lib.lr_layer_norm_backward(g, y, st, 4, count, y, w, ws, None) == 7     # dx over the normalised maps
    assert lib.lr_layer_norm_backward(g, y, st, 4, count, P(0x50000000 + 4), w, ws, None) == 7
    assert lib.lr_layer_norm_backward(g, y, st, 4, 0, x, w, ws, None) == 2


@needs_lib
def test_skip_field_must_not_alias_the_field_output():
    lib = lb.load()
    P = ctypes.c_void_p
    net = _net()
    net.d_skip = 0x3000
    dummy = P(0x1000)
    need = lib.lr_workspace_size(ctypes.byref(net), 2, lb.LR_OP_FORWARD)
    assert need > 0
    assert lib.lr_donn_forward(ctypes.byref(net), 2, dummy, dummy, None, None, None, P(0x3000), dummy, need,
                               None) == 7


@needs_lib
def test_layer_norm_stats_outside_the_workspace():
    lib = lb.load()
    P = ctypes.c_void_p
    count = 4096 * 3
    ws = lib.lr_layer_norm_workspace_size(2, count)
    x, y, w = P(0x10000000), P(0x20000000), P(0x40000000)
    assert lib.lr_layer_norm(x, 2, count, 1e-5, y, P(0x40000000 + 8), w, ws, None) == 7


@needs_lib
def test_detector_origins_near_int_max_are_rejected():
    """Region origins whose end overflows int32 must fail validation, not wrap."""
    lib = lb.load()
    P = ctypes.POINTER(ctypes.c_int32)
    big = 2147483642
    for ys, xs in (((big,), (0,)), ((0,), (big,)), ((-big,), (0,))):
        y = (ctypes.c_int32 * 1)(*ys)
        x = (ctypes.c_int32 * 1)(*xs)
        det = lb.LrDetector(1, 20, ctypes.cast(y, P), ctypes.cast(x, P))
        assert _ws(_net(det=det)) == -3
        assert lib.lr_detector_readout(ctypes.c_void_p(0x1000), 2, 200, ctypes.byref(det), ctypes.c_void_p(0x9000000),
                                       None) == 3
        net = _net(det=det)
        assert lib.lr_donn_forward(ctypes.byref(net), 2, ctypes.c_void_p(0x1000), ctypes.c_void_p(0x1000), None,
                                   None, None, None, ctypes.c_void_p(0x40000000), 1 << 30, None) == 3


@needs_lib
def test_partially_overlapping_buffers_are_rejected():
    """Outputs overlapping an input (or another output) by part of their range
    are aliasing errors, not only equal pointers; nothing is launched."""
    lib = lb.load()
    P = ctypes.c_void_p
    net = _net()
    ref = ctypes.byref(net)
    field = 2 * 200 * 200 * 8
    a, w = 0x10000000, 0x40000000
    ws = lib.lr_workspace_size(ref, 2, lb.LR_OP_PROPAGATE)
    # propagate: output starting inside the input, or the workspace over either
    assert lib.lr_propagate(ref, 2, P(a), P(a + field - 8), 0, P(w), ws, None) == 7
    assert lib.lr_propagate(ref, 2, P(a), P(a + field), 0, P(a + 2 * field - 64), ws, None) == 7
    # forward: intensity over the amplitudes, field output over the phases
    wf = lib.lr_workspace_size(ref, 2, lb.LR_OP_FORWARD)
    amp, phi = 0x10000000, 0x20000000
    assert lib.lr_donn_forward(ref, 2, P(amp), P(phi), None, None, P(amp + 4096), None, P(w), wf, None) == 7
    assert lib.lr_donn_forward(ref, 2, P(amp), P(phi), None, None, None, P(phi + 8), P(w), wf, None) == 7
    # backward: dphi over the saved state
    det_y = (ctypes.c_int32 * 1)(0)
    det = lb.LrDetector(1, 20, ctypes.cast(det_y, ctypes.POINTER(ctypes.c_int32)),
                        ctypes.cast(det_y, ctypes.POINTER(ctypes.c_int32)))
    nd = _net(det=det)
    wb = lib.lr_workspace_size(ctypes.byref(nd), 2, lb.LR_OP_BACKWARD)
    saved = 0x30000000
    gi = 0x50000000
    assert lib.lr_donn_backward(ctypes.byref(nd), 2, P(phi), P(saved), None, None, None, P(gi), None,
                                P(saved + 800), P(w), wb, None) == 7
    # Adam: a moment buffer starting inside the phases
    f = ctypes.c_float
    assert lib.lr_adam_update(P(0x1000), P(0x9000), P(0x1000 + 16), P(0x5000), 8, 1, f(0.5), f(0.9), f(0.999),
                              f(1e-8), None) == 7


@needs_lib
def test_noalloc_propagate_limits_without_touching_the_gpu():
    lib = lb.load()
    P = ctypes.c_void_p
    limit = lib.lr_propagate_noalloc_limit()
    assert limit == 32 << 20
    net = _net(num_layers=1)
    ref = ctypes.byref(net)
    # a batch whose workspace exceeds the scratch array is rejected before any launch
    per = lib.lr_workspace_size(ref, 1, lb.LR_OP_PROPAGATE)
    big = limit // (200 * 200 * 8) + 2
    assert lib.lr_workspace_size(ref, big, lb.LR_OP_PROPAGATE) > limit > per
    assert lib.lr_propagate_noalloc(ref, big, P(0x1000), P(0x40000000), 0, None) == 6
    assert lib.lr_propagate_noalloc(ref, 2, None, P(0x40000000), 0, None) == 1
    assert lib.lr_propagate_noalloc(ref, -1, P(0x1000), P(0x40000000), 0, None) == 2
    assert lib.lr_propagate_noalloc(ref, 0, None, None, 0, None) == 0
    bad = _net(d_H=ctypes.c_void_p(0))
    assert lib.lr_propagate_noalloc(ctypes.byref(bad), 2, P(0x1000), P(0x40000000), 0, None) == 1


@needs_lib
def test_binding_shares_torchs_hip_runtime():
    """Loading the library through the binding maps one HIP runtime, torch's:
    loaded first on its own, the library would bind a second copy from the
    ROCm install, and torch's device pointers and streams would be foreign to
    it."""
    import subprocess
    import sys
    code = ("import paper_2306_11268_amd.binding as lb; lb.load(); "
            "m = open('/proc/self/maps').read(); "
            "print(len({l.split()[-1] for l in m.splitlines() if 'libamdhip64' in l}))")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, cwd=ROOT, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    assert r.stdout.strip().splitlines()[-1] == "1"
