"""Thin Python binding of liblr.so (the C ABI in include/lr.h).

Argument marshalling only: torch tensors supply device memory and the
current HIP stream; every computation runs in the library's HIP kernels.
Importing this module does not load the library; the first call does, and
raises if liblr.so has not been built.  There is no fallback.
"""

from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int32, c_int64, c_size_t, c_void_p
from typing import Optional, Sequence

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblr.so")

LR_FRESNEL = 0
LR_ANGULAR_SPECTRUM = 1
LR_FRESNEL_IR = 2
LR_RS_IR = 3
LR_FRAUNHOFER = 4
LR_ACCUMULATE = 1
LR_LAYER_PASSES = 2
LR_WHOLE_FIELD = 4
LR_OP_PROPAGATE = 0
LR_OP_FORWARD = 1
LR_OP_BACKWARD = 2
LR_LOSS_SOFTMAX_CE = 0
LR_LOSS_SOFTMAX_MSE = 1

EXPORTS = (
    "lr_tf_build", "lr_workspace_size", "lr_saved_size",
    "lr_propagate", "lr_propagate_noalloc", "lr_propagate_noalloc_limit",
    "lr_detector_readout", "lr_donn_forward", "lr_donn_backward",
    "lr_loss", "lr_adam_update", "lr_codesign_phase", "lr_codesign_backward",
    "lr_layer_norm_workspace_size", "lr_layer_norm", "lr_layer_norm_backward",
    "lr_status_string", "lr_kernel_timing", "lr_kernel_timing_report", "lr_version",
)


class LrDetector(ctypes.Structure):
    _fields_ = [("num", c_int32), ("size", c_int32), ("y0", POINTER(c_int32)), ("x0", POINTER(c_int32))]


class LrDonn(ctypes.Structure):
    _fields_ = [
        ("wavelength", c_double), ("pixel_pitch", c_double), ("distance", c_double),
        ("approx", c_int32), ("n", c_int32), ("n_fft", c_int32), ("num_layers", c_int32),
        ("gamma", c_float), ("det", LrDetector), ("d_H", c_void_p), ("flags", c_int32),
        ("d_skip", c_void_p),
    ]


class LrError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} (status {status})")
        self.status = status


_lib = None


def load() -> ctypes.CDLL:
    """Load liblr.so and declare the ABI; raises if the library is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run paper_2306_11268_amd.build.build() first")
    # torch first: its HIP runtime is then the one the library binds to, so
    # device pointers and streams from torch are valid in the library's calls
    _torch()
    lib = ctypes.CDLL(LIB_PATH)
    P = c_void_p
    lib.lr_tf_build.argtypes = [c_double, c_double, c_double, c_int32, c_int32, P, P]
    lib.lr_workspace_size.argtypes = [POINTER(LrDonn), c_int32, c_int32]
    lib.lr_workspace_size.restype = c_int64
    lib.lr_saved_size.argtypes = [POINTER(LrDonn), c_int32]
    lib.lr_saved_size.restype = c_int64
    lib.lr_propagate.argtypes = [POINTER(LrDonn), c_int32, P, P, c_int32, P, c_size_t, P]
    lib.lr_propagate_noalloc.argtypes = [POINTER(LrDonn), c_int32, P, P, c_int32, P]
    lib.lr_propagate_noalloc_limit.argtypes = []
    lib.lr_propagate_noalloc_limit.restype = c_int64
    lib.lr_detector_readout.argtypes = [P, c_int32, c_int32, POINTER(LrDetector), P, P]
    lib.lr_donn_forward.argtypes = [POINTER(LrDonn), c_int32, P, P, P, P, P, P, P, c_size_t, P]
    lib.lr_donn_backward.argtypes = [POINTER(LrDonn), c_int32, P, P, P, P, P, P, P, P, P, c_size_t, P]
    lib.lr_loss.argtypes = [c_int32, P, P, c_int32, c_int32, P, P, P]
    lib.lr_adam_update.argtypes = [P, P, P, P, c_int64, c_int32, c_float, c_float, c_float, c_float, P]
    lib.lr_codesign_phase.argtypes = [P, P, P, c_int32, c_int64, c_float, c_int32, P, P]
    lib.lr_codesign_backward.argtypes = [P, P, P, c_int32, c_int64, c_float, P, P, P]
    lib.lr_layer_norm_workspace_size.argtypes = [c_int32, c_int64]
    lib.lr_layer_norm_workspace_size.restype = c_int64
    lib.lr_layer_norm.argtypes = [P, c_int32, c_int64, c_float, P, P, P, c_size_t, P]
    lib.lr_layer_norm_backward.argtypes = [P, P, P, c_int32, c_int64, P, P, c_size_t, P]
    lib.lr_status_string.argtypes = [ctypes.c_int]
    lib.lr_status_string.restype = c_char_p
    lib.lr_kernel_timing.argtypes = [c_int32]
    lib.lr_kernel_timing_report.argtypes = [ctypes.c_char_p, c_size_t]
    lib.lr_version.restype = c_int32
    for name in EXPORTS:
        getattr(lib, name).restype = getattr(lib, name).restype or ctypes.c_int
    _lib = lib
    return lib


def status_string(status: int) -> str:
    try:
        return load().lr_status_string(int(status)).decode()
    except Exception:  # library missing while formatting an error
        return "unknown"


def _check(status: int, what: str) -> None:
    if status != 0:
        raise LrError(status, what)


# ---------------------------------------------------------------------------
# torch marshalling helpers
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _stream(device) -> c_void_p:
    torch = _torch()
    return c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _ptr(t, dtype=None, shape=None, name="tensor") -> Optional[c_void_p]:
    if t is None:
        return None
    torch = _torch()
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return c_void_p(t.data_ptr())


class Detector:
    """Host copy of a detector layout (square regions of side ``size``)."""

    def __init__(self, size: int, y0: Sequence[int], x0: Sequence[int]):
        if len(y0) != len(x0):
            raise ValueError("y0 and x0 differ in length")
        self.size = int(size)
        self.y0 = [int(v) for v in y0]
        self.x0 = [int(v) for v in x0]
        k = len(self.y0)
        self._y = (c_int32 * max(k, 1))(*self.y0)
        self._x = (c_int32 * max(k, 1))(*self.x0)
        self.c = LrDetector(k, self.size, ctypes.cast(self._y, POINTER(c_int32)),
                            ctypes.cast(self._x, POINTER(c_int32)))

    @property
    def num(self) -> int:
        return len(self.y0)

    @classmethod
    def none(cls) -> "Detector":
        return cls(1, [], [])


class Network:
    """An lr_donn descriptor with its transfer function and workspace cache."""

    def __init__(self, wavelength: float, pixel_pitch: float, distance: float, approx: int, n: int,
                 n_fft: Optional[int] = None, num_layers: int = 1, gamma: float = 1.0,
                 detector: Optional[Detector] = None, device="cuda"):
        torch = _torch()
        self.device = torch.device(device)
        self.n = int(n)
        self.n_fft = int(n if n_fft is None else n_fft)
        self.num_layers = int(num_layers)
        self.detector = detector if detector is not None else Detector.none()
        self.H = torch.empty((self.n_fft, self.n_fft), dtype=torch.complex64, device=self.device)
        lr_tf_build(wavelength, pixel_pitch, distance, approx, self.n_fft, out=self.H)
        self.c = LrDonn(float(wavelength), float(pixel_pitch), float(distance), int(approx), self.n,
                        self.n_fft, self.num_layers, float(gamma), self.detector.c, c_void_p(self.H.data_ptr()))
        self._work = {}

    def workspace_size(self, batch: int, op: int) -> int:
        r = load().lr_workspace_size(ctypes.byref(self.c), int(batch), int(op))
        if r < 0:
            raise LrError(int(-r), "lr_workspace_size")
        return int(r)

    def saved_size(self, batch: int) -> int:
        r = load().lr_saved_size(ctypes.byref(self.c), int(batch))
        if r < 0:
            raise LrError(int(-r), "lr_saved_size")
        return int(r)

    def workspace(self, batch: int, op: int):
        torch = _torch()
        nbytes = max(self.workspace_size(batch, op), 1)
        buf = self._work.get(op)
        if buf is None or buf.numel() < nbytes:
            buf = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
            self._work[op] = buf
        return buf

    def new_saved(self, batch: int):
        torch = _torch()
        return torch.empty(max(self.saved_size(batch), 1), dtype=torch.uint8, device=self.device)


# ---------------------------------------------------------------------------
# The five entry points, same names as the C ABI
# ---------------------------------------------------------------------------

def lr_tf_build(wavelength: float, pixel_pitch: float, distance: float, approx: int, n_fft: int,
                out=None, device="cuda"):
    """Transfer function H [n_fft, n_fft] complex64 (float64 host evaluation)."""
    torch = _torch()
    if out is None:
        out = torch.empty((n_fft, n_fft), dtype=torch.complex64, device=device)
    p = _ptr(out, torch.complex64, (n_fft, n_fft), "out")
    _check(load().lr_tf_build(float(wavelength), float(pixel_pitch), float(distance), int(approx),
                              int(n_fft), p, _stream(out.device)), "lr_tf_build")
    return out


def lr_propagate(net: Network, field, adjoint: bool = False, out=None):
    """One hop P_z (or its adjoint) of a complex64 batch [B, n, n]; with
    LR_FRAUNHOFER the far field [B, n_fft, n_fft]."""
    torch = _torch()
    b = int(field.shape[0])
    m = net.n_fft if net.c.approx == LR_FRAUNHOFER else net.n
    if out is None:
        out = torch.empty((b, m, m), dtype=torch.complex64, device=field.device)
    w = net.workspace(b, LR_OP_PROPAGATE)
    _check(load().lr_propagate(ctypes.byref(net.c), b,
                               _ptr(field, torch.complex64, (b, net.n, net.n), "field"),
                               _ptr(out, torch.complex64, (b, m, m), "out"),
                               1 if adjoint else 0, _ptr(w), w.numel(), _stream(net.device)), "lr_propagate")
    return out


def lr_propagate_noalloc(net: Network, field, adjoint: bool = False, out=None):
    """lr_propagate with the library's fixed device scratch array as the
    workspace (no allocation inside the call; batches whose workspace exceeds
    lr_propagate_noalloc_limit() bytes are rejected).  Calls that overlap on
    one GPU share that array: order them."""
    torch = _torch()
    b = int(field.shape[0])
    m = net.n_fft if net.c.approx == LR_FRAUNHOFER else net.n
    if out is None:
        out = torch.empty((b, m, m), dtype=torch.complex64, device=field.device)
    _check(load().lr_propagate_noalloc(ctypes.byref(net.c), b,
                                       _ptr(field, torch.complex64, (b, net.n, net.n), "field"),
                                       _ptr(out, torch.complex64, (b, m, m), "out"),
                                       1 if adjoint else 0, _stream(net.device)), "lr_propagate_noalloc")
    return out


def lr_propagate_noalloc_limit() -> int:
    """Bytes of the device scratch array lr_propagate_noalloc uses as its workspace."""
    return int(load().lr_propagate_noalloc_limit())


def lr_detector_readout(field, detector: Detector, out=None):
    """Region sums of |field|^2, float32 [B, K]."""
    torch = _torch()
    b, n = int(field.shape[0]), int(field.shape[-1])
    if out is None:
        out = torch.empty((b, detector.num), dtype=torch.float32, device=field.device)
    _check(load().lr_detector_readout(_ptr(field, torch.complex64, (b, n, n), "field"), b, n,
                                      ctypes.byref(detector.c), _ptr(out, torch.float32, (b, detector.num), "out"),
                                      _stream(field.device)), "lr_detector_readout")
    return out


def _with_skip(desc, skip, b: int, n: int):
    """The descriptor with d_skip set to a complex64 [b, n, n] field (a copy), or desc."""
    if skip is None:
        return desc
    torch = _torch()
    d = LrDonn.from_buffer_copy(desc)
    d.d_skip = _ptr(skip, torch.complex64, (b, n, n), "skip").value
    return d


def lr_donn_forward(net: Network, amp, phi, saved=None, sums: bool = True, intensity: bool = False,
                    field: bool = False, out_sums=None, out_intensity=None, out_field=None,
                    accumulate: bool = False, skip=None, layer_passes: bool = False, whole_field: bool = False):
    """Forward pass; returns a dict with the requested outputs (device tensors).
    With accumulate the sums / intensity are added into out_sums / out_intensity
    (LR_ACCUMULATE), which must then be given.  skip: complex64 [B, n, n]
    added to the detector-plane field (lr_donn.d_skip); give the same field
    to lr_donn_backward.  layer_passes: one pass per layer even where the
    whole-field kernel would run (LR_LAYER_PASSES: Fresnel, n == n_fft in
    {64, 100, 128}, no saved state, no skip).  whole_field: the whole-field
    kernel wherever it applies, also at n == n_fft == 200 (LR_WHOLE_FIELD)."""
    torch = _torch()
    b = int(amp.shape[0])
    n, L = net.n, net.num_layers
    dev = net.device
    desc = _with_skip(net.c, skip, b, n)
    if accumulate:
        if (sums and out_sums is None) or (intensity and out_intensity is None) or field:
            raise ValueError("accumulate needs out_sums / out_intensity and no field output")
        desc = LrDonn.from_buffer_copy(desc)
        desc.flags = LR_ACCUMULATE
    if layer_passes and whole_field:
        raise ValueError("layer_passes and whole_field exclude each other")
    if layer_passes:
        desc = LrDonn.from_buffer_copy(desc)
        desc.flags |= LR_LAYER_PASSES
    if whole_field:
        desc = LrDonn.from_buffer_copy(desc)
        desc.flags |= LR_WHOLE_FIELD
    if sums and net.detector.num > 0 and out_sums is None:
        out_sums = torch.empty((b, net.detector.num), dtype=torch.float32, device=dev)
    if intensity and out_intensity is None:
        out_intensity = torch.empty((b, n, n), dtype=torch.float32, device=dev)
    if field and out_field is None:
        out_field = torch.empty((b, n, n), dtype=torch.complex64, device=dev)
    w = net.workspace(b, LR_OP_FORWARD)
    if saved is not None and saved.numel() < net.saved_size(b):
        raise ValueError("saved buffer too small")
    k = net.detector.num
    _check(load().lr_donn_forward(
        ctypes.byref(desc), b,
        _ptr(amp, torch.float32, (b, n, n), "amp"), _ptr(phi, torch.float32, (L, n, n), "phi"),
        _ptr(saved, torch.uint8, None, "saved"),
        _ptr(out_sums, torch.float32, (b, k), "sums"), _ptr(out_intensity, torch.float32, (b, n, n), "intensity"),
        _ptr(out_field, torch.complex64, (b, n, n), "field"),
        _ptr(w), w.numel(), _stream(dev)), "lr_donn_forward")
    return {"sums": out_sums, "intensity": out_intensity, "field": out_field, "saved": saved}


def lr_donn_backward(net: Network, phi, saved, sums=None, labels=None, grad_sums=None, grad_intensity=None,
                     out_grad_phi=None, want_loss: bool = True, skip=None):
    """dL/dphi [L, n, n] (and the loss when labels are given); skip as given
    to lr_donn_forward."""
    torch = _torch()
    n, L = net.n, net.num_layers
    dev = net.device
    seed = next(t for t in (labels, grad_sums, grad_intensity) if t is not None)
    b = int(seed.shape[0])
    if out_grad_phi is None:
        out_grad_phi = torch.empty((L, n, n), dtype=torch.float32, device=dev)
    loss = torch.empty((), dtype=torch.float32, device=dev) if (labels is not None and want_loss) else None
    if saved is None or saved.numel() < net.saved_size(b):
        raise ValueError("saved buffer missing or smaller than the forward pass of this batch fills")
    k = net.detector.num
    w = net.workspace(b, LR_OP_BACKWARD)
    desc = _with_skip(net.c, skip, b, n)
    _check(load().lr_donn_backward(
        ctypes.byref(desc), b, _ptr(phi, torch.float32, (L, n, n), "phi"), _ptr(saved, torch.uint8, None, "saved"),
        _ptr(sums, torch.float32, (b, k), "sums"), _ptr(labels, torch.int32, (b,), "labels"),
        _ptr(grad_sums, torch.float32, (b, k), "grad_sums"),
        _ptr(grad_intensity, torch.float32, (b, n, n), "grad_intensity"),
        _ptr(loss, torch.float32, None, "loss"), _ptr(out_grad_phi, torch.float32, (L, n, n), "grad_phi"),
        _ptr(w), w.numel(), _stream(dev)), "lr_donn_backward")
    return out_grad_phi, loss


def lr_loss(sums, labels, kind: int = LR_LOSS_SOFTMAX_CE, out_grad_sums=None, want_loss: bool = True):
    """Loss of detector sums [B, K] with int32 labels [B] (batch mean) and dL/dS [B, K]."""
    torch = _torch()
    b, k = int(sums.shape[0]), int(sums.shape[1])
    if out_grad_sums is None:
        out_grad_sums = torch.empty((b, k), dtype=torch.float32, device=sums.device)
    loss = torch.empty((), dtype=torch.float32, device=sums.device) if want_loss else None
    _check(load().lr_loss(int(kind), _ptr(sums, torch.float32, (b, k), "sums"),
                          _ptr(labels, torch.int32, (b,), "labels"), b, k, _ptr(loss, torch.float32, None, "loss"),
                          _ptr(out_grad_sums, torch.float32, (b, k), "grad_sums"), _stream(sums.device)), "lr_loss")
    return loss, out_grad_sums


def lr_adam_update(phi, grad, m, v, step: int, lr: float = 0.5, beta1: float = 0.9, beta2: float = 0.999,
                   eps: float = 1e-8):
    """One in-place Adam step on phi (and its moments m, v), all float32 of one shape."""
    torch = _torch()
    shape = tuple(phi.shape)
    count = int(phi.numel())
    _check(load().lr_adam_update(_ptr(phi, torch.float32, shape, "phi"), _ptr(grad, torch.float32, shape, "grad"),
                                 _ptr(m, torch.float32, shape, "m"), _ptr(v, torch.float32, shape, "v"), count,
                                 int(step), float(lr), float(beta1), float(beta2), float(eps),
                                 _stream(phi.device)), "lr_adam_update")
    return phi


def _ln_workspace(batch: int, count: int, device):
    torch = _torch()
    r = load().lr_layer_norm_workspace_size(int(batch), int(count))
    if r < 0:
        raise LrError(int(-r), "lr_layer_norm_workspace_size")
    return torch.empty(max(int(r), 1), dtype=torch.uint8, device=device)


def lr_layer_norm(x, eps: float = 1e-5, out=None, out_stats=None):
    """Per-sample layer normalisation of maps x [B, ...] (float32): returns
    (normalised maps, stats [B, 2] = (mean, 1/sqrt(var + eps)))."""
    torch = _torch()
    b = int(x.shape[0])
    shape = tuple(x.shape)
    count = int(x.numel()) // max(b, 1)
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=x.device)
    if out_stats is None:
        out_stats = torch.empty((b, 2), dtype=torch.float32, device=x.device)
    w = _ln_workspace(b, count, x.device)
    _check(load().lr_layer_norm(_ptr(x, torch.float32, shape, "x"), b, count, float(eps),
                                _ptr(out, torch.float32, shape, "y"), _ptr(out_stats, torch.float32, (b, 2), "stats"),
                                _ptr(w), w.numel(), _stream(x.device)), "lr_layer_norm")
    return out, out_stats


def lr_layer_norm_backward(grad_y, y, stats, out=None):
    """dL/dx [B, ...] from dL/dy, the normalised maps y and their stats."""
    torch = _torch()
    b = int(y.shape[0])
    shape = tuple(y.shape)
    count = int(y.numel()) // max(b, 1)
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=y.device)
    w = _ln_workspace(b, count, y.device)
    _check(load().lr_layer_norm_backward(_ptr(grad_y, torch.float32, shape, "grad_y"), _ptr(y, torch.float32, shape, "y"),
                                         _ptr(stats, torch.float32, (b, 2), "stats"), b, count,
                                         _ptr(out, torch.float32, shape, "grad_x"), _ptr(w), w.numel(),
                                         _stream(y.device)), "lr_layer_norm_backward")
    return out


def kernel_timing(enable: bool) -> None:
    _check(load().lr_kernel_timing(1 if enable else 0), "lr_kernel_timing")


def kernel_timing_report() -> dict:
    import json
    lib = load()
    need = lib.lr_kernel_timing_report(None, 0)
    if need < 0:
        raise LrError(-need, "lr_kernel_timing_report")
    buf = ctypes.create_string_buffer(need + 1)
    lib.lr_kernel_timing_report(buf, need + 1)
    return json.loads(buf.value.decode())


def lr_codesign_phase(logits, noise, levels, tau: float, hard: bool = False, out=None):
    """Phase masks [...] from scores and Gumbel draws [..., K] over the device's
    phase levels [K] (soft sum or, with hard, the chosen level)."""
    torch = _torch()
    shape = tuple(logits.shape)
    k = int(shape[-1])
    count = int(logits.numel()) // max(k, 1)
    if out is None:
        out = torch.empty(shape[:-1], dtype=torch.float32, device=logits.device)
    _check(load().lr_codesign_phase(_ptr(logits, torch.float32, shape, "logits"), _ptr(noise, torch.float32, shape, "noise"),
                                    _ptr(levels, torch.float32, (k,), "levels"), k, count, float(tau),
                                    1 if hard else 0, _ptr(out, torch.float32, shape[:-1], "phi"),
                                    _stream(logits.device)), "lr_codesign_phase")
    return out


def lr_codesign_backward(logits, noise, levels, tau: float, grad_phi, out=None):
    """dL/dlogits [..., K] from dL/dphi [...]."""
    torch = _torch()
    shape = tuple(logits.shape)
    k = int(shape[-1])
    count = int(logits.numel()) // max(k, 1)
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=logits.device)
    _check(load().lr_codesign_backward(_ptr(logits, torch.float32, shape, "logits"),
                                       _ptr(noise, torch.float32, shape, "noise"),
                                       _ptr(levels, torch.float32, (k,), "levels"), k, count, float(tau),
                                       _ptr(grad_phi, torch.float32, shape[:-1], "grad_phi"),
                                       _ptr(out, torch.float32, shape, "grad_logits"), _stream(logits.device)),
           "lr_codesign_backward")
    return out


def multichannel_train_step(nets, amps, phis, saveds, labels, kind: int = LR_LOSS_SOFTMAX_CE):
    """One training step of the multi-channel DONN of §5.6.1 through the C ABI.

    Channel c (its own lr_donn, masks phis[c] and input amps[c]) runs its
    forward pass; the detector sums of all channels add into one merged
    array (LR_ACCUMULATE from the second channel on), the loss is taken on
    the merged sums, and every channel's backward pass receives the same
    dL/dS.  Returns (loss, merged sums, [dL/dphi of each channel])."""
    merged = None
    for c, (net, amp, phi, saved) in enumerate(zip(nets, amps, phis, saveds)):
        merged = lr_donn_forward(net, amp, phi, saved=saved, sums=True, out_sums=merged, accumulate=c > 0)["sums"]
    loss, grad_sums = lr_loss(merged, labels, kind=kind)
    grads = [lr_donn_backward(net, phi, saved, grad_sums=grad_sums)[0]
             for net, phi, saved in zip(nets, phis, saveds)]
    return loss, merged, grads
