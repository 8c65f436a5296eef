"""Seeded synthetic workloads shared by the tests, the benchmark and the oracle checks.

This module holds no diffraction arithmetic: it only names the five workload
shapes and draws their random inputs (amplitudes, phase masks, labels,
upstream gradients) with numpy, in float64, cast once to float32.  The
oracle and the HIP library receive the very same arrays.

Every stream is ``np.random.default_rng([230611268, workload_id, stream])``
with stream 0 = input amplitudes, 1 = phase masks, 2 = labels, 3 = upstream
intensity gradient, 4 = device levels, 5 = codesign scores, 6 = Gumbel draws.  Samples are drawn one after another, so the first B'
samples of a batch of B are the batch of B'.

The paper's datasets (MNIST-style digits, CityScapes scenes) are not
available; the stroke and shape generators below stand in for them with the
sizes and value ranges the paper describes (28 x 28 digits extended to the
200 x 200 system, §5.2; binary segmentation targets, §5.6.2).
"""

from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

import numpy as np

SEED = 230611268
FRESNEL = 0
ANGULAR_SPECTRUM = 1


@dataclasses.dataclass(frozen=True)
class DetectorLayout:
    size: int
    y0: Tuple[int, ...]
    x0: Tuple[int, ...]

    @property
    def num(self) -> int:
        return len(self.y0)


# Ten 20 x 20 regions on a 200 x 200 plane in rows of 4, 3 and 3, centred
# about the plane centre and pairwise disjoint (the prototype's "ten regions
# placed evenly", §5.1).
TEN_CLASS_LAYOUT_200 = DetectorLayout(
    size=20,
    y0=(50, 50, 50, 50, 90, 90, 90, 130, 130, 130),
    x0=(30, 70, 110, 150, 50, 90, 130, 50, 90, 130),
)


@dataclasses.dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    wavelength: float
    pixel_pitch: float
    distance: float
    approx: int
    n: int
    n_fft: int
    layers: int
    batch: int
    kind: str                 # "propagate", "forward", "train"
    detector: Optional[DetectorLayout]
    output: str               # "field+intensity", "sums", "intensity"
    input_kind: str           # "uniform", "strokes", "blobs", "shapes"
    grad: Optional[str] = None  # "ce" or "intensity" for training workloads


WORKLOADS = {
    1: Workload(1, "fresnel_n64_b4_single_hop", 532e-9, 36e-6, 0.3, FRESNEL, 64, 64, 1, 4,
                "forward", None, "field+intensity", "uniform"),
    2: Workload(2, "donn5_n200_b256_forward", 532e-9, 36e-6, 0.3, FRESNEL, 200, 200, 5, 256,
                "forward", TEN_CLASS_LAYOUT_200, "sums", "strokes"),
    3: Workload(3, "donn5_n200_b500_train", 532e-9, 36e-6, 0.3, FRESNEL, 200, 200, 5, 500,
                "train", TEN_CLASS_LAYOUT_200, "sums", "strokes", grad="ce"),
    4: Workload(4, "donn10_as_n512_fft1024_b64_forward", 1550e-9, 8e-6, 0.05, ANGULAR_SPECTRUM,
                512, 1024, 10, 64, "forward", None, "intensity", "blobs"),
    5: Workload(5, "donn3_n1000_b16_train_fullmap", 532e-9, 36e-6, 0.5, FRESNEL, 1000, 1000, 3, 16,
                "train", None, "intensity", "shapes", grad="intensity"),
}


def rng(wid: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([SEED, wid, stream])


# ---------------------------------------------------------------------------
# Input amplitude generators (stream 0)
# ---------------------------------------------------------------------------

def _segment_distance(py, px, y0, x0, y1, x1):
    """Distance from pixel centres (py, px) to the segment (y0,x0)-(y1,x1)."""
    dy, dx = y1 - y0, x1 - x0
    ll = dy * dy + dx * dx
    if ll <= 0.0:
        return np.hypot(py - y0, px - x0)
    t = np.clip(((py - y0) * dy + (px - x0) * dx) / ll, 0.0, 1.0)
    return np.hypot(py - (y0 + t * dy), px - (x0 + t * dx))


def stroke_image(g: np.random.Generator) -> np.ndarray:
    """One 28 x 28 grey image of 3-6 random anti-aliased line segments in [0, 1]."""
    c = np.arange(28, dtype=np.float64) + 0.5
    py, px = np.meshgrid(c, c, indexing="ij")
    img = np.zeros((28, 28))
    for _ in range(int(g.integers(3, 7))):
        y0, x0, y1, x1 = g.uniform(2.0, 26.0, size=4)
        thick = g.uniform(1.0, 2.0)
        val = g.uniform(0.5, 1.0)
        d = _segment_distance(py, px, y0, x0, y1, x1)
        img = np.maximum(img, val * np.clip(thick / 2.0 + 0.5 - d, 0.0, 1.0))
    return np.clip(img, 0.0, 1.0)


def stroke_scale(n: int) -> int:
    """Nearest-upsampling factor of the 28 x 28 strokes on an n x n plane: the
    image spans about 70 % of the plane (x5, 140 px, at n = 200)."""
    return max(1, (7 * n) // 280)


def strokes_batch(wid: int, batch: int, n: int = 200) -> np.ndarray:
    """Stroke digits upsampled (nearest, x stroke_scale(n); x5 to 140 x 140 at
    n = 200), centred in n x n."""
    g = rng(wid, 0)
    f = stroke_scale(n)
    s = 28 * f
    out = np.zeros((batch, n, n))
    o = (n - s) // 2
    block = np.ones((f, f))
    for b in range(batch):
        out[b, o:o + s, o:o + s] = np.kron(stroke_image(g), block)
    return out.astype(np.float32)


def blobs_batch(wid: int, batch: int, n: int) -> np.ndarray:
    """1-4 Gaussian blobs (sigma 10-40 px, peak 0.5-1) per sample, not clipped."""
    g = rng(wid, 0)
    c = np.arange(n, dtype=np.float64)
    yy, xx = np.meshgrid(c, c, indexing="ij")
    out = np.zeros((batch, n, n))
    for b in range(batch):
        for _ in range(int(g.integers(1, 5))):
            sigma = g.uniform(10.0, 40.0)
            cy, cx = g.uniform(sigma, n - sigma, size=2)
            a = g.uniform(0.5, 1.0)
            out[b] += a * np.exp(-((yy - cy) ** 2 + (xx - cx) ** 2) / (2.0 * sigma * sigma))
    return out.astype(np.float32)


def shapes_batch(wid: int, batch: int, n: int) -> np.ndarray:
    """Union of 2-5 random ellipses / axis-aligned rectangles, values in {0, 1}."""
    g = rng(wid, 0)
    c = np.arange(n, dtype=np.float64)
    yy, xx = np.meshgrid(c, c, indexing="ij")
    lo, hi = 0.1 * n, 0.9 * n
    out = np.zeros((batch, n, n), dtype=bool)
    for b in range(batch):
        for _ in range(int(g.integers(2, 6))):
            ellipse = g.uniform() < 0.5
            cy, cx = g.uniform(lo, hi, size=2)
            ry, rx = g.uniform(0.03 * n, 0.2 * n, size=2)
            if ellipse:
                m = ((yy - cy) / ry) ** 2 + ((xx - cx) / rx) ** 2 <= 1.0
            else:
                m = (np.abs(yy - cy) <= ry) & (np.abs(xx - cx) <= rx)
            out[b] |= m
    return out.astype(np.float32)


def uniform_batch(wid: int, batch: int, n: int) -> np.ndarray:
    return rng(wid, 0).uniform(0.0, 1.0, size=(batch, n, n)).astype(np.float32)


def amplitudes(w: Workload, batch: Optional[int] = None) -> np.ndarray:
    b = w.batch if batch is None else batch
    if w.input_kind == "uniform":
        return uniform_batch(w.wid, b, w.n)
    if w.input_kind == "strokes":
        return strokes_batch(w.wid, b, w.n)
    if w.input_kind == "blobs":
        return blobs_batch(w.wid, b, w.n)
    if w.input_kind == "shapes":
        return shapes_batch(w.wid, b, w.n)
    raise ValueError(w.input_kind)


def phases(w: Workload) -> np.ndarray:
    """Phase masks phi ~ U[0, 2*pi), float32 [L, n, n] (stream 1)."""
    return rng(w.wid, 1).uniform(0.0, 2.0 * np.pi, size=(w.layers, w.n, w.n)).astype(np.float32)


def labels(w: Workload, batch: Optional[int] = None, classes: int = 10) -> np.ndarray:
    """Class labels, int32 [B] (stream 2)."""
    b = w.batch if batch is None else batch
    g = rng(w.wid, 2)
    return np.array([g.integers(0, classes) for _ in range(b)], dtype=np.int32)


def upstream_intensity_grad(w: Workload, batch: Optional[int] = None) -> np.ndarray:
    """dL/dI ~ N(0, 1), float32 [B, n, n] (stream 3)."""
    b = w.batch if batch is None else batch
    g = rng(w.wid, 3)
    return np.stack([g.standard_normal((w.n, w.n)) for _ in range(b)]).astype(np.float32)


def ten_class_layout(n: int) -> DetectorLayout:
    """The ten-region layout of the 200 x 200 prototype scaled to an n x n plane."""
    if n == 200:
        return TEN_CLASS_LAYOUT_200
    f = n / 200.0
    t = TEN_CLASS_LAYOUT_200
    return DetectorLayout(max(1, int(round(t.size * f))), tuple(int(round(v * f)) for v in t.y0),
                          tuple(int(round(v * f)) for v in t.x0))


def scaled(w: Workload, n: Optional[int] = None, layers: Optional[int] = None) -> Workload:
    """Workload w on an unpadded n x n grid with `layers` layers: the depth and
    size variants of the paper's runtime study (§5.3: {1, 3, 5, 7, 10} layers
    on grids up to 500 x 500, and deeper networks).  The random streams stay
    those of w, so a variant with w's own n and depth is w itself."""
    n = w.n if n is None else int(n)
    layers = w.layers if layers is None else int(layers)
    if n == w.n and layers == w.layers:
        return w
    det = ten_class_layout(n) if w.detector is not None else None
    name = f"donn{layers}_n{n}_b{w.batch}_{w.kind}"
    return dataclasses.replace(w, name=name, n=n, n_fft=n, layers=layers, detector=det)


def layout_grid(n: int, num: int, size: int) -> DetectorLayout:
    """A simple layout of ``num`` disjoint size x size regions spread on an n x n plane."""
    cols = int(np.ceil(np.sqrt(num)))
    rows = int(np.ceil(num / cols))
    if rows * size > n or cols * size > n:
        raise ValueError("regions do not fit")
    gy = (n - rows * size) // (rows + 1)
    gx = (n - cols * size) // (cols + 1)
    y0, x0 = [], []
    for k in range(num):
        r, c = divmod(k, cols)
        y0.append(gy + r * (size + gy))
        x0.append(gx + c * (size + gx))
    return DetectorLayout(size, tuple(y0), tuple(x0))


# ---------------------------------------------------------------------------
# Codesign layer inputs (§3.2): a device's discrete phase responses, per-pixel
# scores over them and the Gumbel draws of one training step.  No measured
# device vector is available; the synthetic one has the paper's 256 states
# covering [0, 2*pi) with a smooth non-linear (SLM-like) response curve.
# ---------------------------------------------------------------------------

def device_levels(wid: int, levels: int = 256) -> np.ndarray:
    """Monotone phase responses in [0, 2*pi), float32 [levels] (stream 4)."""
    g = rng(wid, 4)
    x = (np.arange(levels, dtype=np.float64) + g.uniform(0.0, 0.3, levels)) / levels
    return np.sort(2.0 * np.pi * x ** 1.3).astype(np.float32)


def codesign_scores(wid: int, shape, levels: int) -> np.ndarray:
    """Per-pixel scores ~ N(0, 1), float32 [*shape, levels] (stream 5)."""
    return rng(wid, 5).standard_normal(tuple(shape) + (levels,)).astype(np.float32)


def gumbel_draws(wid: int, shape, levels: int) -> np.ndarray:
    """Gumbel(0, 1) draws -log(-log U), float32 [*shape, levels] (stream 6)."""
    u = rng(wid, 6).uniform(1e-12, 1.0, tuple(shape) + (levels,))
    return (-np.log(-np.log(u))).astype(np.float32)
