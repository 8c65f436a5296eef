"""The synthetic workloads carry the paper's stated parameters and are reproducible."""

import json
import os

import numpy as np

from paper_2306_11268_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_parameters.json")


def test_n200_workloads_match_paper_parameters():
    p = json.load(open(GOLDEN))
    for wid in (2, 3):
        w = wl.WORKLOADS[wid]
        assert w.wavelength == p["prototype"]["wavelength_m"]
        assert w.pixel_pitch == p["prototype"]["pixel_pitch_m"]
        assert w.distance == p["artifact_defaults"]["distance_m"]
        assert w.n == p["prototype"]["system_size"]
        assert w.layers == p["artifact_defaults"]["num_layers"]
        assert w.detector.num == p["prototype"]["detector_regions"]
    assert wl.WORKLOADS[3].batch == p["prototype"]["batch"]


def test_ten_class_layout_disjoint_inside_and_centred():
    d = wl.TEN_CLASS_LAYOUT_200
    occ = np.zeros((200, 200), int)
    for y, x in zip(d.y0, d.x0):
        occ[y:y + d.size, x:x + d.size] += 1
    assert occ.max() == 1 and occ.sum() == 10 * d.size ** 2
    rows = sorted(set(d.y0))
    assert [y + d.size / 2 for y in rows] == [60, 100, 140]       # rows symmetric about y = 100
    for r in rows:
        xs = [x + d.size / 2 for x, y in zip(d.x0, d.y0) if y == r]
        assert abs(np.mean(xs) - 100) < 1e-9                       # each row centred on x = 100


def test_generators_are_seeded_and_prefix_stable():
    w = wl.WORKLOADS[3]
    a = wl.amplitudes(w, batch=6)
    b = wl.amplitudes(w, batch=3)
    assert a.dtype == np.float32 and a.shape == (6, 200, 200)
    np.testing.assert_array_equal(a[:3], b)
    assert a.min() >= 0 and a.max() <= 1
    assert np.all(a[:, :30, :] == 0) and np.all(a[:, :, 170:] == 0)
    np.testing.assert_array_equal(wl.labels(w, 7)[:4], wl.labels(w, 4))
    p = wl.phases(w)
    assert p.shape == (5, 200, 200) and p.min() >= 0 and p.max() < 2 * np.pi


def test_other_generators_shapes_and_ranges():
    s = wl.amplitudes(wl.WORKLOADS[5], batch=2)
    assert s.shape == (2, 1000, 1000) and set(np.unique(s)) <= {0.0, 1.0} and s.sum() > 0
    bl = wl.amplitudes(wl.WORKLOADS[4], batch=2)
    assert bl.shape == (2, 512, 512) and bl.min() >= 0 and bl.max() > 0.4
    g = wl.upstream_intensity_grad(wl.WORKLOADS[5], batch=2)
    assert g.shape == (2, 1000, 1000) and abs(float(g.mean())) < 0.01


def test_scaled_variants():
    w = wl.WORKLOADS[3]
    assert wl.scaled(w) is w and wl.scaled(w, n=200, layers=5) is w
    v = wl.scaled(w, n=500, layers=30)
    assert (v.n, v.n_fft, v.layers, v.batch, v.wid) == (500, 500, 30, w.batch, w.wid)
    d = v.detector
    assert d.num == 10 and d.size == 50
    for y0, x0 in zip(d.y0, d.x0):
        assert 0 <= y0 and y0 + d.size <= 500 and 0 <= x0 and x0 + d.size <= 500
    # the regions stay pairwise disjoint when scaled
    boxes = list(zip(d.y0, d.x0))
    for i in range(len(boxes)):
        for k in range(i + 1, len(boxes)):
            (ya, xa), (yb, xb) = boxes[i], boxes[k]
            assert abs(ya - yb) >= d.size or abs(xa - xb) >= d.size
    a = wl.amplitudes(v, 2)
    assert a.shape == (2, 500, 500) and a.min() >= 0.0 and a.max() <= 1.0
    f = wl.stroke_scale(500)
    o = (500 - 28 * f) // 2
    assert np.all(a[:, :o, :] == 0) and np.all(a[:, :, :o] == 0)
