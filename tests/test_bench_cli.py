"""Host-side checks of bench.py: the one-GPU guard, the algorithmic byte
counts behind `roofline.achieved`, and the traffic lookup that reports
counter bytes only for the device sources they were measured on."""

import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    doc = json.loads(r.stdout.strip().splitlines()[-1])
    assert doc["n_gpus"] == 2 and "one GPU" in doc["error"]


def test_algorithmic_bytes_per_sample():
    # one field read and one written (complex64) forward; gradient read, saved field read,
    # gradient written backward
    assert bench.algorithmic_bytes_per_sample("fwd_mid", 200) == 16 * 200 * 200
    assert bench.algorithmic_bytes_per_sample("bwd_mid", 200) == 24 * 200 * 200


def test_traffic_reported_only_for_matching_sources(tmp_path, monkeypatch):
    from paper_2306_11268_amd import build as lb

    prof = tmp_path / "profiles"
    prof.mkdir()
    name = "wl"
    doc = {"source_digest": lb.source_digest(), "kernels": {"k": {"hbm_bytes_per_dispatch": 123}}}
    (prof / f"fresnel_passes__{name}__traffic.json").write_text(json.dumps(doc))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.recorded_traffic(name, "k") == 123
    assert bench.recorded_traffic(name, "other") is None
    doc["source_digest"] = "0" * 16
    (prof / f"fresnel_passes__{name}__traffic.json").write_text(json.dumps(doc))
    assert bench.recorded_traffic(name, "k") is None


def test_valu_counts_reported_only_for_matching_sources(tmp_path, monkeypatch):
    from paper_2306_11268_amd import build as lb

    prof = tmp_path / "profiles"
    prof.mkdir()
    name = "wl"
    doc = {"source_digest": lb.source_digest(), "kernels": {"k": {"valu_instr_per_dispatch": 4.5e7}}}
    (prof / f"fresnel_passes__{name}__valu.json").write_text(json.dumps(doc))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.recorded_valu(name, "k") == 4.5e7
    assert bench.recorded_valu(name, "other") is None
    doc["source_digest"] = "0" * 16
    (prof / f"fresnel_passes__{name}__valu.json").write_text(json.dumps(doc))
    assert bench.recorded_valu(name, "k") is None
    # 1024 SIMDs, one wave64 instruction per 4 cycles at 2.4 GHz
    assert bench.VALU_PEAK_WAVE_INSTR_PER_S == 614.4e9


def test_step_byte_models():
    """Per-sample step bytes: the method's one-pass bound (40 L - 10.4) n^2 at
    the 4-3-3 layout, and this path's passes counted by hand for L = 5 at
    200 x 200 with 60 covered rows."""
    from paper_2306_11268_amd import workloads as wl

    w = wl.WORKLOADS[3]

    class Det:
        num = len(w.detector.y0)
        size = w.detector.size
        y0 = w.detector.y0
        x0 = w.detector.x0

    one_pass, path = bench.step_bytes_per_sample(w, Det)
    nn = 200 * 200
    assert abs(one_pass - 189.6 * nn) < 1e-6 * nn
    # prop 12, five forward layers 80, detector read 2.4, seed 4.8, layer 5 adjoint 2.4 + 16,
    # layers 4..2 adjoint 72, layer 1 adjoint 16 (units of n^2)
    assert abs(path - (12 + 80 + 2.4 + 4.8 + 18.4 + 72 + 16) * nn) < 1e-6 * nn


def test_source_digest_ignores_comments_but_not_code():
    from paper_2306_11268_amd import build as lb

    base = 'int f(int x) { return x + 1; }  // add one\n/* note */ const char* s = "a // b";'
    assert lb._code_only(base) == lb._code_only(base.replace("add one", "increment").replace("note", "n"))
    assert lb._code_only(base) != lb._code_only(base.replace("x + 1", "x + 2"))
    assert lb._code_only(base) != lb._code_only(base.replace('"a // b"', '"a // c"'))
