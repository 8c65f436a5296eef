#!/usr/bin/env python3
"""Benchmark of the DONN physics kernel on one MI355X.

One step = one training step of the 5-layer, 200 x 200 Fresnel DONN on a
batch of 500 synthetic stroke images: forward pass (saving activations),
softmax cross-entropy over the ten detector sums, adjoint backward pass to
dL/dphi for all five masks.  Inputs are resident in HBM before timing.

Prints one JSON line.  `value` is samples per second over exactly --steps
steps bracketed by device synchronisation (with --graph the step is recorded
once as a HIP graph and the timed steps replay it).  The defaults (100 timed
steps after 20 warm-up steps, about 0.15 s of GPU time at the headline size)
measure the steady state: over 20 steps after 5 the first steps' clock ramp
costs about 3%.  The per-kernel durations used for the roofline come
from HIP events recorded around every kernel launch on the launch stream
during a second, instrumented run of the same steps.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", type=int, default=3,
                    help="workload id (3 = 5-layer N=200 train, batch 500, the headline line; 1, 2, 4 and 5 print "
                         "a timing line of their own)")
    ap.add_argument("--batch", type=int, default=None, help="override the batch size")
    ap.add_argument("--n", type=int, default=None,
                    help="grid size of a runtime-study variant of the workload (unpadded n x n)")
    ap.add_argument("--layers", type=int, default=None, help="depth of a runtime-study variant")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--layer-passes", action="store_true",
                    help="one pass per layer in the forward call even where the whole-field kernel applies "
                         "(Fresnel, n = n_fft in 64, 100, 128)")
    ap.add_argument("--whole-field", action="store_true",
                    help="the whole-field forward kernel wherever it applies, also at n = n_fft = 200 where the "
                         "layer passes are the default")
    ap.add_argument("--graph", action="store_true",
                    help="record the step once as a HIP graph and time its replays (measured slower than "
                         "launching the kernels one by one on this stack, so not the default)")
    ap.add_argument("--cpu-samples", type=int, default=None, help="samples in the oracle timing run")
    ap.add_argument("--copy-calibration", type=int, default=None, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB three times (the reference "
                         "kernel whose FETCH_SIZE / WRITE_SIZE counters calibrate HBM traffic)")
    return ap.parse_args()


def copy_calibration(mib: int):
    import torch

    nbytes = mib * 1024 * 1024
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "copies": 3}))


def recorded_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` from the committed counter summary of
    this workload, or None when there is none or the device sources have
    changed since the counters were taken."""
    from paper_2306_11268_amd.build import source_digest

    path = os.path.join(ROOT, "profiles", f"fresnel_passes__{workload}__traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        doc = json.load(fh)
    if doc.get("source_digest") != source_digest() or kernel not in doc.get("kernels", {}):
        return None
    return doc["kernels"][kernel]["hbm_bytes_per_dispatch"]


# Vector-ALU issue ceiling of the chip without packed FP32 instructions: 256
# CUs x 4 SIMDs, one wave64 FP32 instruction per SIMD every 4 cycles (16
# lanes per cycle) at the 2.4 GHz peak engine clock, in wave instructions/s.
VALU_PEAK_WAVE_INSTR_PER_S = 256 * 4 * 2.4e9 / 4


def recorded_valu(workload: str, kernel: str):
    """Wave-level VALU instructions per launch of `kernel` (SQ_INSTS_VALU) from
    the committed counter summary of this workload, or None when there is none
    or the device sources have changed since the counters were taken."""
    from paper_2306_11268_amd.build import source_digest

    path = os.path.join(ROOT, "profiles", f"fresnel_passes__{workload}__valu.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        doc = json.load(fh)
    if doc.get("source_digest") != source_digest() or kernel not in doc.get("kernels", {}):
        return None
    return doc["kernels"][kernel]["valu_instr_per_dispatch"]


def algorithmic_bytes_per_sample(kind: str, n: int) -> float:
    """Bytes one sample must move through HBM in one launch of each kernel kind.

    Per layer the method reads the incoming field and writes the modulated
    field (forward, 16 n^2 bytes of complex64), and reads the adjoint field and
    the saved activation and writes the adjoint field (backward, 24 n^2).
    Tables (chirps, modulation) are shared by the batch and not counted.
    """
    nn = n * n
    return {
        "fwd_mid": 16.0 * nn,
        "bwd_mid": 24.0 * nn,
    }[kind]


def step_bytes_per_sample(w, det):
    """HBM bytes one sample moves in one training step (complex64 fields, n x n).

    One-pass bound of the method (a field crosses HBM once in and once out per
    layer, the detector plane restricted to the region rows): forward
    (16 L + 4) n^2 and backward (24 L - 14.4) n^2 at the 4-3-3 layout,
    (40 L - 10.4) n^2 together (L = 5: 189.6 n^2).

    This path's passes: the first reads the amplitude and writes W_0 (12 n^2);
    each forward layer pass reads W_{l-1} and writes W_l (16 n^2); the
    detector-plane passes read (forward) and read and write (backward) the c
    vectors the regions cover along their axis (8 c n and 16 c n); the
    adjoint layer passes read G and W_{l-1} and write G (24 n^2; for layer L
    G only on the c covered vectors when the seed pass ran along rows), and
    layer 1 reads G and W_0 (16 n^2)."""
    n, L = w.n, w.layers
    nn = n * n
    one_pass = (40.0 * L - 10.4) * nn
    detector_rows = (L + 2) % 2 == 1  # the detector-plane pass runs along rows
    covered = set()
    for k in range(det.num):
        lo = det.y0[k] if detector_rows else det.x0[k]
        covered.update(range(lo, lo + det.size))
    c = len(covered)
    g_last = 8.0 * c * n if detector_rows else 8.0 * nn
    path = 12.0 * nn + 16.0 * L * nn + 8.0 * c * n + 16.0 * c * n
    path += (g_last + 16.0 * nn) + 24.0 * nn * max(L - 2, 0) + 16.0 * nn
    return one_pass, path


def oracle_baseline(w, batch, amp, phi, labels, min_seconds=10.0):
    """Time the float64 oracle on the host: forward, loss and backward."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import oracle.donn as od

    h = od.transfer_function(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n_fft)
    det = od.Detector(w.detector.size, tuple(w.detector.y0), tuple(w.detector.x0))

    def one_pass(b):
        fwd = od.donn_forward(amp[:b], phi, h, 1.0, det)
        _, gs = od.softmax_cross_entropy(fwd["sums"], labels[:b])
        od.donn_backward(fwd, phi, h, 1.0, det, grad_sums=gs)

    # a one-sample probe sizes the sample so that a pass takes at most about
    # min_seconds; then whole passes until at least min_seconds have passed
    # (under 2 * min_seconds in all, since one pass takes at most about that)
    tp = time.perf_counter()
    one_pass(1)
    t1 = time.perf_counter() - tp
    batch = max(1, min(batch, int(min_seconds / max(t1, 1e-6))))
    passes = 0
    t0 = time.perf_counter()
    while True:
        one_pass(batch)
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = max([i.get("num_threads", 1) for i in blas] or [1])
    vendor = ", ".join(sorted({f"{i.get('internal_api', '?')} {i.get('version', '')}".strip() for i in blas})) or "none"
    return {"value": passes * batch / dt, "unit": "samples/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{passes} pass(es) over {batch} samples of the same workload (forward + cross-entropy "
                      f"+ backward), {dt:.1f} s on the host, numpy float64 naive DFT",
            "seconds": round(dt, 3), "blas_threads": int(threads), "blas": vendor,
            "host_cpus": len(os.sched_getaffinity(0))}


def other_workload(w, batch, args):
    """Time one of the other workloads (not the headline line): a forward pass
    with region sums or the intensity map, or a training step with an
    upstream intensity gradient; per-kernel averages from HIP events."""
    import torch

    from paper_2306_11268_amd import binding as lb
    from paper_2306_11268_amd import workloads as wl

    det = lb.Detector(w.detector.size, w.detector.y0, w.detector.x0) if w.detector is not None else None
    net = lb.Network(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n, w.n_fft, w.layers, 1.0, det)
    amp = torch.from_numpy(wl.amplitudes(w, batch)).cuda()
    phi = torch.from_numpy(wl.phases(w)).cuda()
    train = w.kind == "train"
    saved = net.new_saved(batch) if train else None
    gi = torch.from_numpy(wl.upstream_intensity_grad(w, batch)).cuda() if train else None

    def step():
        if det is not None and not train:
            lb.lr_donn_forward(net, amp, phi, sums=True, layer_passes=args.layer_passes,
                               whole_field=args.whole_field)
        else:
            lb.lr_donn_forward(net, amp, phi, saved=saved, sums=False, intensity=True)
        if train:
            lb.lr_donn_backward(net, phi, saved, grad_intensity=gi)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = ev0.elapsed_time(ev1) / args.steps
    lb.kernel_timing(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    kt = lb.kernel_timing_report()
    lb.kernel_timing(False)
    print(json.dumps({
        "metric": f"{w.name} samples/sec (not the headline workload)",
        "value": round(batch / (ms_per_step / 1e3), 1),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "n": w.n, "n_fft": w.n_fft, "layers": w.layers, "batch": batch,
                   "approx": "fresnel" if w.approx == 0 else "angular_spectrum", "kind": w.kind,
                   "layer_passes": bool(args.layer_passes), "whole_field": bool(args.whole_field)},
        "kernels": {k: {"count": v["count"], "avg_us": 1e3 * v["ms"] / v["count"], "total_ms": v["ms"]}
                    for k, v in kt.items()},
    }))


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py measures one GPU only; the batch-sharded design for more "
                                   "GPUs is documented but not launched", "n_gpus": args.gpus}))
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2306_11268_amd import binding as lb
    from paper_2306_11268_amd import workloads as wl

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    if args.copy_calibration is not None:
        copy_calibration(args.copy_calibration)
        return
    lb.load()
    w = wl.scaled(wl.WORKLOADS[args.workload], n=args.n, layers=args.layers)
    batch = w.batch if args.batch is None else args.batch
    if w.kind != "train" or w.grad != "ce":
        other_workload(w, batch, args)
        return
    amp_np = wl.amplitudes(w, batch)
    phi_np = wl.phases(w)
    lab_np = wl.labels(w, batch)

    det = lb.Detector(w.detector.size, w.detector.y0, w.detector.x0)
    net = lb.Network(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n, w.n_fft, w.layers, 1.0, det)
    amp = torch.from_numpy(amp_np).cuda()
    phi = torch.from_numpy(phi_np).cuda()
    labels = torch.from_numpy(lab_np).cuda()
    saved = net.new_saved(batch)
    sums = torch.empty((batch, det.num), dtype=torch.float32, device="cuda")
    grad = torch.empty_like(phi)
    net.workspace(batch, lb.LR_OP_FORWARD)
    net.workspace(batch, lb.LR_OP_BACKWARD)

    def step():
        lb.lr_donn_forward(net, amp, phi, saved=saved, sums=True, out_sums=sums, layer_passes=args.layer_passes)
        return lb.lr_donn_backward(net, phi, saved, sums=sums, labels=labels, out_grad_phi=grad)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    run = step
    if args.graph:
        # The step's launches (kernels only: no copies, fills or host waits)
        # recorded once as a HIP graph and replayed: the same kernels on the
        # same buffers, without the per-launch dispatch gaps.
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            _, loss_graph = step()
        torch.cuda.synchronize()

        def run():
            graph.replay()
            return grad, loss_graph

        run()
        torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        _, loss = run()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    ms_per_step = gpu_ms / args.steps
    value = batch / (ms_per_step / 1e3)

    # instrumented replay: HIP events around every kernel launch on its stream
    lb.kernel_timing(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    kt = lb.kernel_timing_report()
    lb.kernel_timing(False)

    per_kernel = {k: {"count": v["count"], "avg_us": 1e3 * v["ms"] / v["count"], "total_ms": v["ms"]}
                  for k, v in kt.items()}
    dom = max(kt.items(), key=lambda kv: kv[1]["ms"])[0]
    kind = "bwd_mid" if "bwd_mid" in dom else ("fwd_mid" if "fwd_mid" in dom else None)
    roof = None
    if kind is not None:
        avg_s = kt[dom]["ms"] / kt[dom]["count"] / 1e3
        bytes_launch = algorithmic_bytes_per_sample(kind, w.n) * batch
        achieved = bytes_launch / avg_s / 1e9
        traffic = recorded_traffic(w.name, dom) if batch == w.batch else None
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic, "kernel": dom,
                "avg_launch_us": round(avg_s * 1e6, 2), "algorithmic_bytes_per_launch": int(bytes_launch),
                "traffic_unit": "HBM bytes per launch (FETCH_SIZE, WRITE_SIZE scaled by a copy calibration)",
                "traffic_gbps": round(traffic / avg_s / 1e9, 1) if traffic else None}
    # what actually bounds the layer passes: vector-ALU issue (counted
    # instructions of the same kernel over its measured launch time)
    valu = None
    if kind is not None:
        instr = recorded_valu(w.name, dom) if batch == w.batch else None
        if instr:
            rate = instr / avg_s
            valu = {"kernel": dom, "instr_per_launch": int(instr), "achieved": round(rate / 1e9, 1),
                    "peak": round(VALU_PEAK_WAVE_INSTR_PER_S / 1e9, 1), "unit": "G wave instructions/s",
                    "frac": round(rate / VALU_PEAK_WAVE_INSTR_PER_S, 4),
                    "floor_us": round(instr / VALU_PEAK_WAVE_INSTR_PER_S * 1e6, 1),
                    "peak_basis": "256 CUs x 4 SIMDs x 2.4 GHz / 4 cycles per wave64 FP32 instruction "
                                  "(no packed FP32)"}

    nn = w.n * w.n
    step_one_pass, step_path = step_bytes_per_sample(w, det)
    out = {
        "metric": "DONN samples/sec (5-layer N=200 fwd+bwd) and achieved HBM GB/s vs peak",
        "value": round(value, 1),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "execution": "graph_replay" if args.graph else "eager",
        "config": {"workload": w.name, "n": w.n, "n_fft": w.n_fft, "layers": w.layers, "batch": batch,
                   "approx": "fresnel" if w.approx == 0 else "angular_spectrum",
                   "wavelength_m": w.wavelength, "pixel_pitch_m": w.pixel_pitch, "distance_m": w.distance,
                   "loss": "softmax_cross_entropy", "detector_regions": det.num},
        "roofline": roof,
        "valu_issue": valu,
        "fields_per_s": round(value * (2 * w.layers + 1), 1),
        # whole-step GB/s under two byte counts: the one-pass lower bound of the
        # method and the bytes this path's passes move by design
        "step_gbps_one_pass_bound": round(batch * step_one_pass / (ms_per_step / 1e3) / 1e9, 1),
        "step_gbps_path_bytes": round(batch * step_path / (ms_per_step / 1e3) / 1e9, 1),
        "wall_s": round(wall, 3),
        "loss": float(loss) if loss is not None else None,
        "kernels": per_kernel,
    }
    if not args.no_cpu_baseline:
        cpu_b = args.cpu_samples if args.cpu_samples is not None else min(batch, 500)
        out["cpu_baseline"] = oracle_baseline(w, cpu_b, amp_np, phi_np, lab_np)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
