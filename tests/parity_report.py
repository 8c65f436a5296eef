"""Parity and oracle timing at the five workloads (measurement record).

    python tests/parity_report.py [--workloads 1 2 3 4 5]

For each workload: the HIP path through the C ABI and the float64 oracle on
the same seeded inputs, relative L2 error of every output (fields, intensity
maps, detector sums, the loss, dL/dphi), and the oracle's own throughput on
the host (samples per second, with the BLAS threads and library).  Workloads
1-3 compare the whole batch; the large ones compare a stated slice of it
(forward: the first and last samples of the full-batch run; training: a
two-sample batch on both sides, since dL/dphi sums over the batch).  Prints
one JSON line per workload.  Test infrastructure: needs a GPU and the built
library.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle.donn as od  # noqa: E402
from paper_2306_11268_amd import binding as lb  # noqa: E402
from paper_2306_11268_amd import workloads as wl  # noqa: E402


def rel(a, b) -> float:
    a = np.asarray(a, np.complex128 if np.iscomplexobj(a) or np.iscomplexobj(b) else np.float64)
    b = np.asarray(b)
    return float(np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(b.ravel()), 1e-300))


def blas_info():
    from threadpoolctl import threadpool_info
    blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = max([i.get("num_threads", 1) for i in blas] or [1])
    vendor = ", ".join(sorted({f"{i.get('internal_api', '?')} {i.get('version', '')}".strip() for i in blas}))
    return int(threads), vendor or "none"


def report(wid: int) -> dict:
    import torch

    w = wl.WORKLOADS[wid]
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    host = lambda t: t.detach().cpu().numpy()  # noqa: E731
    d = w.detector
    det = lb.Detector(d.size, d.y0, d.x0) if d is not None else None
    odet = od.Detector(d.size, tuple(d.y0), tuple(d.x0)) if d is not None else None
    net = lb.Network(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n, w.n_fft, w.layers, 1.0, det)
    h = od.transfer_function(w.wavelength, w.pixel_pitch, w.distance, w.approx, w.n_fft)
    phi = wl.phases(w)
    out = {"workload": w.name}
    par = {}
    if w.kind == "forward":
        amp = wl.amplitudes(w, w.batch)
        full = w.wid != 4
        g = lb.lr_donn_forward(net, dev(amp), dev(phi), sums=det is not None, intensity=w.output != "sums",
                               field=w.output == "field+intensity")
        torch.cuda.synchronize()
        idx = list(range(w.batch)) if full else [0, w.batch - 1]
        t0 = time.perf_counter()
        if full:
            refs = [od.donn_forward(amp, phi, h, 1.0, odet)]
        else:
            refs = [od.donn_forward(amp[i:i + 1], phi, h, 1.0, odet) for i in idx]
        dt = time.perf_counter() - t0
        if g["sums"] is not None:
            par["sums"] = rel(host(g["sums"])[idx], np.concatenate([r["sums"] for r in refs]))
        if g["intensity"] is not None:
            par["intensity"] = rel(host(g["intensity"])[idx], np.concatenate([r["intensity"] for r in refs]))
        if g["field"] is not None:
            par["field"] = rel(host(g["field"])[idx], np.concatenate([r["field"] for r in refs]))
        out["checked"] = "whole batch" if full else f"samples {idx} of the batch of {w.batch}"
        ns = len(idx)
    else:
        b = w.batch if w.grad == "ce" else 2
        amp = wl.amplitudes(w, b)
        saved = net.new_saved(b)
        if w.grad == "ce":
            labels = wl.labels(w, b)
            g = lb.lr_donn_forward(net, dev(amp), dev(phi), saved=saved, sums=True)
            grad, loss = lb.lr_donn_backward(net, dev(phi), saved, sums=g["sums"], labels=dev(labels))
        else:
            gi = wl.upstream_intensity_grad(w, b)
            g = lb.lr_donn_forward(net, dev(amp), dev(phi), saved=saved, sums=False, intensity=True)
            grad, loss = lb.lr_donn_backward(net, dev(phi), saved, grad_intensity=dev(gi))
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ref = od.donn_forward(amp, phi, h, 1.0, odet)
        if w.grad == "ce":
            ref_loss, gs = od.softmax_cross_entropy(ref["sums"], labels)
            ref_g = od.donn_backward(ref, phi, h, 1.0, odet, grad_sums=gs)
        else:
            ref_g = od.donn_backward(ref, phi, h, 1.0, grad_intensity=gi)
        dt = time.perf_counter() - t0
        if w.grad == "ce":
            par["sums"] = rel(host(g["sums"]), ref["sums"])
            par["loss"] = abs(float(host(loss)) - ref_loss) / abs(ref_loss)
        else:
            par["intensity"] = rel(host(g["intensity"]), ref["intensity"])
        par["dphi"] = rel(host(grad), ref_g)
        out["checked"] = "whole batch" if b == w.batch else f"a batch of {b} on both sides (dL/dphi sums over the batch)"
        ns = b
    threads, vendor = blas_info()
    out["parity_rel_l2"] = {k: float(f"{v:.3e}") for k, v in par.items()}
    out["oracle"] = {"samples_per_s": round(ns / dt, 3), "seconds": round(dt, 3), "samples": ns,
                     "what": "forward" if w.kind == "forward" else "forward + loss seed + backward",
                     "blas_threads": threads, "blas": vendor, "host_cpus": len(os.sched_getaffinity(0))}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workloads", type=int, nargs="+", default=[1, 2, 3, 4, 5])
    args = ap.parse_args()
    lb.load()
    for wid in args.workloads:
        print(json.dumps(report(wid)), flush=True)


if __name__ == "__main__":
    main()
