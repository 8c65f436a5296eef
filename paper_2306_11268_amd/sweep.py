"""Depth and grid-size sweep of the training step (the paper's runtime study).

The paper times its emulator over {1, 3, 5, 7, 10} layers on grids from
100 x 100 to 500 x 500 and on deeper networks (§5.3, Fig. runtime_breakdown
and the text around it).  This module runs `bench.py` once per (grid,
depth) point in a fresh process, on the training workload of the benchmark
(softmax cross-entropy over ten detector regions, batch 500, Fresnel,
unpadded grids), and prints one markdown table row per point plus the JSON
lines of the runs.

    python -m paper_2306_11268_amd.sweep [--grids 100 200 400 500] [--layers 1 3 5 7 10 30]
                                         [--steps 5] [--warmup 2] [--json OUT]
"""

from __future__ import annotations

import argparse
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_point(n: int, layers: int, steps: int, warmup: int, batch: int | None) -> dict:
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--n", str(n), "--layers", str(layers),
           "--steps", str(steps), "--warmup", str(warmup), "--no-cpu-baseline"]
    if batch is not None:
        cmd += ["--batch", str(batch)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise SystemExit(f"bench failed at n={n} layers={layers}:\n{r.stderr[-4000:]}")
    return json.loads(r.stdout.strip().splitlines()[-1])


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--grids", type=int, nargs="+", default=[100, 200, 400, 500])
    ap.add_argument("--layers", type=int, nargs="+", default=[1, 3, 5, 7, 10, 30])
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--batch", type=int, default=None)
    ap.add_argument("--json", default=None, help="also write the JSON lines here")
    args = ap.parse_args(argv)
    print("| grid | layers | batch | ms / step | samples/s | one-pass GB/s |", flush=True)
    print("|---:|---:|---:|---:|---:|---:|", flush=True)
    lines = []
    for n in args.grids:
        for layers in args.layers:
            d = run_point(n, layers, args.steps, args.warmup, args.batch)
            lines.append(d)
            c = d["config"]
            print(f"| {n} | {layers} | {c['batch']} | {d['ms_per_step']:.3f} | {d['value']:.0f} | "
                  f"{d['step_effective_gbps']:.0f} |", flush=True)
    if args.json:
        with open(args.json, "w") as fh:
            for d in lines:
                fh.write(json.dumps(d) + "\n")


if __name__ == "__main__":
    main()
