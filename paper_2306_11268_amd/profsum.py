"""Summaries of rocprofv3 CSV output for the DONN kernels.

    # per-kernel durations from `rocprofv3 --kernel-trace --stats --output-format csv -d DIR`
    python -m paper_2306_11268_amd.profsum stats DIR --command "<rocprofv3 command>"

    # HBM traffic per dispatch from two counter runs (FETCH_SIZE, WRITE_SIZE) of the
    # workload and the same two counters read on a plain copy of known size
    python -m paper_2306_11268_amd.profsum traffic --fetch D1 --write D2 \\
        --copy-fetch D3 --copy-write D4 --copy-bytes 536870912 --workload NAME \\
        --command-fetch "..." --command-write "..." --command-copy "..." \\
        --out-md FILE --out-json FILE

Kernel template names are shown with the short label the library's own
timing report uses (e.g. fresnel_pass_fwd_mid_col_N200).  The JSON written
by `traffic` carries the digest of the device sources it was measured on,
so that a reader can tell when the figures have gone stale.
"""

from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import re
import sys
from collections import defaultdict

FR_KINDS = ("prop", "fwd_mid", "fwd_last", "bwd_first", "bwd_mid", "bwd_last")
AS_KINDS = ("row_first", "col", "row_mid", "row_last", "row_bwd_first", "row_bwd_mid", "row_bwd_last", "row_ifft",
            "col_far")
AXES = ("row", "col")


def label(name: str) -> str:
    """Short label of a demangled kernel name."""
    m = re.search(r"(fresnel|detector)_pass<.*?Plan2<(\d+), (\d+).*, (\d+), (\d+)>\(", name)
    if m:
        n = int(m.group(2)) * int(m.group(3))
        return f"fresnel_pass_{FR_KINDS[int(m.group(4))]}_{AXES[int(m.group(5))]}_N{n}"
    m = re.search(r"as_pass<.*?Plan2<(\d+), (\d+).*, (\d+)>\(", name)
    if m:
        n = int(m.group(1)) * int(m.group(2))
        return f"as_pass_{AS_KINDS[int(m.group(3))]}_N{n}"
    m = re.search(r"lr::(\w+?)(_kernel)?[<(]", name)
    if m:
        return m.group(1)
    return name.split("(")[0].replace("void ", "")


def _one(pattern: str, d: str) -> str:
    hits = sorted(glob.glob(os.path.join(d, "**", pattern), recursive=True))
    if not hits:
        raise SystemExit(f"no {pattern} under {d}")
    return hits[0]


def kernel_stats(d: str):
    rows = []
    with open(_one("*kernel_stats.csv", d)) as fh:
        for r in csv.DictReader(fh):
            rows.append({"name": r["Name"], "label": label(r["Name"]), "calls": int(r["Calls"]),
                         "total_ns": float(r["TotalDurationNs"]), "avg_ns": float(r["AverageNs"]),
                         "pct": float(r["Percentage"]), "min_ns": float(r["MinNs"]), "max_ns": float(r["MaxNs"])})
    return rows


def counter_means(d: str, counter: str):
    """Mean counter value per dispatch, by kernel label: {label: (mean, dispatches, meta)}."""
    acc = defaultdict(list)
    meta = {}
    with open(_one("*counter_collection.csv", d)) as fh:
        for r in csv.DictReader(fh):
            if r["Counter_Name"] != counter:
                continue
            lab = label(r["Kernel_Name"])
            acc[lab].append(float(r["Counter_Value"]))
            meta[lab] = {"vgpr": int(r["VGPR_Count"]), "agpr": int(r.get("Accum_VGPR_Count", 0) or 0),
                         "sgpr": int(r["SGPR_Count"]), "lds": int(r["LDS_Block_Size"]),
                         "scratch": int(r["Scratch_Size"]), "wg": int(r["Workgroup_Size"]),
                         "grid": int(r["Grid_Size"])}
    return {k: (sum(v) / len(v), len(v), meta[k]) for k, v in acc.items()}


def cmd_stats(args):
    rows = kernel_stats(args.dir)
    out = [f"# Kernel durations: {args.title}", "", "Command:", "", "```", args.command, "```", "",
           "| kernel | calls | avg (us) | min (us) | max (us) | total (ms) | % |", "|---|---:|---:|---:|---:|---:|---:|"]
    for r in sorted(rows, key=lambda r: -r["total_ns"]):
        out.append(f"| {r['label']} | {r['calls']} | {r['avg_ns'] / 1e3:.1f} | {r['min_ns'] / 1e3:.1f} | "
                   f"{r['max_ns'] / 1e3:.1f} | {r['total_ns'] / 1e6:.3f} | {r['pct']:.1f} |")
    out += ["", "Template names:", ""]
    for r in sorted(rows, key=lambda r: -r["total_ns"]):
        out.append(f"- `{r['label']}`: `{r['name']}`")
    text = "\n".join(out) + "\n"
    if args.out:
        with open(args.out, "w") as fh:
            fh.write(text)
    else:
        sys.stdout.write(text)


def cmd_traffic(args):
    from . import build as lb

    fetch = counter_means(args.fetch, "FETCH_SIZE")
    write = counter_means(args.write, "WRITE_SIZE")
    cf = counter_means(args.copy_fetch, "FETCH_SIZE")
    cw = counter_means(args.copy_write, "WRITE_SIZE")
    copy_key = max(cf, key=lambda k: cf[k][0])
    kib = args.copy_bytes / 1024.0
    fetch_scale = kib / cf[copy_key][0]
    write_scale = kib / cw[copy_key][0]
    kernels = {}
    for lab in sorted(set(fetch) & set(write)):
        f_kib, nf, meta = fetch[lab]
        w_kib, nw, _ = write[lab]
        kernels[lab] = {"fetch_kib_per_dispatch": round(f_kib, 1), "write_kib_per_dispatch": round(w_kib, 1),
                        "dispatches": min(nf, nw),
                        "hbm_bytes_per_dispatch": round(f_kib * fetch_scale * 1024 + w_kib * write_scale * 1024),
                        **meta}
    doc = {"workload": args.workload, "source_digest": lb.source_digest(),
           "copy_kernel": copy_key, "copy_bytes": args.copy_bytes,
           "copy_fetch_kib": round(cf[copy_key][0], 1), "copy_write_kib": round(cw[copy_key][0], 1),
           "fetch_scale": round(fetch_scale, 4), "write_scale": round(write_scale, 4),
           "commands": {"fetch": args.command_fetch, "write": args.command_write, "copy": args.command_copy},
           "kernels": kernels}
    with open(args.out_json, "w") as fh:
        json.dump(doc, fh, indent=1)
        fh.write("\n")
    lines = [f"# HBM traffic per dispatch: {args.workload}", "",
             "Counters: `FETCH_SIZE` and `WRITE_SIZE` (KiB per dispatch, mean over dispatches), "
             "each from its own rocprofv3 run.", "",
             f"Calibration on a plain device copy of {args.copy_bytes} bytes (`{copy_key}`): "
             f"FETCH_SIZE reads {cf[copy_key][0]:.0f} KiB for {kib:.0f} KiB read (scale {fetch_scale:.4f}), "
             f"WRITE_SIZE reads {cw[copy_key][0]:.0f} KiB for {kib:.0f} KiB written (scale {write_scale:.4f}).", "",
             f"Device-source digest: `{doc['source_digest']}`", "", "Commands:", "", "```",
             args.command_fetch, args.command_write, args.command_copy, "```", "",
             "| kernel | FETCH KiB | WRITE KiB | HBM MB / dispatch (scaled) | VGPR | AGPR | LDS B | scratch B |",
             "|---|---:|---:|---:|---:|---:|---:|---:|"]
    for lab, k in sorted(kernels.items(), key=lambda kv: -kv[1]["hbm_bytes_per_dispatch"]):
        lines.append(f"| {lab} | {k['fetch_kib_per_dispatch']:.0f} | {k['write_kib_per_dispatch']:.0f} | "
                     f"{k['hbm_bytes_per_dispatch'] / 1e6:.1f} | {k['vgpr']} | {k['agpr']} | {k['lds']} | "
                     f"{k['scratch']} |")
    with open(args.out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    s.add_argument("--command", required=True)
    s.add_argument("--title", default="")
    s.add_argument("--out", default=None)
    t = sub.add_parser("traffic")
    for k in ("fetch", "write", "copy-fetch", "copy-write", "workload", "command-fetch", "command-write",
              "command-copy", "out-md", "out-json"):
        t.add_argument("--" + k, required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    args = ap.parse_args(argv)
    {"stats": cmd_stats, "traffic": cmd_traffic}[args.cmd](args)


if __name__ == "__main__":
    main()
