"""Profiling helpers: HBM traffic of a kernel class from rocprofv3 counters.

    python -m paper_2609_34977_amd.profiling traffic --fetch F.csv --write W.csv \
        --copy-mib 256 --kernel-class gemm_gateup --out profiles/gemm_gateup_traffic

F.csv / W.csv are rocprofv3 counter-collection CSVs of two runs of
`bench.py --copy-probe-mib 256` (one with `--pmc FETCH_SIZE`, one with
`--pmc WRITE_SIZE`).  The plain copy of known size in the same runs calibrates
both counters (bytes the copy must read / write divided by what the counter
reports for it); the per-launch traffic of the kernel class is the mean over
its dispatches, scaled by that factor.  Writes <out>.json (read by bench.py,
which reports the figure only while the kernel sources still hash to the
recorded value) and <out>.md (the summary).
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import statistics

HERE = os.path.dirname(os.path.abspath(__file__))

# kernel class -> (source files whose text defines its kernels, dispatch-name pattern)
CLASSES = {
    "gemm_gateup": (("csrc/gemm.hip", "csrc/kernels.h", "csrc/common.h"),
                    r"gemm_stream_kernel<\d+, \d+, true\b|gemm_bf16_kernel<\d+, \d+, \d+, \d+, \d+, true"),
}


def kernel_source_hash(kernel_class: str) -> str:
    h = hashlib.sha256()
    for rel in CLASSES[kernel_class][0]:
        with open(os.path.join(HERE, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def recorded_traffic(path: str, kernel_class: str):
    """Bytes per launch recorded for the class, or None if absent or stale."""
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_class") != kernel_class:
        return None
    if rec.get("source_sha256") != kernel_source_hash(kernel_class):
        return None
    return rec.get("bytes_per_launch")


def _dispatches(path: str, counter: str):
    rows = []
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] == counter:
                rows.append((r["Kernel_Name"], float(r["Counter_Value"])))
    return rows


def _calibration(rows, expect_kib: float):
    # the probe is a device-to-device copy, run by the HIP runtime's blit kernel;
    # it is the largest such dispatch of the run
    copies = [v for name, v in rows if "copyBuffer" in name]
    if not copies:
        raise SystemExit("no device-to-device copy dispatch found in the counter CSV")
    measured = max(copies)
    return expect_kib / measured, measured


def traffic(args):
    pat = re.compile(CLASSES[args.kernel_class][1])
    expect_kib = args.copy_mib * 1024.0
    out = {"kernel_class": args.kernel_class,
           "source_sha256": kernel_source_hash(args.kernel_class)}
    per = {}
    for counter, path in (("FETCH_SIZE", args.fetch), ("WRITE_SIZE", args.write)):
        rows = _dispatches(path, counter)
        factor, measured = _calibration(rows, expect_kib)
        vals = [v for name, v in rows if pat.search(name)]
        if not vals:
            raise SystemExit(f"no {args.kernel_class} dispatch in {path}")
        per[counter] = {"mean_kib_per_dispatch": statistics.fmean(vals), "dispatches": len(vals),
                        "copy_kib_measured": measured, "copy_kib_expected": expect_kib,
                        "factor": factor,
                        "bytes_per_launch": statistics.fmean(vals) * factor * 1024.0}
    out["counters"] = per
    out["bytes_per_launch"] = per["FETCH_SIZE"]["bytes_per_launch"] + per["WRITE_SIZE"]["bytes_per_launch"]
    out["commands"] = args.command or []
    with open(args.out + ".json", "w") as f:
        json.dump(out, f, indent=1)
    lines = [f"# HBM traffic of `{args.kernel_class}` (rocprofv3 counters)", "",
             "Commands (from the repository root, one MI355X):", "", "```"]
    lines += out["commands"] + ["```", "",
                                "| counter | dispatches | mean KiB / dispatch | copy KiB measured | copy KiB expected | factor | bytes / launch |",
                                "|---|---|---|---|---|---|---|"]
    for c, v in per.items():
        lines.append(f"| {c} | {v['dispatches']} | {v['mean_kib_per_dispatch']:.1f} | "
                     f"{v['copy_kib_measured']:.1f} | {v['copy_kib_expected']:.1f} | {v['factor']:.4f} | "
                     f"{v['bytes_per_launch']:.4g} |")
    lines += ["", f"Traffic per launch (fetch + write): {out['bytes_per_launch']:.4g} bytes.",
              f"Kernel sources sha256: `{out['source_sha256']}`."]
    with open(args.out + ".md", "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    p = argparse.ArgumentParser()
    sub = p.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--copy-mib", type=float, required=True)
    t.add_argument("--kernel-class", default="gemm_gateup")
    t.add_argument("--out", required=True)
    t.add_argument("--command", action="append")
    args = p.parse_args()
    if args.cmd == "traffic":
        traffic(args)


if __name__ == "__main__":
    main()
