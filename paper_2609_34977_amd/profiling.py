"""Profiling helpers: kernel statistics and HBM traffic from rocprofv3 output.

    python -m paper_2609_34977_amd.profiling stats --csv S_kernel_stats.csv \
        --bench-log bench.log --out profiles/NAME.md --command "..."
    python -m paper_2609_34977_amd.profiling traffic --fetch F.csv --write W.csv \
        --copy-mib 256 --kernel-class gemm_gateup --workload W --rows R \
        --out profiles/gemm_gateup_traffic_W

`bench-table` turns bench.py JSON lines (one per workload) into a markdown
table of step time, throughput and the dominant kernel's roofline fraction.
`stats` turns a `rocprofv3 --kernel-trace --stats` kernel-statistics CSV into
a markdown table of this library's kernels (namespace spider::), sorted by
total time, with the bench line of the same run.

F.csv / W.csv are rocprofv3 counter-collection CSVs of two runs of
`bench.py --copy-probe-mib 256` (one with `--pmc FETCH_SIZE`, one with
`--pmc WRITE_SIZE`) on one workload; the record names that workload
(config.workload of the bench line) and its decoder row count, and bench.py
uses it only for the same workload and rows.  The plain copy of known size in the same runs calibrates
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
import sys
import statistics

HERE = os.path.dirname(os.path.abspath(__file__))

# kernel class -> (source files whose text defines its kernels, pattern of the dispatches
# that make one launch of the class, pattern of the one dispatch counted per launch)
_GEMM_SRC = ("csrc/gemm.hip", "csrc/kernels.h", "csrc/common.h")
CLASSES = {
    "gemm_gateup": (_GEMM_SRC,
                    r"gemm_stream_kernel<\d+, \d+, true\b|gemm_bf16_kernel<\d+, \d+, \d+, \d+, \d+, true"
                    r"|gemm_tile_kernel<\d+, true\b|swiglu_tail_reduce_kernel",
                    r"gemm_stream_kernel<\d+, \d+, true\b|gemm_bf16_kernel<\d+, \d+, \d+, \d+, \d+, true"
                    r"|gemm_tile_kernel<\d+, true\b"),
}


def kernel_source_hash(kernel_class: str) -> str:
    h = hashlib.sha256()
    for rel in CLASSES[kernel_class][0]:
        with open(os.path.join(HERE, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def recorded_traffic(path: str, kernel_class: str, workload: str, rows: int):
    """Bytes per launch recorded for the class on this workload and decoder row count,
    or None if there is no such record or the kernel sources changed since."""
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_class") != kernel_class or kernel_class not in CLASSES:
        return None
    if rec.get("workload") != workload or rec.get("rows") != rows:
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
    primary = re.compile(CLASSES[args.kernel_class][2])
    expect_kib = args.copy_mib * 1024.0
    out = {"kernel_class": args.kernel_class, "workload": args.workload, "rows": args.rows,
           "source_sha256": kernel_source_hash(args.kernel_class)}
    per = {}
    for counter, path in (("FETCH_SIZE", args.fetch), ("WRITE_SIZE", args.write)):
        rows = _dispatches(path, counter)
        factor, measured = _calibration(rows, expect_kib)
        vals = [v for name, v in rows if pat.search(name)]
        launches = sum(1 for name, _ in rows if primary.search(name))
        if not vals or not launches:
            raise SystemExit(f"no {args.kernel_class} dispatch in {path}")
        # a launch of the class may be more than one dispatch (e.g. the SwiGLU tail reduction)
        per[counter] = {"mean_kib_per_dispatch": sum(vals) / launches, "dispatches": launches,
                        "copy_kib_measured": measured, "copy_kib_expected": expect_kib,
                        "factor": factor,
                        "bytes_per_launch": sum(vals) / launches * factor * 1024.0}
    out["counters"] = per
    out["bytes_per_launch"] = per["FETCH_SIZE"]["bytes_per_launch"] + per["WRITE_SIZE"]["bytes_per_launch"]
    out["commands"] = args.command or []
    with open(args.out + ".json", "w") as f:
        json.dump(out, f, indent=1)
    lines = [f"# HBM traffic of `{args.kernel_class}` on `{args.workload}` ({args.rows} decoder rows; "
             "rocprofv3 counters)", "",
             "Commands (from the repository root, one MI355X):", "", "```"]
    lines += out["commands"] + ["```", "",
                                "| counter | launches | mean KiB / launch | copy KiB measured | copy KiB expected | factor | bytes / launch |",
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


def _short_name(name: str) -> str:
    # drop the namespace and the argument list, keep template arguments
    name = name.replace("void ", "", 1) if name.startswith("void ") else name
    name = re.sub(r"^spider::(\(anonymous namespace\)::)?", "", name)
    depth = 0
    for i, ch in enumerate(name):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return name[:i]
    return name


def stats(args):
    rows = []
    with open(args.csv) as f:
        for r in csv.DictReader(f):
            name = r["Name"]
            if "spider::" not in name:
                continue
            rows.append((_short_name(name), int(r["Calls"]), float(r["AverageNs"]) / 1e3,
                         float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3, float(r["TotalDurationNs"]) / 1e6))
    rows.sort(key=lambda t: -t[5])
    cls_line = []
    if getattr(args, "kernel_class", None):
        pat, prim = re.compile(CLASSES[args.kernel_class][1]), re.compile(CLASSES[args.kernel_class][2])
        tot_ms = sum(t for n, c, a, mn, mx, t in rows if pat.search(n))
        launches = sum(c for n, c, a, mn, mx, t in rows if prim.search(n))
        if launches:
            cls_line = [f"Kernel class `{args.kernel_class}` (every dispatch of its kernels, the SwiGLU tail "
                        f"reduction included): {launches} launches, {tot_ms * 1e3 / launches:.2f} us per launch "
                        f"on average, {tot_ms:.3f} ms in total."]
    lines = [f"# {args.title}", "", "Command (run from the repository root on one MI355X):", "", "```"]
    lines += (args.command or []) + ["```", "",
                                      "Kernels of this library (spider::), sorted by total time; the torch kernels that "
                                      "generate the synthetic inputs once at start-up are omitted (not part of the "
                                      "timed step).", "",
                                      "| kernel | calls | avg us | min us | max us | total ms |",
                                      "|---|---|---|---|---|---|"]
    for n, c, a, mn, mx, t in rows:
        lines.append(f"| `{n}` | {c} | {a:.2f} | {mn:.2f} | {mx:.2f} | {t:.3f} |")
    if cls_line:
        lines += [""] + cls_line
    if args.bench_log:
        with open(args.bench_log) as f:
            js = [ln for ln in f if ln.startswith("{")]
        if js:
            rec = json.loads(js[-1])
            lines += ["", "Bench line of the profiled run:", "",
                      f"- ms_per_step {rec['ms_per_step']:.3f}, value {rec['value']:.0f} {rec['unit']}",
                      f"- roofline: {json.dumps(rec.get('roofline'))}"]
    with open(args.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


_KERNEL_SYM = re.compile(r"spider::\(anonymous namespace\)::([A-Za-z0-9_]+_kernel(?:<[^()]*>)?)")


def library_kernels(lib_path=None, names_file=None):
    """Kernel instantiations of the library: the host-side launch stubs that
    `nm -C` lists for the built shared object (one per template instantiation),
    or the names in a text file, one per line."""
    if names_file:
        with open(names_file) as f:
            text = f.read()
    else:
        import subprocess
        text = subprocess.run(["nm", "-C", lib_path], check=True, capture_output=True, text=True).stdout
    out = set()
    for line in text.splitlines():
        line = line.replace("__device_stub__", "")
        m = _KERNEL_SYM.search(line)
        if m:
            out.add(m.group(1))
        elif re.fullmatch(r"[A-Za-z0-9_]+_kernel(<[^()]*>)?", line.strip()):
            out.add(line.strip())
    return sorted(out)


def coverage(args):
    """Every kernel instantiation of the library with the number of its
    dispatches in a traced run (rocprofv3 --kernel-trace --stats), zero flagged."""
    calls = {}
    with open(args.csv) as f:
        for r in csv.DictReader(f):
            m = _KERNEL_SYM.search(r["Name"])
            if m:
                calls[m.group(1)] = calls.get(m.group(1), 0) + int(r["Calls"])
    kernels = library_kernels(args.lib, args.names)
    never = [k for k in kernels if not calls.get(k)]
    lines = [f"# {args.title}", "", "Commands (run from the repository root on one MI355X):", "", "```"]
    lines += (args.command or []) + ["```", "",
              f"{len(kernels)} kernel instantiations in the library, {len(kernels) - len(never)} dispatched "
              f"during the run, {len(never)} never" + (": " + ", ".join(f"`{k}`" for k in never) if never else "") + ".",
              "", "| kernel | dispatches |", "|---|---|"]
    for k in kernels:
        lines.append(f"| `{k}` | {calls.get(k, 0)} |")
    with open(args.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines[:12]))
    return 0 if not never else 1


def bench_table(args):
    lines = [f"# {args.title}", "", "Commands (repository root, one MI355X), one per row:", "", "```"]
    lines += (args.command or []) + ["```", "",
                                      "| workload | skip p | decoder rows | ms / step | prefill TFLOP / step | "
                                      "TFLOP/s (whole step) | dominant kernel | its avg us / launch | "
                                      "achieved | frac of peak | GEMM ms (qkv/o/gateup/down) | attention ms |",
                                      "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    with open(args.jsonl) as f:
        for ln in f:
            if not ln.startswith("{"):
                continue
            r = json.loads(ln)
            ro, km, c = r["roofline"], r["kernel_ms_per_step"], r["config"]
            g = "/".join(f"{km.get(k, 0):.2f}" for k in ("gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down"))
            lines.append(f"| {c['workload']} | {c.get('skip_p')} | {c['decoder_rows']} | {r['ms_per_step']:.2f} | "
                         f"{r['prefill_tflop_per_step']:.2f} | {r['prefill_tflop_per_step'] / r['ms_per_step'] * 1e3:.0f} | "
                         f"{ro['kernel']} ({ro['bound']}) | {ro['avg_launch_us']:.1f} | {ro['achieved']:.0f} {ro['unit']} | "
                         f"{ro['frac']:.3f} | {g} | {km.get('attention', 0):.2f} |")
    with open(args.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


# kernels of the decoder step grouped for the counter table (name pattern, label)
_MFMA_GROUPS = [
    (r"gemm_tile_kernel<\d+, true\b", "tile GEMM, SwiGLU epilogue (gate/up, > 256 rows)"),
    (r"gemm_tile_kernel<\d+, false, true>", "tile GEMM, RoPE/bf16 epilogue (QKV, > 256 rows)"),
    (r"gemm_tile_kernel<\d+, false, false>", "tile GEMM, fp32 partials (O and down, > 256 rows)"),
    (r"gemm_stream_kernel<\d+, \d+, true", "streaming GEMM, SwiGLU (<= 256 rows)"),
    (r"gemm_stream_kernel<\d+, \d+, false", "streaming GEMM, fp32 partials (<= 256 rows)"),
    (r"attention_wide_kernel", "attention, many queries"),
    (r"attention_bf16_kernel", "attention, few queries"),
]


def mfma(args):
    """MFMA counters per kernel group from a rocprofv3 counter CSV with SQ_BUSY_CYCLES,
    SQ_VALU_MFMA_BUSY_CYCLES and SQ_INSTS_VALU_MFMA_MOPS_BF16 (one pass).  SQ_BUSY_CYCLES
    sums the 32 shader engines (8 XCDs x 4), so a dispatch lasts SQ_BUSY_CYCLES / 32
    cycles; MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x those cycles); one MOP
    is 512 flops."""
    per = {}
    with open(args.csv) as f:
        for r in csv.DictReader(f):
            name = r["Kernel_Name"]
            for pat, label in _MFMA_GROUPS:
                if re.search(pat, name):
                    d = per.setdefault(label, {}).setdefault(r["Dispatch_Id"], {})
                    d[r["Counter_Name"]] = float(r["Counter_Value"])
                    d["ns"] = float(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
                    break
    lines = [f"# {args.title}", "", "Command (repository root, one MI355X; `cd /tmp && export TMPDIR=/tmp` first):",
             "", "```"] + (args.command or []) + ["```", "",
             "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x SQ_BUSY_CYCLES / 32 shader engines), "
             "summed over the group's dispatches; flops = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 (an exact "
             "count of the MFMA work issued).  Counter runs serialise dispatches, so these fractions "
             "describe the kernels themselves, not the step's overlap.  Clock = GRBM_GUI_ACTIVE / 8 XCDs "
             "over the dispatches' own durations (their timestamps): the clock the chip sustained while "
             "they ran.  TFLOP/s = the issued flops over those durations; the last column divides it by "
             "the bf16 peak at that clock (2.5 PFLOP/s x clock / 2.4 GHz).  The GRBM window of a dispatch "
             "includes some time around it, so for dispatches of tens of microseconds the clock reads above "
             "the part's 2.4 GHz maximum: the column means something for the long dispatches only.", "",
             "| kernel group | dispatches | MFMA busy | TFLOP issued (all dispatches) | clock GHz | TFLOP/s | "
             "frac of 2.5 PFLOP/s | frac of the peak at that clock |",
             "|---|---|---|---|---|---|---|---|"]
    for _, label in _MFMA_GROUPS:
        if label not in per:
            continue
        ds = per[label].values()
        busy = sum(d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0) for d in ds)
        cyc = sum(d.get("SQ_BUSY_CYCLES", 0) for d in ds) / 32.0
        mops = sum(d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0) for d in ds)
        tf = mops * 512 / 1e12
        secs = sum(d.get("ns", 0) for d in ds) * 1e-9
        ghz = sum(d.get("GRBM_GUI_ACTIVE", 0) for d in ds) / 8.0 / max(secs, 1e-12) / 1e9
        rate = tf / max(secs, 1e-12)
        lines.append(f"| {label} | {len(per[label])} | {busy / max(1024 * cyc, 1):.3f} | {tf:.2f} | {ghz:.2f} | "
                     f"{rate:.0f} | {rate / 2500:.3f} | {rate / (2500 * ghz / 2.4):.3f} |")
    with open(args.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def sweep_table(args):
    """Markdown table of bench.py JSON lines (score / select sweeps, the stress curve, the
    hipBLASLt context)."""
    rows = []
    with open(args.jsonl) as f:
        for ln in f:
            if ln.startswith("{"):
                rows.append(json.loads(ln))
    lines = [f"# {args.title}", "", "Command (repository root, one MI355X):", "", "```"] + \
        (args.command or []) + ["```", ""] + (args.note or [])
    if rows and rows[0].get("mode") == "curve":
        lines += ["", "| keep / tile | skip p | decoder rows | ms / step | rows / s | prefill TFLOP | "
                      "TFLOP/s (step) | dominant kernel | bound | achieved | frac of peak |",
                  "|---|---|---|---|---|---|---|---|---|---|---|"]
        for r in rows:
            ro = r["roofline"]
            lines.append(f"| {r['keep_per_tile']} | {r['skip_p']} | {r['decoder_rows']} | {r['ms_per_step']:.2f} | "
                         f"{r['tokens_per_s']:.0f} | {r['prefill_tflop_per_step']:.1f} | "
                         f"{r['prefill_tflop_per_step'] / r['ms_per_step'] * 1e3:.0f} | {ro['kernel']} | "
                         f"{ro['bound']} | {ro['achieved']:.0f} {ro['unit']} | {ro['frac']:.3f} |")
    elif rows and rows[0].get("mode") == "vendor_gemm":
        cls = ("gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down")
        lines += ["", "Per launch, microseconds (TFLOP/s); last column: the library's time over hipBLASLt's.", "",
                  "| workload | rows | class | library us (TFLOP/s) | hipBLASLt us (TFLOP/s) | ratio |",
                  "|---|---|---|---|---|---|"]
        for r in rows:
            for c in cls:
                if c not in r["ours_us"]:
                    continue
                lines.append(f"| {r['workload']} | {r['rows']} | {c} | {r['ours_us'][c]:.1f} "
                             f"({r['ours_tflops'][c]:.0f}) | {r['hipblaslt_us'][c]:.1f} "
                             f"({r['hipblaslt_tflops'][c]:.0f}) | {r['ours_us'][c] / r['hipblaslt_us'][c]:.2f} |")
    elif rows and rows[0].get("mode") == "select_sweep":
        lines += ["", "| keep / tile | tiles | kept rows | select ms | select frac of HBM | gather ms | "
                      "gather MB | gather frac of HBM |", "|---|---|---|---|---|---|---|---|"]
        for r in rows:
            lines.append(f"| {r['keep_per_tile']} | {r['tiles']} | {r['kept_rows']} | {r['select_ms']:.4f} | "
                         f"{r['select_frac_of_hbm_peak']:.3f} | {r['gather_ms']:.4f} | {r['gather_bytes'] / 1e6:.1f} | "
                         f"{r['gather_frac_of_hbm_peak']:.3f} |")
    elif rows and rows[0].get("mode") == "score_sweep":
        ks = list(rows[0]["kernel_ms_per_call"])
        lines += ["", "| tiles | ms / call | compulsory MB | frac of HBM (compulsory / call) | " +
                  " | ".join(f"{k} ms" for k in ks) + " |", "|---|---|---|---|" + "---|" * len(ks)]
        for r in rows:
            lines.append(f"| {r['tiles']} | {r['ms_per_call']:.3f} | {r['compulsory_bytes'] / 1e6:.1f} | "
                         f"{r['frac_of_hbm_peak']:.3f} | " +
                         " | ".join(f"{r['kernel_ms_per_call'].get(k, 0):.4f}" for k in ks) + " |")
        if "kernel_effective_GBs" in rows[0]:
            ke = list(rows[0]["kernel_effective_GBs"])
            lines += ["", "Per kernel class: effective MB (what its design reads and writes once per pass), "
                          "GB/s and fraction of the 8 TB/s HBM peak.", "",
                      "| tiles | K-means working passes | " +
                      " | ".join(f"{k} MB / GB/s / frac" for k in ke) + " |", "|---|---|" + "---|" * len(ke)]
            for r in rows:
                lines.append(f"| {r['tiles']} | {r['kmeans_working_passes']} | " + " | ".join(
                    f"{r['kernel_effective_bytes'][k] / 1e6:.1f} / {r['kernel_effective_GBs'].get(k, 0):.0f} / "
                    f"{r['kernel_effective_GBs'].get(k, 0) / 8000:.2f}" for k in ke) + " |")
    with open(args.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    p = argparse.ArgumentParser()
    sub = p.add_subparsers(dest="cmd", required=True)
    b = sub.add_parser("bench-table")
    b.add_argument("--jsonl", required=True)
    b.add_argument("--out", required=True)
    b.add_argument("--title", default="bench.py over workloads")
    b.add_argument("--command", action="append")
    s = sub.add_parser("stats")
    s.add_argument("--csv", required=True)
    s.add_argument("--bench-log")
    s.add_argument("--out", required=True)
    s.add_argument("--title", default="rocprofv3 kernel statistics")
    s.add_argument("--kernel-class", default=None, help="also report this class's average per launch")
    s.add_argument("--command", action="append")
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--copy-mib", type=float, required=True)
    t.add_argument("--kernel-class", default="gemm_gateup")
    t.add_argument("--workload", required=True, help="config.workload of the bench line")
    t.add_argument("--rows", type=int, required=True, help="decoder rows of the bench line")
    t.add_argument("--out", required=True)
    t.add_argument("--command", action="append")
    m = sub.add_parser("mfma")
    m.add_argument("--csv", required=True)
    m.add_argument("--out", required=True)
    m.add_argument("--title", default="MFMA counters")
    m.add_argument("--command", action="append")
    c = sub.add_parser("coverage")
    c.add_argument("--csv", required=True, help="kernel statistics of the traced run")
    c.add_argument("--lib", default=None, help="the built library (its kernel instantiations via nm -C)")
    c.add_argument("--names", default=None, help="or a file of kernel instantiation names")
    c.add_argument("--out", required=True)
    c.add_argument("--title", default="Kernel coverage")
    c.add_argument("--command", action="append")
    w = sub.add_parser("sweep-table")
    w.add_argument("--jsonl", required=True)
    w.add_argument("--out", required=True)
    w.add_argument("--title", default="bench.py sweep")
    w.add_argument("--command", action="append")
    w.add_argument("--note", action="append")
    args = p.parse_args()
    if args.cmd == "mfma":
        mfma(args)
    elif args.cmd == "sweep-table":
        sweep_table(args)
    elif args.cmd == "traffic":
        traffic(args)
    elif args.cmd == "stats":
        stats(args)
    elif args.cmd == "bench-table":
        bench_table(args)
    elif args.cmd == "coverage":
        sys.exit(coverage(args))


if __name__ == "__main__":
    main()
