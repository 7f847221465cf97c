"""Host logic of the profiling helpers (CPU only): the counter-traffic record
and its keying, kernel-name shortening, the MFMA counter table and the kernel
statistics table, each on small synthetic rocprofv3-style CSVs."""
import argparse
import csv
import json

import pytest

from paper_2609_34977_amd import profiling as P

TILE = "void spider::(anonymous namespace)::gemm_tile_kernel<4, true, false>(spider::GemmArgs)"
TAIL = "void spider::(anonymous namespace)::swiglu_tail_reduce_kernel(float const*, int)"
STREAM = "void spider::(anonymous namespace)::gemm_stream_kernel<6, 2, true, false>(spider::GemmArgs)"
OTHER = "void spider::(anonymous namespace)::norm_kernel<unsigned short, 4>(spider::NormArgs)"
COPY = "__amd_rocclr_copyBuffer.kd"


def _counter_csv(path, counter, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, v) in enumerate(rows):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": v})


def _traffic_args(tmp_path, workload="stress_keep288", rows=6014):
    # the copy of 1 MiB reads as 2048 KiB on FETCH (factor 0.5) and 1024 KiB on WRITE (factor 1)
    _counter_csv(tmp_path / "f.csv", "FETCH_SIZE",
                 [(COPY, 2048.0), (TILE, 100.0), (TAIL, 10.0), (TILE, 300.0), (OTHER, 999.0), (COPY, 16.0)])
    _counter_csv(tmp_path / "w.csv", "WRITE_SIZE",
                 [(COPY, 1024.0), (TILE, 40.0), (TAIL, 4.0), (TILE, 60.0), (OTHER, 999.0)])
    return argparse.Namespace(fetch=str(tmp_path / "f.csv"), write=str(tmp_path / "w.csv"), copy_mib=1.0,
                              kernel_class="gemm_gateup", workload=workload, rows=rows,
                              out=str(tmp_path / "rec"), command=["cmd one", "cmd two"])


def test_traffic_record_scales_by_copy_calibration(tmp_path):
    args = _traffic_args(tmp_path)
    P.traffic(args)
    rec = json.load(open(args.out + ".json"))
    f, w = rec["counters"]["FETCH_SIZE"], rec["counters"]["WRITE_SIZE"]
    # two launches of the class; the tail reduction's dispatch counts toward them, the norm does not
    assert f["dispatches"] == 2 and w["dispatches"] == 2
    assert f["factor"] == pytest.approx(0.5) and w["factor"] == pytest.approx(1.0)
    assert f["mean_kib_per_dispatch"] == pytest.approx((100 + 10 + 300) / 2)
    assert f["bytes_per_launch"] == pytest.approx(205.0 * 0.5 * 1024)
    assert w["bytes_per_launch"] == pytest.approx(52.0 * 1.0 * 1024)
    assert rec["bytes_per_launch"] == pytest.approx(205.0 * 512 + 52.0 * 1024)
    assert rec["workload"] == "stress_keep288" and rec["rows"] == 6014
    assert rec["source_sha256"] == P.kernel_source_hash("gemm_gateup")
    md = open(args.out + ".md").read()
    assert "cmd one" in md and "stress_keep288" in md


def test_recorded_traffic_is_keyed_by_workload_rows_and_sources(tmp_path, monkeypatch):
    args = _traffic_args(tmp_path)
    P.traffic(args)
    path = args.out + ".json"
    want = json.load(open(path))["bytes_per_launch"]
    assert P.recorded_traffic(path, "gemm_gateup", "stress_keep288", 6014) == pytest.approx(want)
    assert P.recorded_traffic(path, "gemm_gateup", "llava15_7b_keep128", 6014) is None
    assert P.recorded_traffic(path, "gemm_gateup", "stress_keep288", 192) is None
    assert P.recorded_traffic(path, "no_such_class", "stress_keep288", 6014) is None
    assert P.recorded_traffic(str(tmp_path / "missing.json"), "gemm_gateup", "stress_keep288", 6014) is None
    # a changed kernel source invalidates the record
    monkeypatch.setattr(P, "kernel_source_hash", lambda cls: "0" * 64)
    assert P.recorded_traffic(path, "gemm_gateup", "stress_keep288", 6014) is None


def test_traffic_without_copy_probe_fails(tmp_path):
    args = _traffic_args(tmp_path)
    _counter_csv(tmp_path / "f.csv", "FETCH_SIZE", [(TILE, 100.0)])
    with pytest.raises(SystemExit):
        P.traffic(args)


def test_gateup_class_patterns():
    _, every, primary = P.CLASSES["gemm_gateup"]
    import re
    for name in (TILE, STREAM):
        assert re.search(every, name) and re.search(primary, name)
    assert re.search(every, TAIL) and not re.search(primary, TAIL)
    for name in (OTHER, TILE.replace("<4, true, false>", "<4, false, false>"),
                 STREAM.replace("<6, 2, true, false>", "<6, 2, false, false>")):
        assert not re.search(every, name)


def test_short_name_keeps_template_arguments():
    assert P._short_name(TILE) == "gemm_tile_kernel<4, true, false>"
    assert P._short_name("spider::f(int)") == "f"
    assert P._short_name("plain") == "plain"


def test_mfma_table_busy_clock_and_rate(tmp_path):
    # one dispatch of 1 ms: 2e6 busy cycles per shader engine, half of it MFMA,
    # GRBM_GUI_ACTIVE 8 x 2.0e6 (2.0 GHz), 2e12 flops issued (2 PFLOP/s)
    rows = []
    vals = {"SQ_BUSY_CYCLES": 32 * 2.0e6, "SQ_VALU_MFMA_BUSY_CYCLES": 0.5 * 1024 * 2.0e6,
            "SQ_INSTS_VALU_MFMA_MOPS_BF16": 2e12 / 512, "GRBM_GUI_ACTIVE": 8 * 2.0e6}
    for k, v in vals.items():
        rows.append({"Dispatch_Id": 7, "Kernel_Name": TILE, "Counter_Name": k, "Counter_Value": v,
                     "Start_Timestamp": 1_000_000, "End_Timestamp": 2_000_000})
    path = tmp_path / "m.csv"
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0]))
        w.writeheader()
        w.writerows(rows)
    out = tmp_path / "m.md"
    P.mfma(argparse.Namespace(csv=str(path), out=str(out), title="t", command=["c"]))
    line = [ln for ln in open(out) if ln.startswith("| tile GEMM, SwiGLU")][0]
    cells = [c.strip() for c in line.strip().strip("|").split("|")]
    assert cells[1] == "1"
    assert float(cells[2]) == pytest.approx(0.5)
    assert float(cells[3]) == pytest.approx(2.0)
    assert float(cells[4]) == pytest.approx(2.0)
    assert float(cells[5]) == pytest.approx(2000)
    assert float(cells[6]) == pytest.approx(0.8)
    assert float(cells[7]) == pytest.approx(2000 / (2500 * 2.0 / 2.4), abs=1e-3)


def test_stats_table_keeps_library_kernels_and_class_line(tmp_path):
    path = tmp_path / "s.csv"
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Name", "Calls", "AverageNs", "MinNs", "MaxNs", "TotalDurationNs"])
        w.writeheader()
        w.writerow({"Name": TILE, "Calls": 4, "AverageNs": 1000, "MinNs": 900, "MaxNs": 1100,
                    "TotalDurationNs": 4000})
        w.writerow({"Name": TAIL, "Calls": 4, "AverageNs": 100, "MinNs": 90, "MaxNs": 110,
                    "TotalDurationNs": 400})
        w.writerow({"Name": "at::native::fill_kernel", "Calls": 9, "AverageNs": 5, "MinNs": 5, "MaxNs": 5,
                    "TotalDurationNs": 45})
    out = tmp_path / "s.md"
    P.stats(argparse.Namespace(csv=str(path), out=str(out), title="t", command=["c"], bench_log=None,
                               kernel_class="gemm_gateup"))
    text = open(out).read()
    assert "fill_kernel" not in text
    assert "| `gemm_tile_kernel<4, true, false>` | 4 | 1.00 |" in text
    # 4 launches; the tail reduction's time is part of the class
    assert "4 launches, 1.10 us per launch" in text


def test_vendor_gemm_table_rows_and_ratio(tmp_path):
    line = {"mode": "vendor_gemm", "workload": "stress_keep288_skip0", "rows": 6014, "d": 4096, "d_ff": 11008,
            "ours_us": {"gemm_qkv": 500.0, "gemm_o": 180.0, "gemm_gateup": 900.0},
            "hipblaslt_us": {"gemm_qkv": 550.0, "gemm_o": 200.0, "gemm_gateup": 880.0, "gemm_down": 480.0},
            "ours_tflops": {"gemm_qkv": 1210.0, "gemm_o": 1120.0, "gemm_gateup": 1205.0},
            "hipblaslt_tflops": {"gemm_qkv": 1100.0, "gemm_o": 1008.0, "gemm_gateup": 1232.0, "gemm_down": 1100.0}}
    src = tmp_path / "v.jsonl"
    src.write_text("# a comment line\n" + json.dumps(line) + "\n")
    out = tmp_path / "v.md"
    P.sweep_table(argparse.Namespace(jsonl=str(src), out=str(out), title="t", command=["cmd"], note=None))
    rows = [ln for ln in out.read_text().splitlines() if ln.startswith("| stress")]
    # a class the library did not launch is left out; the ratio is library / hipBLASLt
    assert len(rows) == 3
    assert rows[0].split("|")[3].strip() == "gemm_qkv" and rows[0].rstrip("| ").endswith("0.91")
    assert "900.0 (1205)" in rows[2] and rows[2].rstrip("| ").endswith("1.02")


def test_coverage_lists_every_instantiation_and_flags_the_idle_ones(tmp_path):
    names = tmp_path / "names.txt"
    names.write_text("__device_stub__gemm_tile_kernel<4, true, false>\nnorm_kernel<float, 8>\nselect_kernel\n")
    stats = tmp_path / "stats.csv"
    with open(stats, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs", "StdDev"])
        w.writerow(["void spider::(anonymous namespace)::gemm_tile_kernel<4, true, false>(spider::GemmArgs)",
                    "12", "100", "8", "1", "1", "9", "0"])
        w.writerow(["spider::(anonymous namespace)::select_kernel(int, int)", "3", "30", "10", "1", "9", "11", "0"])
        w.writerow(["at::native::vectorized_elementwise_kernel<4>(int)", "99", "5", "1", "1", "1", "1", "0"])
    out = tmp_path / "cov.md"
    rc = P.coverage(argparse.Namespace(csv=str(stats), lib=None, names=str(names), out=str(out), title="t",
                                       command=["cmd"]))
    text = out.read_text()
    assert rc == 1
    assert "3 kernel instantiations in the library, 2 dispatched during the run, 1 never: `norm_kernel<float, 8>`" in text
    assert "| `gemm_tile_kernel<4, true, false>` | 12 |" in text and "| `norm_kernel<float, 8>` | 0 |" in text
