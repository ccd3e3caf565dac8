"""Host logic of bench.py (no GPU): the HBM-traffic bookkeeping built from
rocprofv3 counter CSVs, and its gate on the kernel-source hash."""
import csv
import json

import bench


def _csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Value"])
        w.writeheader()
        for name, value in rows:
            w.writerow({"Kernel_Name": name, "Counter_Value": value})


def test_write_traffic_sums_the_launches_of_a_split_call(tmp_path, monkeypatch):
    # a split prefill call is three kinds of launch; each kind is averaged
    # over its launches and the averages added; the count variant is left out
    main = "void attn::prefill_kernel<128, 128, true, false, 1, false, 2>(attn::Params)"
    count = "void attn::prefill_kernel<128, 128, true, true, 1, false, 2>(attn::Params)"
    p1 = "void attn::prefill_kernel<128, 128, true, false, 0, false, 1>(attn::Params)"
    merge = "void attn::prefill_merge<128>(attn::Params)"
    copy = "__amd_rocclr_copyBuffer"
    fetch = tmp_path / "fetch.csv"
    write = tmp_path / "write.csv"
    _csv(fetch, [(main, 100), (main, 110), (count, 999), (p1, 40), (p1, 44), (merge, 6), (copy, 10),
                 (copy, 2 * 1024 * 1024 / 4)])
    _csv(write, [(main, 10), (main, 10), (count, 999), (p1, 1), (p1, 1), (merge, 2), (copy, 1024 * 1024)])
    monkeypatch.setattr(bench, "traffic_file", lambda w: str(tmp_path / f"traffic_{w}.json"))
    t = bench.write_traffic(str(fetch), str(write), "wl", copy_mib=1024)
    assert t["fetch_kib_per_launch_raw"] == 105 + 42 + 6
    assert t["write_kib_per_launch_raw"] == 10 + 1 + 2
    # FETCH is scaled by 1 GiB / the largest copy reading (2x), WRITE by 1x
    assert t["fetch_scale"] == 2.0 and t["write_scale"] == 1.0
    assert t["hbm_bytes_per_launch"] == (153 * 2 + 13) * 1024
    assert json.load(open(tmp_path / "traffic_wl.json"))["kernel_source_sha256"] == bench.kernel_source_hash()


def test_measured_traffic_only_for_the_current_sources(tmp_path, monkeypatch):
    path = tmp_path / "traffic_wl.json"
    monkeypatch.setattr(bench, "traffic_file", lambda w: str(path))
    assert bench.measured_traffic("wl") is None                     # no file
    rec = {"workload": "wl", "kernel_source_sha256": bench.kernel_source_hash(),
           "hbm_bytes_per_launch": 123.0}
    path.write_text(json.dumps(rec))
    assert bench.measured_traffic("wl") == 123.0
    assert bench.measured_traffic("other") is None                  # another workload
    path.write_text(json.dumps(dict(rec, kernel_source_sha256="0" * 64)))
    assert bench.measured_traffic("wl") is None                     # kernels changed since


def test_more_than_one_gpu_is_refused_with_a_message():
    # one GPU only: --gpus N > 1 exits non-zero before touching a device
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr and r.stdout == ""


def test_report_markdown_and_paper_context(tmp_path):
    # the report's markdown summary from one synthetic run record, and the
    # paper context attached only where the paper has a figure for the run
    import json
    import bench
    rec = {"config": "C2", "workload": "w", "mode": "faithful", "S": 1.0, "order": "forward",
           "delta": 7.0, "delta_eff": 7.0, "gpu_ms_median": 1.0, "timed_launches": 20,
           "tflops": 68.7, "peak_tflops": 157.3, "frac_of_peak": 0.437,
           "mse_gpu_vs_fp64": 5.5e-5, "mse_oracle_vs_fp64": 5.5e-5,
           "max_abs_gpu_minus_oracle": 1e-6, "max_abs_lse_gpu_minus_oracle": 1e-7,
           "zero_fraction_nonsink": 0.81, "collapse_fraction_F": 0.86,
           "counts_equal_on_oracle_rows": True,
           "oracle": {"rows": 8192, "rows_total": 32768, "sample": "every 4th flat row",
                      "pairs": 1, "seconds": 0.5, "cores": 16, "tflops": 0.1},
           "paper_context": bench._paper_context("C2", "forward", 1.0, 7.0)}
    p = tmp_path / "r.jsonl"
    p.write_text(json.dumps(rec) + "\n")
    md = open(bench.write_report_md(str(p))).read()
    assert "| C2 | 7.0 | 1 | forward |" in md
    assert "table1_frac_zeroed=0.82" in md and "table2_mse=5.65e-05" in md
    assert bench._paper_context("C2", "reverse", 16.0, 7.0) == {}
    assert bench._paper_context("C4", "forward", 1.0, 9.0) == {}
