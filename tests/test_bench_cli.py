"""bench.py's host-side contract (no GPU needed): more than one GPU is refused
with a message, the traffic record matches its kernels' code (comments
aside), and the counter summary keeps only full-size dispatches."""
from __future__ import annotations

import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_record_is_used_only_for_its_kernels():
    """The counter record is reported only while it was taken on the kernels'
    current code; then measured traffic equals the algorithmic bytes."""
    rec = json.load(open(bench.TRAFFIC_FILE))
    if rec["kernel_source_hash"] != bench.kernel_source_hash():
        assert bench.measured_traffic() is None
        return
    assert bench.measured_traffic() is not None
    for k in ("fwd_lane_kernel", "bwd_lane_kernel"):
        assert abs(rec["kernels"][k]["traffic_over_algorithmic"] - 1.0) < 1e-3


def test_source_hash_ignores_comments_only():
    """The record stays valid across comment and layout edits of the kernel
    sources, and no longer matches once their code changes."""
    src = 'int f(int a) { // add one\n  return a + 1; /* done */ }\nconst char* s = "x//y";'
    assert bench.code_only(src) == bench.code_only(
        "/* header */\nint f(int a)\n{\n    return a + 1;\n}\nconst char* s = \"x//y\";  // end")
    assert bench.code_only(src) != bench.code_only(src.replace("a + 1", "a + 2"))
    assert bench.code_only(src) != bench.code_only(src.replace('"x//y"', '"x/y"'))


def _counters(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                          "Counter_Value"])
        w.writeheader()
        for r in rows:
            w.writerow(r)


def _pass_rows(dispatches, counters_of):
    """CSV rows of one counter pass: dispatches is [(id, kernel, read, write)]."""
    rows = []
    for did, name, rd, wr in dispatches:
        for c, v in counters_of(rd, wr).items():
            rows.append({"Dispatch_Id": did, "Kernel_Name": name, "Counter_Name": c,
                         "Counter_Value": v})
    return rows


# what each pass reads for `rd` bytes read and `wr` written, on a device
# whose FETCH_SIZE sees half the bytes read (128-byte requests counted as 64)
PASSES = {
    "fetch": lambda rd, wr: {"FETCH_SIZE": rd / 2 / 1024},
    "write": lambda rd, wr: {"WRITE_SIZE": wr / 1024, "TCC_WRITE_SECTORS_sum": wr / 32},
    "reads": lambda rd, wr: {"TCC_EA0_RDREQ_128B_sum": rd / 128, "TCC_EA0_RDREQ_64B_sum": 0,
                             "TCC_EA0_RDREQ_32B_sum": 0},
}


def test_traffic_summary_calibrates_and_keeps_full_size_dispatches(tmp_path, monkeypatch):
    """Two full-size dispatches and a small one of each kernel: the small one
    does not dilute the per-launch figure; FETCH_SIZE is scaled by what it
    reads for the calibration copy, and the read-only, write-only and
    request-size figures are recorded against the known bytes."""
    numel, n, m = 1 << 20, 2, 4
    bf, bb = bench.algorithmic_bytes(n, m)
    fwd_rd, fwd_wr = 6 * numel, (bf - 6) * numel
    bench_disp = [("1", "fwd_lane_kernel<4,2>", fwd_rd, fwd_wr),
                  ("2", "fwd_lane_kernel<4,2>", fwd_rd, fwd_wr),
                  ("3", "fwd_lane_kernel<4,2>", fwd_rd / 50, fwd_wr / 50),
                  ("4", "bwd_lane_kernel<4,2>", 8 * numel, 4 * numel)]
    B = 1 << 30
    # the library splits the sum and the fill into several launches
    calib_disp = [("1", "roi::stream_copy_kernel(...)", B, B),
                  ("2", "at::native::reduce_kernel<...>", B / 4, 0),
                  ("3", "at::native::reduce_kernel<...>", 3 * B / 4, 0),
                  ("4", "at::native::FillFunctor<...>", 0, B / 2),
                  ("5", "at::native::FillFunctor<...>", 0, B / 2)]
    paths = []
    for who, disp in (("b", bench_disp), ("c", calib_disp)):
        for name, fn in PASSES.items():
            path = tmp_path / f"{who}_{name}.csv"
            _counters(path, _pass_rows(disp, fn))
            paths.append(str(path))
    out = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(out))
    assert bench.traffic_summary(paths[0:3], paths[3:6], B, numel, n, m) == 0
    rec = json.load(open(out))
    assert rec["fetch_scale"] == pytest.approx(2.0) and rec["write_scale"] == pytest.approx(1.0)
    cal = rec["calibration"]
    assert cal["reduce"]["fetch_size_over_known"] == pytest.approx(0.5)
    assert cal["reduce"]["read_requests_over_known"] == pytest.approx(1.0)
    assert cal["fill"]["write_size_over_known"] == pytest.approx(1.0)
    assert cal["fill"]["write_requests_over_known"] == pytest.approx(1.0)
    for k in ("fwd_lane_kernel", "bwd_lane_kernel"):
        assert rec["kernels"][k]["traffic_over_algorithmic"] == pytest.approx(1.0)
        assert rec["kernels"][k]["request_counters_over_algorithmic"] == pytest.approx(1.0)


def test_backward_flops_tally():
    """19 flops per entry and step plus 3 per weight (keys 6, upstream 1,
    output 1, less the 5 of the steps that have no successor)."""
    assert bench.backward_flops(1) == 22
    for n in range(1, 33):
        assert bench.backward_flops(n) == 19 * n + 3


def test_roofline_bound_follows_the_pattern():
    """m = 4 and 8 report the HBM roofline first, m = 16 and 32 the ALU one;
    each line carries both, and the ALU figure is the backward's flops over
    its event time against the fp32 vector peak."""
    numel = 1 << 30
    r = bench.step_rooflines("none", 2, 4, numel, 8.0, 12.0, None)
    assert r["roofline"]["bound"] == "hbm" and r["alu_roofline"]["bound"] == "alu"
    assert r["roofline"]["achieved"] == pytest.approx(12 * numel / 12e-3 / 1e9)
    r = bench.step_rooflines("none", 16, 32, numel, 3.0, 10.0, None)
    assert r["roofline"]["bound"] == "alu" and r["hbm_roofline"]["bound"] == "hbm"
    alu = r["roofline"]
    assert alu["achieved"] == pytest.approx(307 * numel / 10e-3 / 1e12)
    assert alu["frac"] == pytest.approx(alu["achieved"] / 157.3)
    assert alu["valu"] is None  # no counter record for an unknown workload


def test_valu_record_is_used_only_for_its_kernels():
    rec = json.load(open(bench.VALU_FILE))
    if rec["kernel_source_hash"] != bench.kernel_source_hash(bench.ALL_KERNEL_SOURCES):
        assert bench.measured_valu("qwen2.5-1.5b-stack-16:32") is None
        return
    wide = rec["workloads"]["qwen2.5-1.5b-stack-16:32"]["bwd_wide_kernel"]
    assert wide["valu_lane_insts_per_weight"] > bench.backward_flops(16) / 2
