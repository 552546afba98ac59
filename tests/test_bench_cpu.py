"""bench.py's host-side contract, without a GPU: more than one GPU is refused with a
message, and the HBM-traffic summary rescales each counter by what it read for the
calibration copy and averages it over the conv launches between the two copies that
bench.py runs around its first traced pass."""
import csv
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

FIELDS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
          "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
          "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _write(d, counter, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "x_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for i, (name, kib) in enumerate(rows):
            w.writerow({k: 0 for k in FIELDS} | {"Dispatch_Id": i + 1, "Kernel_Name": name,
                                                 "Counter_Name": counter, "Counter_Value": kib})


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_pmc_summary_rescales_by_the_copy(tmp_path):
    conv = "void rafiki::conv_mfma_kernel<128, 128, 2, 2, 3, true, 8, false, false, 0>(rafiki::ConvArgs)"
    copy = "void at::native::elementwise_kernel<mul>(x)"
    fill = "void at::native::vectorized_elementwise_kernel<fill>(x)"
    copy_bytes = 1 << 20
    # the buffer's fill (writes only), timed-step conv launches before the first copy and
    # the concurrent traced pass after the second are ignored; the copy read half its bytes
    _write(str(tmp_path / "f"), "FETCH_SIZE", [(conv, 999.0), (fill, 0.5), (conv, 777.0), (copy, 512.0),
                                                (conv, 100.0), ("void rafiki::pool(x)", 7.0), (conv, 300.0),
                                                (copy, 512.0), (conv, 5000.0)])
    _write(str(tmp_path / "w"), "WRITE_SIZE", [(conv, 5.0), (fill, 1024.0), (conv, 77.0), (copy, 1024.0),
                                                (conv, 40.0), (conv, 60.0), (copy, 1024.0), (conv, 900.0)])
    out = bench.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"), copy_bytes)
    assert out["fetch"]["launches"] == 2 and out["write"]["launches"] == 2
    assert abs(out["fetch"]["scale"] - 2.0) < 1e-12 and abs(out["write"]["scale"] - 1.0) < 1e-12
    assert abs(out["fetch"]["bytes_per_launch"] - 2.0 * 200.0 * 1024) < 1e-6
    assert abs(out["write"]["bytes_per_launch"] - 50.0 * 1024) < 1e-6
    assert abs(out["traffic_bytes_per_launch"] - (400.0 + 50.0) * 1024) < 1e-6
    assert out["source_sha256"] == bench.kernel_source_sha()


def test_pmc_summary_needs_both_marker_copies(tmp_path):
    conv = "void rafiki::conv_mfma_kernel<128, 128, 2, 2, 3, true, 8, false, false, 0>(rafiki::ConvArgs)"
    _write(str(tmp_path / "f"), "FETCH_SIZE", [("copy", 512.0), (conv, 100.0)])
    _write(str(tmp_path / "w"), "WRITE_SIZE", [("copy", 1024.0), (conv, 40.0)])
    try:
        bench.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"), 1 << 20)
    except SystemExit as e:
        assert "marker" in str(e)
    else:
        raise AssertionError("a single copy was accepted")


def test_pmc_summary_counts_both_conv_kernels(tmp_path):
    """The traced class conv_mfma holds the GEMM and the direct 3x3 launches; the
    counter summary averages over both."""
    gemm = "void rafiki::conv_mfma_kernel<128, 128, 2, 2, 3, true, 8, false, false, 0>(rafiki::ConvArgs)"
    direct = "rafiki::conv_direct_kernel(rafiki::ConvArgs)"
    copy = "void at::native::elementwise_kernel<mul>(x)"
    _write(str(tmp_path / "f"), "FETCH_SIZE", [(copy, 512.0), (gemm, 100.0), (direct, 300.0), (copy, 512.0)])
    _write(str(tmp_path / "w"), "WRITE_SIZE", [(copy, 1024.0), (gemm, 10.0), (direct, 30.0), (copy, 1024.0)])
    out = bench.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"), 1 << 20)
    assert out["fetch"]["launches"] == 2 and out["write"]["launches"] == 2
    assert abs(out["fetch"]["bytes_per_launch"] - 2.0 * 200.0 * 1024) < 1e-6
    assert abs(out["write"]["bytes_per_launch"] - 20.0 * 1024) < 1e-6


def test_source_hash_ignores_comments_not_code():
    """The stored traffic counters stay valid across comment edits, not code edits."""
    src = "int f(int a) {  // add one\n  /* the sum */ return a + 1;\n}\n"
    assert bench.strip_comments(src) == bench.strip_comments("// header\nint f(int a) {\n\n  return a + 1;  }\n".replace("  }", "\n}"))
    assert bench.strip_comments(src) != bench.strip_comments(src.replace("a + 1", "a + 2"))
    assert "add one" not in bench.strip_comments(src) and "sum" not in bench.strip_comments(src)

