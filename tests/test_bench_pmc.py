"""The traffic summary of bench.py: FETCH_SIZE / WRITE_SIZE counts (KiB per dispatch) are
scaled by what the counters read for the calibration copies, which are the first three
dispatches of the runtime's copy kernel; later, larger copies must not move the factors."""
import csv
import importlib.util
import json
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return m


def _write(path, counter, rows):
    with open(path, "w", newline="") as fh:
        wr = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                            "Counter_Value"])
        wr.writeheader()
        for disp, name, kib in rows:
            wr.writerow({"Dispatch_Id": disp, "Kernel_Name": name, "Counter_Name": counter,
                         "Counter_Value": kib})


def test_traffic_summary_calibrates_on_the_first_three_copies(tmp_path):
    b = _bench()
    copy, scan = "__amd_rocclr_copyBuffer", "void hsa::(anonymous namespace)::decode_scan<>(...)"
    calib_kib = b.CALIB_BYTES / 1024.0
    # the counters read half of each calibration copy's reads and all of its writes; a later
    # copy 16 times larger comes after the workload's first kernel
    fetch = [(1, copy, calib_kib / 2), (2, copy, calib_kib / 2), (3, copy, calib_kib / 2),
             (4, scan, 1000.0), (5, copy, 8 * calib_kib), (6, scan, 1000.0)]
    write = [(1, copy, calib_kib), (2, copy, calib_kib), (3, copy, calib_kib),
             (4, scan, 10.0), (5, copy, 16 * calib_kib), (6, scan, 30.0)]
    # rows out of dispatch order must not matter
    _write(tmp_path / "f.csv", "FETCH_SIZE", fetch[::-1])
    _write(tmp_path / "w.csv", "WRITE_SIZE", write)
    out = tmp_path / "t.json"
    b.pmc_summarize("decode_1M_bf16", str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), str(out))
    rec = json.loads(out.read_text())
    assert abs(rec["calibration"]["fetch_factor"] - 2.0) < 1e-9
    assert abs(rec["calibration"]["write_factor"] - 1.0) < 1e-9
    k = rec["kernels"]["decode_scan"]
    assert k["dispatches"] == 2
    assert k["fetch_bytes_per_launch"] == round(1000.0 * 1024 * 2.0)
    assert k["write_bytes_per_launch"] == round(20.0 * 1024)
    assert k["hbm_bytes_per_launch"] == k["fetch_bytes_per_launch"] + k["write_bytes_per_launch"]
    assert rec["source_sha256"] == b.source_digest()


def test_traffic_summary_adds_kernels_that_share_a_name(tmp_path):
    """stream_rowcount and stream_plan both report as 'plan': their bytes add up per launch of
    the stage instead of the later one replacing the earlier."""
    b = _bench()
    copy = "__amd_rocclr_copyBuffer"
    rc = "void hsa::(anonymous namespace)::stream_rowcount(...)"
    pl = "void hsa::(anonymous namespace)::stream_plan(...)"
    calib_kib = b.CALIB_BYTES / 1024.0
    fetch = [(1, copy, calib_kib / 2), (2, copy, calib_kib / 2), (3, copy, calib_kib / 2),
             (4, rc, 100.0), (5, pl, 3.0), (6, rc, 100.0), (7, pl, 5.0)]
    write = [(1, copy, calib_kib), (2, copy, calib_kib), (3, copy, calib_kib),
             (4, rc, 1.0), (5, pl, 2.0), (6, rc, 1.0), (7, pl, 2.0)]
    _write(tmp_path / "f.csv", "FETCH_SIZE", fetch)
    _write(tmp_path / "w.csv", "WRITE_SIZE", write)
    out = tmp_path / "t.json"
    b.pmc_summarize("L4K_bf16", str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), str(out))
    rec = json.loads(out.read_text())
    k = rec["kernels"]["plan"]
    assert k["dispatches"] == 2
    assert k["fetch_bytes_per_launch"] == round((100.0 + 4.0) * 1024 * 2.0)
    assert k["write_bytes_per_launch"] == round(3.0 * 1024)
    assert rec["by_kernel"][pl]["fetch_bytes_per_launch"] == round(4.0 * 1024 * 2.0)
    assert rec["by_kernel"][rc]["short"] == "plan"
