"""bench.py's HBM-traffic bookkeeping on synthetic counter files (CPU only).

The FETCH_SIZE and WRITE_SIZE counters come per dispatch in KiB-like units; a
1 GiB device copy calibrates them. A scan in two passes is two scan-kernel
dispatches and one list-bound dispatch per batch, and its record must be their
sum; a one-pass scan is one dispatch.
"""
import csv
import json
import os

import pytest

import bench

HEADER = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id",
          "Grid_Size", "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size",
          "Scratch_Size", "VGPR_Count", "Accum_VGPR_Count", "SGPR_Count", "Counter_Name",
          "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def write_counters(path, rows):
    """rows: (kernel name, counter, value) in dispatch order."""
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.writer(f, quoting=csv.QUOTE_NONNUMERIC)
        w.writerow(HEADER)
        for i, (name, counter, value) in enumerate(rows):
            w.writerow([i, i, "Agent 1", 2, 1, 1, 1024, 7, name, 512, 0, 0, 128, 0, 80, counter,
                        float(value), 1000 * i, 1000 * i + 500])


SCAN = "void rb::(anonymous namespace)::rq_scan_kernel<12, 4, 1, 1, 4>(rb::ScanArgs)"
LIST_BOUND = "rb::(anonymous namespace)::list_bound_kernel(int const*, unsigned int const*, int)"
COPY = "__amd_rocclr_copyBuffer"


def calibrate(pmc, fetch_kib=524288.0, write_kib=1048576.0):
    write_counters(os.path.join(pmc, "copyfetch"), [(COPY, "FETCH_SIZE", fetch_kib)] * 3)
    write_counters(os.path.join(pmc, "copywrite"), [(COPY, "WRITE_SIZE", write_kib)] * 3)


def record(pmc, workload, capsys):
    bench.record_traffic(str(pmc), workload)
    capsys.readouterr()
    with open(os.path.join(pmc, "scan_traffic.json")) as f:
        return json.load(f)["workloads"][workload]


def test_one_pass_scan_is_one_dispatch(tmp_path, capsys):
    calibrate(tmp_path)
    # three batches of one dispatch each (one unit = 2,048 bytes fetched, 1,024 written)
    write_counters(tmp_path / "highload" / "fetch", [(SCAN, "FETCH_SIZE", 1000.0)] * 3)
    write_counters(tmp_path / "highload" / "write", [(SCAN, "WRITE_SIZE", 10.0)] * 3)
    r = record(tmp_path, "highload", capsys)
    assert r["passes"] == 1
    assert r["fetch_bytes"] == 1000 * 2048
    assert r["write_bytes"] == 10 * 1024
    assert r["bytes_per_launch"] == 1000 * 2048 + 10 * 1024
    assert r["sources_sha256"] == bench.scan_source_digest()


def test_two_pass_scan_sums_both_passes_and_the_list_bound(tmp_path, capsys):
    calibrate(tmp_path)
    # per batch: the first pass, the list bound, the second pass
    batch_f = [(SCAN, "FETCH_SIZE", 100.0), (LIST_BOUND, "FETCH_SIZE", 3.0),
               (SCAN, "FETCH_SIZE", 700.0)]
    batch_w = [(SCAN, "WRITE_SIZE", 4.0), (LIST_BOUND, "WRITE_SIZE", 1.0),
               (SCAN, "WRITE_SIZE", 6.0)]
    write_counters(tmp_path / "wide" / "fetch", batch_f * 2)
    write_counters(tmp_path / "wide" / "write", batch_w * 2)
    r = record(tmp_path, "wide", capsys)
    assert r["passes"] == 2
    assert r["fetch_bytes"] == (100 + 700 + 3) * 2048
    assert r["write_bytes"] == (4 + 6 + 1) * 1024


def test_records_of_other_workloads_are_kept(tmp_path, capsys):
    calibrate(tmp_path)
    for w in ("highload", "online"):
        write_counters(tmp_path / w / "fetch", [(SCAN, "FETCH_SIZE", 50.0)])
        write_counters(tmp_path / w / "write", [(SCAN, "WRITE_SIZE", 5.0)])
    record(tmp_path, "highload", capsys)
    r = record(tmp_path, "online", capsys)
    with open(tmp_path / "scan_traffic.json") as f:
        recs = json.load(f)["workloads"]
    assert recs["highload"]["fetch_bytes"] == r["fetch_bytes"] == 50 * 2048


def test_missing_scan_counters_are_an_error(tmp_path):
    calibrate(tmp_path)
    write_counters(tmp_path / "highload" / "fetch", [(LIST_BOUND, "FETCH_SIZE", 1.0)])
    write_counters(tmp_path / "highload" / "write", [(SCAN, "WRITE_SIZE", 1.0)])
    with pytest.raises(SystemExit):
        bench.record_traffic(str(tmp_path), "highload")
