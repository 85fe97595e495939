"""The traffic record that bench.py reports as roofline.traffic: per-dispatch
averages of the counter CSVs, scaled by the copy probe, keyed to the hash of
the kernel sources (bench.py drops a record taken on other sources)."""
import csv
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2609_33477_amd import traffic_record as tr  # noqa: E402
import bench  # noqa: E402

FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]


def _csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, FIELDS)
        w.writeheader()
        for i, (name, counter, value) in enumerate(rows):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value})


def test_record_scales_by_the_copy_probe_and_averages_dispatches(tmp_path):
    proj, scan = "void sr::proj_conv_kernel<sr::bf16_t, 128>(x)", "void sr::gdn_scan_bf16_kernel<128>(y)"
    copy = "void at::native::vectorized_elementwise_kernel<4>(z)"
    _csv(tmp_path / "f.csv", [(proj, "FETCH_SIZE", 100.0), (proj, "FETCH_SIZE", 300.0), (scan, "FETCH_SIZE", 50.0),
                              (copy, "FETCH_SIZE", 1.0)])
    _csv(tmp_path / "w.csv", [(proj, "WRITE_SIZE", 40.0), (proj, "WRITE_SIZE", 40.0), (scan, "WRITE_SIZE", 8.0)])
    # the copy reads and writes 1 GiB: FETCH_SIZE reports half of it, WRITE_SIZE all of it
    _csv(tmp_path / "cf.csv", [(copy, "FETCH_SIZE", 524288.0), (copy, "FETCH_SIZE", 524288.0)])
    _csv(tmp_path / "cw.csv", [(copy, "WRITE_SIZE", 1048576.0)])
    rec = tr.make_record(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), str(tmp_path / "cf.csv"),
                         str(tmp_path / "cw.csv"))
    assert rec["copy_probe"]["fetch_scale"] == 2.0 and rec["copy_probe"]["write_scale"] == 1.0
    p = rec["kernels"]["proj_conv"]
    assert p["dispatches"] == 2 and p["fetch_kib_raw"] == 200.0 and p["write_kib_raw"] == 40.0
    assert p["fetch_bytes"] == 200 * 1024 * 2 and p["write_bytes"] == 40 * 1024
    assert p["traffic_bytes"] == p["fetch_bytes"] + p["write_bytes"]
    assert rec["kernels"]["gdn_scan"]["traffic_bytes"] == 50 * 1024 * 2 + 8 * 1024


def test_record_hashes_match_what_bench_checks():
    for key in tr.KERNELS:
        assert tr.source_sha256(tr.KERNELS[key][1]) == bench.kernel_source_hash(key)
