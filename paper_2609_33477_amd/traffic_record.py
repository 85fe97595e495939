"""Writes profiles/traffic_<workload>.json from two rocprofv3 --pmc runs of
bench.py (FETCH_SIZE, then WRITE_SIZE) and the same two counters read on
bench.py --copy-probe, a plain copy that reads and writes exactly 1 GiB.

    python -m paper_2609_33477_amd.traffic_record <fetch.csv> <write.csv> \
        <copy_fetch.csv> <copy_write.csv> [workload]

Each counter is averaged per dispatch of a kernel (KiB), then scaled by
what it reads for the copy of known size; the record carries the hash of
the sources each kernel is built from (bench.py drops it when they change).
"""
import csv
import hashlib
import json
import os
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")

# kernel key -> (name fragment in the trace, sources)
KERNELS = {
    "proj_conv": ("proj_conv_kernel", ("proj_conv.hip", "tail_q.hpp", "sr_device.hpp", "sr_internal.hpp")),
    "gdn_scan": ("gdn_scan_bf16_kernel", ("gdn_scan_bf16.hip", "sr_device.hpp", "sr_internal.hpp")),
    "decay_state": ("decay_state_kernel", ("decay_state.hip", "sr_device.hpp", "sr_internal.hpp")),
    "anchor_gather": ("gather_kernel", ("sidecar.hip", "sr_internal.hpp")),
    "anchor_write": ("write_kernel", ("sidecar.hip", "sr_internal.hpp")),
}
COPY_BYTES = 1 << 30


def source_sha256(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def per_dispatch_kib(path, fragment):
    vals = [float(r["Counter_Value"]) for r in csv.DictReader(open(path)) if fragment in r["Kernel_Name"]]
    if not vals:
        raise SystemExit(f"no dispatch of {fragment} in {path}")
    return sum(vals) / len(vals), len(vals)


def make_record(fetch, write, cfetch, cwrite, workload="varlen16"):
    """The traffic record from the four counter CSV files."""
    cf, _ = per_dispatch_kib(cfetch, "elementwise")
    cw, _ = per_dispatch_kib(cwrite, "elementwise")
    fscale, wscale = COPY_BYTES / (cf * 1024), COPY_BYTES / (cw * 1024)
    rec = {"workload": workload,
           "copy_probe": {"read_bytes": COPY_BYTES, "write_bytes": COPY_BYTES, "fetch_kib": cf, "write_kib": cw,
                          "fetch_scale": fscale, "write_scale": wscale},
           "kernels": {}}
    for key, (frag, files) in KERNELS.items():
        if not any(frag in r["Kernel_Name"] for r in csv.DictReader(open(fetch))):
            continue   # not launched by this workload
        fk, n = per_dispatch_kib(fetch, frag)
        wk, _ = per_dispatch_kib(write, frag)
        fb, wb = fk * 1024 * fscale, wk * 1024 * wscale
        rec["kernels"][key] = {"dispatches": n, "fetch_kib_raw": fk, "write_kib_raw": wk, "fetch_bytes": int(fb),
                               "write_bytes": int(wb), "traffic_bytes": int(fb + wb),
                               "source_sha256": source_sha256(files)}
    return rec


def main():
    fetch, write, cfetch, cwrite = sys.argv[1:5]
    workload = sys.argv[5] if len(sys.argv) > 5 else "varlen16"
    rec = make_record(fetch, write, cfetch, cwrite, workload)
    out = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    with open(out, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec, indent=1))


if __name__ == "__main__":
    main()
