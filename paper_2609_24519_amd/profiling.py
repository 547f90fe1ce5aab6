"""Summaries of rocprofv3 output for the profiles/ folder.

    python -m paper_2609_24519_amd.profiling stats  <kernel_stats.csv> <out.md> "<command>"
    python -m paper_2609_24519_amd.profiling traffic <fetch_counter_collection.csv> \\
        <write_counter_collection.csv> <out.json> <out.md> "<fetch command>" "<write command>"

``stats`` turns a ``--kernel-trace --stats`` kernel_stats.csv into a short
Markdown table.  ``traffic`` takes two ``--pmc`` runs (FETCH_SIZE, then
WRITE_SIZE, each in KiB per dispatch) of a command that also ran a plain
device copy of a known size (``bench.py --calibrate-copy``), scales every
kernel's counters by what the counters read for that copy, and records the
per-dispatch HBM bytes of the GEMM together with a hash of the kernel source
they were taken on, so that a later change to the kernel makes them stale.
"""
import csv
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCE = os.path.join(HERE, "csrc", "awe_kernels.hip")
COPY_BYTES = 1 << 30  # bench.py --calibrate-copy copies 1 GiB


def kernel_source_hash():
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def _short(name):
    for key in ("gemm_kernel", "encode_kernel<true>", "encode_kernel<false>", "fill_zero_kernel"):
        if key in name:
            return {"encode_kernel<true>": "encode_kernel (B side, transposed)",
                    "encode_kernel<false>": "encode_kernel (A side)"}.get(key, key)
    return name[:60]


def stats(csv_path, out_md, command):
    rows = list(csv.DictReader(open(csv_path)))
    lines = ["# Kernel time summary (rocprofv3 --kernel-trace --stats)", "",
             "Command: `%s`" % command, "",
             "| kernel | calls | average (us) | min (us) | max (us) | share |",
             "|---|---|---|---|---|---|"]
    for r in rows:
        lines.append("| %s | %s | %.1f | %.1f | %.1f | %.1f%% |" % (
            _short(r["Name"]), r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
            float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


def _per_kernel(csv_path, counter):
    out = {}
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] != counter:
            continue
        out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]) * 1024.0)
    return out


def traffic(fetch_csv, write_csv, out_json, out_md, fetch_cmd, write_cmd):
    fetch = _per_kernel(fetch_csv, "FETCH_SIZE")
    write = _per_kernel(write_csv, "WRITE_SIZE")
    copy_name = [k for k in fetch if "gemm_kernel" not in k and "encode_kernel" not in k
                 and max(fetch[k]) > 0.5 * COPY_BYTES]
    if not copy_name:
        raise SystemExit("no copy kernel of the calibration size found")
    cname = copy_name[0]
    f_scale = COPY_BYTES / max(fetch[cname])
    w_scale = COPY_BYTES / max(write[cname])
    res = {"kernel_source_sha": kernel_source_hash(), "copy_kernel": cname[:80],
           "fetch_scale": f_scale, "write_scale": w_scale, "kernels": {}}
    lines = ["# HBM traffic per dispatch (rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE)", "",
             "FETCH command: `%s`" % fetch_cmd, "", "WRITE command: `%s`" % write_cmd, "",
             "Scale factors from the 1 GiB device copy (%s): fetch x%.4f, write x%.4f." % (
                 _short(cname), f_scale, w_scale), "",
             "| kernel | dispatches | fetch (MB, scaled) | write (MB, scaled) |", "|---|---|---|---|"]
    for k in fetch:
        if k == cname:
            continue
        fb = sum(fetch[k]) / len(fetch[k]) * f_scale
        wb = (sum(write.get(k, [0])) / max(len(write.get(k, [1])), 1)) * w_scale
        res["kernels"][_short(k)] = {"fetch_bytes": fb, "write_bytes": wb, "dispatches": len(fetch[k])}
        lines.append("| %s | %d | %.1f | %.1f |" % (_short(k), len(fetch[k]), fb / 1e6, wb / 1e6))
    lines += ["", "Kernel source hash: %s" % res["kernel_source_sha"]]
    with open(out_json, "w") as f:
        json.dump(res, f, indent=1)
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    if sys.argv[1] == "stats":
        stats(sys.argv[2], sys.argv[3], sys.argv[4])
    elif sys.argv[1] == "traffic":
        traffic(*sys.argv[2:8])
    else:
        raise SystemExit(__doc__)
