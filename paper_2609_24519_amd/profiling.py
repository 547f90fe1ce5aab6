"""Summaries of rocprofv3 output for the profiles/ folder.

    python -m paper_2609_24519_amd.profiling stats  <kernel_stats.csv | kernel_trace.csv> <out.md> \
        "<command>" [<warm-up dispatches to skip, kernel_trace.csv only>]
    python -m paper_2609_24519_amd.profiling traffic <fetch_counter_collection.csv> \\
        <write_counter_collection.csv> <out.json> <out.md> "<fetch command>" "<write command>"
    python -m paper_2609_24519_amd.profiling counters <out.md> <fp4_flop_per_gemm> \\
        "<command>" <counter_collection.csv> [<counter_collection.csv> ...]
    python -m paper_2609_24519_amd.profiling clock <bench output> <out.md> "<command>"

``stats`` turns a ``--kernel-trace --stats`` kernel_stats.csv into a short
Markdown table.  ``traffic`` takes two ``--pmc`` runs (FETCH_SIZE, then
WRITE_SIZE, each in KiB per dispatch) of a command that also ran a plain
device copy of a known size (``bench.py --calibrate-copy``), scales every
kernel's counters by what the counters read for that copy, and records the
per-dispatch HBM bytes of the GEMM together with a hash of the kernel sources
they were taken on (the kernels, the GEMM's addressing header and the encoders'
plane packing), so that a
later change to either makes them stale.
``counters`` summarises one or more ``--pmc`` passes over the same command:
per kernel the FP4 MFMA operation count (checked against the algorithmic
r 2MNK), MFMA busy cycles, LDS bank conflicts and activity, L2 hit rate and
request latency.  ``clock`` renders the engine clocks and socket power that
``bench.py --clock-sample`` read under each load.
"""
import csv
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
# the GEMM's kernel code and its addressing (tile configurations, copy / LDS / fragment offsets)
KERNEL_SOURCES = tuple(os.path.join(HERE, "csrc", f) for f in ("awe_kernels.hip", "gemm_layout.h", "plane_pack.h"))
COPY_BYTES = 1 << 30  # bench.py --calibrate-copy copies 1 GiB


def kernel_source_hash():
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


_LABELS = (  # first match wins
    ("residue_encode_kernel<true>", "residue_encode_kernel (B side, transposed)"),
    ("residue_encode_kernel<false>", "residue_encode_kernel (A side)"),
    ("residues_kernel", "residues_kernel"),
    ("crt_kernel", "crt_kernel"),
    ("gemm_group_kernel", "gemm_group_kernel"),
    ("gemm_kernel", "gemm_kernel"),
    ("encode16_kernel<true>", "encode16_kernel (B side, transposed)"),
    ("encode16_kernel<false>", "encode16_kernel (A side)"),
    ("encode_kernel<true>", "encode_kernel (B side, transposed)"),
    ("encode_kernel<false>", "encode_kernel (A side)"),
    ("zero_tiles_kernel", "zero_tiles_kernel"),
    ("fill_zero_kernel", "fill_zero_kernel"),
    ("distribution_elementwise", "input generation (torch random)"),
)


def _short(name):
    for key, label in _LABELS:
        if key in name:
            return label
    return name[:60]


def stats(csv_path, out_md, command, skip=0):
    """Per-kernel times from a kernel_stats.csv, or from a kernel_trace.csv with the first
    ``skip`` dispatches of every kernel left out (the untimed warm-up steps of the command,
    so that the averages cover the same dispatches as the command's own timing)."""
    rows = list(csv.DictReader(open(csv_path)))
    lines = ["# Kernel time summary (rocprofv3 --kernel-trace --stats)", "",
             "Command: `%s`" % command, ""]
    if rows and "Start_Timestamp" in rows[0]:
        per = {}
        for r in rows:
            per.setdefault(r["Kernel_Name"], []).append(
                (int(r["Start_Timestamp"]), (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3))
        if skip:
            lines += ["Per-dispatch durations from the kernel trace, the first %d dispatches of each kernel "
                      "(the warm-up steps) left out." % skip, ""]
        else:
            lines += ["Per-dispatch durations from the kernel trace, every dispatch (the command's own warm-up "
                      "calls included).", ""]
        table = []
        for name, d in per.items():
            d = [us for _, us in sorted(d)][skip:]
            if d:
                table.append((name, len(d), sum(d) / len(d), min(d), max(d), sum(d)))
        total = sum(t[5] for t in table) or 1.0
        rows_out = [(n, c, a, lo, hi, 100.0 * t / total) for n, c, a, lo, hi, t in
                    sorted(table, key=lambda t: -t[5])]
    else:
        rows_out = [(r["Name"], int(r["Calls"]), float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
                     float(r["MaxNs"]) / 1e3, float(r["Percentage"])) for r in rows]
    lines += ["| kernel | calls | average (us) | min (us) | max (us) | share |", "|---|---|---|---|---|---|"]
    for n, c, a, lo, hi, pct in rows_out:
        lines.append("| %s | %d | %.1f | %.1f | %.1f | %.1f%% |" % (_short(n), c, a, lo, hi, pct))
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


def _dispatch_counters(paths):
    """{kernel: {"n": dispatches, counter: mean per dispatch, "_res": resources}} over CSV files."""
    per = {}
    for path in paths:
        seen = {}
        for r in csv.DictReader(open(path)):
            key = (path, r["Dispatch_Id"])
            d = seen.setdefault(key, {"kernel": r["Kernel_Name"], "vals": {}, "res": {
                "arch_vgpr": r.get("Arch_VGPR_Count", r.get("VGPR_Count", "")),
                "accum_vgpr": r.get("Accum_VGPR_Count", ""), "sgpr": r.get("SGPR_Count", ""),
                "lds_bytes": r.get("LDS_Block_Size", ""), "scratch": r.get("Scratch_Size", ""),
                "ns": float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
                if r.get("End_Timestamp") else 0.0}})
            d["vals"][r["Counter_Name"]] = d["vals"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        for d in seen.values():
            k = per.setdefault(_short(d["kernel"]), {"sums": {}, "cnt": {}, "res": d["res"], "ns": []})
            k["ns"].append(d["res"]["ns"])
            for c, v in d["vals"].items():
                k["sums"][c] = k["sums"].get(c, 0.0) + v
                k["cnt"][c] = k["cnt"].get(c, 0) + 1
    out = {}
    for name, k in per.items():
        mean = {c: k["sums"][c] / k["cnt"][c] for c in k["sums"]}
        mean["_ns"] = sum(k["ns"]) / len(k["ns"])
        mean["_res"] = k["res"]
        out[name] = mean
    return out


# Engine clock under the GEMM (amd-smi, `bench.py --clock-sample`) and the CU count, for
# turning per-chip cycle counters into per-CU rates and shares of the kernel's cycles.
CLOCK_HZ = 2.05e9
CUS = 256


def counters(out_md, fp4_flop, command, paths):
    fp4_flop = float(fp4_flop)
    data = _dispatch_counters(paths)
    lines = ["# GEMM counters (rocprofv3 --pmc, one pass per counter group)", "",
             "Command (each pass): `%s`" % command, "",
             "Per-dispatch means.  MOPS counts units of 512 FLOP; a 32x32x64 FP4 MFMA is",
             "256 MOPS and keeps its SIMD busy 32 cycles.  Expected FP4 work per GEMM",
             "dispatch: r 2MNK = %.4g FLOP." % fp4_flop, ""]
    for name, m in data.items():
        if "gemm_kernel" not in name:
            continue
        lines += ["## %s" % name, "", "| quantity | value |", "|---|---|"]
        lines.append("| duration (us) | %.1f |" % (m["_ns"] / 1e3))
        mops = m.get("SQ_INSTS_VALU_MFMA_MOPS_F6F4")
        if mops is not None:
            lines.append("| FP4 MFMA FLOP (MOPS x 512) | %.6g (expected %.6g, ratio %.6f) |" % (
                mops * 512, fp4_flop, mops * 512 / fp4_flop))
            busy = m.get("SQ_VALU_MFMA_BUSY_CYCLES")
            if busy is not None:
                lines.append("| MFMA busy SIMD-cycles | %.6g (= %.3f x 32 per MFMA) |" % (
                    busy, busy / (mops / 256.0) / 32.0 if mops else 0.0))
        for c, label in (("SQ_LDS_BANK_CONFLICT", "LDS bank-conflict cycles"),
                         ("SQ_LDS_IDX_ACTIVE", "LDS active cycles"),
                         ("SQ_WAIT_INST_LDS", "wave-cycles waiting on LDS instructions"),
                         ("SQ_BUSY_CYCLES", "SQ busy cycles"), ("GRBM_GUI_ACTIVE", "GRBM GUI active")):
            if c in m:
                lines.append("| %s (%s) | %.6g |" % (label, c, m[c]))
        if "TCC_HIT" in m and "TCC_MISS" in m:
            lines.append("| L2 hit rate (TCC_HIT / (HIT + MISS)) | %.3f |" % (
                m["TCC_HIT"] / max(m["TCC_HIT"] + m["TCC_MISS"], 1.0)))
        if "TCP_TCC_READ_REQ" in m:
            lines.append("| L1 -> L2 read requests (x 128 B) | %.4g (%.2f GB) |" % (
                m["TCP_TCC_READ_REQ"], m["TCP_TCC_READ_REQ"] * 128 / 1e9))
            if "TCP_TCC_READ_REQ_LATENCY" in m:
                lines.append("| mean L2 read latency (cycles) | %.0f |" % (
                    m["TCP_TCC_READ_REQ_LATENCY"] / max(m["TCP_TCC_READ_REQ"], 1.0)))
                # Little's law: requests in flight = total latency / elapsed cycles
                cyc = m["_ns"] * 1e-9 * CLOCK_HZ
                lines.append("| L1 -> L2 reads in flight per CU at %.2f GHz (total latency / cycles / CUs) "
                             "| %.1f |" % (CLOCK_HZ / 1e9, m["TCP_TCC_READ_REQ_LATENCY"] / cyc / CUS))
        for c, label in (("TCP_PENDING_STALL_CYCLES", "L1 cycles stalled on pending misses, per CU"),
                         ("TA_ADDR_STALLED_BY_TC_CYCLES", "address unit cycles stalled by L1, per CU")):
            if c in m:
                cyc = m["_ns"] * 1e-9 * CLOCK_HZ
                lines.append("| %s (%s) | %.4g (%.0f %% of the cycles at %.2f GHz) |" % (
                    label, c, m[c] / CUS, 100.0 * m[c] / CUS / cyc, CLOCK_HZ / 1e9))
        lines.append("")
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


CLOCK_LOADS = (
    ("gemm", "AWE6 GEMM (awe_gemm_planes, 8192^3, 6 FP4 products)"),
    ("gemm_e2m3", "E2M3 GEMM, 3 products (FP6 Karatsuba, 8192^3)"),
    ("gemm_e2m3_scaled", "E2M3 GEMM, 4 products with the weights in the scales (8192^3)"),
    ("probe_static", "FP4 MFMA probe, constant operands (8 waves/CU)"),
    ("probe_varied", "FP4 MFMA probe, operands changing between MFMAs (8 waves/CU)"),
    ("probe_varied_e2m3", "E2M3 MFMA probe, operands changing between MFMAs (8 waves/CU)"),
)


def clock(bench_log, out_md, command):
    """The `clock_under_load` field of a `bench.py --clock-sample` line as a table."""
    line = None
    with open(bench_log) as f:
        for l in f:
            if l.startswith("{") and "clock_under_load" in l:
                line = json.loads(l)
    if line is None:
        raise SystemExit("no bench line with clock_under_load in " + bench_log)
    loads = line["clock_under_load"]
    lines = ["# Engine clock and socket power under load (amd-smi metric -c -p)", "",
             "Command: `%s`" % command, "",
             "Each load runs in a loop; `amd-smi metric -c -p` is read once 2 s after it starts (a child",
             "process started before the GPU is touched).  Clock = mean of the 8 XCDs' GFX clocks; the",
             "peak at that clock is 256 CUs x 16,384 FP4 (or FP6) FLOP per clock; rates count the",
             "products' FP4/FP6 work, r 2MNK per GEMM.", "",
             "| load | GFX clock mean (min..max) MHz | socket power W | TFLOP/s | fraction of the peak at that "
             "clock | fraction of the 10.1 PF spec |", "|---|---|---|---|---|---|"]
    for key, label in CLOCK_LOADS:
        r = loads.get(key)
        if not r or "fp4_TFLOPs" not in r:
            continue
        clk = "%.0f (%.0f..%.0f)" % (r["gfx_clock_mhz_mean"], r["gfx_clock_mhz_min"], r["gfx_clock_mhz_max"]) \
            if "gfx_clock_mhz_mean" in r else "n/a"
        pw = "%.0f" % r["socket_power_w"] if r.get("socket_power_w") is not None else "n/a"
        fr = "%.3f" % r["frac_of_peak_at_this_clock"] if "frac_of_peak_at_this_clock" in r else "n/a"
        lines.append("| %s | %s | %s | %.1f | %s | %.3f |" % (label, clk, pw, r["fp4_TFLOPs"], fr,
                                                            r["fp4_TFLOPs"] / 10100.0))
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    if sys.argv[1] == "stats":
        stats(sys.argv[2], sys.argv[3], sys.argv[4], int(sys.argv[5]) if len(sys.argv) > 5 else 0)
    elif sys.argv[1] == "traffic":
        traffic(*sys.argv[2:8])
    elif sys.argv[1] == "counters":
        counters(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5:])
    elif sys.argv[1] == "clock":
        clock(sys.argv[2], sys.argv[3], sys.argv[4])
    else:
        raise SystemExit(__doc__)
