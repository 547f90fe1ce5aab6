"""Benchmark of the exact INT8 x INT8 product as 6 FP4 GEMMs (AWE) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

One step is the whole hot path on one batch of resident synthetic input:
encode A, encode B, the r FP4 products with their fused reconstruction
(the calls awe_encode, awe_encode, awe_gemm_planes, i.e. awe_gemm_exact).
The workload is M = N = K = 8192 with int8 entries uniform in [-128, 127]
(seed 0) and int32 C.  Printed: one JSON line with the end-to-end exact TOPS
as ``value``, the roofline of the dominant kernel (the GEMM) from HIP events
on its stream, the 9-product base-13 baseline, the 2 FP8 + 1 FP4 scheme, the
3-product {0,+-1} x INT8 GEMM, the 12-product FP16-significand GEMM, the
native INT8 MFMA GEMM
(hipBLASLt through torch._int_mm), one plain MXFP4 GEMM of the vendor library
(torch._scaled_mm), the residue-number-system route for 53-bit
integers (the integer layer of Ozaki scheme II) and the sustained rate of the
FP4 MFMA alone timed in the same run as context, the other workloads (INT4 x INT8 in 4
products at 8192^3; C mod m at 4096^3 for every modulus of the FP64-significand residue set;
the 4096 x 4096 x 65,536 accumulation stress with int64 C), and the oracle timed on the
host's cores on a bounded sample.  ``--only <workload>`` times one of those workloads alone.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "exact INT8xINT8 GEMM TOPS at 8192^3 (6 FP4 GEMMs) + % of FP4 MFMA peak"
FP4_PEAK_TFLOPS = 10100.0  # MI355X dense MXFP4 MFMA
HBM_PEAK_GBS = 8000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    # the first ~15 GEMMs of a process run ~10 % slower (clocks still settling), so the default
    # warms up past them
    p.add_argument("--warmup", type=int, default=30)
    p.add_argument("--size", type=int, default=8192)
    p.add_argument("--no-cpu", action="store_true", help="skip the oracle timing")
    p.add_argument("--no-context", action="store_true", help="skip base-13 and INT8 context")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="also run a plain 1 GiB device copy (the reference for rocprofv3 byte counters)")
    p.add_argument("--only", choices=sorted(WORKLOADS), default=None,
                   help="only time this one workload of the other configurations and print its fields "
                        "(for kernel traces of that workload)")
    p.add_argument("--ozaki2-only", type=int, default=0, metavar="CALLS",
                   help="only run the residue-number-system route (the ozaki2_int53 context) CALLS "
                        "times and print its timing (for kernel traces of that route)")
    p.add_argument("--clock-sample", action="store_true",
                   help="also read the engine clocks and socket power (amd-smi) while the GEMM and the "
                        "MFMA probes run in a loop")
    return p.parse_args()


WORKLOADS = ("awe4_int4xint8", "residues_per_modulus", "stress_65536")

CLOCK_PHASES = ("gemm", "gemm_e2m3", "gemm_e2m3_scaled", "probe_static", "probe_varied", "probe_varied_e2m3")


def start_clock_sampler(tmpdir):
    """Child process (started before the GPU is touched) that waits for each phase's marker
    file, lets the load settle for 2 s, reads `amd-smi metric -c -p` once and signals done."""
    import shutil
    import subprocess

    smi = "/opt/rocm/bin/amd-smi" if os.path.exists("/opt/rocm/bin/amd-smi") else shutil.which("amd-smi")
    if not smi:
        return None
    lines = []
    for ph in CLOCK_PHASES:
        lines.append('for i in $(seq 600); do [ -f "{d}/go_{p}" ] && break; sleep 0.1; done; sleep 2; '
                     'timeout 20 "{smi}" metric -c -p > "{d}/smi_{p}.txt" 2>&1; touch "{d}/done_{p}"'
                     .format(d=tmpdir, p=ph, smi=smi))
    return subprocess.Popen(["bash", "-c", "; ".join(lines)], stdout=subprocess.DEVNULL,
                            stderr=subprocess.DEVNULL)


def read_smi(path):
    """Mean GFX (per-XCD) engine clock and socket power from an `amd-smi metric -c -p` dump."""
    import re

    try:
        text = open(path).read()
    except OSError:
        return {"error": "no amd-smi output"}
    clks = [int(m.group(2)) for m in re.finditer(r"GFX_(\d+):\s*\n\s*CLK:\s*(\d+)\s*MHz", text)]
    pw = re.search(r"SOCKET_POWER:\s*([\d.]+)\s*W", text)
    if not clks:
        return {"error": "no GFX clocks in amd-smi output"}
    return {"gfx_clock_mhz_mean": round(sum(clks) / len(clks), 1), "gfx_clock_mhz_min": min(clks),
            "gfx_clock_mhz_max": max(clks), "socket_power_w": float(pw.group(1)) if pw else None}


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path; use --gpus 1",
              file=sys.stderr)
        sys.exit(2)
    sampler = None
    if args.clock_sample:
        import tempfile
        clock_dir = tempfile.mkdtemp(prefix="awe_clock_")
        sampler = start_clock_sampler(clock_dir)
    import numpy as np
    import torch

    from paper_2609_24519_amd import awe, inputs

    if not os.path.exists(awe.LIB_PATH):
        from paper_2609_24519_amd import build as hip_build
        hip_build.build()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    if args.ozaki2_only:
        print(json.dumps({"ozaki2_int53": ozaki2_context(dev, reps=args.ozaki2_only)}), flush=True)
        return
    if args.only:
        print(json.dumps({args.only: WORKLOAD_FNS[args.only](dev)}), flush=True)
        return
    M = N = K = args.size
    A_h, B_h = inputs.int8_pair(M, N, K, seed=0)
    A = torch.from_numpy(A_h).to(dev)
    B = torch.from_numpy(B_h).to(dev)
    C = torch.empty((M, N), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()

    def setup(enc):
        info = awe.get_encoding_info(enc)
        pa = torch.empty(awe.plane_bytes(enc, 0, awe.SIDE_A, M, K), dtype=torch.uint8, device=dev)
        pb = torch.empty(awe.plane_bytes(enc, 0, awe.SIDE_B, N, K), dtype=torch.uint8, device=dev)
        return info, pa, pb

    def step(enc, pa, pb, ev=None):
        if ev is not None:
            ev[0].record(stream)
        awe.encode(enc, 0, awe.SIDE_A, A, M, K, K, pa, None, stream)
        awe.encode(enc, 0, awe.SIDE_B, B, N, K, N, pb, None, stream)
        if ev is not None:
            ev[1].record(stream)
        awe.gemm_planes(enc, 0, M, N, K, pa, pb, C, N, awe.I32, 0, stream)
        if ev is not None:
            ev[2].record(stream)

    def run(enc, steps, warmup):
        info, pa, pb = setup(enc)
        for _ in range(warmup):
            step(enc, pa, pb)
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
        t0 = time.perf_counter()
        for s in range(steps):
            step(enc, pa, pb, evs[s])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        enc_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / steps
        gemm_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / steps
        return info, wall, enc_ms, gemm_ms

    info, wall, enc_ms, gemm_ms = run(awe.ENC_AWE6, args.steps, args.warmup)
    C_awe6 = C.clone()  # the headline product, compared with the INT8 GEMM below
    ms_step = wall / args.steps * 1e3
    ops = 2.0 * M * N * K
    r = info["r"]
    gemm_tflops = r * ops / (gemm_ms * 1e-3) / 1e12
    enc_bytes = (M * K + N * K) * (1 + info["planes_a"] / 2.0)
    line = {
        "metric": METRIC,
        "value": round(ops / (ms_step * 1e-3) / 1e12, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "e2m1",
        "data": "synthetic",
        "config": {"workload": "AWE 6-product exact INT8xINT8 GEMM, M=N=K=%d, int8 uniform "
                               "[-128,127] seed 0, int32 C (encode A + encode B + GEMM)" % M,
                   "M": M, "N": N, "K": K, "encoding": "awe6", "products": r},
        "gemm_only": {"ms": round(gemm_ms, 4), "exact_TOPS": round(ops / (gemm_ms * 1e-3) / 1e12, 2),
                      "fp4_TFLOPs": round(gemm_tflops, 1),
                      "fp4_peak_frac": round(gemm_tflops / FP4_PEAK_TFLOPS, 4)},
        "encode": {"ms": round(enc_ms, 4), "GB_s": round(enc_bytes / (enc_ms * 1e-3) / 1e9, 1)},
        "roofline": {"bound": "mfma", "achieved": round(gemm_tflops, 1), "peak": FP4_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(gemm_tflops / FP4_PEAK_TFLOPS, 4),
                     "traffic": gemm_traffic()},
    }
    if not args.no_context:
        binfo, bwall, benc_ms, bgemm_ms = run(awe.ENC_B13, max(3, args.steps // 2), 2)
        line["base13_9_products"] = {
            "ms_per_step": round(bwall / max(3, args.steps // 2) * 1e3, 4),
            "gemm_ms": round(bgemm_ms, 4),
            "gemm_exact_TOPS": round(ops / (bgemm_ms * 1e-3) / 1e12, 2),
            "fp4_peak_frac": round(binfo["r"] * ops / (bgemm_ms * 1e-3) / 1e12 / FP4_PEAK_TFLOPS, 4),
            "equal_to_awe6_C": bool(torch.equal(C, C_awe6))}
        try:
            Ci = torch._int_mm(A, B)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(5):
                Ci = torch._int_mm(A, B)
            e1.record(stream)
            torch.cuda.synchronize()
            ims = e0.elapsed_time(e1) / 5
            line["int8_mfma_context"] = {"library": "hipBLASLt via torch._int_mm", "ms": round(ims, 4),
                                         "TOPS": round(ops / (ims * 1e-3) / 1e12, 1)}
            # both products are exact, so the timed AWE6 result must equal the INT8 GEMM bit for bit
            line["int8_mfma_context"]["equal_to_awe6_C"] = bool(torch.equal(Ci, C_awe6))
        except Exception as ex:  # noqa: BLE001 - context only
            line["int8_mfma_context"] = {"error": str(ex)[:200]}
        line["fp4_vendor_gemm_context"] = fp4_vendor_context(dev, M, N, K, stream)
    if not args.no_context:
        # INT8 x INT8 with 2 E4M3 products and 1 E2M1 product (App. A) on the same A and B;
        # an E4M3 MFMA runs at half the E2M1 rate, so the work is 5 FP4-product equivalents
        finfo, fwall, fenc_ms, fgemm_ms = run(awe.ENC_FP8FP4, max(3, args.steps // 2), 2)
        line["fp8fp4_2_fp8_1_fp4"] = {
            "ms_per_step": round(fwall / max(3, args.steps // 2) * 1e3, 4),
            "gemm_ms": round(fgemm_ms, 4),
            "gemm_exact_TOPS": round(ops / (fgemm_ms * 1e-3) / 1e12, 2),
            "fp4_equiv_peak_frac": round(5 * ops / (fgemm_ms * 1e-3) / 1e12 / FP4_PEAK_TFLOPS, 4)}
        # INT8 x INT8 in 3 E2M3 (FP6) products on the same A and B (one Karatsuba-type step,
        # which Sec. 3.3 admits from a 3-bit significand); E2M3 MFMAs run at the E2M1 rate
        sinfo, swall, senc_ms, sgemm_ms = run(awe.ENC_FP6K3, max(3, args.steps // 2), 2)
        line["fp6k3_3_fp6_products"] = {
            "ms_per_step": round(swall / max(3, args.steps // 2) * 1e3, 4),
            "exact_TOPS": round(ops / (swall / max(3, args.steps // 2)) / 1e12, 2),
            "encode_ms": round(senc_ms, 4),
            "gemm_ms": round(sgemm_ms, 4),
            "gemm_exact_TOPS": round(ops / (sgemm_ms * 1e-3) / 1e12, 2),
            "fp6_TFLOPs": round(sinfo["r"] * ops / (sgemm_ms * 1e-3) / 1e12, 1),
            "fp6_peak_frac": round(sinfo["r"] * ops / (sgemm_ms * 1e-3) / 1e12 / FP4_PEAK_TFLOPS, 4)}
        # the same limbs with the weights in the block scales (Sec. 4.5): 4 E2M3 products into
        # one accumulator, each stage bringing both planes of each side once
        pinfo, pwall, penc_ms, pgemm_ms = run(awe.ENC_FP6P4, max(3, args.steps // 2), 2)
        line["fp6p4_4_fp6_products_weights_in_scales"] = {
            "ms_per_step": round(pwall / max(3, args.steps // 2) * 1e3, 4),
            "exact_TOPS": round(ops / (pwall / max(3, args.steps // 2)) / 1e12, 2),
            "encode_ms": round(penc_ms, 4),
            "gemm_ms": round(pgemm_ms, 4),
            "gemm_exact_TOPS": round(ops / (pgemm_ms * 1e-3) / 1e12, 2),
            "fp6_TFLOPs": round(pinfo["r"] * ops / (pgemm_ms * 1e-3) / 1e12, 1),
            "fp6_peak_frac": round(pinfo["r"] * ops / (pgemm_ms * 1e-3) / 1e12 / FP4_PEAK_TFLOPS, 4)}
        # {0, +-1} x INT8 (Sec. 6.2) on the same B: 3 products
        At = torch.from_numpy(inputs.int8_pair(M, 8, K, seed=5, a_range=(-1, 1))[0]).to(dev)
        tinfo, pta, ptb = setup(awe.ENC_TERNARY)
        awe.encode(awe.ENC_TERNARY, 0, awe.SIDE_A, At, M, K, K, pta, None, stream)
        awe.encode(awe.ENC_TERNARY, 0, awe.SIDE_B, B, N, K, N, ptb, None, stream)
        tms = _time_ms(lambda: awe.gemm_planes(awe.ENC_TERNARY, 0, M, N, K, pta, ptb, C, N, awe.I32, 0, stream),
                       10, stream, warm=3)
        line["ternary_3_products"] = {
            "gemm_ms": round(tms, 4), "gemm_exact_TOPS": round(ops / (tms * 1e-3) / 1e12, 2),
            "fp4_peak_frac": round(tinfo["r"] * ops / (tms * 1e-3) / 1e12 / FP4_PEAK_TFLOPS, 4)}
        del At, pta, ptb
        line["fp16_12_products"] = fp16_context(dev, M)
        for name in WORKLOADS:
            line[name] = WORKLOAD_FNS[name](dev)
        line["ozaki2_int53"] = ozaki2_context(dev)
        probe = mfma_sustained()
        if probe and "error" not in probe:
            probe["gemm_frac_of_8_wave_rate"] = round(gemm_tflops / probe["8_waves_per_cu_TFLOPs"], 4)
            probe["gemm_frac_of_varied_operand_rate"] = round(
                gemm_tflops / probe["varied_operands_8_waves_per_cu_TFLOPs"], 4)
            probe["gemm_frac_of_varied_operand_16x16x128_rate"] = round(
                gemm_tflops / probe["varied_operands_16x16x128_8_waves_per_cu_TFLOPs"], 4)
        line["mfma_sustained"] = probe
    if sampler is not None:
        line["clock_under_load"] = clock_under_load(sampler, clock_dir, awe, M, N, K, stream)
    if args.calibrate_copy:
        src = torch.ones(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(A_h, B_h)
    print(json.dumps(line), flush=True)


def _time_ms(fn, reps, stream, warm=1):
    """Average milliseconds of fn() over reps calls, HIP events on `stream` after `warm` warm-up
    calls."""
    import torch

    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def _time_steps(encode, gemm, reps, stream):
    """Average milliseconds of a step (encode() then gemm()) and of the GEMM within it, over reps
    steps after three warm-up steps: HIP events on `stream` around each step's GEMM, as for the
    headline, so that both figures come from the same sequence of launches."""
    import torch

    for _ in range(3):
        encode()
        gemm()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(reps)]
    for e in evs:
        e[0].record(stream)
        encode()
        e[1].record(stream)
        gemm()
        e[2].record(stream)
    torch.cuda.synchronize()
    step = sum(e[0].elapsed_time(e[2]) for e in evs) / reps
    g = sum(e[1].elapsed_time(e[2]) for e in evs) / reps
    return step, g


def awe4_workload(dev, n=8192):
    """INT4 x INT8 in 4 FP4 products (App. A): A int4 uniform in [-8, 7] (one per int8 byte), B
    int8 uniform in [-128, 127], seed 0, n^3, int32 C.  Steps of both encoders + GEMM on the
    resident planes (awe_gemm_planes), timed whole and GEMM alone within each step; the FP4 work
    is 4 products of 2 n^3."""
    import torch

    from paper_2609_24519_amd import awe, inputs

    A_h, B_h = inputs.int8_pair(n, n, n, seed=0, a_range=(-8, 7))
    A, B = torch.from_numpy(A_h).to(dev), torch.from_numpy(B_h).to(dev)
    enc = awe.ENC_AWE4
    r = awe.get_encoding_info(enc)["r"]
    pa = torch.empty(awe.plane_bytes(enc, 0, awe.SIDE_A, n, n), dtype=torch.uint8, device=dev)
    pb = torch.empty(awe.plane_bytes(enc, 0, awe.SIDE_B, n, n), dtype=torch.uint8, device=dev)
    C = torch.empty((n, n), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()

    def enc_both():
        awe.encode(enc, 0, awe.SIDE_A, A, n, n, n, pa, None, stream)
        awe.encode(enc, 0, awe.SIDE_B, B, n, n, n, pb, None, stream)

    def gemm():
        awe.gemm_planes(enc, 0, n, n, n, pa, pb, C, n, awe.I32, 0, stream)

    ems, gms = _time_steps(enc_both, gemm, 10, stream)
    ops = 2.0 * n ** 3
    tf = r * ops / (gms * 1e-3) / 1e12
    out = {"workload": "INT4xINT8 exact GEMM, M=N=K=%d, A uniform [-8,7], B uniform [-128,127], seed 0, "
                       "int32 C, %d FP4 products" % (n, r),
           "gemm_ms": round(gms, 4), "gemm_exact_TOPS": round(ops / (gms * 1e-3) / 1e12, 1),
           "fp4_TFLOPs": round(tf, 1), "fp4_peak_frac": round(tf / FP4_PEAK_TFLOPS, 4),
           "end_to_end_ms": round(ems, 4), "end_to_end_exact_TOPS": round(ops / (ems * 1e-3) / 1e12, 1)}
    del A, B, pa, pb, C
    torch.cuda.empty_cache()
    return out


def residues_workload(dev, n=4096):
    """C mod m at n^3 for every modulus of the FP64-significand residue set (Sec. 5.3), operands
    uniform in [0, m - 1] (seed m), int32 C in [0, m): the mod-m GEMM on resident planes
    (awe_gemm_planes) and awe_gemm_mod end to end, summed over the moduli; the FP4 work is
    sum_m r_m 2 n^3."""
    import torch

    from paper_2609_24519_amd import awe, inputs

    with open(os.path.join(ROOT, "tests", "golden", "moduli_fp64_k16384.txt")) as f:
        rows = [l for l in f if l.strip() and not l.startswith("#")]
    moduli = [int(x) for x in rows[0].split()]
    stream = torch.cuda.current_stream()
    C = torch.empty((n, n), dtype=torch.int32, device=dev)
    g_ms = e_ms = 0.0
    products = 0
    for m in moduli:
        A_h, B_h = inputs.residue_pair(n, n, n, m)
        A, B = torch.from_numpy(A_h).to(dev), torch.from_numpy(B_h).to(dev)
        r = awe.get_encoding_info(awe.ENC_MOD, m)["r"]
        products += r
        pa = torch.empty(awe.plane_bytes(awe.ENC_MOD, m, awe.SIDE_A, n, n), dtype=torch.uint8, device=dev)
        pb = torch.empty(awe.plane_bytes(awe.ENC_MOD, m, awe.SIDE_B, n, n), dtype=torch.uint8, device=dev)
        awe.encode(awe.ENC_MOD, m, awe.SIDE_A, A, n, n, n, pa, None, stream)
        awe.encode(awe.ENC_MOD, m, awe.SIDE_B, B, n, n, n, pb, None, stream)
        g_ms += _time_ms(lambda: awe.gemm_planes(awe.ENC_MOD, m, n, n, n, pa, pb, C, n, awe.I32, 0, stream),
                         5, stream)
        wsn = awe.workspace_bytes(awe.ENC_MOD, m, n, n, n)
        ws = torch.empty(wsn, dtype=torch.uint8, device=dev)
        e_ms += _time_ms(lambda: awe.gemm_mod(m, n, n, n, A, n, B, n, C, n, ws, wsn, None, stream), 5, stream)
        del A, B, pa, pb, ws
    ops = 2.0 * n ** 3
    tf = products * ops / (g_ms * 1e-3) / 1e12
    out = {"workload": "C mod m, M=N=K=%d, operands uniform [0,m-1] seed m, for the %d moduli of the "
                       "FP64-significand residue set (%d FP4 products in all)" % (n, len(moduli), products),
           "gemm_ms_sum": round(g_ms, 4), "fp4_TFLOPs": round(tf, 1), "fp4_peak_frac": round(tf / FP4_PEAK_TFLOPS, 4),
           "end_to_end_ms_sum": round(e_ms, 4)}
    del C
    torch.cuda.empty_cache()
    return out


def stress_workload(dev, M=4096, N=4096, K=65536):
    """Accumulation stress (every entry -128 or 127, structured rows and columns), AWE6, int64 C:
    the GEMM on resident planes with the default fold segment and with a forced one of 4096, timed
    alternately twice (the second pass is reported: the first GEMMs on freshly written planes run
    slower)."""
    import torch

    from paper_2609_24519_amd import awe, inputs

    A_h, B_h = inputs.stress_operands(M, N, K, seed=0)
    A, B = torch.from_numpy(A_h).to(dev), torch.from_numpy(B_h).to(dev)
    enc = awe.ENC_AWE6
    r = awe.get_encoding_info(enc)["r"]
    pa = torch.empty(awe.plane_bytes(enc, 0, awe.SIDE_A, M, K), dtype=torch.uint8, device=dev)
    pb = torch.empty(awe.plane_bytes(enc, 0, awe.SIDE_B, N, K), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    awe.encode(enc, 0, awe.SIDE_A, A, M, K, K, pa, None, stream)
    awe.encode(enc, 0, awe.SIDE_B, B, N, K, N, pb, None, stream)
    del A, B
    C = torch.empty((M, N), dtype=torch.int64, device=dev)
    ops = 2.0 * M * N * K
    out = {"workload": "AWE6 exact GEMM, M=N=%d, K=%d, entries -128 or 127 (structured stress operands), "
                       "int64 C" % (M, K)}
    for _ in range(2):
        for name, kseg in (("default_fold_segment", 0), ("fold_segment_4096", 4096)):
            ms = _time_ms(lambda: awe.gemm_planes(enc, 0, M, N, K, pa, pb, C, N, awe.I64, kseg, stream), 5, stream)
            tf = r * ops / (ms * 1e-3) / 1e12
            out[name] = {"gemm_ms": round(ms, 4), "gemm_exact_TOPS": round(ops / (ms * 1e-3) / 1e12, 1),
                         "fp4_TFLOPs": round(tf, 1), "fp4_peak_frac": round(tf / FP4_PEAK_TFLOPS, 4)}
    del pa, pb, C
    torch.cuda.empty_cache()
    return out


WORKLOAD_FNS = {"awe4_int4xint8": awe4_workload, "residues_per_modulus": residues_workload,
                "stress_65536": stress_workload}


def fp16_context(dev, n):
    """App. A's FP16-significand scheme: 12-bit integers (int16 in [-2048, 2047]) in 12 FP4
    products (one launch), n^3, int64 C, awe_gemm_planes on resident planes: 10 calls timed after
    3 warm-up calls (the first calls on freshly written planes run slower)."""
    import numpy as np
    import torch

    from paper_2609_24519_amd import awe, inputs

    rng = np.random.default_rng(7)
    A = torch.from_numpy(inputs.uniform(rng, (n, n), -2048, 2047, np.int16)).to(dev)
    B = torch.from_numpy(inputs.uniform(rng, (n, n), -2048, 2047, np.int16)).to(dev)
    enc = awe.ENC_FP16
    info = awe.get_encoding_info(enc)
    pa = torch.empty(awe.plane_bytes(enc, 0, awe.SIDE_A, n, n), dtype=torch.uint8, device=dev)
    pb = torch.empty(awe.plane_bytes(enc, 0, awe.SIDE_B, n, n), dtype=torch.uint8, device=dev)
    C = torch.empty((n, n), dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()
    awe.encode(enc, 0, awe.SIDE_A, A, n, n, n, pa, None, stream)
    awe.encode(enc, 0, awe.SIDE_B, B, n, n, n, pb, None, stream)
    ms = _time_ms(lambda: awe.gemm_planes(enc, 0, n, n, n, pa, pb, C, n, awe.I64, 0, stream), 10, stream, warm=3)
    ops = 2.0 * n * n * n
    out = {"workload": "M=N=K=%d, int16 entries uniform in [-2048, 2047], int64 C" % n,
           "gemm_ms": round(ms, 3), "gemm_exact_TOPS": round(ops / (ms * 1e-3) / 1e12, 1),
           "fp4_peak_frac": round(info["r"] * ops / (ms * 1e-3) / 1e12 / FP4_PEAK_TFLOPS, 4)}
    del A, B, pa, pb, C
    torch.cuda.empty_cache()
    return out


def ozaki2_context(dev, M=4096, N=4096, K=16384, reps=3):
    """The residue route of Sec. 5.3 as the integer layer of Ozaki scheme II: exact product of
    53-bit integer matrices through the 23-modulus FP64-significand set (60 FP4 products),
    awe_gemm_crt end to end (residues, mod-m GEMMs, reconstruction to 128-bit words and the
    nearest double).  Timed with HIP events on the current stream."""
    import torch

    from paper_2609_24519_amd import awe

    with open(os.path.join(ROOT, "tests", "golden", "moduli_fp64_k16384.txt")) as f:
        rows = [l for l in f if l.strip() and not l.startswith("#")]
    moduli = [int(x) for x in rows[0].split()]
    b53 = (1 << 53) - 1
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    A = torch.randint(-b53, b53, (M, K), dtype=torch.int64, device=dev, generator=g)
    B = torch.randint(-b53, b53, (K, N), dtype=torch.int64, device=dev, generator=g)
    c128 = torch.empty((M, N, 2), dtype=torch.int64, device=dev)
    c64 = torch.empty((M, N), dtype=torch.float64, device=dev)
    wsn = awe.crt_workspace_bytes(moduli, M, N, K)
    ws = torch.empty(wsn, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def run():
        awe.gemm_crt(M, N, K, A, K, B, N, b53, b53, moduli, c128, c64, N, ws, wsn, None, stream)

    run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    products = sum(awe.get_encoding_info(awe.ENC_MOD, m)["r"] for m in moduli)
    out = {"workload": "M=N=%d, K=%d, int64 entries uniform in [-(2^53-1), 2^53-1], %d moduli, "
                       "%d FP4 products" % (M, K, len(moduli), products),
           "ms": round(ms, 3), "fp64_equiv_TFLOPs": round(2.0 * M * N * K / (ms * 1e-3) / 1e12, 1),
           "fp4_products_TFLOPs": round(products * 2.0 * M * N * K / (ms * 1e-3) / 1e12, 1)}
    del A, B, c128, c64, ws
    torch.cuda.empty_cache()
    return out


def fp4_vendor_context(dev, M, N, K, stream):
    """One plain MXFP4 GEMM of the same shape from the vendor library (hipBLASLt through
    torch._scaled_mm: E2M1 operands with E8M0 block scales of 2^0, bf16 output) on random codes:
    what one FP4 GEMM reaches on this board, next to the r plane products of the AWE GEMM.  Its
    output is rounded to bf16, so it is checked only to one bf16 ulp on a 64 x 64 corner."""
    import torch

    try:
        g = torch.Generator(device=dev).manual_seed(0)
        a8 = torch.randint(0, 256, (M, K // 2), dtype=torch.uint8, device=dev, generator=g)
        b8 = torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device=dev, generator=g)
        a, b = a8.view(torch.float4_e2m1fn_x2), b8.view(torch.float4_e2m1fn_x2)
        sa = torch.full((M, K // 32), 127, dtype=torch.uint8, device=dev).view(torch.float8_e8m0fnu)
        sb = torch.full((N, K // 32), 127, dtype=torch.uint8, device=dev).view(torch.float8_e8m0fnu)
        with torch.cuda.stream(stream):
            out = torch._scaled_mm(a, b.t(), sa, sb, out_dtype=torch.bfloat16)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(10):
                out = torch._scaled_mm(a, b.t(), sa, sb, out_dtype=torch.bfloat16)
            e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 10
        lut = torch.tensor([0, .5, 1, 1.5, 2, 3, 4, 6, 0, -.5, -1, -1.5, -2, -3, -4, -6], device=dev)

        def decode(x8):
            return torch.stack([lut[(x8 & 15).long()], lut[(x8 >> 4).long()]], -1).reshape(x8.shape[0], -1)

        ref = decode(a8[:64]) @ decode(b8[:64]).t()
        err = (out[:64, :64].float() - ref).abs()
        # within one bf16 unit in the last place (its conversion does not round to nearest)
        ok = bool((err <= ref.abs() * 2.0 ** -7 + 1e-6).all())
        tf = 2.0 * M * N * K / (ms * 1e-3) / 1e12
        return {"library": "hipBLASLt via torch._scaled_mm (MXFP4, bf16 output)", "ms": round(ms, 4),
                "fp4_TFLOPs": round(tf, 1), "fp4_peak_frac": round(tf / FP4_PEAK_TFLOPS, 4),
                "within_1_bf16_ulp_64x64": ok}
    except Exception as ex:  # noqa: BLE001 - context only
        return {"error": str(ex)[:200]}


def mfma_sustained(iters=20000):
    """Dense FP4 rate of the GEMM's MFMA issued back to back from registers with 8 and
    with 4 waves per compute unit (libawe_probe.so), with constant operands and with operands
    that change between MFMAs: the practical ceilings, at the clock the chip holds under full
    MFMA load, next to the data-sheet peak."""
    import ctypes

    from paper_2609_24519_amd import build as hip_build

    if not os.path.exists(hip_build.PROBE_LIB):
        return None
    lib = ctypes.CDLL(hip_build.PROBE_LIB)
    lib.awe_mfma_peak.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    out = {}
    for waves in (8, 4):
        tf = ctypes.c_double(0.0)
        rc = lib.awe_mfma_peak(waves, iters, ctypes.byref(tf))
        if rc != 0:
            return {"error": "HIP error %d" % rc}
        out["%d_waves_per_cu_TFLOPs" % waves] = round(tf.value, 1)
        out["%d_waves_frac_of_peak" % waves] = round(tf.value / FP4_PEAK_TFLOPS, 4)
    # the same probe with E2M3 (FP6) and E4M3 (FP8) operands, 8 waves per CU: the data
    # sheet lists FP6 at the FP4 rate and FP8 at half of it
    lib.awe_mfma_peak_fmt.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      ctypes.POINTER(ctypes.c_double)]
    for fmt, name in ((2, "e2m3"), (0, "e4m3")):
        tf = ctypes.c_double(0.0)
        rc = lib.awe_mfma_peak_fmt(fmt, 8, iters, ctypes.byref(tf))
        if rc != 0:
            return {"error": "HIP error %d" % rc}
        out["%s_8_waves_per_cu_TFLOPs" % name] = round(tf.value, 1)
    # E2M1 operands that change between MFMAs, as real data does: the matrix unit then draws
    # more power and the clock falls under the board's power limit (a longer run, so that the
    # clock has settled)
    lib.awe_mfma_peak_varied.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    best = 0.0
    for _ in range(2):
        tf = ctypes.c_double(0.0)
        rc = lib.awe_mfma_peak_varied(8, 10 * iters, ctypes.byref(tf))
        if rc != 0:
            return {"error": "HIP error %d" % rc}
        best = tf.value
    out["varied_operands_8_waves_per_cu_TFLOPs"] = round(best, 1)
    out["varied_operands_frac_of_peak"] = round(best / FP4_PEAK_TFLOPS, 4)
    # the same on the 16x16x128 form of the MFMA, which sustains more on changing operands
    lib.awe_mfma_peak_varied16.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    for _ in range(2):
        tf = ctypes.c_double(0.0)
        rc = lib.awe_mfma_peak_varied16(8, 10 * iters, ctypes.byref(tf))
        if rc != 0:
            return {"error": "HIP error %d" % rc}
    out["varied_operands_16x16x128_8_waves_per_cu_TFLOPs"] = round(tf.value, 1)
    out["varied_operands_16x16x128_frac_of_peak"] = round(tf.value / FP4_PEAK_TFLOPS, 4)
    lib.awe_mfma_peak_varied_fmt.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                             ctypes.POINTER(ctypes.c_double)]
    for fmt, name in ((2, "e2m3"), (0, "e4m3")):
        for _ in range(2):
            tf = ctypes.c_double(0.0)
            rc = lib.awe_mfma_peak_varied_fmt(fmt, 8, 10 * iters, ctypes.byref(tf))
            if rc != 0:
                return {"error": "HIP error %d" % rc}
        out["%s_varied_operands_8_waves_per_cu_TFLOPs" % name] = round(tf.value, 1)
    return out


def clock_under_load(sampler, d, awe, M, N, K, stream):
    """Runs the AWE6 GEMM, the 3-product E2M3 GEMM, the 4-product E2M3 GEMM with the weights in
    the scales, then the MFMA probe with constant and with changing E2M1 operands and with
    changing E2M3 operands, each in a loop until the sampler has read the clocks and power under
    that load.  The rates are FP4/FP6 FLOP/s (r 2MNK / t)."""
    import ctypes

    import torch

    from paper_2609_24519_amd import build as hip_build
    from paper_2609_24519_amd import inputs

    out = {}
    A_h, B_h = inputs.int8_pair(M, N, K, seed=0)
    A = torch.from_numpy(A_h).cuda()
    B = torch.from_numpy(B_h).cuda()
    C = torch.empty((M, N), dtype=torch.int32, device="cuda")
    planes = {}
    for enc in (awe.ENC_AWE6, awe.ENC_FP6K3, awe.ENC_FP6P4):
        pa = torch.empty(awe.plane_bytes(enc, 0, awe.SIDE_A, M, K), dtype=torch.uint8, device="cuda")
        pb = torch.empty(awe.plane_bytes(enc, 0, awe.SIDE_B, N, K), dtype=torch.uint8, device="cuda")
        awe.encode(enc, 0, awe.SIDE_A, A, M, K, K, pa, None, stream)
        awe.encode(enc, 0, awe.SIDE_B, B, N, K, N, pb, None, stream)
        planes[enc] = (pa, pb, awe.get_encoding_info(enc)["r"])
    lib = ctypes.CDLL(hip_build.PROBE_LIB)
    for f in (lib.awe_mfma_peak, lib.awe_mfma_peak_varied):
        f.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    lib.awe_mfma_peak_varied_fmt.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                             ctypes.POINTER(ctypes.c_double)]
    for ph in CLOCK_PHASES:
        open(os.path.join(d, "go_" + ph), "w").close()
        t0 = time.time()
        rates = []
        while not os.path.exists(os.path.join(d, "done_" + ph)) and time.time() - t0 < 90:
            if ph.startswith("gemm"):
                enc = {"gemm_e2m3": awe.ENC_FP6K3, "gemm_e2m3_scaled": awe.ENC_FP6P4}.get(ph, awe.ENC_AWE6)
                pa, pb, r = planes[enc]
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for _ in range(20):
                    awe.gemm_planes(enc, 0, M, N, K, pa, pb, C, N, awe.I32, 0, stream)
                e1.record(stream)
                torch.cuda.synchronize()
                rates.append(r * 2.0 * M * N * K / (e0.elapsed_time(e1) / 20 * 1e-3) / 1e12)
            else:
                tf = ctypes.c_double(0.0)
                if ph == "probe_static":
                    rc = lib.awe_mfma_peak(8, 100000, ctypes.byref(tf))
                elif ph == "probe_varied":
                    rc = lib.awe_mfma_peak_varied(8, 100000, ctypes.byref(tf))
                else:
                    rc = lib.awe_mfma_peak_varied_fmt(2, 8, 100000, ctypes.byref(tf))
                if rc != 0:
                    break
                rates.append(tf.value)
        r = read_smi(os.path.join(d, "smi_" + ph + ".txt"))
        if rates:
            r["fp4_TFLOPs"] = round(sum(rates[1:] or rates) / len(rates[1:] or rates), 1)
            if "gfx_clock_mhz_mean" in r:
                peak_at_clock = 256 * 16384 * r["gfx_clock_mhz_mean"] * 1e6 / 1e12
                r["frac_of_peak_at_this_clock"] = round(r["fp4_TFLOPs"] / peak_at_clock, 4)
        out[ph] = r
    try:
        sampler.wait(timeout=30)
    except Exception:  # noqa: BLE001 - the sampler is best effort
        sampler.kill()
    return out


def gemm_traffic():
    """HBM bytes per GEMM dispatch from the committed rocprofv3 counter summary, or None
    when that summary was taken on a different kernel source."""
    from paper_2609_24519_amd import profiling

    path = os.path.join(ROOT, "profiles", "traffic_gemm_awe6_int8_8192.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except OSError:
        return None
    if rec.get("kernel_source_sha") != profiling.kernel_source_hash():
        return None
    k = rec["kernels"].get("gemm_kernel")
    return None if k is None else round(k["fetch_bytes"] + k["write_bytes"])


def cpu_baseline(A_h, B_h, target_s=15.0):
    """The oracle (plain int64 triple loop, OpenMP over rows) on a bounded sample of
    the same workload: a block of rows of C over the full N and K, sized from two short
    calibration runs (the first warms the threads and caches) to take about ``target_s``
    seconds, scaled to exact TOPS; ``other_workloads`` holds the same oracle's rate on the
    other workloads (cpu_oracle_timings)."""
    import numpy as np

    from oracle import gemm as og

    if not os.path.exists(os.path.join(ROOT, "oracle", "liboracle_gemm.so")):
        og.build()
    K, N = B_h.shape
    threads = og.num_threads()
    rows = max(2 * threads, 32)
    for _ in range(2):
        t0 = time.perf_counter()
        og.gemm_i64(np.ascontiguousarray(A_h[:rows]), B_h)
        dt = time.perf_counter() - t0
    rows = int(min(A_h.shape[0], max(rows, rows * target_s / max(dt, 1e-3))))
    rows = max(threads, rows // threads * threads)
    sub = np.ascontiguousarray(A_h[:rows])
    t0 = time.perf_counter()
    og.gemm_i64(sub, B_h)
    dt = time.perf_counter() - t0
    macs = rows * N * K
    return {"value": round(2.0 * macs / dt / 1e12, 6), "unit": "TOPS", "cores": threads,
            "kind": "oracle", "host_cpus": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": "rows 0..%d of C over full N=%d, K=%d (%d MACs), %.1f s"
                      % (rows - 1, N, K, macs, dt),
            "other_workloads": cpu_oracle_timings()}


def cpu_model():
    """The host CPU's model name (/proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_oracle_timings():
    """The same oracle on the other workloads, each whole or on a stated block of rows (a few
    seconds in all): 256^3 int8, 2048^3 int8, the 4096 x 4096 x 65,536 stress operands (rows
    0..63), and one modulus of the residue set at 4096^3 (m = 251, rows 0..255).  MAC/s."""
    import numpy as np

    from oracle import gemm as og
    from paper_2609_24519_amd import inputs

    out = {}

    def timed(name, A, B, full_rows, fn):
        t0 = time.perf_counter()
        fn(A, B)
        dt = time.perf_counter() - t0
        macs = A.shape[0] * A.shape[1] * B.shape[1]
        out[name] = {"MAC_per_s": round(macs / dt, 1), "seconds": round(dt, 3),
                     "rows": "%d of %d" % (A.shape[0], full_rows)}

    A, B = inputs.int8_pair(256, 256, 256, seed=0)
    og.gemm_i64(A, B)  # loads the library and starts its threads
    timed("int8_256^3", A, B, 256, og.gemm_i64)
    A, B = inputs.int8_pair(2048, 2048, 2048, seed=0)
    timed("int8_2048^3", A, B, 2048, og.gemm_i64)
    A, B = inputs.stress_operands(64, 4096, 65536, seed=0)
    timed("stress_4096x4096x65536", np.ascontiguousarray(A), B, 4096, og.gemm_i64)
    A, B = inputs.residue_pair(256, 4096, 4096, 251)
    timed("residues_mod251_4096^3", A, B, 4096, lambda a, b: og.gemm_mod(251, a, b))
    return out


if __name__ == "__main__":
    main()
