"""Host-side checks of the benchmark and profiling helpers (CPU only, no GPU calls)."""
import csv
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    # the library has no multi-GPU path: --gpus N > 1 exits with a message before touching a GPU
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""


def test_read_smi_parses_clocks_and_power(tmp_path):
    sys.path.insert(0, ROOT)
    import bench

    p = tmp_path / "smi.txt"
    p.write_text("GPU: 0\n    POWER:\n        SOCKET_POWER: 1362 W\n    CLOCK:\n        GFX_0:\n"
                 "            CLK: 2106 MHz\n            MIN_CLK: 500 MHz\n        GFX_1:\n"
                 "            CLK: 2000 MHz\n")
    r = bench.read_smi(str(p))
    assert r == {"gfx_clock_mhz_mean": 2053.0, "gfx_clock_mhz_min": 2000, "gfx_clock_mhz_max": 2106,
                 "socket_power_w": 1362.0}
    assert "error" in bench.read_smi(str(tmp_path / "missing.txt"))


def test_stats_from_trace_skips_warmup(tmp_path):
    from paper_2609_24519_amd import profiling

    trace = tmp_path / "trace.csv"
    with open(trace, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        t = 0
        for us in (900, 800, 100, 110, 120):  # two slow warm-up dispatches, then three timed ones
            w.writerow(["void k<1>(int)", t, t + us * 1000])
            t += 1_000_000
    out = tmp_path / "out.md"
    profiling.stats(str(trace), str(out), "cmd", 2)
    row = [l for l in out.read_text().splitlines() if l.startswith("| void k")][0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells[1:5] == ["3", "110.0", "100.0", "120.0"]


def test_kernel_source_hash_tracks_the_kernel_file():
    from paper_2609_24519_amd import profiling

    h = profiling.kernel_source_hash()
    assert h == profiling.kernel_source_hash() and len(h) >= 8


def test_clock_table_from_bench_line(tmp_path):
    import json

    from paper_2609_24519_amd import profiling

    line = {"metric": "m", "clock_under_load": {
        "gemm": {"gfx_clock_mhz_mean": 2000.0, "gfx_clock_mhz_min": 1950, "gfx_clock_mhz_max": 2050,
                 "socket_power_w": 1380.0, "fp4_TFLOPs": 4040.0, "frac_of_peak_at_this_clock": 0.4817},
        "probe_varied": {"gfx_clock_mhz_mean": 1600.0, "gfx_clock_mhz_min": 1500, "gfx_clock_mhz_max": 1700,
                         "socket_power_w": None, "fp4_TFLOPs": 6363.0}}}
    log = tmp_path / "bench.log"
    log.write_text("noise\n" + json.dumps(line) + "\n")
    out = tmp_path / "clock.md"
    profiling.clock(str(log), str(out), "cmd")
    rows = [l for l in out.read_text().splitlines() if l.startswith("| AWE6") or l.startswith("| FP4 MFMA")]
    assert len(rows) == 2
    gemm = [c.strip() for c in rows[0].strip("|").split("|")]
    assert gemm[1:] == ["2000 (1950..2050)", "1380", "4040.0", "0.482", "0.400"]
    probe = [c.strip() for c in rows[1].strip("|").split("|")]
    assert probe[2] == "n/a" and probe[4] == "n/a" and probe[5] == "0.630"


def test_kernel_labels():
    from paper_2609_24519_amd import profiling

    ns = "void awe::(anonymous namespace)::"
    assert profiling._short(ns + "residue_encode_kernel<true>(awe::ResidueEncodeArgs)") == \
        "residue_encode_kernel (B side, transposed)"
    assert profiling._short(ns + "encode_kernel<true>(unsigned char const*)") == "encode_kernel (B side, transposed)"
    assert profiling._short(ns + "encode_kernel<false>(unsigned char const*)") == "encode_kernel (A side)"
    assert profiling._short(ns + "gemm_group_kernel<Cfg<4> >(GroupArgs)") == "gemm_group_kernel"
    assert profiling._short(ns + "gemm_kernel<Cfg<4> >(GemmArgs)") == "gemm_kernel"


def test_cpu_model_and_workload_names():
    sys.path.insert(0, ROOT)
    import bench

    m = bench.cpu_model()
    assert m is None or (isinstance(m, str) and m)
    assert set(bench.WORKLOADS) == set(bench.WORKLOAD_FNS)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--only", "nonsense"],
                       stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=120)
    assert r.returncode == 2 and "invalid choice" in r.stderr
