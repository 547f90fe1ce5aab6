"""Builds libawe.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree, and
the benchmark helper libawe_probe.so (the sustained-MFMA-rate probe).

    python -m paper_2609_24519_amd.build [--resources <out.md>]

``--resources`` also compiles the kernels to assembly and writes the register,
spill and LDS figures the compiler assigned to every kernel (from the code
object metadata).

Every HIP translation unit is compiled with packed FP32 instructions disabled
(-packed-fp32-ops): the kernels' float code must not be turned into
v_pk_*_f32 forms.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libawe.so")
SOURCES = ["awe_kernels.hip", "awe_rns.hip", "awe_tables.cpp", "awe_api.cpp"]
PROBE_LIB = os.path.join(HERE, "libawe_probe.so")
PROBE_SOURCES = ["mfma_peak.hip"]
ARCH = "gfx950"


def hipcc():
    for c in (os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc"), "hipcc"):
        if os.path.sep not in c or os.path.exists(c):
            return c
    return "hipcc"


def _compile(sources, lib, verbose):
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Wall", "-Wno-unused-function",
           "-I", os.path.join(ROOT, "include")]
    cmd += [os.path.join(CSRC, s) for s in sources]
    cmd += ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in res.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if res.returncode != 0:
        if os.path.exists(tmp):
            os.remove(tmp)
        raise RuntimeError("hipcc failed:\n" + out)
    if verbose and out.strip():
        print(out)
    os.replace(tmp, lib)
    return lib


def build(verbose=False):
    _compile(PROBE_SOURCES, PROBE_LIB, verbose)
    return _compile(SOURCES, LIB, verbose)


def kernel_resources():
    """Per-kernel register / spill / LDS figures from the gfx950 code object metadata: a list of
    (name, vgpr, agpr, sgpr, vgpr spill, sgpr spill, static LDS, scratch, max workgroup) with the
    mangled name's namespace prefix removed."""
    import re
    import tempfile

    import yaml

    rows = []
    for src in ["awe_kernels.hip", "awe_rns.hip"]:
        with tempfile.TemporaryDirectory() as td:
            asm = os.path.join(td, "k.s")
            cmd = [hipcc(), "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
                   "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                   "-I", os.path.join(ROOT, "include"), "--cuda-device-only", "-S",
                   os.path.join(CSRC, src), "-o", asm]
            res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
            if res.returncode != 0:
                raise RuntimeError("hipcc failed:\n" + res.stdout)
            text = open(asm).read()
        meta = text.split(".amdgpu_metadata", 1)[1].split(".end_amdgpu_metadata", 1)[0].replace("\t", " ")
        for k in yaml.safe_load(meta)["amdhsa.kernels"]:
            name = re.sub(r"^_ZN3awe12_GLOBAL__N_1", "", k[".name"])
            rows.append((name, k.get(".vgpr_count"), k.get(".agpr_count"), k.get(".sgpr_count"),
                         k.get(".vgpr_spill_count"), k.get(".sgpr_spill_count"),
                         k.get(".group_segment_fixed_size"), k.get(".private_segment_fixed_size"),
                         k.get(".max_flat_workgroup_size")))
    return rows


def resources(out_md):
    """kernel_resources() as a Markdown table."""
    rows = kernel_resources()
    lines = ["# Kernel resources (gfx950 code object metadata)", "",
             "Command: `python -m paper_2609_24519_amd.build --resources %s`" % out_md, "",
             "VGPR is the unified count (arch + accumulation registers); the GEMM's LDS ring is",
             "dynamic (set at launch) and not part of the static LDS column.", "",
             "| kernel (mangled tail) | VGPR | AGPR | SGPR | VGPR spill | SGPR spill | static LDS | scratch | max WG |",
             "|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append("| %s | %s | %s | %s | %s | %s | %s | %s | %s |" % r)
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    build(verbose=True)
    if len(sys.argv) == 3 and sys.argv[1] == "--resources":
        resources(sys.argv[2])
    sys.exit(0)
