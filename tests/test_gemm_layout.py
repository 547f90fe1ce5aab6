"""Bounds of the GEMM's copy, LDS-ring, fragment and LDS-fold addressing for every tile
configuration the library builds (CPU only): tests/layout_check/gemm_layout_check.cpp includes
the kernels' own address helpers (paper_2609_24519_amd/csrc/gemm_layout.h), is compiled for the
host with hipcc and enumerates every wave, lane, copy, stage and k-step."""
import os
import shutil
import subprocess

import pytest

from paper_2609_24519_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_every_configuration_addresses_within_bounds(tmp_path):
    h = build.hipcc()
    if not (os.path.exists(h) or shutil.which(h)):
        pytest.skip("hipcc not found")
    exe = str(tmp_path / "gemm_layout_check")
    subprocess.run([h, "-std=c++17", "-O1", "-I", os.path.join(ROOT, "include"), "-I",
                    os.path.join(ROOT, "paper_2609_24519_amd", "csrc"),
                    os.path.join(ROOT, "tests", "layout_check", "gemm_layout_check.cpp"), "-o", exe],
                   check=True, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=300)
    assert r.returncode == 0, r.stdout
    lines = [l for l in r.stdout.splitlines() if l.startswith("ok ")]
    assert len(lines) >= 20, r.stdout
