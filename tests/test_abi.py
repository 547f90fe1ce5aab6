"""The C ABI on the host (CPU only): symbols, configuration records, tables, errors.

Loads libawe.so without touching a GPU: every call here either queries host
tables or is rejected by argument checks before anything is enqueued.  The
library's own tables (C++) are compared with the oracle's (Python), which were
written independently from the same reading of the paper.
"""
import ctypes
import math
from functools import lru_cache

import numpy as np
import pytest

from oracle import modm, schemes as sc
from paper_2609_24519_amd import awe

EXACT = {"b13": awe.ENC_B13, "awe6": awe.ENC_AWE6, "awe6_alt": awe.ENC_AWE6ALT, "awe4": awe.ENC_AWE4,
         "ternary": awe.ENC_TERNARY, "fp16_12": awe.ENC_FP16, "fp8fp4": awe.ENC_FP8FP4,
         "fp6k3": awe.ENC_FP6K3, "fp6p4": awe.ENC_FP6P4}


@lru_cache(maxsize=None)
def oracle_mod(m):
    return modm.find_scheme(m)


def test_k_pad_matches_header():
    import re
    with open(awe.HEADER) as f:
        assert int(re.search(r"#define AWE_K_PAD (\d+)", f.read()).group(1)) == awe.K_PAD


def test_exports_every_declared_symbol():
    L = awe.lib()
    names = awe.header_symbols()
    assert len(names) >= 10
    for n in names:
        assert hasattr(L, n), n


@pytest.mark.parametrize("name", sorted(EXACT))
def test_encoding_info_matches_oracle(name):
    s = sc.ALL_SCHEMES[name]()
    info = awe.get_encoding_info(EXACT[name])
    assert info["r"] == s.r
    assert info["w"] == s.w and info["v"] == s.v
    assert info["ell"] == [l for _, _, l in s.products]
    assert 2 ** info["log2_D"] == s.D
    assert info["alpha"] == s.planes_a and info["beta"] == s.planes_b
    assert [info["alpha"][k] for k in info["pair_a"]] == [a for a, _, _ in s.products]
    assert [info["beta"][k] for k in info["pair_b"]] == [b for _, b, _ in s.products]
    c_a, c_b = sc.stored_cap(s, "a"), sc.stored_cap(s, "b")
    assert (info["c_a"], info["c_b"]) == (c_a, c_b)
    if name == "fp6p4":  # weights in the scales: one accumulator for all products
        kstar, per_index = sc.shared_accumulator_kstar(s)
        assert info["n_g"] == s.r and info["k_star"] == kstar
        assert 0 < info["k_seg"] <= kstar and info["k_seg"] % awe.K_PAD == 0
        assert info["k_seg"] * per_index <= 2 ** 24
    else:
        assert info["n_g"] == s.n_g
        assert info["k_star"] == sc.k_star(s.n_g, c_a, c_b)
        assert info["k_seg"] % awe.K_PAD == 0 and 0 < info["k_seg"] <= info["k_star"]
        assert info["k_seg"] * s.n_g * c_a * c_b < 2 ** 23
    assert info["range_a"] == s.range_a and info["range_b"] == s.range_b
    assert info["formats_a"] == (s.formats_a or ["e2m1"] * len(s.planes_a))
    assert info["formats_b"] == (s.formats_b or ["e2m1"] * len(s.planes_b))


def test_coverages(paper):
    assert awe.get_encoding_info(awe.ENC_AWE6)["coverage_a"] == paper["awe6.coverage_cap6"][0]
    assert awe.get_encoding_info(awe.ENC_AWE6ALT)["coverage_a"] == paper["awe6_alt.coverage"][0]
    assert awe.get_encoding_info(awe.ENC_B13)["coverage_a"] == paper["b13.xcarry"][2]


@pytest.mark.parametrize("name", sorted(EXACT))
def test_plane_tables_match_oracle(name):
    s = sc.ALL_SCHEMES[name]()
    for side, oside in ((awe.SIDE_A, "a"), (awe.SIDE_B, "b")):
        lo, T = awe.get_plane_table(EXACT[name], 0, side)
        olo, OT = sc.plane_table(s, oside)
        assert lo == olo
        assert np.array_equal(T, OT)


def test_mod_families_match_oracle():
    for m in range(2, 257):
        o = oracle_mod(m)
        if o is None:
            with pytest.raises(awe.AweError) as ei:
                awe.get_encoding_info(awe.ENC_MOD, m)
            assert ei.value.status == awe.ERR_UNSUPPORTED
            continue
        info = awe.get_encoding_info(awe.ENC_MOD, m)
        assert info["r"] == o.r, m
        assert info["w"] == o.w, m
        assert info["ell"] == [l for _, _, l in o.products], m
        assert info["alpha"] == o.planes_a, m


@pytest.mark.parametrize("m", [5, 8, 13, 31, 61, 89, 149, 151, 157])
def test_mod_tables_match_oracle(m):
    lo, T = awe.get_plane_table(awe.ENC_MOD, m, awe.SIDE_A)
    assert lo == 0
    assert np.array_equal(T, modm.plane_table(oracle_mod(m)))


def test_selected_moduli_have_schemes(paper):
    with open("tests/golden/moduli_fp64_k16384.txt") as f:
        lines = [l for l in f if l.strip() and not l.startswith("#")]
    ms = [int(x) for x in lines[0].split()]
    assert sum(awe.get_encoding_info(awe.ENC_MOD, m)["r"] for m in ms) == int(lines[1])


def test_plane_bytes():
    for enc, npl in ((awe.ENC_AWE6, 6), (awe.ENC_B13, 3), (awe.ENC_AWE4, 4)):
        assert awe.plane_bytes(enc, 0, awe.SIDE_A, 8192, 8192) == npl * 8192 * 8192 // 2
        # ragged: rows up to a multiple of 32, K up to a multiple of K_PAD
        assert awe.plane_bytes(enc, 0, awe.SIDE_A, 33, 129) == npl * 64 * awe.K_PAD // 2
        assert awe.plane_bytes(enc, 0, awe.SIDE_A, 33, awe.K_PAD + 1) == npl * 64 * 2 * awe.K_PAD // 2
        assert awe.plane_bytes(enc, 0, awe.SIDE_A, 0, 100) == 0
    ws = awe.workspace_bytes(awe.ENC_AWE4, 0, 100, 50, 300)
    a = awe.plane_bytes(awe.ENC_AWE4, 0, awe.SIDE_A, 100, 300)
    b = awe.plane_bytes(awe.ENC_AWE4, 0, awe.SIDE_B, 50, 300)
    assert ws == (a + 255) // 256 * 256 + b


def test_residue_number_system_host_checks():
    fp64 = [5, 7, 8, 9, 11, 13, 31, 37, 41, 43, 47, 53, 59, 61, 67, 71, 73, 79, 83, 89, 149, 151, 157]
    assert awe.crt_workspace_bytes(fp64, 4096, 4096, 16384) > 23 * 4096 * 4096 * 6
    for bad in ([4, 6], [1, 3], [300], [], list(range(2, 40))):
        with pytest.raises(awe.AweError) as e:
            awe.crt_workspace_bytes(bad, 4, 4, 4)
        assert e.value.status == awe.ERR_INVALID_VALUE
    # product above 2^127
    big = [251, 241, 239, 233, 229, 227, 223, 211, 199, 197, 193, 191, 181, 179, 173, 167, 163]
    with pytest.raises(awe.AweError):
        awe.crt_workspace_bytes(big, 4, 4, 4)
    L = awe.lib()
    fake = ctypes.c_void_p(4096)
    arr = (ctypes.c_int32 * 3)(3, 5, 7)
    # uniqueness: 105 <= 2 K bound_a bound_b, rejected before anything is enqueued
    assert L.awe_gemm_crt(8, 8, 16384, fake, 16384, fake, 8, 1, 1, arr, 3, fake, None, 8, fake,
                          1 << 40, None, None) == awe.ERR_OVERFLOW
    # a modulus without a scheme in the supported families
    arr2 = (ctypes.c_int32 * 2)(251, 3)
    assert L.awe_gemm_crt(8, 8, 1, fake, 1, fake, 8, 1, 1, arr2, 2, fake, None, 8, fake, 1 << 40,
                          None, None) == awe.ERR_UNSUPPORTED
    # residues accept moduli that are not coprime; reconstruction does not
    arr3 = (ctypes.c_int32 * 2)(4, 6)
    assert L.awe_residues(fake, 0, 4, 4, 1, arr3, 2, fake, 16, None, None) == awe.OK
    assert L.awe_crt(fake, 16, 4, 4, 4, arr3, 2, fake, None, 4, None) == awe.ERR_INVALID_VALUE
    assert L.awe_residues(fake, 4, 4, 4, 1, arr, 3, fake, 15, None, None) == awe.ERR_INVALID_VALUE


def test_error_paths_host_only():
    L = awe.lib()
    i = awe.EncodingInfo()
    assert L.awe_get_encoding_info(99, 0, ctypes.byref(i)) == awe.ERR_INVALID_VALUE
    assert L.awe_get_encoding_info(awe.ENC_MOD, 1, ctypes.byref(i)) == awe.ERR_INVALID_VALUE
    assert L.awe_get_encoding_info(awe.ENC_MOD, 300, ctypes.byref(i)) == awe.ERR_UNSUPPORTED
    assert L.awe_get_encoding_info(awe.ENC_AWE6, 0, None) == awe.ERR_INVALID_VALUE
    fake = 1 << 40  # never dereferenced: every call below fails its argument checks first
    # int32 output overflow: 128 * 128 * 131072 > 2^31 - 1
    assert L.awe_gemm_exact(awe.ENC_AWE6, 64, 64, 131072, fake, 131072, fake, 64, fake, 64, awe.I32,
                            fake, 1 << 40, None, None) == awe.ERR_OVERFLOW
    # workspace too small
    assert L.awe_gemm_exact(awe.ENC_AWE6, 64, 64, 64, fake, 64, fake, 64, fake, 64, awe.I32,
                            fake, 10, None, None) == awe.ERR_WORKSPACE
    assert L.awe_gemm_exact(awe.ENC_AWE6, 64, 64, 64, fake, 64, fake, 64, fake, 64, awe.I32,
                            None, 0, None, None) == awe.ERR_WORKSPACE
    # leading dimensions and sizes
    assert L.awe_gemm_exact(awe.ENC_AWE6, 64, 64, 64, fake, 63, fake, 64, fake, 64, awe.I32,
                            fake, 1 << 40, None, None) == awe.ERR_INVALID_VALUE
    assert L.awe_gemm_exact(awe.ENC_AWE6, -1, 64, 64, fake, 64, fake, 64, fake, 64, awe.I32,
                            fake, 1 << 40, None, None) == awe.ERR_INVALID_VALUE
    assert L.awe_gemm_exact(awe.ENC_MOD, 64, 64, 64, fake, 64, fake, 64, fake, 64, awe.I32,
                            fake, 1 << 40, None, None) == awe.ERR_INVALID_VALUE
    assert L.awe_gemm_exact(awe.ENC_AWE6, 64, 64, 64, None, 64, fake, 64, fake, 64, awe.I32,
                            fake, 1 << 40, None, None) == awe.ERR_INVALID_VALUE
    assert L.awe_gemm_exact(awe.ENC_AWE6, 64, 64, 64, fake, 64, fake, 64, fake, 64, 7,
                            fake, 1 << 40, None, None) == awe.ERR_INVALID_VALUE
    # fold segment must be a multiple of K_PAD within the encoding's bound
    assert L.awe_gemm_planes(awe.ENC_AWE6, 0, 64, 64, 1024, fake, fake, fake, 64, awe.I32, 100,
                             None) == awe.ERR_INVALID_VALUE
    assert L.awe_gemm_planes(awe.ENC_AWE6, 0, 64, 64, 1024, fake, fake, fake, 64, awe.I32,
                             awe.K_PAD // 2, None) == awe.ERR_INVALID_VALUE
    big = awe.get_encoding_info(awe.ENC_AWE6)["k_seg"] + awe.K_PAD
    assert L.awe_gemm_planes(awe.ENC_AWE6, 0, 64, 64, 1024, fake, fake, fake, 64, awe.I32, big,
                             None) == awe.ERR_INVALID_VALUE
    # residues are written as int32 only
    assert L.awe_gemm_planes(awe.ENC_MOD, 13, 64, 64, 64, fake, fake, fake, 64, awe.I64, 0,
                             None) == awe.ERR_INVALID_VALUE
    assert L.awe_gemm_mod(126, 64, 64, 64, fake, 64, fake, 64, fake, 64, fake, 1 << 40, None,
                          None) == awe.ERR_UNSUPPORTED
    # encode: bad side, small leading dimension, NULL
    assert L.awe_encode(awe.ENC_AWE6, 0, 5, fake, 64, 64, 64, fake, None, None) == awe.ERR_INVALID_VALUE
    assert L.awe_encode(awe.ENC_AWE6, 0, awe.SIDE_A, fake, 64, 64, 32, fake, None, None) == awe.ERR_INVALID_VALUE
    assert L.awe_encode(awe.ENC_AWE6, 0, awe.SIDE_B, fake, 64, 64, 32, fake, None, None) == awe.ERR_INVALID_VALUE
    assert L.awe_encode(awe.ENC_AWE6, 0, awe.SIDE_A, None, 64, 64, 64, fake, None, None) == awe.ERR_INVALID_VALUE
    assert L.awe_last_error().decode() != ""
    assert L.awe_status_string(awe.ERR_OVERFLOW).decode() != ""


def test_empty_problems_are_noops():
    L = awe.lib()
    # M = 0 or N = 0: success, nothing enqueued (pointers are never touched)
    assert L.awe_gemm_exact(awe.ENC_AWE6, 0, 64, 64, None, 64, None, 64, None, 64, awe.I32,
                            None, 0, None, None) == awe.OK
    assert L.awe_gemm_planes(awe.ENC_AWE6, 0, 64, 0, 64, None, None, None, 0, awe.I32, 0,
                             None) == awe.OK
    assert L.awe_encode(awe.ENC_AWE6, 0, awe.SIDE_A, None, 0, 64, 64, None, None, None) == awe.OK


def test_library_imports_no_device_allocation_routine():
    # the library allocates no memory itself (awe_gemm_exact_noalloc relies on it): its dynamic
    # imports hold no HIP allocation or free routine
    import shutil
    import subprocess

    if not shutil.which("nm"):
        pytest.skip("nm not found")
    out = subprocess.run(["nm", "-D", "--undefined-only", awe.LIB_PATH], stdout=subprocess.PIPE,
                         text=True, check=True).stdout
    names = [l.split()[-1].split("@")[0] for l in out.splitlines() if l.strip()]
    assert "hipGetSymbolAddress" in names
    bad = [n for n in names if n.startswith("hip") and any(w in n for w in ("Malloc", "Free", "Alloc", "MemPool"))]
    assert not bad, bad


def test_noalloc_limit_matches_header():
    import re
    with open(awe.HEADER) as f:
        m = re.search(r"#define AWE_NOALLOC_MAX_BYTES \(\(size_t\)(\d+) << (\d+)\)", f.read())
    assert int(m.group(1)) << int(m.group(2)) == awe.NOALLOC_MAX_BYTES
