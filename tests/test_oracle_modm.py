"""Pins for the oracle's congruence (mod m) schemes (CPU only).

Ties the residue code to the facts the paper prints in Sec. 5.3: the moduli a
single product handles, the moduli two base-13 limbs cover, and the free
weights that extend that set, plus the CRT bound and exhaustive congruence
checks of every scheme used.
"""
import math
import os
from functools import lru_cache

import numpy as np
import pytest

from oracle import modm

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@lru_cache(maxsize=None)
def scheme(m):
    return modm.find_scheme(m)


def test_single_product_moduli(paper):
    got = [m for m in range(2, 257) if modm.single_limb_surjective(m)]
    assert got == paper["mod.single_product"]


def test_base13_two_limb_coverage(paper):
    got = [m for m in range(2, 226) if modm.two_limb_covers(13, m)]
    want = list(range(2, paper["mod.base13_upto"][0] + 1)) + paper["mod.base13_extra"]
    assert got == want


def test_free_weights(paper):
    for m, W in zip(paper["mod.free_weight_moduli"], paper["mod.free_weights"]):
        assert modm.two_limb_covers(W, m)
        assert not modm.two_limb_covers(13, m)


def test_crt_bound(paper):
    K, width = paper["crt.k"][0], paper["crt.width"][0]
    bits = modm.crt_bits_needed(K, width)
    assert abs(bits - (1 + math.log2(K) + 2 * math.log2(2 ** (width - 1) - 1))) < 1e-9
    assert 120.9 < bits < 121.1


@pytest.mark.parametrize("m", [2, 9, 11, 13, 31, 47, 89, 149, 157])
def test_schemes_are_valid(m):
    sch = scheme(m)
    assert sch is not None
    assert modm.identity_mod_all_pairs(sch)
    T = modm.plane_table(sch)
    limbs = modm.residue_table(sch)
    for x in range(m):
        assert modm.dot(sch.w, limbs[x]) % m == x
    assert set(np.unique(T)).issubset(set(modm.S))


@pytest.mark.parametrize("m", [7, 37, 151])
def test_scheme_gemm_mod(m):
    sch = scheme(m)
    rng = np.random.default_rng(m)
    A = rng.integers(0, m - 1, (11, 30), endpoint=True)
    B = rng.integers(0, m - 1, (30, 7), endpoint=True)
    assert np.array_equal(modm.scheme_gemm_mod(sch, A, B), (A @ B) % m)


def test_family_sizes():
    assert scheme(13).r == 1 and scheme(11).r == 1
    assert scheme(31).r == 3 and scheme(89).r == 3
    assert scheme(149).r == 4 and scheme(151).r == 4 and scheme(157).r == 4


def test_mutation_wrong_lambda_caught():
    sch = modm.find_scheme(31)
    a, b, lam = sch.products[2]
    sch.products[2] = (a, b, lam + 1)
    assert not modm.identity_mod_all_pairs(sch)


def test_selected_moduli_golden():
    with open(os.path.join(GOLDEN, "moduli_fp64_k16384.txt")) as f:
        lines = [l for l in f if l.strip() and not l.startswith("#")]
    want = [int(x) for x in lines[0].split()]
    total = int(lines[1])
    got, cost = modm.select_moduli(16384, 54)
    assert got == want and cost == total
    assert sum(scheme(m).r for m in got) == total
    assert all(math.gcd(a, b) == 1 for i, a in enumerate(got) for b in got[i + 1:])
    assert sum(math.log2(m) for m in got) > modm.crt_bits_needed(16384, 54)
