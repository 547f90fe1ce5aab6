"""Pins of the residue-number-system oracle (oracle/crt.py) and of the 128-bit
integer product (oracle/gemm.c) that the Ozaki-II path is checked against.

The theorem fixes the reconstruction (Sec. 5.3: unique for a modulus product
above 2 K B_A B_B); these tests pin the oracle to textbook facts, closed forms
and exact Python-integer arithmetic, so that a wrong inverse, a missing shift
into the symmetric range or a lost carry between the two 64-bit words fails.
"""
import math
import os

import numpy as np
import pytest

from oracle import crt
from oracle import gemm as og

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
B53 = (1 << 53) - 1


def _moduli():
    with open(os.path.join(GOLDEN, "moduli_fp64_k16384.txt")) as f:
        lines = [l for l in f if l.strip() and not l.startswith("#")]
    return [int(x) for x in lines[0].split()]


def test_textbook_example():
    # x = 2 mod 3, 3 mod 5, 2 mod 7 has the least solution 23 (the classical example)
    assert crt.reconstruct([2, 3, 2], [3, 5, 7]) == 23
    # the symmetric range (-M/2, M/2]: 105 - 23 = 82 is represented as -23
    assert crt.reconstruct([(-23) % 3, (-23) % 5, (-23) % 7], [3, 5, 7]) == -23


def test_fp64_set_meets_the_uniqueness_bound():
    ms = _moduli()
    assert crt.pairwise_coprime(ms)
    M = crt.modulus_product(ms)
    assert M > 2 * 16384 * B53 * B53                     # Sec. 5.3 condition at K = 16,384
    # and it is not met with any one modulus left out (the set is minimal for the bound)
    for m in ms:
        assert M // m <= 2 * 16384 * B53 * B53


def test_round_trip_over_the_symmetric_range():
    ms = _moduli()
    M = crt.modulus_product(ms)
    rng = np.random.default_rng(7)
    xs = [0, 1, -1, M // 2, -(M // 2) + 1, 16384 * B53 * B53, -16384 * B53 * B53]
    xs += [int.from_bytes(rng.bytes(16), "little") % M - M // 2 for _ in range(200)]
    for x in xs:
        assert crt.reconstruct([x % m for m in ms], ms) == x
    # vectorised form agrees with the scalar one
    arr = np.array(xs, dtype=object)
    rec = crt.reconstruct([np.array([x % m for x in xs], dtype=np.int64) for m in ms], ms)
    assert list(rec) == xs


def test_residues_are_non_negative():
    x = np.array([-1, -128, 0, 127, -(1 << 62), (1 << 62) - 1], dtype=np.int64)
    for m in (5, 13, 157, 256):
        r = crt.residues(x, m)
        assert r.min() >= 0 and r.max() < m
        assert all((int(v) - int(rv)) % m == 0 for v, rv in zip(x, r))


def test_words_round_trip():
    vals = [0, 1, -1, (1 << 64) - 1, -(1 << 64), (1 << 120) + 12345, -(1 << 126) + 7]
    lo, hi = crt.split_words(np.array(vals, dtype=object))
    assert [int(h) * (1 << 64) + int(l) for l, h in zip(lo, hi)] == vals


def test_double_rounding_facts():
    # IEEE round to nearest, ties to even (what float() of a Python int does)
    assert crt.to_double((1 << 53) + 1) == float(1 << 53)
    assert crt.to_double((1 << 53) + 3) == float((1 << 53) + 4)
    assert crt.to_double((1 << 64) + (1 << 11)) == float(1 << 64)
    assert crt.to_double((1 << 64) + (1 << 11) + 1) == float((1 << 64) + (1 << 12))
    assert crt.to_double(-((1 << 64) + (1 << 11) + 1)) == -float((1 << 64) + (1 << 12))


def test_int128_product_closed_forms():
    K = 16384
    A = np.full((2, K), B53, np.int64)
    B = np.full((K, 3), -B53, np.int64)
    C = og.gemm_i128(A, B)
    assert (C == -K * B53 * B53).all()                 # needs the high word
    lo, hi = og.gemm_i128(A, B, words=True)
    assert int(hi[0, 0]) < 0 and all(int(h) * (1 << 64) + int(l) == -K * B53 * B53
                                     for l, h in zip(lo.ravel(), hi.ravel()))
    # rank one: A = u 1^T, B = 1 v^T  =>  C = K u v^T
    rng = np.random.default_rng(3)
    u = rng.integers(-B53, B53, size=5, endpoint=True)
    v = rng.integers(-B53, B53, size=4, endpoint=True)
    K = 1000
    C = og.gemm_i128(np.repeat(u[:, None], K, 1), np.repeat(v[None, :], K, 0))
    assert all(C[i, j] == K * int(u[i]) * int(v[j]) for i in range(5) for j in range(4))
    # identity on the right returns A
    A = rng.integers(-B53, B53, size=(6, 9), endpoint=True)
    assert (og.gemm_i128(A, np.eye(9, dtype=np.int64)) == A.astype(object)).all()


def test_int128_product_against_python_integers():
    rng = np.random.default_rng(11)
    A = rng.integers(-B53, B53, size=(7, 37), endpoint=True)
    B = rng.integers(-B53, B53, size=(37, 5), endpoint=True)
    ref = np.array([[sum(int(A[i, k]) * int(B[k, j]) for k in range(37)) for j in range(5)]
                    for i in range(7)], dtype=object)
    assert (og.gemm_i128(A, B) == ref).all()
    rows, cols = np.array([6, 0, 3]), np.array([4, 1])
    assert (og.gemm_i128_sampled(A, B, rows, cols) == ref[rows][:, cols]).all()


def test_product_through_residues():
    # the whole residue route on the CPU: residues of A and B, products mod m, CRT
    ms = _moduli()
    rng = np.random.default_rng(5)
    A = rng.integers(-B53, B53, size=(4, 64), endpoint=True)
    B = rng.integers(-B53, B53, size=(64, 3), endpoint=True)
    res = [og.gemm_mod(m, crt.residues(A, m), crt.residues(B, m)) for m in ms]
    assert (crt.reconstruct(res, ms) == og.gemm_i128(A, B)).all()
