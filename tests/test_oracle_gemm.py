"""Pins for the oracle's plain integer product (CPU only).

The oracle is a C triple loop; these tests tie it to things other than itself:
numpy's int64 matmul (a library routine the oracle does not use), Python's
arbitrary-precision integers on tiny inputs, permutation and transposition
identities that catch swapped or transposed operands, and the closed forms of
the structured accumulation-stress operands.
"""
import numpy as np
import pytest

from oracle import gemm as og
from paper_2609_24519_amd import inputs


def _np_ref(A, B):
    return A.astype(np.int64) @ B.astype(np.int64)


@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (3, 5, 7), (17, 33, 65), (64, 48, 129), (5, 0, 3), (0, 4, 4)])
def test_matches_numpy_int64(M, N, K):
    A, B = inputs.int8_pair(M, N, K, seed=M * 100 + N * 10 + K)
    assert np.array_equal(og.gemm_i64(A, B), _np_ref(A, B))


def test_zero_reduction_length():
    A = np.zeros((4, 0), np.int8)
    B = np.zeros((0, 3), np.int8)
    assert np.array_equal(og.gemm_i64(A, B), np.zeros((4, 3), np.int64))


def test_python_bigint_bruteforce():
    A, B = inputs.int8_pair(4, 3, 6, seed=7)
    C = og.gemm_i64(A, B)
    for i in range(4):
        for j in range(3):
            assert C[i, j] == sum(int(A[i, k]) * int(B[k, j]) for k in range(6))


def test_permutation_and_transpose():
    rng = np.random.default_rng(3)
    A, B = inputs.int8_pair(9, 11, 13, seed=5)
    perm = rng.permutation(11)
    P = np.zeros((11, 11), np.int8)
    P[np.arange(11), perm] = 1  # (B P)[:, perm[i]] = B[:, i]
    C = og.gemm_i64(A, B)
    CP = og.gemm_i64(A, np.ascontiguousarray(B @ P))
    assert np.array_equal(CP[:, perm], C)
    # (A B)^T = B^T A^T
    CT = og.gemm_i64(np.ascontiguousarray(B.T), np.ascontiguousarray(A.T))
    assert np.array_equal(CT, C.T)
    # identity right factor
    I = np.eye(13, dtype=np.int8)
    assert np.array_equal(og.gemm_i64(A, I), A.astype(np.int64))


def test_extreme_values_closed_form():
    K = 1000
    A = np.full((2, K), -128, np.int8)
    A[1] = 127
    B = np.full((K, 2), -128, np.int8)
    B[:, 1] = 127
    C = og.gemm_i64(A, B)
    assert C.tolist() == [[16384 * K, -16256 * K], [-16256 * K, 16129 * K]]


def test_stress_operands_closed_forms():
    M = N = 8
    K = 4096
    A, B = inputs.stress_operands(M, N, K, seed=0)
    C = og.gemm_i64(A, B)
    h = K // 2
    lo, hi = -128, 127
    closed = {
        (0, 0): K * lo * lo, (0, 1): K * lo * hi, (1, 1): K * hi * hi,
        (3, 3): h * (lo * lo + hi * hi), (0, 3): h * (lo * lo + lo * hi), (1, 3): h * (hi * lo + hi * hi),
    }
    for i in range(M):
        for j in range(N):
            ti, tj = i % 4, j % 4
            key = (min(ti, tj), max(ti, tj))
            if key in closed:
                assert C[i, j] == closed[key], (i, j)
    assert C[0, 0] == 2 ** 14 * K  # the largest magnitude an int8 dot product of length K reaches
    # random-sign rows against constant columns: sums of the row's entries times the constant
    for i in range(M):
        if i % 4 == 2:
            s = int(A[i].astype(np.int64).sum())
            assert C[i, 0] == s * lo and C[i, 1] == s * hi


def test_sampled_matches_full():
    A, B = inputs.int8_pair(70, 90, 50, seed=11)
    C = og.gemm_i64(A, B)
    rows = np.array([0, 5, 69, 33])
    cols = np.array([89, 0, 7])
    assert np.array_equal(og.gemm_i64_sampled(A, B, rows, cols), C[rows][:, cols])


@pytest.mark.parametrize("m", [2, 13, 89, 157])
def test_mod_matches_numpy(m):
    A, B = inputs.residue_pair(21, 19, 77, m)
    ref = (A.astype(np.int64) @ B.astype(np.int64)) % m
    C = og.gemm_mod(m, A, B)
    assert C.dtype == np.int32 and np.array_equal(C, ref)
    rows, cols = np.array([3, 0, 20]), np.array([18, 1])
    assert np.array_equal(og.gemm_mod_sampled(m, A, B, rows, cols), ref[rows][:, cols])


def test_mod_python_ints():
    m = 151
    A, B = inputs.residue_pair(3, 2, 9, m)
    C = og.gemm_mod(m, A, B)
    for i in range(3):
        for j in range(2):
            assert C[i, j] == sum(int(A[i, k]) * int(B[k, j]) for k in range(9)) % m


def _py_product(A, B):
    M, K = A.shape
    N = B.shape[1]
    return [[sum(int(A[i, k]) * int(B[k, j]) for k in range(K)) for j in range(N)] for i in range(M)]


def test_wide_product_python_ints_fp16_extremes():
    """gemm_i64_wide (the checker of the 12-bit significand scheme) against Python integers on
    int16 inputs in [-2048, 2047], with the -2048 / 2047 extremes placed so that some results are
    negative (their low word, read as int64, is negative) and some reach K * 2048^2."""
    rng = np.random.default_rng(21)
    K = 37
    A = inputs.uniform(rng, (6, K), -2048, 2047, np.int16)
    B = inputs.uniform(rng, (K, 5), -2048, 2047, np.int16)
    A[0, :] = -2048
    B[:, 0] = -2048  # C[0, 0] = K 2^22
    B[:, 1] = 2047   # C[0, 1] = -K 2048 2047 < 0
    A[1, :] = 2047
    C = og.gemm_i64_wide(A, B)
    assert C.dtype == np.int64
    assert C.tolist() == _py_product(A, B)
    assert C[0, 0] == K * 2048 * 2048 and C[0, 1] == -K * 2048 * 2047
    assert (C < 0).any() and (C > 0).any()


def test_wide_product_int64_boundaries():
    """Results at the edges of int64: -2^63 and 2^63 - 1 fit and come back exactly; 2^63 and a
    product far beyond int64 (low word alone would look like a valid int64) must be refused."""
    lo_edge = og.gemm_i64_wide(np.array([[-(1 << 31)]]), np.array([[1 << 32]]))
    assert int(lo_edge[0, 0]) == -(1 << 63)
    x = 3037000499  # x^2 = 2^63 - 5,928,526,806 < 2^63 - 1
    hi_edge = og.gemm_i64_wide(np.array([[x, 1]]), np.array([[x], [(1 << 63) - 1 - x * x]]))
    assert int(hi_edge[0, 0]) == (1 << 63) - 1
    with pytest.raises(AssertionError):
        og.gemm_i64_wide(np.array([[1 << 31]]), np.array([[1 << 32]]))  # 2^63: low word reads as -2^63
    with pytest.raises(AssertionError):
        og.gemm_i64_wide(np.array([[1 << 40, 3]]), np.array([[1 << 40], [5]]))  # 2^80 + 15


def test_full_oracle_hash_file_matches_oracle():
    """tests/golden/full_oracle_sha256.txt (used by the GPU tests of the large workloads) lists
    the two 8192^3 products, every modulus of the residue set and the stress workload, and its
    entry for m = 5 is the SHA-256 of the oracle's C recomputed here (8 s on a few cores)."""
    import hashlib
    import os

    golden = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
    with open(os.path.join(golden, "moduli_fp64_k16384.txt")) as f:
        moduli = [int(x) for x in [l for l in f if l.strip() and not l.startswith("#")][0].split()]
    rows = {}
    with open(os.path.join(golden, "full_oracle_sha256.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                name, dims, dtype, digest = [x.strip() for x in line.split("|")]
                rows[name] = (dims, dtype, digest)
    assert set(rows) == {"residues mod %d" % m for m in moduli} | {"stress", "int8 8192", "int4xint8 8192"}
    assert rows["stress"][:2] == ("4096 4096 65536", "int64")
    assert rows["int8 8192"][:2] == rows["int4xint8 8192"][:2] == ("8192 8192 8192", "int32")
    A, B = inputs.residue_pair(4096, 4096, 4096, 5)
    C = og.gemm_mod(5, A, B)
    assert rows["residues mod 5"][:2] == ("4096 4096 4096", "int32")
    assert hashlib.sha256(np.ascontiguousarray(C).tobytes()).hexdigest() == rows["residues mod 5"][2]
