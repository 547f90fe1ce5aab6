"""Oracle (test infrastructure only): ctypes wrapper of ``gemm.c``.

``gemm.c`` is the plain definition of the exact integer product C = A B
(Sec. 1 and the postcondition of Alg. 1), of its residue C mod m (Sec. 5.3),
and of the wide product of int64 matrices a residue number system
reconstructs (Sec. 5.3), accumulated in 128 bits.  ``build()`` compiles it with gcc; nothing here touches a GPU.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gemm.c")
_LIB = os.path.join(_HERE, "liboracle_gemm.so")
_lib = None

_I64 = ctypes.c_int64
_P = ctypes.c_void_p


def build(force=True):
    """Compile gemm.c into liboracle_gemm.so (gcc, OpenMP)."""
    if not force and os.path.exists(_LIB):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", _SRC, "-o", tmp])
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        lib.oracle_gemm_i8_i64.argtypes = [_I64, _I64, _I64, _P, _I64, _P, _I64, _P, _I64]
        lib.oracle_gemm_i8_i64_sampled.argtypes = [_I64, _P, _I64, _P, _I64, _P, _I64, _P, _I64, _P]
        lib.oracle_gemm_u8_mod.argtypes = [_I64, _I64, _I64, _I64, _P, _I64, _P, _I64, _P, _I64]
        lib.oracle_gemm_u8_mod_sampled.argtypes = [_I64, _I64, _P, _I64, _P, _I64, _P, _I64, _P, _I64, _P]
        lib.oracle_gemm_i64_i128.argtypes = [_I64, _I64, _I64, _P, _I64, _P, _I64, _P, _P, _I64]
        lib.oracle_gemm_i64_i128_sampled.argtypes = [_I64, _P, _I64, _P, _I64, _P, _I64, _P, _I64,
                                                     _P, _P]
        lib.oracle_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def num_threads():
    """OpenMP threads the oracle loops use."""
    return int(_load().oracle_num_threads())


def gemm_i64(A, B):
    """Exact C = A B for int8 A (M x K) and int8 B (K x N); returns int64 M x N."""
    A = np.ascontiguousarray(A, dtype=np.int8)
    B = np.ascontiguousarray(B, dtype=np.int8)
    M, K = A.shape
    K2, N = B.shape
    assert K == K2
    C = np.empty((M, N), dtype=np.int64)
    if M and N:
        _load().oracle_gemm_i8_i64(M, N, K, _ptr(A), K, _ptr(B), N, _ptr(C), N)
    return C


def gemm_i64_sampled(A, B, rows, cols):
    """Exact (A B)[rows][:, cols] without forming the full product."""
    A = np.ascontiguousarray(A, dtype=np.int8)
    B = np.ascontiguousarray(B, dtype=np.int8)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    M, K = A.shape
    K2, N = B.shape
    assert K == K2
    assert rows.size == 0 or (rows.min() >= 0 and rows.max() < M)
    assert cols.size == 0 or (cols.min() >= 0 and cols.max() < N)
    C = np.empty((rows.size, cols.size), dtype=np.int64)
    if rows.size and cols.size:
        _load().oracle_gemm_i8_i64_sampled(rows.size, _ptr(rows), cols.size, _ptr(cols), K,
                                           _ptr(A), K, _ptr(B), N, _ptr(C))
    return C


def gemm_mod(m, A, B):
    """(A B) mod m as non-negative int32, for uint8 residue operands."""
    A = np.ascontiguousarray(A, dtype=np.uint8)
    B = np.ascontiguousarray(B, dtype=np.uint8)
    M, K = A.shape
    K2, N = B.shape
    assert K == K2 and m >= 1
    C = np.empty((M, N), dtype=np.int32)
    if M and N:
        _load().oracle_gemm_u8_mod(m, M, N, K, _ptr(A), K, _ptr(B), N, _ptr(C), N)
    return C


def gemm_mod_sampled(m, A, B, rows, cols):
    """(A B)[rows][:, cols] mod m without forming the full product."""
    A = np.ascontiguousarray(A, dtype=np.uint8)
    B = np.ascontiguousarray(B, dtype=np.uint8)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    M, K = A.shape
    K2, N = B.shape
    assert K == K2
    assert rows.size == 0 or (rows.min() >= 0 and rows.max() < M)
    assert cols.size == 0 or (cols.min() >= 0 and cols.max() < N)
    C = np.empty((rows.size, cols.size), dtype=np.int32)
    if rows.size and cols.size:
        _load().oracle_gemm_u8_mod_sampled(m, rows.size, _ptr(rows), cols.size, _ptr(cols), K,
                                           _ptr(A), K, _ptr(B), N, _ptr(C))
    return C


def _join128(lo, hi):
    """Two int64 words per entry -> numpy object array of Python ints hi * 2^64 + lo."""
    out = np.empty(lo.shape, dtype=object)
    flat_lo, flat_hi, flat = lo.ravel(), hi.ravel(), out.ravel()
    for i in range(flat.size):
        flat[i] = (int(flat_hi[i]) << 64) + int(flat_lo[i])
    return out


def gemm_i128(A, B, words=False):
    """Exact C = A B for int64 A (M x K) and B (K x N), with sum_k |a b| < 2^127.

    Returns a numpy object array of Python ints, or with ``words=True`` the pair
    (lo uint64, hi int64) with C = hi * 2^64 + lo."""
    A = np.ascontiguousarray(A, dtype=np.int64)
    B = np.ascontiguousarray(B, dtype=np.int64)
    M, K = A.shape
    K2, N = B.shape
    assert K == K2
    lo = np.zeros((M, N), dtype=np.uint64)
    hi = np.zeros((M, N), dtype=np.int64)
    if M and N:
        _load().oracle_gemm_i64_i128(M, N, K, _ptr(A), K, _ptr(B), N, _ptr(lo), _ptr(hi), N)
    return (lo, hi) if words else _join128(lo, hi)


def gemm_i128_sampled(A, B, rows, cols, words=False):
    """Exact (A B)[rows][:, cols] for int64 operands without forming the full product."""
    A = np.ascontiguousarray(A, dtype=np.int64)
    B = np.ascontiguousarray(B, dtype=np.int64)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    M, K = A.shape
    K2, N = B.shape
    assert K == K2
    assert rows.size == 0 or (rows.min() >= 0 and rows.max() < M)
    assert cols.size == 0 or (cols.min() >= 0 and cols.max() < N)
    lo = np.zeros((rows.size, cols.size), dtype=np.uint64)
    hi = np.zeros((rows.size, cols.size), dtype=np.int64)
    if rows.size and cols.size:
        _load().oracle_gemm_i64_i128_sampled(rows.size, _ptr(rows), cols.size, _ptr(cols), K,
                                             _ptr(A), K, _ptr(B), N, _ptr(lo), _ptr(hi))
    return (lo, hi) if words else _join128(lo, hi)


def gemm_i64_wide(A, B):
    """Exact C = A B for integer operands of any width up to int64 whose product fits int64
    (e.g. int16 significands): the 128-bit loop, checked to fit, as int64."""
    lo, hi = gemm_i128(np.asarray(A, dtype=np.int64), np.asarray(B, dtype=np.int64), words=True)
    C = lo.view(np.int64)
    assert np.array_equal(hi, np.where(C < 0, -1, 0)), "product exceeds int64"
    return C
