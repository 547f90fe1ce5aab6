"""Seeded synthetic inputs for the exact integer products.

This module draws random matrices and nothing else: it holds none of the
method's arithmetic, so both the library's tests and the oracle may consume
its arrays.  The paper measures no datasets; every workload here is synthetic
and uniform over the operand's integer range, with the structured
accumulation-stress pattern described in ``stress_operands``.
"""
import numpy as np


def uniform(rng, shape, lo, hi, dtype=np.int8):
    """Integers uniform in [lo, hi] (both ends included)."""
    return rng.integers(lo, hi, size=shape, endpoint=True, dtype=dtype)


def int8_pair(M, N, K, seed, a_range=(-128, 127), b_range=(-128, 127)):
    """A (M x K) then B (K x N) from one generator seeded with ``seed``."""
    rng = np.random.default_rng(seed)
    A = uniform(rng, (M, K), *a_range)
    B = uniform(rng, (K, N), *b_range)
    return A, B


def residue_pair(M, N, K, m, seed=None):
    """Residue operands uniform in [0, m - 1] as uint8; seed defaults to m."""
    rng = np.random.default_rng(m if seed is None else seed)
    A = uniform(rng, (M, K), 0, m - 1, np.uint8)
    B = uniform(rng, (K, N), 0, m - 1, np.uint8)
    return A, B


def _stress_rows(n, K, rng):
    """Rows of {-128, 127}: row type i mod 4 = all -128, all 127, random sign, alternating."""
    X = np.empty((n, K), dtype=np.int8)
    kk = np.arange(K)
    alt = np.where(kk % 2 == 0, -128, 127).astype(np.int8)
    for i in range(n):
        t = i % 4
        if t == 0:
            X[i] = -128
        elif t == 1:
            X[i] = 127
        elif t == 2:
            X[i] = np.where(rng.integers(0, 2, size=K, dtype=np.int8) == 0, -128, 127)
        else:
            X[i] = alt
    return X


def stress_operands(M, N, K, seed=0):
    """Accumulation stress: every entry -128 or 127.

    Row i of A and column j of B follow type i mod 4 (resp. j mod 4): all -128,
    all 127, random sign, or alternating -128/127 along k (even k gives -128).
    Dot products of the constant types reach the largest magnitudes an int8
    product can, e.g. 16384 K for two all -128 vectors.
    """
    rng = np.random.default_rng(seed)
    A = _stress_rows(M, K, rng)
    Bt = _stress_rows(N, K, rng)
    return A, np.ascontiguousarray(Bt.T)


def sample_tiles(M, N, ntiles, tile, seed):
    """Row/column index lists of ``ntiles`` random tile x tile output tiles plus the 4 corners."""
    rng = np.random.default_rng(seed)
    tiles = []
    tm, tn = min(tile, M), min(tile, N)
    for _ in range(ntiles):
        i0 = int(rng.integers(0, M - tm + 1))
        j0 = int(rng.integers(0, N - tn + 1))
        tiles.append((i0, j0))
    tiles += [(0, 0), (0, N - tn), (M - tm, 0), (M - tm, N - tn)]
    return [(np.arange(i0, i0 + tm), np.arange(j0, j0 + tn)) for i0, j0 in tiles]
