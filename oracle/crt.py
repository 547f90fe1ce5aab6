"""Oracle (test infrastructure only): the residue number system around the
mod-m products (Sec. 5.3).

A residue number system represents an integer by its residues modulo
pairwise coprime moduli m_1..m_n and recovers it by the Chinese remainder
theorem; the recovery is unique for integers in a range of width
M = m_1 ... m_n, here the symmetric range (-M/2, M/2], which is why the
paper asks for M > 2 K B_A B_B (the product C = A B satisfies |C| <= K B_A B_B).

Written with Python integers, in the textbook form of the theorem:
X = sum_i r_i (M/m_i) [(M/m_i)^-1 mod m_i]  mod M, then shifted into the
symmetric range.  Nothing here touches a GPU or shares code with the library.
"""
import math

import numpy as np


def residues(x, m):
    """x mod m in [0, m) for an int64 array (Python's remainder has the divisor's sign)."""
    x = np.asarray(x, dtype=np.int64)
    return np.remainder(x, m).astype(np.uint8 if m <= 256 else np.int64)


def modulus_product(moduli):
    return math.prod(int(m) for m in moduli)


def pairwise_coprime(moduli):
    ms = [int(m) for m in moduli]
    return all(math.gcd(a, b) == 1 for i, a in enumerate(ms) for b in ms[i + 1:])


def reconstruct(res, moduli):
    """The integer X in (-M/2, M/2] with X = res[i] (mod moduli[i]) for every i.

    ``res`` is a list of equal-shape integer arrays (or scalars), one per modulus;
    returns a numpy object array of Python ints (or an int for scalar input)."""
    ms = [int(m) for m in moduli]
    assert pairwise_coprime(ms)
    Mtot = modulus_product(ms)
    scalar = np.isscalar(res[0]) or np.ndim(res[0]) == 0
    acc = 0 if scalar else np.zeros(np.shape(res[0]), dtype=object)
    for r, m in zip(res, ms):
        q = Mtot // m
        coef = q * pow(q % m, -1, m)  # = 1 mod m, = 0 mod every other modulus
        rr = int(r) if scalar else np.asarray(r).astype(object)
        acc = acc + rr * coef
    if scalar:
        x = acc % Mtot
        return x - Mtot if 2 * x > Mtot else x
    x = np.vectorize(lambda v: v % Mtot, otypes=[object])(acc)
    return np.vectorize(lambda v: v - Mtot if 2 * v > Mtot else v, otypes=[object])(x)


def to_double(x):
    """Python ints -> float64, rounded to nearest (ties to even), as Python's float() does."""
    if np.ndim(x) == 0:
        return float(int(x))
    return np.vectorize(lambda v: float(int(v)), otypes=[np.float64])(x)


def split_words(x):
    """Python ints (|x| < 2^127) -> (lo uint64, hi int64) with x = hi * 2^64 + lo."""
    x = np.asarray(x, dtype=object)
    lo = np.vectorize(lambda v: int(v) & ((1 << 64) - 1), otypes=[np.uint64])(x)
    hi = np.vectorize(lambda v: int(v) >> 64, otypes=[np.int64])(x)
    return lo, hi
