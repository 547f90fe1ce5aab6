"""Oracle (test infrastructure only): congruence (mod m) schemes, Sec. 5.3.

A mod-m scheme relaxes the identity of Definition 4.1 to a congruence modulo m,
with integer reconstruction coefficients, and requires the encoding of each
side to represent every residue (a -> w . a mod m surjective on the admissible
tuples).  The paper gives the moduli with a single product and the weights
that make two-limb encodings cover Z/m; its three-product records are not
part of the text.  This module restates the three families used here:

* single limb (r = 1): w = (1); S itself must be a complete residue system;
* one Karatsuba-type step (r = 3): two limbs, w = v = (1, W), planes a0, a1 and
  p a0 + u a1 on both sides; matching the coefficients of a0b0, a0b1 + a1b0 and
  a1b1 gives t = W (p u)^-1, lambda_00 = 1 - t p^2, lambda_11 = W^2 - t u^2,
  lambda_c = t (all mod m);
* two limbs, all four pairs (r = 4): w = v = (1, W), lambda_ij = W^(i+j).

Search order (a reading: the paper's search space for these records is not
given): the smallest family that exists; within the Karatsuba family the plane
(p, u) in the order listed in KARATSUBA_PLANES, then the smallest W; within the
direct family the smallest W.  Residue tables use the same choice rule as the
exact schemes (smallest largest |plane|, then smallest sum of |limb|, then the
reversed limb tuple in ascending order), with the full set S (cap 12).
Reconstruction coefficients are kept as balanced residues in (-m/2, m/2].
"""
import math
from itertools import product as _cartesian

import numpy as np

from .schemes import S, S_SET, dot

KARATSUBA_PLANES = ((1, 1), (1, -1), (1, 2), (1, -2), (2, 1), (2, -1))
CAP = 12


def balanced(x, m):
    x %= m
    return x - m if x > m // 2 else x


def single_limb_surjective(m):
    """S covers every residue mod m with one limb (Sec. 5.3: one product)."""
    return {s % m for s in S} == set(range(m))


def two_limb_residues(W, m, plane=None):
    """Residues a0 + W a1 mod m over limb pairs in S^2 (with plane value in S if given)."""
    out = set()
    for a0, a1 in _cartesian(S, repeat=2):
        if plane is not None and (plane[0] * a0 + plane[1] * a1) not in S_SET:
            continue
        out.add((a0 + W * a1) % m)
    return out


def two_limb_covers(W, m, plane=None):
    return len(two_limb_residues(W, m, plane)) == m


class ModScheme:
    def __init__(self, m, family, w, products, planes_a, planes_b, params):
        self.m = m
        self.family = family          # "single", "karatsuba" or "direct"
        self.w = tuple(w)             # same weights on both sides
        self.products = products      # list of (alpha, beta, lam) with integer lam
        self.planes_a = planes_a
        self.planes_b = planes_b
        self.params = params

    @property
    def r(self):
        return len(self.products)


def find_scheme(m):
    """The mod-m scheme used for modulus m (search order in the module header), or None."""
    if m < 2:
        return None
    if single_limb_surjective(m):
        e = (1,)
        return ModScheme(m, "single", (1,), [(e, e, 1)], [e], [e], {})
    for p, u in KARATSUBA_PLANES:
        if math.gcd(p * u, m) != 1:
            continue
        for W in range(2, m):
            if not two_limb_covers(W, m, (p, u)):
                continue
            t = (W * pow(p * u, -1, m)) % m
            lam00 = balanced(1 - t * p * p, m)
            lam11 = balanced(W * W - t * u * u, m)
            lamc = balanced(t, m)
            e0, e1, c = (1, 0), (0, 1), (p, u)
            prods = [(e0, e0, lam00), (e1, e1, lam11), (c, c, lamc)]
            return ModScheme(m, "karatsuba", (1, W), prods, [e0, e1, c], [e0, e1, c],
                             {"p": p, "u": u, "W": W})
    for W in range(2, m):
        if two_limb_covers(W, m):
            e0, e1 = (1, 0), (0, 1)
            prods = [(e0, e0, balanced(1, m)), (e0, e1, balanced(W, m)),
                     (e1, e0, balanced(W, m)), (e1, e1, balanced(W * W, m))]
            return ModScheme(m, "direct", (1, W), prods, [e0, e1], [e0, e1], {"W": W})
    return None


def _admissible(planes, p):
    out = []
    for a in _cartesian(S, repeat=p):
        if all(dot(c, a) in S_SET and abs(dot(c, a)) <= CAP for c in planes):
            out.append(a)
    return out


def _key(a, planes):
    return (max(abs(dot(c, a)) for c in planes), sum(abs(x) for x in a), tuple(reversed(a)))


def residue_table(sch):
    """residue x in [0, m) -> chosen limb tuple."""
    best = {}
    for a in _admissible(sch.planes_a, len(sch.w)):
        x = dot(sch.w, a) % sch.m
        k = _key(a, sch.planes_a)
        if x not in best or k < best[x][0]:
            best[x] = (k, a)
    assert len(best) == sch.m, "encoding not surjective"
    return {x: best[x][1] for x in range(sch.m)}


def plane_table(sch):
    """T[x, k] = value of stored plane k for residue x (int64)."""
    limbs = residue_table(sch)
    T = np.zeros((sch.m, len(sch.planes_a)), dtype=np.int64)
    for x in range(sch.m):
        for k, c in enumerate(sch.planes_a):
            T[x, k] = dot(c, limbs[x])
    return T


def encode_planes(sch, X):
    """Table lookup per residue -> array [planes, *X.shape]."""
    T = plane_table(sch)
    X = np.asarray(X, dtype=np.int64)
    if X.size and (X.min() < 0 or X.max() >= sch.m):
        raise ValueError("residue outside [0, m)")
    return np.moveaxis(T[X], -1, 0)


def identity_mod_all_pairs(sch):
    """Congruence identity over every admissible pair of limb tuples (Sec. 5.3)."""
    TA = _admissible(sch.planes_a, len(sch.w))
    PA = np.array([[dot(c, a) for c in sch.planes_a] for a in TA], dtype=np.int64)
    WA = np.array([dot(sch.w, a) for a in TA], dtype=np.int64)
    acc = np.zeros((len(TA), len(TA)), dtype=np.int64)
    for a, b, lam in sch.products:
        acc += lam * np.outer(PA[:, sch.planes_a.index(a)], PA[:, sch.planes_b.index(b)])
    return bool(np.all((acc - np.outer(WA, WA)) % sch.m == 0))


def scheme_gemm_mod(sch, A, B):
    """The mod-m run-time procedure in plain int64: (sum_k lam_k P_k) mod m."""
    PA = encode_planes(sch, A)
    PB = encode_planes(sch, B)
    acc = np.zeros((A.shape[0], B.shape[1]), dtype=np.int64)
    for a, b, lam in sch.products:
        acc += lam * (PA[sch.planes_a.index(a)] @ PB[sch.planes_b.index(b)])
    return (acc % sch.m).astype(np.int32)


def crt_bits_needed(K, width):
    """log2 of the bound the product of the moduli must exceed: 2 K B^2, B = 2^(M-1) - 1 (Sec. 5.3)."""
    B = 2 ** (width - 1) - 1
    return math.log2(2 * K * B * B)


def select_moduli(K, width, m_max=256):
    """Pairwise-coprime moduli with the fewest products whose product exceeds 2 K B^2.

    Sec. 5.3 chooses the set by an integer program over the per-modulus table.
    Here: depth-first branch and bound over the moduli that have a scheme, in
    order of decreasing bits per product (ties: larger m first); a set replaces
    the incumbent only when it needs strictly fewer products.
    """
    need = crt_bits_needed(K, width)
    cands = []
    for m in range(2, m_max + 1):
        sch = find_scheme(m)
        if sch is not None:
            cands.append((m, sch.r, math.log2(m)))
    cands.sort(key=lambda c: (-c[2] / c[1], -c[0]))
    best = [None, math.inf]

    def dfs(i, chosen, bits, cost):
        if bits > need:
            if cost < best[1]:
                best[0], best[1] = list(chosen), cost
            return
        if i >= len(cands):
            return
        eff = cands[i][2] / cands[i][1]
        if cost + (need - bits) / eff >= best[1] - 1e-12:
            return
        m, r, b = cands[i]
        if all(math.gcd(m, c) == 1 for c in chosen):
            chosen.append(m)
            dfs(i + 1, chosen, bits + b, cost + r)
            chosen.pop()
        dfs(i + 1, chosen, bits, cost)

    dfs(0, [], 0.0, 0)
    return sorted(best[0]), best[1]
