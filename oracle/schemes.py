"""Oracle (test infrastructure only): the paper's exact encodings, written out.

Everything here follows the paper's definitions in plain Python / numpy int64,
for checking by eye against the paper.  Nothing here is shared with the HIP
library.

* The storable set S (Sec. 3.1): the E2M1 values doubled.
* Limb decomposition N = sum_i w_i a_i with a_i in S (Sec. 3.2), and the
  base-13 positional form with carries and its coverage recurrence.
* A scheme (Definition 4.1): products k = 1..r, each with an A-side plane
  coefficient vector alpha_k, a B-side vector beta_k and an integer ell_k, a
  power-of-two denominator D and weights w, v, such that
  sum_k (ell_k / D) (alpha_k . a)(beta_k . b) = (w . a)(v . b)
  for all admissible limb tuples a, b.
* Admissible tuples (Definition 4.1): limb tuples in S^p whose every plane
  value lies in S (here also within a stated cap on |stored value|).
* Coverage (Sec. 4.2): the half-width of the contiguous range of w . a.
* The exact-accumulation bound K* = floor(2^24 / (n_g c_A c_B)) (Sec. 3.4).
* The run-time procedure (Alg. 1): table lookup -> planes -> r integer
  products -> (sum_k ell_k P_k) / D.

Reading adopted where the paper is silent (which admissible tuple encodes a
given integer; the paper only says "table lookup"): among the admissible tuples
with every stored plane value within the cap and w . a = x, take the one that
minimises, in order, (1) the largest |plane value|, (2) the sum of |limb|,
(3) the limb tuple (a_{p-1}, ..., a_0) in ascending lexicographic order.
Base-13 digits instead follow the positional carry rule with the
least-magnitude representative of each residue class (its worked example in
the paper is a figure whose content is lost).
"""
from fractions import Fraction
from itertools import product as _cartesian

import numpy as np

# Sec. 3.1: doubling the E2M1 values gives these 15 integers.
S = (0, 1, -1, 2, -2, 3, -3, 4, -4, 6, -6, 8, -8, 12, -12)
S_SET = frozenset(S)

# E2M1 values (undoubled), OCP MX element format: sign, 2 exponent bits, 1 mantissa bit.
E2M1_VALUES = (0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0)


def e2m1_value(code):
    """Value of a 4-bit E2M1 code (bit 3 = sign), from the format's fields."""
    sign = -1.0 if code & 8 else 1.0
    e = (code >> 1) & 3
    m = code & 1
    if e == 0:  # subnormal: m * 2^(1-bias) * 0.5 with bias 1
        mag = 0.5 * m
    else:
        mag = (1.0 + 0.5 * m) * 2.0 ** (e - 1)
    return sign * mag


class Scheme:
    """One exact scheme in the form of Definition 4.1.

    products: list of (alpha, beta, ell) with alpha a length-p tuple, beta a
    length-q tuple and ell an integer (lambda = ell / D).
    """

    def __init__(self, name, w, v, products, D, cap_a, cap_b, range_a, range_b, n_g=1):
        self.name = name
        self.w = tuple(w)
        self.v = tuple(v)
        self.products = [(tuple(a), tuple(b), int(l)) for a, b, l in products]
        self.D = int(D)
        self.cap_a = cap_a
        self.cap_b = cap_b
        self.range_a = range_a  # inclusive input range the A table must cover
        self.range_b = range_b
        self.n_g = n_g
        # sides whose limbs are base-13 positional digits instead of the choice rule
        self.positional = ()
        # side -> (x -> limb tuple) for encodings whose limbs a rule fixes outright
        self.limb_rule = {}
        # element format of every stored plane ("e2m1" unless stated)
        self.formats_a = None
        self.formats_b = None
        # distinct stored planes per side, in order of first use
        self.planes_a = []
        self.planes_b = []
        for a, b, _ in self.products:
            if a not in self.planes_a:
                self.planes_a.append(a)
            if b not in self.planes_b:
                self.planes_b.append(b)

    @property
    def r(self):
        return len(self.products)

    @property
    def p(self):
        return len(self.w)

    @property
    def q(self):
        return len(self.v)


def dot(c, a):
    return sum(ci * ai for ci, ai in zip(c, a))


# ---------------------------------------------------------------------------
# The paper's schemes (Sec. 4.3 and App. A coefficient tables)
# ---------------------------------------------------------------------------
def _e(i, n):
    return tuple(1 if j == i else 0 for j in range(n))


def _pair(i, j, n):
    return tuple(1 if t in (i, j) else 0 for t in range(n))


INT8_RANGE = (-128, 127)
INT4_RANGE = (-8, 7)


def awe6():
    """INT8 x INT8 in 6 products, weights (1, 29, 37), Sec. 4.3 / App. A.

    Products in the paper's order P00, P11, P22, P01, P02, P12 with
    P_ii = a_i b_i and P_ij = (a_i + a_j)(b_i + b_j); every stored value
    capped at 6 (App. A), which still covers 148.
    """
    ell = (-65, -261, 259, 29, 37, 1073)
    planes = [_e(0, 3), _e(1, 3), _e(2, 3), _pair(0, 1, 3), _pair(0, 2, 3), _pair(1, 2, 3)]
    prods = [(pl, pl, l) for pl, l in zip(planes, ell)]
    return Scheme("awe6", (1, 29, 37), (1, 29, 37), prods, 1, 6, 6, INT8_RANGE, INT8_RANGE)


def awe6_alt():
    """The alternative 6-product solution, weights (1, 11, 39), App. A.

    Same plane structure as awe6; coverage 134 uses the full set S (cap 12).
    """
    ell = (-49, -319, 1053, 11, 39, 429)
    planes = [_e(0, 3), _e(1, 3), _e(2, 3), _pair(0, 1, 3), _pair(0, 2, 3), _pair(1, 2, 3)]
    prods = [(pl, pl, l) for pl, l in zip(planes, ell)]
    return Scheme("awe6_alt", (1, 11, 39), (1, 11, 39), prods, 1, 12, 12, INT8_RANGE, INT8_RANGE)


def awe4():
    """INT4 x INT8 in 4 products, App. A: A = 3a0 + 5a1, B = 5b0 + 3b1 + 42b2.

    A planes (a1, a0, a0 + 2a1, 2a0 + a1); B planes (b0, b1 - b2, b2, b0 + 2b1);
    2AB = 35 P1 - 42 P2 + 210 P3 + 15 P4 (D = 2); plane values within 3 on A
    and 8 on B.
    """
    alpha = [(0, 1), (1, 0), (1, 2), (2, 1)]
    beta = [(1, 0, 0), (0, 1, -1), (0, 0, 1), (1, 2, 0)]
    ell = (35, -42, 210, 15)
    prods = list(zip(alpha, beta, ell))
    return Scheme("awe4", (3, 5), (5, 3, 42), prods, 2, 3, 8, INT4_RANGE, INT8_RANGE)


def b13():
    """Base-13 positional baseline (Sec. 3.2): weights (1, 13, 169), all 9 limb pairs.

    ell_ij = 13^(i+j); equal coefficients may share an accumulator (n_g = 3,
    Sec. 3.4 and Alg. 1), so the products are listed grouped by coefficient.
    """
    prods = []
    for s in range(5):
        for i in range(3):
            j = s - i
            if 0 <= j < 3:
                prods.append((_e(i, 3), _e(j, 3), 13 ** s))
    s = Scheme("b13", (1, 13, 169), (1, 13, 169), prods, 1, 8, 8, INT8_RANGE, INT8_RANGE, n_g=3)
    s.positional = ("a", "b")
    return s


def ternary():
    """{0, +-1} x INT8 in 3 products (Sec. 6.2): a ternary weight is one limb (w = (1,)),
    the INT8 side takes base-13 positional limbs, and C = sum_j 13^j (a)(b_j)."""
    prods = [((1,), _e(j, 3), 13 ** j) for j in range(3)]
    s = Scheme("ternary", (1,), (1, 13, 169), prods, 1, 1, 8, (-1, 1), INT8_RANGE)
    s.positional = ("b",)
    return s


def fp16_12():
    """FP16 x FP16 significands in 12 products, App. A: weights (1, 9, 71, 639) on both sides.

    With P_ij = a_i b_j and Q_kl = (a_{2k} + 2 a_{2k+1})(b_{2l} + 2 b_{2l+1}), k, l in {0, 1}:
    2AB = sum_{k,l} 71^(k+l) (-7 P_{2k,2l} + 126 P_{2k+1,2l+1} + 9 Q_kl), D = 2; stored values
    within 12.  Products are listed grouped by (k, l), in that order inside each group.
    The input range is the 12-bit two's-complement range (coverage 2160 reaches past it).
    """
    def q(k):
        return tuple(1 if t == 2 * k else (2 if t == 2 * k + 1 else 0) for t in range(4))

    prods = []
    for k in (0, 1):
        for l in (0, 1):
            o = 71 ** (k + l)
            prods.append((_e(2 * k, 4), _e(2 * l, 4), -7 * o))
            prods.append((_e(2 * k + 1, 4), _e(2 * l + 1, 4), 126 * o))
            prods.append((q(k), q(l), 9 * o))
    w = (1, 9, 71, 639)
    return Scheme("fp16_12", w, w, prods, 2, 12, 12, (-2048, 2047), (-2048, 2047))


# ---------------------------------------------------------------------------
# E4M3 (OCP FP8): sign, 4 exponent bits (bias 7), 3 mantissa bits; no infinities,
# S.1111.111 is NaN.  Small integers (|v| <= 16) are exact.
# ---------------------------------------------------------------------------
def e4m3_value(code):
    sign = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 15
    m = code & 7
    if e == 15 and m == 7:
        return float("nan")
    if e == 0:
        return sign * (m / 8.0) * 2.0 ** (1 - 7)
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)


def e4m3_code(v):
    """Code of an exactly representable value (searched over all codes)."""
    for c in range(256):
        if e4m3_value(c) == v and not (v == 0 and c & 0x80):
            return c
    raise ValueError("%r is not an E4M3 value" % (v,))


FP8FP4_EPS = (0, 1, -1, 2, -2, 3, -3, 4, -4, 6, -6, 8, -8)


def fp8fp4_limbs(x):
    """App. A: x = 13 h + 5 eps with eps in FP8FP4_EPS; eps is fixed by x mod 13, since
    5 eps = x (mod 13) and the set holds every residue class mod 13 exactly once."""
    eps = next(e for e in FP8FP4_EPS if (5 * e - x) % 13 == 0)
    return ((x - 5 * eps) // 13, eps)


def fp8fp4():
    """INT8 x INT8 with 2 FP8 products and 1 FP4 product, App. A.

    A = 13 h + 5 eps, B = 13 h' + 5 eps'; P1 = h h' and P2 = (h + eps)(h' + eps') with the
    planes h, h + eps stored in FP8 (E4M3), P3 = eps eps' in FP4; AB = 104 P1 + 65 P2 - 40 P3,
    D = 1.  Plane values stay within 14 (c_A = c_B = 14).
    """
    planes = [(1, 0), (1, 1), (0, 1)]
    prods = [(pl, pl, l) for pl, l in zip(planes, (104, 65, -40))]
    s = Scheme("fp8fp4", (13, 5), (13, 5), prods, 1, 14, 14, INT8_RANGE, INT8_RANGE)
    s.limb_rule = {"a": fp8fp4_limbs, "b": fp8fp4_limbs}
    s.formats_a = s.formats_b = ["e4m3", "e4m3", "e2m1"]
    return s


PAPER_SCHEMES = {"b13": b13, "awe6": awe6, "awe6_alt": awe6_alt, "awe4": awe4, "ternary": ternary,
                 "fp16_12": fp16_12, "fp8fp4": fp8fp4}


# ---------------------------------------------------------------------------
# E2M3 (OCP MX FP6): sign bit 5, 2 exponent bits (bias 1), 3 mantissa bits;
# every one of the 64 codes is finite.
# ---------------------------------------------------------------------------
def e2m3_value(code):
    sign = -1.0 if code & 0x20 else 1.0
    e = (code >> 3) & 3
    m = code & 7
    if e == 0:  # subnormal: m / 8 * 2^(1 - bias)
        return sign * (m / 8.0)
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 1)


def e2m3_code(v):
    """Code of an exactly representable value (searched over all codes)."""
    for c in range(64):
        if e2m3_value(c) == v and not (v == 0 and c & 0x20):
            return c
    raise ValueError("%r is not an E2M3 value" % (v,))


def contiguous_half_width(values, scale):
    """Largest X such that every integer in [-X, X] is scale times a value of the format
    (the contiguous integer part that Sec. 3.3 measures)."""
    ints = {int(scale * v) for v in values if float(scale * v).is_integer()}
    X = 0
    while X + 1 in ints and -(X + 1) in ints:
        X += 1
    return X


# Integers n of an E2M3 plane are stored as the E2M3 value n / 8; a block scale of
# 2^3 on each operand restores n_a n_b in every product (Sec. 4.5 form of the scale).
FP6_SCALE = 8


def fp6k3_limbs(x):
    """x = a0 + 16 a1 with the balanced base-16 digit a0 in [-8, 7]."""
    a0 = (x + 8) % 16 - 8
    return (a0, (x - a0) // 16)


def fp6k3():
    """INT8 x INT8 in 3 E2M3 (FP6) products: one Karatsuba-type step on base-16 limbs.

    Sec. 3.3: a Karatsuba-type step forms a product of limb sums, and the sums must be
    storable; for a format with an m-bit significand the contiguous integer part is
    [-2^(m+1), 2^(m+1)], wide enough only from m = 3.  E2M3 has m = 3: with n stored as
    n / 8 it holds every integer of [-16, 16].  Base-16 limbs of an INT8 value lie in
    [-8, 8], so a0 + a1 fits.  With P1 = a0 b0, P2 = a1 b1, P3 = (a0 + a1)(b0 + b1):
    AB = P1 + 16 (P3 - P1 - P2) + 256 P2 = -15 P1 + 240 P2 + 16 P3, D = 1.
    Not one of the paper's catalogued schemes: the same construction on the FP6 format.
    """
    planes = [(1, 0), (0, 1), (1, 1)]
    prods = [(pl, pl, l) for pl, l in zip(planes, (-15, 240, 16))]
    s = Scheme("fp6k3", (1, 16), (1, 16), prods, 1, 16, 16, INT8_RANGE, INT8_RANGE)
    s.limb_rule = {"a": fp6k3_limbs, "b": fp6k3_limbs}
    s.formats_a = s.formats_b = ["e2m3", "e2m3", "e2m3"]
    return s


def e8m0_value(code):
    """OCP MX E8M0 scale: 2^(code - 127) for code 0..254 (255 is NaN); powers of two only."""
    if code == 255:
        return float("nan")
    return 2.0 ** (code - 127)


def fp6p4():
    """INT8 x INT8 in 4 E2M3 products with the limb weights in the block scales (Sec. 4.5).

    The same base-16 limbs as fp6k3, x = a0 + 16 a1, but every limb pair is its own product:
    AB = a0 b0 + 16 a0 b1 + 16 a1 b0 + 256 a1 b1.  The weights are powers of two, which an
    E8M0 scale represents (Sec. 4.5), so each product's weight 16^(i+j) can ride in the
    scales of its two operands and all four products add into one FP32 accumulator.
    """
    planes = [(1, 0), (0, 1)]
    prods = [(planes[i], planes[j], 16 ** (i + j)) for i in range(2) for j in range(2)]
    s = Scheme("fp6p4", (1, 16), (1, 16), prods, 1, 16, 16, INT8_RANGE, INT8_RANGE)
    s.limb_rule = {"a": fp6k3_limbs, "b": fp6k3_limbs}
    s.formats_a = s.formats_b = ["e2m3", "e2m3"]
    return s


def shared_accumulator_kstar(s, F=24):
    """Sec. 3.4's condition for one FP32 accumulator that receives every product with its
    weight: each reduction index adds at most sum_k |ell_k| c_A(k) c_B(k) in magnitude
    (c the largest |value| of the product's planes), so partial sums stay exact integers
    for floor(2^F / that) indices."""
    _, TA = plane_table(s, "a")
    _, TB = plane_table(s, "b")
    ca = np.abs(TA).max(axis=0)
    cb = np.abs(TB).max(axis=0)
    per_index = sum(abs(l) * int(ca[s.planes_a.index(a)]) * int(cb[s.planes_b.index(b)])
                    for a, b, l in s.products)
    return (2 ** F) // per_index, per_index


VARIANT_SCHEMES = {"fp6k3": fp6k3, "fp6p4": fp6p4}
ALL_SCHEMES = dict(PAPER_SCHEMES, **VARIANT_SCHEMES)


# ---------------------------------------------------------------------------
# Identity checks (Sec. 4.2 coefficient-matrix equation; Sec. 4.7 all pairs)
# ---------------------------------------------------------------------------
def coefficient_matrix(s):
    """sum_k ell_k alpha_k beta_k^T as exact integers (p x q)."""
    M = [[0] * s.q for _ in range(s.p)]
    for a, b, l in s.products:
        for i in range(s.p):
            for j in range(s.q):
                M[i][j] += l * a[i] * b[j]
    return M


def coefficient_identity_holds(s):
    """Sec. 4.2: sum_k lambda_k alpha_k beta_k^T = w v^T, with lambda = ell / D."""
    M = coefficient_matrix(s)
    return all(Fraction(M[i][j], s.D) == s.w[i] * s.v[j] for i in range(s.p) for j in range(s.q))


def solve_ell(s):
    """Re-solve the reconstruction coefficients from the planes and weights alone.

    The coefficient-matrix equation is linear in lambda; solve it by exact
    rational Gaussian elimination (Sec. 4.6 decision step; Sec. 4.7 re-solves
    it independently).  Returns the list of Fractions, or None if the system
    has no unique solution.
    """
    rows = []
    rhs = []
    for i in range(s.p):
        for j in range(s.q):
            rows.append([Fraction(a[i] * b[j]) for a, b, _ in s.products])
            rhs.append(Fraction(s.w[i] * s.v[j]))
    n = s.r
    aug = [r + [y] for r, y in zip(rows, rhs)]
    piv_row = 0
    pivots = []
    for col in range(n):
        pr = next((r for r in range(piv_row, len(aug)) if aug[r][col] != 0), None)
        if pr is None:
            return None
        aug[piv_row], aug[pr] = aug[pr], aug[piv_row]
        pv = aug[piv_row][col]
        aug[piv_row] = [x / pv for x in aug[piv_row]]
        for r in range(len(aug)):
            if r != piv_row and aug[r][col] != 0:
                f = aug[r][col]
                aug[r] = [x - f * y for x, y in zip(aug[r], aug[piv_row])]
        pivots.append(col)
        piv_row += 1
    for r in range(piv_row, len(aug)):  # inconsistent rows
        if aug[r][n] != 0:
            return None
    return [aug[i][n] for i in range(n)]


# ---------------------------------------------------------------------------
# Admissible tuples, coverage, encoding tables (Definition 4.1, Sec. 4.2)
# ---------------------------------------------------------------------------
def admissible(planes, p, cap):
    """Limb tuples a in S^p whose every plane value is in S with |value| <= cap."""
    out = []
    for a in _cartesian(S, repeat=p):
        vals = [dot(c, a) for c in planes]
        if all(x in S_SET and abs(x) <= cap for x in vals):
            out.append(a)
    return out


def coverage(weights, tuples):
    """Half-width X of the contiguous range [-X, X] of w . a over the tuples."""
    vals = {dot(weights, a) for a in tuples}
    X = 0
    while (X + 1) in vals and -(X + 1) in vals:
        X += 1
    return X if 0 in vals else -1


def _choice_key(a, planes):
    vals = [abs(dot(c, a)) for c in planes]
    return (max(vals), sum(abs(x) for x in a), tuple(reversed(a)))


def encode_table(weights, planes, cap, lo, hi):
    """x -> chosen admissible limb tuple for every x in [lo, hi] (reading in the header)."""
    p = len(weights)
    best = {}
    for a in admissible(planes, p, cap):
        x = dot(weights, a)
        if lo <= x <= hi:
            k = _choice_key(a, planes)
            if x not in best or k < best[x][0]:
                best[x] = (k, a)
    missing = [x for x in range(lo, hi + 1) if x not in best]
    if missing:
        raise ValueError("range not covered: %s" % missing[:5])
    return {x: best[x][1] for x in range(lo, hi + 1)}


# Base-13 positional digits with carries (Sec. 3.2).
def b13_rep():
    """Least-magnitude element of S in each residue class mod 13."""
    rep = {}
    for s in sorted(S, key=abs):
        rep.setdefault(s % 13, s)
    assert len(rep) == 13  # S holds a complete residue system mod 13 (Sec. 3.2)
    return rep


def b13_digits(x, L=3):
    """x = sum_i 13^i a_i with a_i in S, by carries: a = rep[x mod 13], x <- (x - a) / 13."""
    rep = b13_rep()
    out = []
    for _ in range(L):
        a = rep[x % 13]
        out.append(a)
        x = (x - a) // 13
    if x != 0:
        raise ValueError("needs more than %d limbs" % L)
    return tuple(out)


def x_carry(L):
    """Contiguous half-width of L base-13 limbs: X(1) = 4, X(L) = 13 X(L-1) + 4 (Sec. 3.2)."""
    X = 4
    for _ in range(L - 1):
        X = 13 * X + 4
    return X


def k_star(n_g, c_a, c_b, F=24):
    """Sec. 3.4: K* = floor(2^F / (n_g c_A c_B)), F = 24 for FP32 accumulation."""
    return (2 ** F) // (n_g * c_a * c_b)


# ---------------------------------------------------------------------------
# Per-scheme tables: input value -> plane values
# ---------------------------------------------------------------------------
def limb_table(s, side):
    """x -> limb tuple for every x in the side's input range."""
    lo, hi = s.range_a if side == "a" else s.range_b
    if side in s.limb_rule:
        return {x: s.limb_rule[side](x) for x in range(lo, hi + 1)}
    if side in s.positional:
        return {x: b13_digits(x) for x in range(lo, hi + 1)}
    w = s.w if side == "a" else s.v
    planes = s.planes_a if side == "a" else s.planes_b
    cap = s.cap_a if side == "a" else s.cap_b
    return encode_table(w, planes, cap, lo, hi)


def plane_table(s, side):
    """(lo, T) with T[x - lo, k] = value of stored plane k for input x (int64)."""
    lo, hi = s.range_a if side == "a" else s.range_b
    planes = s.planes_a if side == "a" else s.planes_b
    limbs = limb_table(s, side)
    T = np.zeros((hi - lo + 1, len(planes)), dtype=np.int64)
    for x in range(lo, hi + 1):
        for k, c in enumerate(planes):
            T[x - lo, k] = dot(c, limbs[x])
    return lo, T


def stored_cap(s, side):
    """Largest |stored plane value| the chosen table uses (c_A or c_B)."""
    _, T = plane_table(s, side)
    return int(np.abs(T).max())


def encode_planes(s, side, X):
    """Alg. 1, first two loops: table lookup per entry -> array [planes, *X.shape]."""
    lo, T = plane_table(s, side)
    idx = np.asarray(X, dtype=np.int64) - lo
    if idx.size and (idx.min() < 0 or idx.max() >= T.shape[0]):
        raise ValueError("input outside the encoding's range")
    return np.moveaxis(T[idx], -1, 0)


def scheme_gemm(s, A, B):
    """Alg. 1 in plain int64: C = (sum_k ell_k (plane alpha_k of A)(plane beta_k of B)) / D.

    A is M x K (A-side inputs), B is K x N (B-side inputs).  Each integer
    product is a numpy int64 matmul (exact); the division by D is an exact
    shift whose remainder must be zero.
    """
    PA = encode_planes(s, "a", A)  # [planes_a, M, K]
    PB = encode_planes(s, "b", B)  # [planes_b, K, N]
    acc = np.zeros((A.shape[0], B.shape[1]), dtype=np.int64)
    for a, b, l in s.products:
        ka = s.planes_a.index(a)
        kb = s.planes_b.index(b)
        acc += l * (PA[ka] @ PB[kb])
    assert not np.any(acc % s.D), "reconstruction not divisible by D"
    return acc // s.D


def brute_force_pairs(s):
    """All input pairs (x, y): sum_k ell_k planeA_k(x) planeB_k(y) == D x y (Sec. 4.7)."""
    loa, TA = plane_table(s, "a")
    lob, TB = plane_table(s, "b")
    xs = np.arange(loa, loa + TA.shape[0], dtype=np.int64)
    ys = np.arange(lob, lob + TB.shape[0], dtype=np.int64)
    acc = np.zeros((xs.size, ys.size), dtype=np.int64)
    for a, b, l in s.products:
        ka = s.planes_a.index(a)
        kb = s.planes_b.index(b)
        acc += l * np.outer(TA[:, ka], TB[:, kb])
    return bool(np.array_equal(acc, s.D * np.outer(xs, ys)))


def identity_all_admissible(s, cap_a=None, cap_b=None):
    """Definition 4.1 identity over every admissible pair of limb tuples (Sec. 4.7)."""
    ca = s.cap_a if cap_a is None else cap_a
    cb = s.cap_b if cap_b is None else cap_b
    TA = admissible(s.planes_a, s.p, ca)
    TB = admissible(s.planes_b, s.q, cb)
    PA = np.array([[dot(c, a) for c in s.planes_a] for a in TA], dtype=np.int64)
    PB = np.array([[dot(c, b) for c in s.planes_b] for b in TB], dtype=np.int64)
    WA = np.array([dot(s.w, a) for a in TA], dtype=np.int64)
    VB = np.array([dot(s.v, b) for b in TB], dtype=np.int64)
    acc = np.zeros((len(TA), len(TB)), dtype=np.int64)
    for a, b, l in s.products:
        acc += l * np.outer(PA[:, s.planes_a.index(a)], PB[:, s.planes_b.index(b)])
    return bool(np.array_equal(acc, s.D * np.outer(WA, VB)))
