"""Pins for the oracle's encodings (CPU only).

Each check ties the oracle's scheme code to something the paper or the
mathematics fixes: the printed coverages, K* values and coefficients
(tests/golden/paper_values.txt, each line citing its passage), the E2M1 format
definition, exact rational re-solving of the reconstruction coefficients, and
brute force over every input pair.  The mutation tests plant a mistake in a
copy of a scheme and require the pins to catch it.
"""
import copy
from fractions import Fraction

import numpy as np
import pytest

from oracle import schemes as sc


def test_storable_set(paper):
    assert sorted(sc.S) == sorted(paper["storable_set"])
    # S is the E2M1 value set doubled (format definition, sign-magnitude codes 0..15)
    doubled = {int(2 * sc.e2m1_value(c)) for c in range(16)}
    assert doubled == set(sc.S)
    assert [sc.e2m1_value(c) for c in range(8)] == list(sc.E2M1_VALUES)


def test_b13_positional(paper):
    assert list(sc.b13().w) == paper["b13.weights"]
    assert [sc.x_carry(L) for L in (1, 2, 3)] == paper["b13.xcarry"]
    # X_carry(L) = (13^L - 1) / 3 (App. B closed form)
    assert all(sc.x_carry(L) == (13 ** L - 1) // 3 for L in range(1, 7))
    limbs3 = sc.admissible([(1, 0, 0), (0, 1, 0), (0, 0, 1)], 3, 12)
    assert sc.coverage((1, 13, 169), limbs3) == paper["b13.xcarry"][2]
    limbs2 = sc.admissible([(1, 0), (0, 1)], 2, 12)
    assert sc.coverage((1, 13), limbs2) == paper["b13.xcarry"][1]
    assert sc.b13().r == paper["b13.products"][0]
    for x in range(-128, 128):
        d = sc.b13_digits(x)
        assert sum(a * 13 ** i for i, a in enumerate(d)) == x
        assert all(a in sc.S_SET for a in d)
        assert d[2] in (-1, 0, 1)
    # the INT8 side of the ternary x INT8 construction has K* = 2^24 / (1 * 8): largest limb 8
    assert sc.stored_cap(sc.b13(), "a") == 8
    assert sc.k_star(1, 1, 8) == paper["kstar.ternary_int8"][0]


def test_awe6_printed(paper):
    s = sc.awe6()
    assert list(s.w) == paper["awe6.w"] and list(s.v) == paper["awe6.w"]
    assert [l for _, _, l in s.products] == paper["awe6.ell"]
    assert s.r == paper["awe6.products"][0]
    # re-solve the coefficients from planes and weights alone (independent verification)
    assert [f for f in sc.solve_ell(s)] == paper["awe6.ell"]
    assert sc.coefficient_identity_holds(s)
    cap6 = sc.admissible(s.planes_a, 3, 6)
    assert sc.coverage(s.w, cap6) == paper["awe6.coverage_cap6"][0]
    assert sc.coverage(s.w, sc.admissible(s.planes_a, 3, 12)) >= 127
    assert sc.stored_cap(s, "a") == 6 and sc.stored_cap(s, "b") == 6
    assert sc.k_star(1, 6, 6) == paper["awe6.kstar_cap6"][0]
    assert sc.k_star(1, 12, 12) == paper["awe6.kstar_fullS"][0]


def test_awe6_alt_printed(paper):
    s = sc.awe6_alt()
    assert list(s.w) == paper["awe6_alt.w"]
    assert [l for _, _, l in s.products] == paper["awe6_alt.ell"]
    assert [f for f in sc.solve_ell(s)] == paper["awe6_alt.ell"]
    full = sc.admissible(s.planes_a, 3, 12)
    assert sc.coverage(s.w, full) == paper["awe6_alt.coverage"][0]


def test_awe4_printed(paper):
    s = sc.awe4()
    assert list(s.w) == paper["awe4.w"] and list(s.v) == paper["awe4.v"]
    assert [l for _, _, l in s.products] == paper["awe4.ell"]
    assert s.D == paper["awe4.D"][0]
    lam = sc.solve_ell(s)
    assert [f * s.D for f in lam] == paper["awe4.ell"]
    assert sc.coefficient_identity_holds(s)
    assert [sc.stored_cap(s, "a"), sc.stored_cap(s, "b")] == paper["awe4.cap"]
    assert sc.k_star(1, *paper["awe4.cap"]) == paper["awe4.kstar"][0]


def test_kstar_formula(paper):
    assert sc.k_star(1, 127, 127) == paper["kstar.bf16_int8"][0]
    assert sc.k_star(1, 127, 1) == paper["kstar.bf16_ternary"][0]
    assert sc.k_star(1, 14, 14) == paper["kstar.fp8fp4"][0]


@pytest.mark.parametrize("name", ["b13", "awe6", "awe6_alt", "awe4", "ternary"])
def test_round_trip_and_storability(name):
    s = sc.PAPER_SCHEMES[name]()
    for side in ("a", "b"):
        lo, hi = s.range_a if side == "a" else s.range_b
        w = s.w if side == "a" else s.v
        planes = s.planes_a if side == "a" else s.planes_b
        cap = s.cap_a if side == "a" else s.cap_b
        limbs = sc.limb_table(s, side)
        for x in range(lo, hi + 1):
            a = limbs[x]
            assert sc.dot(w, a) == x
            assert all(l in sc.S_SET for l in a)
            for c in planes:
                assert sc.dot(c, a) in sc.S_SET and abs(sc.dot(c, a)) <= cap


@pytest.mark.parametrize("name", ["b13", "awe6", "awe6_alt", "awe4", "ternary"])
def test_brute_force_all_pairs(name):
    assert sc.brute_force_pairs(sc.PAPER_SCHEMES[name]())


@pytest.mark.parametrize("name", ["awe6", "awe6_alt", "awe4", "ternary"])
def test_identity_all_admissible(name):
    assert sc.identity_all_admissible(sc.PAPER_SCHEMES[name]())


def test_scheme_gemm_equals_plain_product():
    rng = np.random.default_rng(0)
    A = rng.integers(-128, 127, (13, 40), endpoint=True)
    B = rng.integers(-128, 127, (40, 9), endpoint=True)
    A4 = rng.integers(-8, 7, (13, 40), endpoint=True)
    for name in ("b13", "awe6", "awe6_alt"):
        assert np.array_equal(sc.scheme_gemm(sc.PAPER_SCHEMES[name](), A, B), A @ B)
    assert np.array_equal(sc.scheme_gemm(sc.awe4(), A4, B), A4 @ B)


def test_ternary_scheme(paper):
    # Sec. 6.2: {0, +-1} x INT8 takes 3 products; the INT8 side keeps its base-13 digits
    # (largest |digit| 8), the ternary side one limb, so K* = 2^24 / (1 * 8)
    s = sc.ternary()
    assert s.r == 3 and len(s.planes_a) == 1 and len(s.planes_b) == 3
    assert sc.stored_cap(s, "a") == 1 and sc.stored_cap(s, "b") == 8
    assert sc.k_star(1, sc.stored_cap(s, "a"), sc.stored_cap(s, "b")) == paper["kstar.ternary_int8"][0]
    assert sc.coefficient_identity_holds(s)
    rng = np.random.default_rng(4)
    A = rng.integers(-1, 1, (11, 50), endpoint=True)
    B = rng.integers(-128, 127, (50, 7), endpoint=True)
    assert np.array_equal(sc.scheme_gemm(s, A, B), A @ B)
    assert sc.limb_table(s, "b") == {x: sc.b13_digits(x) for x in range(-128, 128)}


def test_endpoints_are_covered():
    # the two's-complement endpoints -128 and -8 are encodable although the paper's
    # symmetric width convention does not require them
    for name in ("b13", "awe6", "awe6_alt"):
        assert -128 in sc.limb_table(sc.PAPER_SCHEMES[name](), "a")
    assert -8 in sc.limb_table(sc.awe4(), "a")


# ---- planted mistakes: the pins must fail ---------------------------------
def _mutate_ell(s, k, new):
    t = copy.deepcopy(s)
    a, b, _ = t.products[k]
    t.products[k] = (a, b, new)
    return t


@pytest.mark.parametrize("k", range(6))
def test_mutation_sign_flip_caught(k):
    s = sc.awe6()
    bad = _mutate_ell(s, k, -s.products[k][2])
    assert not sc.coefficient_identity_holds(bad)
    assert not sc.brute_force_pairs(bad)


def test_mutation_dropped_term_caught():
    s = sc.awe6()
    bad = copy.deepcopy(s)
    bad.products = bad.products[:-1]
    assert not sc.coefficient_identity_holds(bad)
    assert not sc.brute_force_pairs(bad)


def test_mutation_wrong_plane_caught():
    s = sc.awe4()
    bad = copy.deepcopy(s)
    a, b, l = bad.products[1]
    bad.products[1] = (a, (0, -1, 1), l)  # b2 - b1 instead of b1 - b2
    bad.planes_b[bad.planes_b.index(b)] = (0, -1, 1)
    assert not sc.coefficient_identity_holds(bad)
    assert not sc.brute_force_pairs(bad)


def test_mutation_wrong_weight_caught():
    s = sc.awe6()
    bad = copy.deepcopy(s)
    bad.w = (1, 29, 38)
    bad.v = (1, 29, 38)
    assert not sc.coefficient_identity_holds(bad)
    try:
        ok = sc.brute_force_pairs(bad)
    except ValueError:  # the weights may no longer cover the int8 range
        ok = False
    assert not ok


def test_fp16_12_scheme(paper):
    # App. A: FP16 x FP16 significands in 12 products
    s = sc.fp16_12()
    assert s.w == tuple(paper["fp16_12.w"]) and s.r == paper["fp16_12.products"][0]
    assert s.D == paper["fp16_12.D"][0]
    inner = paper["fp16_12.inner_ell"]
    o = paper["fp16_12.outer"][0]
    assert [l for _, _, l in s.products] == [x * o ** (k + l) for k in (0, 1) for l in (0, 1)
                                              for x in inner]
    assert len(s.planes_a) == 6 and len(s.planes_b) == 6
    assert sc.coefficient_identity_holds(s)
    # re-solving the coefficients from planes and weights alone gives the same ell / D
    assert sc.solve_ell(s) == [Fraction(l, s.D) for _, _, l in s.products]
    # coverage of the weights over the admissible tuples at cap 12, and the K* bound
    assert sc.coverage(s.w, sc.admissible(s.planes_a, 4, 12)) == paper["fp16_12.coverage"][0]
    ca, cb = sc.stored_cap(s, "a"), sc.stored_cap(s, "b")
    assert (ca, cb) == tuple(paper["fp16_12.cap"])
    assert sc.k_star(1, ca, cb) == paper["fp16_12.kstar"][0]


def test_fp16_12_all_input_pairs():
    # every pair of 12-bit inputs through the tables: sum_k ell_k planeA planeB = 2 x y
    s = sc.fp16_12()
    assert sc.brute_force_pairs(s)
    limbs = sc.limb_table(s, "a")
    assert all(sc.dot(s.w, limbs[x]) == x for x in range(-2048, 2048))


def test_e4m3_format_facts(paper):
    # OCP FP8 E4M3: 1.0, the largest normal 448, the smallest normal 2^-6 and subnormal 2^-9
    one, big, nmin, smin = paper["e4m3.codes"]
    assert sc.e4m3_value(one) == 1.0 and sc.e4m3_value(big) == 448.0
    assert sc.e4m3_value(nmin) == 2.0 ** -6 and sc.e4m3_value(smin) == 2.0 ** -9
    assert all(sc.e4m3_value(sc.e4m3_code(v)) == v for v in range(-16, 17))


def test_fp8fp4_scheme(paper):
    s = sc.fp8fp4()
    assert s.w == tuple(paper["fp8fp4.w"]) and [l for _, _, l in s.products] == paper["fp8fp4.ell"]
    assert sorted(sc.FP8FP4_EPS) == sorted(paper["fp8fp4.eps"])
    assert sorted(e % 13 for e in sc.FP8FP4_EPS) == list(range(13))  # one per residue class
    assert all(e in sc.S_SET for e in sc.FP8FP4_EPS)                  # the FP4 limb is storable
    assert sc.coefficient_identity_holds(s)
    assert sc.brute_force_pairs(s)                                     # all 65,536 int8 pairs
    limbs = sc.limb_table(s, "a")
    assert all(13 * h + 5 * e == x for x, (h, e) in limbs.items())
    caps = (sc.stored_cap(s, "a"), sc.stored_cap(s, "b"))
    assert caps == tuple(paper["fp8fp4.cap"])
    assert sc.k_star(1, *caps) == paper["kstar.fp8fp4"][0]
    # the FP8 planes hold exact E4M3 integers
    _, T = sc.plane_table(s, "a")
    assert all(sc.e4m3_value(sc.e4m3_code(int(v))) == v for v in np.unique(T[:, :2]))
    rng = np.random.default_rng(9)
    A = rng.integers(-128, 127, (9, 70), endpoint=True)
    B = rng.integers(-128, 127, (70, 6), endpoint=True)
    assert np.array_equal(sc.scheme_gemm(s, A, B), A @ B)


def test_e2m3_format_facts(paper):
    # OCP MX FP6 E2M3: 1.0, the largest value 7.5 and the smallest subnormal 0.125
    one, big, smin = paper["e2m3.codes"]
    assert sc.e2m3_value(one) == 1.0 and sc.e2m3_value(big) == 7.5 and sc.e2m3_value(smin) == 0.125
    vals = [sc.e2m3_value(c) for c in range(64)]
    assert max(vals) == 7.5 and min(vals) == -7.5 and len(set(vals)) == 63  # +0 and -0 coincide


def test_contiguous_part_threshold(paper):
    # Sec. 3.3: a format with an m-bit significand holds the contiguous integer range
    # [-2^(m+1), 2^(m+1)] (at the scale that makes its smallest step 1); E2M1 (m = 1)
    # gives S's [-4, 4], E2M3 and E4M3 (m = 3) give [-16, 16], the first wide enough
    # for a Karatsuba-type step.
    e2m1 = sc.E2M1_VALUES + tuple(-v for v in sc.E2M1_VALUES)
    assert sc.contiguous_half_width(e2m1, 2) == paper["contiguous.S"][0]
    assert sc.contiguous_half_width(e2m1, 2) == 2 ** (1 + 1)
    m = paper["karatsuba.min_m"][0]
    e2m3 = [sc.e2m3_value(c) for c in range(64)]
    assert sc.contiguous_half_width(e2m3, sc.FP6_SCALE) == 2 ** (m + 1)
    assert sc.contiguous_half_width([sc.e4m3_value(c) for c in range(256)], 1) == 2 ** (m + 1)
    # base-16 limb sums of INT8 values need [-16, 16]: inside E2M3's part, outside S's
    sums = {sum(sc.fp6k3_limbs(x)) for x in range(-128, 128)}
    assert max(abs(v) for v in sums) <= 2 ** (m + 1)
    assert max(abs(v) for v in sums) > paper["contiguous.S"][0]


def test_fp6k3_scheme():
    s = sc.fp6k3()
    limbs = sc.limb_table(s, "a")
    assert all(a0 + 16 * a1 == x and -8 <= a0 <= 7 and -8 <= a1 <= 8 for x, (a0, a1) in limbs.items())
    assert sc.coefficient_identity_holds(s)
    assert sc.brute_force_pairs(s)  # all 65,536 int8 pairs
    caps = (sc.stored_cap(s, "a"), sc.stored_cap(s, "b"))
    assert caps == (15, 15)
    assert sc.k_star(1, *caps) == 74565
    # every plane value is n with n / 8 an E2M3 value, coded as sign bit 5 | |n|
    _, T = sc.plane_table(s, "a")
    for n in np.unique(T):
        assert sc.e2m3_value(sc.e2m3_code(n / sc.FP6_SCALE)) * sc.FP6_SCALE == n
        assert sc.e2m3_code(n / sc.FP6_SCALE) == (0x20 if n < 0 else 0) | abs(int(n))
    rng = np.random.default_rng(11)
    A = rng.integers(-128, 127, (9, 70), endpoint=True)
    B = rng.integers(-128, 127, (70, 6), endpoint=True)
    assert np.array_equal(sc.scheme_gemm(s, A, B), A @ B)


@pytest.mark.parametrize("k,delta", [(0, 1), (1, -1), (2, 1)])
def test_fp6k3_mutation_caught(k, delta):
    s = sc.fp6k3()
    bad = _mutate_ell(s, k, s.products[k][2] + delta)
    assert not sc.coefficient_identity_holds(bad)
    assert not sc.brute_force_pairs(bad)


def test_e8m0_scale_format(paper):
    # OCP MX E8M0: an exponent with bias 127 and no significand, so powers of two only
    one, lo, hi, nan = paper["e8m0.codes"]
    assert sc.e8m0_value(one) == 1.0 and sc.e8m0_value(lo) == 2.0 ** -127 and sc.e8m0_value(hi) == 2.0 ** 127
    assert sc.e8m0_value(nan) != sc.e8m0_value(nan)
    values = {sc.e8m0_value(c) for c in range(255)}
    assert all(v == 2.0 ** round(np.log2(v)) for v in values)


def test_weights_in_scales(paper):
    # Sec. 4.5: a limb weight can ride in an E8M0 scale only if it is a power of two; AWE6's
    # weights (1, 29, 37) cannot (the paper's example), the base-16 weights of fp6p4 can, with
    # plane i of each operand carrying 16^i on top of the 2^3 that stores n as n / 8
    scales = {sc.e8m0_value(c) for c in range(255)}
    assert [w in scales for w in sc.awe6().w] == [True, False, False]
    s = sc.fp6p4()
    for a, b, l in s.products:
        i, j = a.index(1), b.index(1)
        sa = sc.e8m0_value(127 + 3 + 4 * i)
        sb = sc.e8m0_value(127 + 3 + 4 * j)
        assert sa in scales and sb in scales
        assert (sa / sc.FP6_SCALE) * (sb / sc.FP6_SCALE) == l


def test_fp6p4_scheme():
    s = sc.fp6p4()
    assert s.r == 4 and s.planes_a == [(1, 0), (0, 1)]
    assert sc.coefficient_identity_holds(s)
    assert sc.brute_force_pairs(s)  # all 65,536 int8 pairs
    # one shared accumulator: each reduction index adds at most (8 + 16*8)^2 = 18496, which
    # the input pair x = y = 120 (a0 = -8, a1 = 8) attains; K* = floor(2^24 / 18496)
    kstar, per_index = sc.shared_accumulator_kstar(s)
    assert (kstar, per_index) == (907, 136 * 136)
    lo, TA = sc.plane_table(s, "a")
    terms = sum(abs(l) * np.outer(np.abs(TA[:, s.planes_a.index(a)]), np.abs(TA[:, s.planes_a.index(b)]))
                for a, b, l in s.products)
    assert terms.max() == per_index and terms[120 - lo, 120 - lo] == per_index
    rng = np.random.default_rng(13)
    A = rng.integers(-128, 127, (9, 70), endpoint=True)
    B = rng.integers(-128, 127, (70, 6), endpoint=True)
    assert np.array_equal(sc.scheme_gemm(s, A, B), A @ B)


@pytest.mark.parametrize("k", range(4))
def test_fp6p4_mutation_caught(k):
    s = sc.fp6p4()
    bad = _mutate_ell(s, k, 2 * s.products[k][2])
    assert not sc.coefficient_identity_holds(bad)
    assert not sc.brute_force_pairs(bad)
