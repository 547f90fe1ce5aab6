// Host-side encoding tables: the schemes of the paper, the limb-tuple choice,
// the packed E2M1 lookup tables the encoder kernel uses, and a self-check of
// every table before it is used (the verifier of Sec. 4.7 applied to the
// tables actually shipped to the GPU).
#include <algorithm>
#include <climits>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <memory>
#include <mutex>
#include <numeric>
#include <tuple>
#include <vector>

#include "awe_internal.h"

namespace awe {
namespace {

// Sec. 3.1: the doubled E2M1 values.
constexpr int kS[15] = {0, 1, -1, 2, -2, 3, -3, 4, -4, 6, -6, 8, -8, 12, -12};
constexpr int kMag[8] = {0, 1, 2, 3, 4, 6, 8, 12};

bool in_S(int x) {
  for (int s : kS)
    if (s == x) return true;
  return false;
}

int64_t pmod(int64_t x, int64_t m) {
  int64_t r = x % m;
  return r < 0 ? r + m : r;
}

int64_t balanced(int64_t x, int64_t m) {
  int64_t r = pmod(x, m);
  return r > m / 2 ? r - m : r;
}

void set_plane(int32_t (&pl)[kMaxPlanes][kMaxLimbs], int k, std::initializer_list<int> c) {
  int i = 0;
  for (int x : c) pl[k][i++] = x;
}

// ---- scheme definitions -------------------------------------------------
// INT8 x INT8 in 6 products (Sec. 4.3, App. A): planes a0, a1, a2, a0+a1,
// a0+a2, a1+a2 on both sides, product k pairs plane k with plane k.
void define_awe6(Scheme& s, bool alt) {
  s.p = s.q = 3;
  const int32_t w0[3] = {1, 29, 37}, w1[3] = {1, 11, 39};
  const int64_t l0[6] = {-65, -261, 259, 29, 37, 1073};
  const int64_t l1[6] = {-49, -319, 1053, 11, 39, 429};
  for (int i = 0; i < 3; ++i) s.w[i] = s.v[i] = alt ? w1[i] : w0[i];
  s.na = s.nb = 6;
  const int comb[6][3] = {{1, 0, 0}, {0, 1, 0}, {0, 0, 1}, {1, 1, 0}, {1, 0, 1}, {0, 1, 1}};
  for (int k = 0; k < 6; ++k)
    for (int i = 0; i < 3; ++i) s.alpha[k][i] = s.beta[k][i] = comb[k][i];
  s.r = 6;
  for (int k = 0; k < 6; ++k) {
    s.pa[k] = s.pb[k] = k;
    s.ell[k] = alt ? l1[k] : l0[k];
  }
  // App. A: capping every stored value at 6 keeps coverage 148 for (1, 29, 37);
  // the (1, 11, 39) solution needs the full set for its coverage 134.
  s.cap_a = s.cap_b = alt ? 12 : 6;
  s.xmin_a = s.xmin_b = -128;
  s.xmax_a = s.xmax_b = 127;
}

// INT4 x INT8 in 4 products (App. A).
void define_awe4(Scheme& s) {
  s.p = 2;
  s.q = 3;
  s.w[0] = 3; s.w[1] = 5;
  s.v[0] = 5; s.v[1] = 3; s.v[2] = 42;
  s.na = s.nb = 4;
  set_plane(s.alpha, 0, {0, 1});
  set_plane(s.alpha, 1, {1, 0});
  set_plane(s.alpha, 2, {1, 2});
  set_plane(s.alpha, 3, {2, 1});
  set_plane(s.beta, 0, {1, 0, 0});
  set_plane(s.beta, 1, {0, 1, -1});
  set_plane(s.beta, 2, {0, 0, 1});
  set_plane(s.beta, 3, {1, 2, 0});
  s.r = 4;
  const int64_t l[4] = {35, -42, 210, 15};
  for (int k = 0; k < 4; ++k) {
    s.pa[k] = s.pb[k] = k;
    s.ell[k] = l[k];
  }
  s.log2D = 1;
  s.cap_a = 3;
  s.cap_b = 8;
  s.xmin_a = -8; s.xmax_a = 7;
  s.xmin_b = -128; s.xmax_b = 127;
}

// Base-13 positional limbs (Sec. 3.2), all 9 limb pairs, ordered so that the
// pairs with equal coefficient 13^(i+j) are adjacent and share an accumulator.
void define_b13(Scheme& s) {
  s.p = s.q = 3;
  s.w[0] = s.v[0] = 1; s.w[1] = s.v[1] = 13; s.w[2] = s.v[2] = 169;
  s.na = s.nb = 3;
  for (int k = 0; k < 3; ++k) s.alpha[k][k] = s.beta[k][k] = 1;
  s.r = 0;
  int64_t pw = 1;
  for (int d = 0; d <= 4; ++d, pw *= 13)
    for (int i = 0; i < 3; ++i) {
      int j = d - i;
      if (j < 0 || j > 2) continue;
      s.pa[s.r] = i;
      s.pb[s.r] = j;
      s.ell[s.r] = pw;
      ++s.r;
    }
  s.positional13_a = s.positional13_b = true;
  s.cap_a = s.cap_b = 12;
  s.xmin_a = s.xmin_b = -128;
  s.xmax_a = s.xmax_b = 127;
}

// {0, +-1} x INT8 in 3 products (Sec. 6.2): a ternary value is one limb of
// weight 1 on A; B takes the three base-13 positional limbs; C = sum_j 13^j P_j.
void define_ternary(Scheme& s) {
  s.p = 1;
  s.q = 3;
  s.w[0] = 1;
  s.v[0] = 1; s.v[1] = 13; s.v[2] = 169;
  s.na = 1;
  s.nb = 3;
  s.alpha[0][0] = 1;
  for (int k = 0; k < 3; ++k) s.beta[k][k] = 1;
  s.r = 3;
  for (int k = 0; k < 3; ++k) {
    s.pa[k] = 0;
    s.pb[k] = k;
    s.ell[k] = k == 0 ? 1 : (k == 1 ? 13 : 169);
  }
  s.positional13_b = true;
  s.cap_a = 1;
  s.cap_b = 12;
  s.xmin_a = -1; s.xmax_a = 1;
  s.xmin_b = -128; s.xmax_b = 127;
}

// FP16 x FP16 significands in 12 products (App. A): w = v = (1, 9, 71, 639),
// planes a_0..a_3, a_0 + 2 a_1, a_2 + 2 a_3; for the outer pair (k, l) the
// products P_{2k,2l}, P_{2k+1,2l+1}, Q_kl with coefficients 71^(k+l) (-7, 126, 9),
// D = 2.  Each (k, l) is a launch group (outer weight 71^(k+l)): its inner sum
// is 2 (a_{2k} + 9 a_{2k+1})(b_{2l} + 9 b_{2l+1}), which fits the int32 fold.
void define_fp16(Scheme& s) {
  s.p = s.q = 4;
  const int32_t w[4] = {1, 9, 71, 639};
  for (int i = 0; i < 4; ++i) s.w[i] = s.v[i] = w[i];
  // stored planes in order of first use: a_0, a_1, a_0 + 2 a_1, a_2, a_3, a_2 + 2 a_3
  s.na = s.nb = 6;
  for (auto* pl : {&s.alpha, &s.beta}) {
    set_plane(*pl, 0, {1, 0, 0, 0});
    set_plane(*pl, 1, {0, 1, 0, 0});
    set_plane(*pl, 2, {1, 2, 0, 0});
    set_plane(*pl, 3, {0, 0, 1, 0});
    set_plane(*pl, 4, {0, 0, 0, 1});
    set_plane(*pl, 5, {0, 0, 1, 2});
  }
  const int64_t inner[3] = {-7, 126, 9};
  s.r = 0;
  // one launch group per outer factor 71^(k+l): the pairs (0, 1) and (1, 0) share 71, so
  // their six products fold into one int32 accumulator (one pass over C fewer)
  s.n_lgroups = 3;
  for (int k = 0; k < 2; ++k)
    for (int l = 0; l < 2; ++l) {
      const int g = k + l;
      const int64_t outer = (k + l == 0) ? 1 : (k + l == 1 ? 71 : 71 * 71);
      s.louter[g] = outer;
      const int pa[3] = {3 * k, 3 * k + 1, 3 * k + 2}, pb[3] = {3 * l, 3 * l + 1, 3 * l + 2};
      for (int t = 0; t < 3; ++t) {
        s.pa[s.r] = pa[t];
        s.pb[s.r] = pb[t];
        s.ell[s.r] = inner[t] * outer;
        s.lgroup[s.r] = g;
        ++s.r;
      }
    }
  s.log2D = 1;
  s.cap_a = s.cap_b = 12;
  s.xmin_a = s.xmin_b = -2048;
  s.xmax_a = s.xmax_b = 2047;
  s.wide = true;
}

// INT8 x INT8 with 2 FP8 products and 1 FP4 product (App. A): A = 13 h + 5 eps,
// planes h, h + eps (E4M3) and eps (E2M1); AB = 104 P1 + 65 P2 - 40 P3.  The two
// E4M3 products form one launch group, the E2M1 product another (outer 1).
void define_fp8fp4(Scheme& s) {
  s.p = s.q = 2;
  s.w[0] = s.v[0] = 13;
  s.w[1] = s.v[1] = 5;
  s.na = s.nb = 3;
  for (auto* pl : {&s.alpha, &s.beta}) {
    set_plane(*pl, 0, {1, 0});
    set_plane(*pl, 1, {1, 1});
    set_plane(*pl, 2, {0, 1});
  }
  s.fmt_a[0] = s.fmt_a[1] = s.fmt_b[0] = s.fmt_b[1] = kFmtE4M3;
  s.r = 3;
  const int64_t l[3] = {104, 65, -40};
  for (int k = 0; k < 3; ++k) {
    s.pa[k] = s.pb[k] = k;
    s.ell[k] = l[k];
    s.lgroup[k] = k < 2 ? 0 : 1;
  }
  s.n_lgroups = 2;
  s.louter[0] = s.louter[1] = 1;
  s.lfmt[0] = kFmtE4M3;
  s.lfmt[1] = kFmtE2M1;
  s.limb_rule = kRuleFp8Fp4;
  s.cap_a = s.cap_b = 14;
  s.xmin_a = s.xmin_b = -128;
  s.xmax_a = s.xmax_b = 127;
}

// INT8 x INT8 in 3 E2M3 (FP6) products: a Karatsuba-type step (Sec. 3.3 gives its
// condition, limb sums inside the format's contiguous integer range, met from a 3-bit
// significand) on balanced base-16 limbs: A = a0 + 16 a1 with a0 in [-8, 7], planes
// a0, a1, a0 + a1 (all within 15); AB = -15 P1 + 240 P2 + 16 P3 with P1 = a0 b0,
// P2 = a1 b1, P3 = (a0 + a1)(b0 + b1), D = 1.
void define_fp6k3(Scheme& s) {
  s.p = s.q = 2;
  s.w[0] = s.v[0] = 1;
  s.w[1] = s.v[1] = 16;
  s.na = s.nb = 3;
  for (auto* pl : {&s.alpha, &s.beta}) {
    set_plane(*pl, 0, {1, 0});
    set_plane(*pl, 1, {0, 1});
    set_plane(*pl, 2, {1, 1});
  }
  for (int k = 0; k < 3; ++k) s.fmt_a[k] = s.fmt_b[k] = kFmtE2M3;
  s.r = 3;
  const int64_t l[3] = {-15, 240, 16};
  for (int k = 0; k < 3; ++k) {
    s.pa[k] = s.pb[k] = k;
    s.ell[k] = l[k];
  }
  s.lfmt[0] = kFmtE2M3;
  s.limb_rule = kRuleBase16;
  s.cap_a = s.cap_b = 16;
  s.xmin_a = s.xmin_b = -128;
  s.xmax_a = s.xmax_b = 127;
}

// INT8 x INT8 in 4 E2M3 products with the limb weights in the block scales (Sec. 4.5):
// the limbs of define_fp6k3, planes a0 and a1, every pair (i, j) a product with weight
// 16^(i+j) = 2^(4 i) 2^(4 j), so plane i's scale carries 2^(4 i).
void define_fp6p4(Scheme& s) {
  s.p = s.q = 2;
  s.w[0] = s.v[0] = 1;
  s.w[1] = s.v[1] = 16;
  s.na = s.nb = 2;
  for (auto* pl : {&s.alpha, &s.beta}) {
    set_plane(*pl, 0, {1, 0});
    set_plane(*pl, 1, {0, 1});
  }
  for (int k = 0; k < 2; ++k) {
    s.fmt_a[k] = s.fmt_b[k] = kFmtE2M3;
    s.sexp_a[k] = s.sexp_b[k] = 4 * k;
  }
  s.r = 4;
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j) {
      s.pa[2 * i + j] = i;
      s.pb[2 * i + j] = j;
      s.ell[2 * i + j] = int64_t(1) << (4 * (i + j));
    }
  s.lfmt[0] = kFmtE2M3;
  s.scale_weights = true;
  s.limb_rule = kRuleBase16;
  s.cap_a = s.cap_b = 16;
  s.xmin_a = s.xmin_b = -128;
  s.xmax_a = s.xmax_b = 127;
}

// ---- limb tuples ----------------------------------------------------------
struct Tuple {
  int a[kMaxLimbs];
};

int plane_value(const int32_t* c, const int* a, int p) {
  int x = 0;
  for (int i = 0; i < p; ++i) x += c[i] * a[i];
  return x;
}

// Enumerate S^p; call f(a) for every tuple whose plane values all lie in S
// within |cap| (the admissible tuples of Definition 4.1 under a cap).
template <class F>
void for_admissible(int p, const int32_t (*planes)[kMaxLimbs], int nplanes, int cap, F f) {
  int idx[kMaxLimbs] = {0, 0, 0, 0};
  int a[kMaxLimbs] = {0, 0, 0, 0};
  for (;;) {
    for (int i = 0; i < p; ++i) a[i] = kS[idx[i]];
    bool ok = true;
    for (int k = 0; k < nplanes && ok; ++k) {
      int x = plane_value(planes[k], a, p);
      ok = in_S(x) && std::abs(x) <= cap;
    }
    if (ok) f(a);
    int i = 0;
    while (i < p && ++idx[i] == 15) idx[i++] = 0;
    if (i == p) break;
  }
}

// Choice among several admissible tuples for one input (the paper leaves it to
// "table lookup"): smallest largest |plane value|, then smallest sum of |limb|,
// then the limb tuple read from the top limb down, ascending.
bool better(const int* a, const int* b, int p, const int32_t (*planes)[kMaxLimbs], int nplanes) {
  int ma = 0, mb = 0, sa = 0, sb = 0;
  for (int k = 0; k < nplanes; ++k) {
    ma = std::max(ma, std::abs(plane_value(planes[k], a, p)));
    mb = std::max(mb, std::abs(plane_value(planes[k], b, p)));
  }
  if (ma != mb) return ma < mb;
  for (int i = 0; i < p; ++i) {
    sa += std::abs(a[i]);
    sb += std::abs(b[i]);
  }
  if (sa != sb) return sa < sb;
  for (int i = p - 1; i >= 0; --i)
    if (a[i] != b[i]) return a[i] < b[i];
  return false;
}

// Least-magnitude element of S in each residue class mod 13 (S holds a full
// residue system mod 13, Sec. 3.2).
void base13_digits(int x, int* out) {
  int rep[13];
  for (int r = 0; r < 13; ++r) rep[r] = INT_MAX;
  for (int s : kS) {
    int r = (int)pmod(s, 13);
    if (rep[r] == INT_MAX || std::abs(s) < std::abs(rep[r])) rep[r] = s;
  }
  for (int i = 0; i < 3; ++i) {
    int d = rep[pmod(x, 13)];
    out[i] = d;
    x = (x - d) / 13;
  }
  if (x != 0) out[0] = INT_MAX;  // not representable in 3 limbs (never for int8)
}

// Builds the limb table of one side: for every table index (input byte, or
// x - xmin for a wide encoding), the chosen limbs, plane values and codes.
// Returns false with a message if an input of the range has no tuple.
bool build_side(Scheme& s, bool sideA, std::string* msg) {
  const int p = sideA ? s.p : s.q;
  const int np = sideA ? s.na : s.nb;
  const int32_t* wts = sideA ? s.w : s.v;
  const int32_t(*planes)[kMaxLimbs] = sideA ? s.alpha : s.beta;
  const int cap = sideA ? s.cap_a : s.cap_b;
  const int xmin = sideA ? s.xmin_a : s.xmin_b;
  const int xmax = sideA ? s.xmax_a : s.xmax_b;
  auto& val = sideA ? s.val_a : s.val_b;
  auto& lut = sideA ? s.lut_a : s.lut_b;
  const int nx = xmax - xmin + 1;
  const int nt = s.table_size(sideA);
  val.assign(nt, std::array<int32_t, kMaxPlanes>{});
  lut.assign(nt, kLutInvalid);

  std::vector<Tuple> best(nx);
  std::vector<char> have(nx, 0);
  const bool by_rule = s.limb_rule == kRuleFp8Fp4 || s.limb_rule == kRuleBase16;
  if (s.modulus == 0 && by_rule) {
    // the rule encodes every input of the range; no admissible-tuple search
    (sideA ? s.coverage_a : s.coverage_b) = std::min(-xmin, xmax);
  } else if (s.modulus == 0) {
    // values of w.a over the admissible tuples, for the coverage (Sec. 4.2)
    int64_t span = 0;
    for (int i = 0; i < p; ++i) span += 12 * (int64_t)std::abs(wts[i]);
    std::vector<char> hit(2 * span + 1, 0);
    for_admissible(p, planes, np, cap, [&](const int* a) {
      int64_t x = 0;
      for (int i = 0; i < p; ++i) x += (int64_t)wts[i] * a[i];
      hit[x + span] = 1;
    });
    int64_t X = 0;
    while (X < span && hit[X + 1 + span] && hit[-(X + 1) + span]) ++X;
    (sideA ? s.coverage_a : s.coverage_b) = (int32_t)X;
  }
  if (s.limb_rule == kRuleFp8Fp4) {
    // App. A: x = 13 h + 5 eps with eps the element of {0, +-1, +-2, +-3, +-4, +-6, +-8} in
    // the residue class 5^-1 x mod 13 (the set holds each class once), h = (x - 5 eps) / 13
    static const int kEps[13] = {0, 1, -1, 2, -2, 3, -3, 4, -4, 6, -6, 8, -8};
    for (int x = xmin; x <= xmax; ++x) {
      for (int e : kEps)
        if (pmod(5 * e - x, 13) == 0) {
          Tuple t{};
          t.a[0] = (x - 5 * e) / 13;
          t.a[1] = e;
          best[x - xmin] = t;
          have[x - xmin] = 1;
        }
    }
  } else if (s.limb_rule == kRuleBase16) {
    // x = a0 + 16 a1 with the balanced digit a0 in [-8, 7]
    for (int x = xmin; x <= xmax; ++x) {
      Tuple t{};
      t.a[0] = (int)pmod(x + 8, 16) - 8;
      t.a[1] = (x - t.a[0]) / 16;
      best[x - xmin] = t;
      have[x - xmin] = 1;
    }
  } else if (sideA ? s.positional13_a : s.positional13_b) {
    for (int x = xmin; x <= xmax; ++x) {
      int d[3];
      base13_digits(x, d);
      if (d[0] == INT_MAX) continue;
      Tuple t{};
      for (int i = 0; i < 3; ++i) t.a[i] = d[i];
      best[x - xmin] = t;
      have[x - xmin] = 1;
    }
  } else {
    for_admissible(p, planes, np, cap, [&](const int* a) {
      int64_t x = 0;
      for (int i = 0; i < p; ++i) x += (int64_t)wts[i] * a[i];
      if (s.modulus) x = pmod(x, s.modulus);
      if (x < xmin || x > xmax) return;
      int ix = (int)x - xmin;
      if (!have[ix] || better(a, best[ix].a, p, planes, np)) {
        for (int i = 0; i < kMaxLimbs; ++i) best[ix].a[i] = i < p ? a[i] : 0;
        have[ix] = 1;
      }
    });
  }
  for (int ix = 0; ix < nx; ++ix)
    if (!have[ix]) {
      *msg = "encoding table misses input " + std::to_string(ix + xmin);
      return false;
    }

  // Packed codes: the leading E4M3 planes take 8 bits each, then 4 bits per E2M1 plane;
  // a side of E2M3 planes (only those) takes 8 bits per plane.
  const uint8_t* fmt = sideA ? s.fmt_a : s.fmt_b;
  const bool f6 = fmt[0] == kFmtE2M3;
  const int n8 = f6 ? np : s.planes8(sideA);
  for (int k = 0; k < np; ++k)
    if (f6 ? fmt[k] != kFmtE2M3 : (k >= n8 && fmt[k] != kFmtE2M1)) {
      *msg = f6 ? "E2M3 planes cannot be mixed with other formats"
                : "E4M3 planes must precede the E2M1 planes";
      return false;
    }
  if (8 * n8 + 4 * (np - n8) > 31) {
    *msg = "packed codes exceed 31 bits";
    return false;
  }
  int cmax = 0;
  for (int b = 0; b < nt; ++b) {
    const int x = s.table_value(sideA, b);
    if (x < xmin || x > xmax) continue;  // stays kLutInvalid
    const int* a = best[x - xmin].a;
    uint32_t packed = 0;
    for (int k = 0; k < np; ++k) {
      int pv = plane_value(planes[k], a, p);
      val[b][k] = pv;
      cmax = std::max(cmax, std::abs(pv));
      const bool f8 = k < n8;
      int code = f6 ? e2m3_code(pv) : (f8 ? e4m3_code(pv) : e2m1_code(pv));
      if (code < 0 || std::abs(pv) > cap) {
        *msg = f6   ? "stored value outside E2M3's integer range or above the cap"
               : f8 ? "stored value not an E4M3 integer or above the cap"
                    : "stored value outside S or above the cap";
        return false;
      }
      packed |= (uint32_t)code << (f8 ? 8 * k : 8 * n8 + 4 * (k - n8));
    }
    // round trip: the limbs reproduce the input (Sec. 3.2), or its residue (Sec. 5.3)
    int64_t back = 0;
    for (int i = 0; i < p; ++i) {
      if (!by_rule && !in_S(a[i])) {
        *msg = "limb outside S";
        return false;
      }
      back += (int64_t)wts[i] * a[i];
    }
    if (s.modulus ? pmod(back - x, s.modulus) != 0 : back != x) {
      *msg = "limb table does not reproduce its input";
      return false;
    }
    lut[b] = packed;
  }
  (sideA ? s.c_a : s.c_b) = cmax;
  return true;
}

// Definition 4.1 identity (or its congruence) on every pair of table inputs.
bool check_identity(const Scheme& s, std::string* msg) {
  const int na = s.table_size(true), nb = s.table_size(false);
  for (int ba = 0; ba < na; ++ba) {
    if (s.lut_a[ba] & kLutInvalid) continue;
    const int x = s.table_value(true, ba);
    for (int bb = 0; bb < nb; ++bb) {
      if (s.lut_b[bb] & kLutInvalid) continue;
      const int y = s.table_value(false, bb);
      int64_t acc = 0;
      for (int k = 0; k < s.r; ++k) acc += s.ell[k] * s.val_a[ba][s.pa[k]] * s.val_b[bb][s.pb[k]];
      bool ok = s.modulus ? pmod(acc - (int64_t)x * y, s.modulus) == 0
                          : acc == ((int64_t)x * y) * (int64_t(1) << s.log2D);
      if (!ok) {
        *msg = "scheme identity fails at x=" + std::to_string(x) + " y=" + std::to_string(y);
        return false;
      }
    }
  }
  return true;
}

// Largest |value| of plane k over the table's inputs.
int plane_cap(const Scheme& s, bool sideA, int k) {
  int c = 0;
  for (int b = 0; b < s.table_size(sideA); ++b)
    if (!((sideA ? s.lut_a : s.lut_b)[b] & kLutInvalid))
      c = std::max(c, std::abs((sideA ? s.val_a : s.val_b)[b][k]));
  return c;
}

void derive_bounds(Scheme& s) {
  if (s.scale_weights) {
    // One FP32 accumulator receives every product with its weight (Sec. 3.4 for a shared,
    // weighted accumulator): a reduction index adds at most sum_k ell_k c_A(k) c_B(k).  The
    // fold adds the accumulator into int32 unmultiplied, so 2^24 is the only bound.
    int64_t per_index = 0;
    for (int k = 0; k < s.r; ++k)
      per_index += std::abs(s.ell[k]) * plane_cap(s, true, s.pa[k]) * plane_cap(s, false, s.pb[k]);
    s.n_g = s.r;
    for (int k = 0; k < s.r; ++k) s.group[k] = 0;
    s.k_star = (int64_t(1) << 24) / per_index;
    s.k_seg = s.k_star / kKPad * kKPad;
    s.lkseg[0] = s.k_seg;
    return;
  }
  // products with equal coefficients that are adjacent share one accumulator (n_g, Sec. 3.4)
  int g = -1, run = 0;
  s.n_g = 1;
  for (int k = 0; k < s.r; ++k) {
    if (k == 0 || s.ell[k] != s.ell[k - 1]) {
      ++g;
      run = 0;
    }
    s.group[k] = g;
    s.n_g = std::max(s.n_g, ++run);
  }
  const int64_t denom = (int64_t)s.n_g * s.c_a * s.c_b;
  s.k_star = (int64_t(1) << 24) / denom;
  // The fold multiplies each FP32 partial by its coefficient with a signed
  // 24-bit multiply, so a partial must stay within 2^23 - 1 in magnitude.  Each
  // launch group may use its own planes' bounds (the E2M1 product of the FP8 +
  // FP4 scheme has c = 8 while its E4M3 products have c = 14).
  s.k_seg = INT64_MAX;
  for (int g = 0; g < s.n_lgroups; ++g) {
    int64_t worst = 1;
    for (int k = 0; k < s.r; ++k) {
      if (s.lgroup[k] != g) continue;
      int ca = 0, cb = 0;
      for (int b = 0; b < s.table_size(true); ++b)
        if (!(s.lut_a[b] & kLutInvalid)) ca = std::max(ca, std::abs(s.val_a[b][s.pa[k]]));
      for (int b = 0; b < s.table_size(false); ++b)
        if (!(s.lut_b[b] & kLutInvalid)) cb = std::max(cb, std::abs(s.val_b[b][s.pb[k]]));
      worst = std::max<int64_t>(worst, (int64_t)ca * cb);
    }
    const int64_t seg = ((int64_t(1) << 23) - 1) / ((int64_t)s.n_g * worst) / kKPad * kKPad;
    s.lkseg[g] = seg;
    s.k_seg = std::min(s.k_seg, seg);
  }
}

// Every launch group must reconstruct D times an integer on its own (its
// coefficient matrix sum_k (ell_k / outer) alpha_k beta_k^T divisible by D), so
// that the shift by log2 D can be applied per launch; its inner coefficients
// must fit the kernel's signed 24-bit fold multiply.
bool check_launch_groups(const Scheme& s, std::string* msg) {
  for (int k = 0; k < s.r; ++k)
    if (s.fmt_a[s.pa[k]] != s.lfmt[s.lgroup[k]] || s.fmt_b[s.pb[k]] != s.lfmt[s.lgroup[k]]) {
      *msg = "a product's planes do not have its launch group's format";
      return false;
    }
  for (int g = 0; g < s.n_lgroups; ++g) {
    int64_t cm[kMaxLimbs][kMaxLimbs] = {};
    for (int k = 0; k < s.r; ++k) {
      if (s.lgroup[k] != g) continue;
      if (s.louter[g] == 0 || s.ell[k] % s.louter[g] != 0) {
        *msg = "coefficient not a multiple of its launch group's outer weight";
        return false;
      }
      const int64_t inner = s.ell[k] / s.louter[g];
      if (inner < -(1 << 23) || inner >= (1 << 23)) {
        *msg = "inner coefficient outside the 24-bit fold multiply";
        return false;
      }
      for (int i = 0; i < s.p; ++i)
        for (int j = 0; j < s.q; ++j) cm[i][j] += inner * s.alpha[s.pa[k]][i] * s.beta[s.pb[k]][j];
    }
    for (int i = 0; i < s.p; ++i)
      for (int j = 0; j < s.q; ++j)
        if (cm[i][j] % (int64_t(1) << s.log2D) != 0) {
          *msg = "launch group does not reconstruct a multiple of D";
          return false;
        }
  }
  return true;
}

// Weights in the scales: every product's ell_k must be 2^(sexp_a + sexp_b) of its planes,
// each side two E2M3 planes, every pair of them a product (the kernel's shared mode).
bool check_scale_weights(const Scheme& s, std::string* msg) {
  if (!s.scale_weights) return true;
  if (s.na != 2 || s.nb != 2 || s.r != 4 || s.n_lgroups != 1 || s.fmt_a[0] != kFmtE2M3) {
    *msg = "weights in scales need two E2M3 planes per side and all four pairs";
    return false;
  }
  for (int k = 0; k < s.r; ++k) {
    const int e = s.sexp_a[s.pa[k]] + s.sexp_b[s.pb[k]];
    if (s.pa[k] != k / 2 || s.pb[k] != k % 2 || e < 0 || e > 24 || s.ell[k] != (int64_t(1) << e)) {
      *msg = "a product's weight is not the product of its planes' scale factors";
      return false;
    }
  }
  return true;
}

bool finish(Scheme& s, std::string* msg) {
  if (!check_scale_weights(s, msg)) return false;
  if (!build_side(s, true, msg) || !build_side(s, false, msg)) return false;
  if (!check_identity(s, msg)) return false;
  if (!check_launch_groups(s, msg)) return false;
  derive_bounds(s);
  if (s.k_seg < kKPad) {
    *msg = "fold segment below one k-tile";
    return false;
  }
  return true;
}

// ---- mod-m schemes (Sec. 5.3) ----------------------------------------------
bool residues_cover(int m, int W, int pp, int uu) {
  std::vector<char> seen(m, 0);
  int count = 0;
  for (int a0 : kS)
    for (int a1 : kS) {
      if (pp != 0 && !in_S(pp * a0 + uu * a1)) continue;
      int r = (int)pmod(a0 + (int64_t)W * a1, m);
      if (!seen[r]) {
        seen[r] = 1;
        ++count;
      }
    }
  return count == m;
}

int64_t inv_mod(int64_t a, int64_t m) {
  int64_t t = 0, nt = 1, r = m, nr = pmod(a, m);
  while (nr) {
    int64_t q = r / nr;
    std::tie(t, nt) = std::make_pair(nt, t - q * nt);
    std::tie(r, nr) = std::make_pair(nr, r - q * nr);
  }
  return r == 1 ? pmod(t, m) : -1;
}

// Families, tried in order: one limb (S a complete residue system mod m);
// one Karatsuba-type step with the plane p a0 + u a1 on both sides; two limbs
// with all four pairs.  Weights w = v = (1, W), W as small as possible.
bool define_mod(Scheme& s, int m, std::string* msg) {
  s.modulus = m;
  s.a_unsigned = s.b_unsigned = true;
  s.xmin_a = s.xmin_b = 0;
  s.xmax_a = s.xmax_b = m - 1;
  s.cap_a = s.cap_b = 12;
  {
    std::vector<char> seen(m, 0);
    int count = 0;
    for (int x : kS)
      if (!seen[pmod(x, m)]) {
        seen[pmod(x, m)] = 1;
        ++count;
      }
    if (count == m) {
      s.p = s.q = 1;
      s.w[0] = s.v[0] = 1;
      s.na = s.nb = 1;
      s.alpha[0][0] = s.beta[0][0] = 1;
      s.r = 1;
      s.ell[0] = 1;
      return true;
    }
  }
  static const int kPlanes[6][2] = {{1, 1}, {1, -1}, {1, 2}, {1, -2}, {2, 1}, {2, -1}};
  for (const auto& pu : kPlanes) {
    const int pp = pu[0], uu = pu[1];
    int64_t inv = inv_mod(pp * uu, m);
    if (inv < 0) continue;
    for (int W = 2; W < m; ++W) {
      if (!residues_cover(m, W, pp, uu)) continue;
      // coefficients of a0b0, a0b1 + a1b0 and a1b1 matched modulo m
      int64_t t = pmod((int64_t)W * inv, m);
      s.p = s.q = 2;
      s.w[0] = s.v[0] = 1;
      s.w[1] = s.v[1] = W;
      s.na = s.nb = 3;
      set_plane(s.alpha, 0, {1, 0});
      set_plane(s.alpha, 1, {0, 1});
      set_plane(s.alpha, 2, {pp, uu});
      for (int k = 0; k < 3; ++k)
        for (int i = 0; i < 2; ++i) s.beta[k][i] = s.alpha[k][i];
      s.r = 3;
      for (int k = 0; k < 3; ++k) s.pa[k] = s.pb[k] = k;
      s.ell[0] = balanced(1 - t * pp * pp, m);
      s.ell[1] = balanced((int64_t)W * W - t * uu * uu, m);
      s.ell[2] = balanced(t, m);
      return true;
    }
  }
  for (int W = 2; W < m; ++W) {
    if (!residues_cover(m, W, 0, 0)) continue;
    s.p = s.q = 2;
    s.w[0] = s.v[0] = 1;
    s.w[1] = s.v[1] = W;
    s.na = s.nb = 2;
    set_plane(s.alpha, 0, {1, 0});
    set_plane(s.alpha, 1, {0, 1});
    set_plane(s.beta, 0, {1, 0});
    set_plane(s.beta, 1, {0, 1});
    s.r = 4;
    const int pr[4][2] = {{0, 0}, {0, 1}, {1, 0}, {1, 1}};
    for (int k = 0; k < 4; ++k) {
      s.pa[k] = pr[k][0];
      s.pb[k] = pr[k][1];
    }
    s.ell[0] = balanced(1, m);
    s.ell[1] = s.ell[2] = balanced(W, m);
    s.ell[3] = balanced((int64_t)W * W, m);
    return true;
  }
  *msg = "no single, Karatsuba-type or two-limb scheme for modulus " + std::to_string(m);
  return false;
}

std::mutex g_mu;
std::map<std::pair<int, int>, std::unique_ptr<Scheme>> g_cache;
std::map<std::pair<int, int>, std::string> g_fail;

}  // namespace

// E4M3 code of a small integer (|v| <= 16 is exact: 3 mantissa bits after the
// leading one), or -1: sign bit 7, exponent field (bias 7) bits 6..3, mantissa 2..0.
int e4m3_code(int v) {
  const int a = std::abs(v);
  if (a == 0) return 0;
  if (a > 16) return -1;
  int e = 31 - __builtin_clz((unsigned)a);  // floor(log2 a)
  const int frac = a - (1 << e);            // a = 2^e (1 + m / 8)
  if ((frac << 3) % (1 << e) != 0) return -1;
  const int m = (frac << 3) >> e;
  return (v < 0 ? 0x80 : 0) | ((e + 7) << 3) | m;
}

// E2M3 code of v / 8 (|v| <= 16): the subnormals m / 8 and the first binade
// 1 + m / 8 give |v| = 0 .. 15 as the 5-bit field itself, and 16 / 8 = 2 is
// exponent field 2 with mantissa 0, again the field value 16; bit 5 is the sign.
int e2m3_code(int v) {
  const int a = std::abs(v);
  if (a > 16) return -1;
  return (v < 0 ? 0x20 : 0) | a;
}

int e2m1_code(int s) {
  int a = std::abs(s);
  for (int i = 0; i < 8; ++i)
    if (kMag[i] == a) return (s < 0 ? 8 : 0) | i;
  return -1;
}

int64_t plane_stride_bytes(int64_t rows, int64_t K) {
  int64_t rb = (rows + kBrickRows - 1) / kBrickRows;
  int64_t kp = (K + kKPad - 1) / kKPad * kKPad;
  return rb * (kp / kBrickK) * kBrickBytes;
}

const Scheme* get_scheme(awe_encoding enc, int32_t modulus, awe_status* st, std::string* msg) {
  if (enc < AWE_ENC_B13 || enc > AWE_ENC_FP6P4) {
    *st = AWE_ERR_INVALID_VALUE;
    *msg = "unknown encoding";
    return nullptr;
  }
  int key_m = enc == AWE_ENC_MOD ? modulus : 0;
  if (enc == AWE_ENC_MOD && (modulus < 2 || modulus > 256)) {
    *st = modulus < 2 ? AWE_ERR_INVALID_VALUE : AWE_ERR_UNSUPPORTED;
    *msg = "modulus must lie in [2, 256] (residues are stored as uint8)";
    return nullptr;
  }
  std::lock_guard<std::mutex> lk(g_mu);
  auto key = std::make_pair((int)enc, key_m);
  auto it = g_cache.find(key);
  if (it != g_cache.end()) return it->second.get();
  auto f = g_fail.find(key);
  if (f != g_fail.end()) {
    *st = enc == AWE_ENC_MOD ? AWE_ERR_UNSUPPORTED : AWE_ERR_TABLE;
    *msg = f->second;
    return nullptr;
  }
  auto s = std::make_unique<Scheme>();
  s->enc = enc;
  bool ok = true;
  std::string m;
  awe_status fail = AWE_ERR_TABLE;
  switch (enc) {
    case AWE_ENC_B13: define_b13(*s); break;
    case AWE_ENC_AWE6: define_awe6(*s, false); break;
    case AWE_ENC_AWE6ALT: define_awe6(*s, true); break;
    case AWE_ENC_AWE4: define_awe4(*s); break;
    case AWE_ENC_TERNARY: define_ternary(*s); break;
    case AWE_ENC_FP16: define_fp16(*s); break;
    case AWE_ENC_FP8FP4: define_fp8fp4(*s); break;
    case AWE_ENC_FP6K3: define_fp6k3(*s); break;
    case AWE_ENC_FP6P4: define_fp6p4(*s); break;
    case AWE_ENC_MOD:
      ok = define_mod(*s, modulus, &m);
      if (!ok) fail = AWE_ERR_UNSUPPORTED;
      break;
  }
  if (ok) ok = finish(*s, &m);
  if (!ok) {
    g_fail[key] = m;
    *st = fail;
    *msg = m;
    return nullptr;
  }
  const Scheme* out = s.get();
  g_cache[key] = std::move(s);
  *st = AWE_OK;
  return out;
}

}  // namespace awe
