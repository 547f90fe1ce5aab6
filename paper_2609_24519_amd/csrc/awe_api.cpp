// The C ABI (include/awe.h): argument checks on the host, reduction-length
// splitting, and the launches of the encoder and GEMM kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <string>

#include <map>
#include <memory>
#include <mutex>
#include <vector>
#include "awe_internal.h"

namespace awe {

namespace {
thread_local std::string g_last_error;

awe_status fail(awe_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

int64_t max_abs_input(const Scheme& s, bool sideA) {
  int32_t lo = sideA ? s.xmin_a : s.xmin_b, hi = sideA ? s.xmax_a : s.xmax_b;
  return std::max<int64_t>(std::abs((int64_t)lo), std::abs((int64_t)hi));
}

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

const Scheme* scheme_or_fail(awe_encoding enc, int32_t modulus, awe_status* st) {
  std::string msg;
  const Scheme* s = get_scheme(enc, modulus, st, &msg);
  if (!s) g_last_error = msg;
  return s;
}

size_t side_bytes(const Scheme& s, bool sideA, int64_t rows, int64_t K) {
  return (size_t)s.plane_halves(sideA, sideA ? s.na : s.nb) * (size_t)(plane_stride_bytes(rows, K) / 2);
}

// Largest reduction length (multiple of kKPad) one GEMM launch may cover so that
// the int32 accumulator's true value fits: |D C| <= D max|A| max|B| K for an
// exact scheme, |sum lambda_k P_k| <= sum|lambda_k| c_A c_B K for a congruence,
// and for launch groups |sum_{k in g} (ell_k / outer_g) P_k| over the worst group.
int64_t launch_k_limit(const Scheme& s) {
  const int64_t lim = 0x7fffffffLL;
  int64_t per_k;
  if (s.n_lgroups > 1) {
    per_k = 1;
    for (int g = 0; g < s.n_lgroups; ++g) {
      int64_t sum = 0;
      for (int k = 0; k < s.r; ++k)
        if (s.lgroup[k] == g) sum += std::abs(s.ell[k] / s.louter[g]);
      per_k = std::max(per_k, sum * s.c_a * s.c_b);
    }
  } else if (s.modulus) {
    int64_t sum = 0;
    for (int k = 0; k < s.r; ++k) sum += std::abs(s.ell[k]);
    per_k = sum * s.c_a * s.c_b;
  } else {
    per_k = (int64_t(1) << s.log2D) * max_abs_input(s, true) * max_abs_input(s, false);
  }
  return std::max<int64_t>(lim / per_k / kKPad * kKPad, kKPad);
}

// Whether the scheme's products are all nine pairs (i, j) of 3 E2M1 planes per side in one
// launch group, with a coefficient that depends on i + j only (base-13: 13^(i + j)); then
// ell_d[i + j] receives it.  AWE_GEMM_ALLPAIRS=0 keeps such schemes on the product-major
// stream (for comparison).
bool all_pairs_by_sum(const Scheme& s, int64_t* ell_d) {
  const char* e = getenv("AWE_GEMM_ALLPAIRS");
  if (e && atoi(e) == 0) return false;
  if (s.n_lgroups != 1 || s.na != 3 || s.nb != 3 || s.r != 9 || s.scale_weights || s.wide) return false;
  for (int k = 0; k < 3; ++k)
    if (s.fmt_a[k] != kFmtE2M1 || s.fmt_b[k] != kFmtE2M1) return false;
  bool seen[3][3] = {};
  bool have[5] = {};
  for (int k = 0; k < s.r; ++k) {
    const int i = s.pa[k], j = s.pb[k];
    if (i < 0 || i > 2 || j < 0 || j > 2 || seen[i][j]) return false;
    seen[i][j] = true;
    const int64_t l = s.ell[k] / s.louter[0];
    if (l * s.louter[0] != s.ell[k] || l >= (1 << 23) || l < -(1 << 23)) return false;
    if (have[i + j] && ell_d[i + j] != l) return false;
    have[i + j] = true;
    ell_d[i + j] = l;
  }
  return true;
}

// Whether the scheme's products are (3k + t, 3l + t) for t < 3 and k, l < 2 with coefficient
// inner[t] * outer[k + l], in launch group k + l of outer weight outer[k + l] (the 12-bit
// significand scheme: two halves of three planes per side, App. A); then inner and outer receive
// them.  Such a scheme runs as one launch: stream product t brings planes t and t + 3 of each
// side, and its four pairs add into three accumulator groups, one per k + l.  AWE_GEMM_ALLPAIRS=0
// keeps it on one launch per group.
bool pairs_of_halves(const Scheme& s, int64_t* inner, int64_t* outer) {
  const char* e = getenv("AWE_GEMM_ALLPAIRS");
  if (e && atoi(e) == 0) return false;
  if (s.n_lgroups != 3 || s.na != 6 || s.nb != 6 || s.r != 12 || s.scale_weights || s.modulus) return false;
  for (int k = 0; k < 6; ++k)
    if (s.fmt_a[k] != kFmtE2M1 || s.fmt_b[k] != kFmtE2M1) return false;
  bool seen[3][2][2] = {}, have[3] = {};
  for (int q = 0; q < s.r; ++q) {
    const int t = s.pa[q] % 3, k = s.pa[q] / 3, l = s.pb[q] / 3;
    if (s.pa[q] < 0 || s.pa[q] > 5 || s.pb[q] < 0 || s.pb[q] > 5 || s.pb[q] % 3 != t || seen[t][k][l] ||
        s.lgroup[q] != k + l)
      return false;
    seen[t][k][l] = true;
    const int64_t o = s.louter[k + l], in = s.ell[q] / o;
    if (in * o != s.ell[q] || in >= (1 << 23) || in < -(1 << 23) || o > 0x7fffffff) return false;
    if (have[t] && inner[t] != in) return false;
    have[t] = true;
    inner[t] = in;
    outer[k + l] = o;
  }
  return true;
}

// The launches of one exact or mod-m GEMM on stored planes, in order (every launch after
// the first adds into C); nothing is enqueued.
awe_status plan_gemm(const Scheme& s, int64_t M, int64_t N, int64_t K, const void* pa, const void* pb,
                     void* C, int64_t ldc, awe_dtype c_type, int64_t k_seg, std::vector<GemmLaunch>* plan) {
  plan->clear();
  if (M < 0 || N < 0 || K < 0) return fail(AWE_ERR_INVALID_VALUE, "negative size");
  if (c_type != AWE_I32 && c_type != AWE_I64) return fail(AWE_ERR_INVALID_VALUE, "bad c_type");
  if (s.modulus && c_type != AWE_I32) return fail(AWE_ERR_INVALID_VALUE, "residues are written as int32");
  if (M == 0 || N == 0) return AWE_OK;
  if (C == nullptr) return fail(AWE_ERR_INVALID_VALUE, "C is NULL");
  if (ldc < N) return fail(AWE_ERR_INVALID_VALUE, "ldc < N");
  if (K > 0 && (pa == nullptr || pb == nullptr)) return fail(AWE_ERR_INVALID_VALUE, "planes are NULL");
  if (M > 0x7fffff00LL || N > 0x7fffff00LL) return fail(AWE_ERR_UNSUPPORTED, "M or N too large");
  if (round_up(K, kKPad) / kKPad > 0x7fffffffLL) return fail(AWE_ERR_UNSUPPORTED, "K too large");
  if (!s.modulus && c_type == AWE_I32 &&
      max_abs_input(s, true) * max_abs_input(s, false) * K > 0x7fffffffLL)
    return fail(AWE_ERR_OVERFLOW, "int32 C cannot hold max|A| max|B| K");
  const bool own_seg = k_seg == 0;  // each launch group folds at its own bound
  if (own_seg) k_seg = s.k_seg;
  if (k_seg < 0 || k_seg % kKPad != 0 || k_seg > s.k_seg)
    return fail(AWE_ERR_INVALID_VALUE,
                "k_seg must be a positive multiple of " + std::to_string(kKPad) +
                    " no larger than " + std::to_string(s.k_seg));

  GemmLaunch L{};
  const int64_t unit_a = plane_stride_bytes(M, K), unit_b = plane_stride_bytes(N, K);
  L.planes_a = reinterpret_cast<const uint8_t*>(pa);
  L.planes_b = reinterpret_cast<const uint8_t*>(pb);
  L.stride_a = unit_a;
  L.stride_b = unit_b;
  L.M = M;
  L.N = N;
  L.K = K;
  L.k_seg = k_seg;
  L.C = C;
  L.ldc = ldc;
  L.c_type = c_type;
  L.log2D = s.log2D;
  L.modulus = s.modulus;
  const int64_t kp = round_up(K, kKPad);
  const int64_t step = launch_k_limit(s);
  if (kp == 0) {
    L.k_begin = L.k_end = 0;
    L.accumulate = false;
    plan->push_back(L);
    return AWE_OK;
  }
  int64_t inner[3] = {}, outer[3] = {};
  if (pairs_of_halves(s, inner, outer)) {
    // one launch per reduction range: stream product t = the four pairs of planes t and t + 3;
    // an FP32 accumulator of group k + l covers at most two products per index
    L.fmt = kFmtE2M1;
    L.r = 3;
    L.allpairs_a = L.allpairs_b = 2;
    L.outer_groups = true;
    for (int t = 0; t < 3; ++t) {
      L.pa[t] = L.pb[t] = t;
      L.fold_ell[t] = (int32_t)inner[t];
      L.outer_g[t] = (int32_t)outer[t];
    }
    L.fold_mask = 7;
    L.outer = 1;
    const int64_t bound = ((int64_t(1) << 23) - 1) / (2 * (int64_t)s.c_a * s.c_b) / kKPad * kKPad;
    L.k_seg = std::max<int64_t>(kKPad, std::min<int64_t>(own_seg ? s.k_seg : k_seg, bound));
    for (int64_t k0 = 0; k0 < kp; k0 += step) {
      L.k_begin = k0;
      L.k_end = std::min(kp, k0 + step);
      L.accumulate = k0 > 0;
      plan->push_back(L);
    }
    return AWE_OK;
  }
  // one launch per (reduction range, launch group); every launch after the first adds into C
  for (int64_t k0 = 0; k0 < kp; k0 += step) {
    for (int g = 0; g < s.n_lgroups; ++g) {
      // the group's planes share one format; address them from the first plane of it
      L.fmt = s.lfmt[g];
      const int first_a = s.first_plane(true, L.fmt), first_b = s.first_plane(false, L.fmt);
      L.planes_a = reinterpret_cast<const uint8_t*>(pa) + s.plane_halves(true, first_a) * (unit_a / 2);
      L.planes_b = reinterpret_cast<const uint8_t*>(pb) + s.plane_halves(false, first_b) * (unit_b / 2);
      L.stride_a = fmt_halves(L.fmt) * (unit_a / 2);
      L.stride_b = fmt_halves(L.fmt) * (unit_b / 2);
      L.k_seg = own_seg ? s.lkseg[g] : k_seg;
      L.r = 0;
      L.fold_mask = 0;
      L.shared = s.scale_weights;
      if (L.shared) {
        // one pass over the reduction: each stage brings both planes of each side and runs
        // the four pair products into one accumulator, the weights in the scales (2^3 stores
        // n as n/8 in E2M3, 2^sexp is the plane's weight); folded with coefficient 1
        for (int k = 0; k < 2; ++k) {
          L.scale_a[k] = 0x01010101u * (uint32_t)(127 + 3 + s.sexp_a[k]);
          L.scale_b[k] = 0x01010101u * (uint32_t)(127 + 3 + s.sexp_b[k]);
        }
        L.r = 1;
        L.pa[0] = L.pb[0] = 0;
        L.fold_ell[0] = 1;
        L.fold_mask = 1;
      }
      L.allpairs_a = L.allpairs_b = 0;
      int64_t ell_d[2 * kMaxPlanes] = {};
      if (!L.shared && all_pairs_by_sum(s, ell_d)) {
        // every pair (i, j) of the 3 + 3 planes is a product with coefficient ell_d[i + j]: one
        // stream in which each stage brings the six planes once and the MFMAs of all nine
        // products add into five accumulators (one per i + j), folded with ell_d
        L.allpairs_a = L.allpairs_b = 3;
        L.r = 1;
        L.pa[0] = L.pb[0] = 0;
        for (int d = 0; d < 5; ++d) L.fold_ell[d] = (int32_t)ell_d[d];
        L.fold_mask = 1;
      }
      for (int k = 0; k < s.r && !L.shared && !L.allpairs_a; ++k) {
        if (s.lgroup[k] != g) continue;
        L.pa[L.r] = s.pa[k] - first_a;
        L.pb[L.r] = s.pb[k] - first_b;
        L.fold_ell[L.r] = (int32_t)(s.ell[k] / s.louter[g]);
        const bool last = k == s.r - 1 || s.group[k + 1] != s.group[k] || s.lgroup[k + 1] != g;
        if (last) L.fold_mask |= 1u << L.r;
        ++L.r;
      }
      L.outer = s.louter[g];
      L.k_begin = k0;
      L.k_end = std::min(kp, k0 + step);
      L.accumulate = k0 > 0 || g > 0;
      plan->push_back(L);
    }
  }
  return AWE_OK;
}

awe_status gemm_planes_impl(const Scheme& s, int64_t M, int64_t N, int64_t K, const void* pa,
                            const void* pb, void* C, int64_t ldc, awe_dtype c_type, int64_t k_seg,
                            hipStream_t stream) {
  std::vector<GemmLaunch> plan;
  awe_status st = plan_gemm(s, M, N, K, pa, pb, C, ldc, c_type, k_seg, &plan);
  for (size_t i = 0; st == AWE_OK && i < plan.size(); ++i) st = launch_gemm(plan[i], stream);
  return st;
}

awe_status encode_impl(const Scheme& s, awe_side side, const void* x, int64_t rows, int64_t K,
                       int64_t ld, void* planes, int32_t* flag, hipStream_t stream) {
  if (side != AWE_SIDE_A && side != AWE_SIDE_B) return fail(AWE_ERR_INVALID_VALUE, "bad side");
  if (rows < 0 || K < 0) return fail(AWE_ERR_INVALID_VALUE, "negative size");
  if (rows == 0 || K == 0) return AWE_OK;  // no bricks
  if (x == nullptr || planes == nullptr) return fail(AWE_ERR_INVALID_VALUE, "NULL pointer");
  const bool sideA = side == AWE_SIDE_A;
  if (sideA ? ld < K : ld < rows) return fail(AWE_ERR_INVALID_VALUE, "leading dimension too small");
  EncodeLaunch e{};
  e.x = x;
  e.rows = rows;
  e.K = K;
  e.ld = ld;
  e.transposed = !sideA;
  e.is_unsigned = sideA ? s.a_unsigned : s.b_unsigned;
  e.nplanes = sideA ? s.na : s.nb;
  e.nplanes8 = s.planes8(sideA);
  e.fp6 = (sideA ? s.fmt_a : s.fmt_b)[0] == kFmtE2M3;
  e.planes = reinterpret_cast<uint8_t*>(planes);
  e.plane_stride = plane_stride_bytes(rows, K);
  e.flag = flag;
  e.lut = sideA ? s.lut_a.data() : s.lut_b.data();
  e.wide = s.wide;
  e.xmin = sideA ? s.xmin_a : s.xmin_b;
  e.nvalues = s.table_size(sideA);
  e.side = sideA ? 0 : 1;
  e.table_key = &s;
  return launch_encode(e, stream);
}

awe_status exact_impl(const Scheme& s, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                      const void* B, int64_t ldb, void* C, int64_t ldc, awe_dtype c_type,
                      void* ws, size_t ws_bytes, int32_t* flag, hipStream_t stream) {
  if (M < 0 || N < 0 || K < 0) return fail(AWE_ERR_INVALID_VALUE, "negative size");
  if (M == 0 || N == 0) return AWE_OK;
  if (K > 0 && (A == nullptr || B == nullptr)) return fail(AWE_ERR_INVALID_VALUE, "A or B is NULL");
  if (K > 0 && (lda < K || ldb < N)) return fail(AWE_ERR_INVALID_VALUE, "leading dimension too small");
  if (C == nullptr || ldc < N) return fail(AWE_ERR_INVALID_VALUE, "bad C or ldc");
  if (c_type != AWE_I32 && c_type != AWE_I64) return fail(AWE_ERR_INVALID_VALUE, "bad c_type");
  if (!s.modulus && c_type == AWE_I32 &&
      max_abs_input(s, true) * max_abs_input(s, false) * K > 0x7fffffffLL)
    return fail(AWE_ERR_OVERFLOW, "int32 C cannot hold max|A| max|B| K");
  const size_t ba = round_up((int64_t)side_bytes(s, true, M, K), 256);
  const size_t bb = side_bytes(s, false, N, K);
  if (ba + bb > 0 && (ws == nullptr || ws_bytes < ba + bb))
    return fail(AWE_ERR_WORKSPACE, "workspace smaller than awe_workspace_bytes");
  uint8_t* pa = reinterpret_cast<uint8_t*>(ws);
  uint8_t* pb = pa + ba;
  awe_status st = AWE_OK;
  if (K > 0) {
    st = encode_impl(s, AWE_SIDE_A, A, M, K, lda, pa, flag, stream);
    if (st != AWE_OK) return st;
    st = encode_impl(s, AWE_SIDE_B, B, N, K, ldb, pb, flag, stream);
    if (st != AWE_OK) return st;
  }
  return gemm_planes_impl(s, M, N, K, pa, pb, C, ldc, c_type, 0, stream);
}

// ---- residue number system ----

uint32_t inverse_mod(uint32_t a, uint32_t m) {  // a^-1 mod m by the extended Euclidean algorithm
  int64_t t = 0, nt = 1, r = m, nr = a % m;
  while (nr != 0) {
    const int64_t q = r / nr;
    std::swap(t, nt);
    nt -= q * t;
    std::swap(r, nr);
    nr -= q * r;
  }
  return r == 1 ? (uint32_t)((t % m + m) % m) : 0;
}

// Checks a moduli set (1..AWE_MAX_MODULI moduli in 2..256; for a
// reconstruction also pairwise coprime with product below 2^127) and derives
// the constants of the residue and reconstruction kernels.
awe_status rns_setup(const int32_t* moduli, int32_t n, ResidueParams* rp, CrtParams* cp,
                     unsigned __int128* prod, bool reconstruct = true) {
  if (moduli == nullptr || n < 1 || n > kMaxModuli)
    return fail(AWE_ERR_INVALID_VALUE, "need 1 to " + std::to_string(kMaxModuli) + " moduli");
  const unsigned __int128 limit = ((unsigned __int128)1 << 127) - 1;
  unsigned __int128 M = 1;
  for (int j = 0; j < n; ++j) {
    const int32_t m = moduli[j];
    if (m < 2 || m > 256) return fail(AWE_ERR_INVALID_VALUE, "moduli must lie in [2, 256]");
    if (!reconstruct) continue;
    for (int i = 0; i < j; ++i)
      if (std::__gcd(moduli[i], m) != 1) return fail(AWE_ERR_INVALID_VALUE, "moduli are not pairwise coprime");
    if (M > limit / (unsigned)m) return fail(AWE_ERR_INVALID_VALUE, "product of the moduli must stay below 2^127");
    M *= (unsigned)m;
  }
  if (rp) {
    std::memset(rp, 0, sizeof(*rp));
    rp->n = n;
    for (int j = 0; j < n; ++j) {
      const uint32_t m = (uint32_t)moduli[j];
      rp->m[j] = m;
      rp->inv[j] = 1.0f / (float)m;
      rp->dinv[j] = 1.0 / (double)m;
      rp->w16[j] = (uint32_t)((uint64_t(1) << 16) % m);
      rp->w32[j] = (uint32_t)((uint64_t(1) << 32) % m);
      rp->w48[j] = (uint32_t)((uint64_t(1) << 48) % m);
      rp->negc[j] = (m - (uint32_t)(((unsigned __int128)1 << 64) % m)) % m;
    }
  }
  if (cp) {
    std::memset(cp, 0, sizeof(*cp));
    cp->n = n;
    for (int j = 0; j < n; ++j) {
      const uint32_t m = (uint32_t)moduli[j];
      cp->mod[j].m = m;
      cp->mod[j].inv = 1.0f / (float)m;
      uint64_t pj = 1;  // m_0 ... m_{j-1} mod m
      for (int i = 0; i < j; ++i) {
        cp->c[j][i] = (uint8_t)pj;
        pj = pj * (uint32_t)moduli[i] % m;
      }
      cp->mod[j].d = inverse_mod((uint32_t)pj, m);
      const uint32_t most = (uint32_t)(kMaxModuli - 1) * 255u * 255u;  // largest subtracted sum
      cp->mod[j].off = (most / m + 1) * m;
    }
    cp->M_lo = (uint64_t)M;
    cp->M_hi = (uint64_t)(M >> 64);
    const unsigned __int128 h = M / 2;
    cp->half_lo = (uint64_t)h;
    cp->half_hi = (uint64_t)(h >> 64);
  }
  if (prod) *prod = M;
  return AWE_OK;
}

struct CrtLayout {  // workspace of awe_gemm_crt
  size_t luts;                   // the moduli's code tables, A side then B side (n x 1 KiB each)
  size_t planes_a, planes_b;     // every modulus's stored planes of A, then of B
  int64_t off_a[kMaxModuli], off_b[kMaxModuli];
  size_t res_c;                  // the n residue products, one byte each (m <= 256)
  size_t total;
};

CrtLayout crt_layout(const int32_t* moduli, int32_t n, int64_t M, int64_t N, int64_t K, awe_status* st) {
  CrtLayout L{};
  *st = AWE_OK;
  L.luts = (size_t)round_up(2 * (int64_t)n * 256 * 4, 256);
  int64_t pa = 0, pb = 0;
  for (int j = 0; j < n; ++j) {
    const Scheme* s = scheme_or_fail(AWE_ENC_MOD, moduli[j], st);
    if (!s) return L;
    L.off_a[j] = pa;
    L.off_b[j] = pb;
    pa += (int64_t)side_bytes(*s, true, M, K);
    pb += (int64_t)side_bytes(*s, false, N, K);
  }
  L.planes_a = (size_t)round_up(pa, 256);
  L.planes_b = (size_t)round_up(pb, 256);
  L.res_c = (size_t)round_up((int64_t)n * M * N, 256);
  L.total = L.luts + L.planes_a + L.planes_b + L.res_c;
  return L;
}

// The code tables of a set of moduli packed for the device (A side, then B side), built once
// per set and kept for the life of the process, so that an asynchronous copy may read them.
const std::vector<uint32_t>* crt_tables(const int32_t* moduli, int32_t n, awe_status* st) {
  static std::mutex mu;
  static std::map<std::vector<int32_t>, std::unique_ptr<std::vector<uint32_t>>> cache;
  std::vector<int32_t> key(moduli, moduli + n);
  {
    std::lock_guard<std::mutex> lk(mu);
    auto it = cache.find(key);
    if (it != cache.end()) return it->second.get();
  }
  auto t = std::make_unique<std::vector<uint32_t>>(2 * (size_t)n * 256);
  for (int j = 0; j < n; ++j) {
    const Scheme* s = scheme_or_fail(AWE_ENC_MOD, moduli[j], st);
    if (!s) return nullptr;
    std::copy(s->lut_a.begin(), s->lut_a.begin() + 256, t->begin() + (size_t)j * 256);
    std::copy(s->lut_b.begin(), s->lut_b.begin() + 256, t->begin() + ((size_t)n + j) * 256);
  }
  std::lock_guard<std::mutex> lk(mu);
  auto& slot = cache[key];
  if (!slot) slot = std::move(t);
  return slot.get();
}

}  // namespace

void set_error(const std::string& msg) { g_last_error = msg; }

}  // namespace awe

using namespace awe;

extern "C" {

awe_status awe_get_encoding_info(awe_encoding enc, int32_t modulus, awe_encoding_info* out) {
  if (out == nullptr) return fail(AWE_ERR_INVALID_VALUE, "out is NULL");
  awe_status st;
  const Scheme* s = scheme_or_fail(enc, modulus, &st);
  if (!s) return st;
  awe_encoding_info info;
  std::memset(&info, 0, sizeof(info));
  info.r = s->r;
  info.limbs_a = s->p;
  info.limbs_b = s->q;
  info.planes_a = s->na;
  info.planes_b = s->nb;
  info.log2_D = s->log2D;
  info.c_a = s->c_a;
  info.c_b = s->c_b;
  info.n_g = s->n_g;
  info.modulus = s->modulus;
  info.xmin_a = s->xmin_a;
  info.xmax_a = s->xmax_a;
  info.xmin_b = s->xmin_b;
  info.xmax_b = s->xmax_b;
  info.coverage_a = s->coverage_a;
  info.coverage_b = s->coverage_b;
  for (int i = 0; i < AWE_MAX_LIMBS; ++i) {
    info.w[i] = s->w[i];
    info.v[i] = s->v[i];
  }
  for (int k = 0; k < AWE_MAX_PLANES; ++k)
    for (int i = 0; i < AWE_MAX_LIMBS; ++i) {
      info.alpha[k][i] = s->alpha[k][i];
      info.beta[k][i] = s->beta[k][i];
    }
  for (int k = 0; k < s->r; ++k) {
    info.pair_a[k] = s->pa[k];
    info.pair_b[k] = s->pb[k];
    info.ell[k] = s->ell[k];
    info.group[k] = s->group[k];
  }
  info.k_star = s->k_star;
  info.k_seg = s->k_seg;
  for (int k = 0; k < AWE_MAX_PLANES; ++k) {
    info.format_a[k] = s->fmt_a[k];
    info.format_b[k] = s->fmt_b[k];
  }
  *out = info;
  return AWE_OK;
}

awe_status awe_get_plane_table(awe_encoding enc, int32_t modulus, awe_side side, int32_t* values,
                               int64_t n_values) {
  awe_status st;
  const Scheme* s = scheme_or_fail(enc, modulus, &st);
  if (!s) return st;
  if (side != AWE_SIDE_A && side != AWE_SIDE_B) return fail(AWE_ERR_INVALID_VALUE, "bad side");
  const bool a = side == AWE_SIDE_A;
  const int lo = a ? s->xmin_a : s->xmin_b, hi = a ? s->xmax_a : s->xmax_b;
  const int np = a ? s->na : s->nb;
  if (values == nullptr || n_values < (int64_t)(hi - lo + 1) * np)
    return fail(AWE_ERR_INVALID_VALUE, "values too small");
  for (int x = lo; x <= hi; ++x) {
    const int b = s->table_index(a, x);
    for (int k = 0; k < np; ++k) values[(int64_t)(x - lo) * np + k] = (a ? s->val_a : s->val_b)[b][k];
  }
  return AWE_OK;
}

awe_status awe_plane_bytes(awe_encoding enc, int32_t modulus, awe_side side, int64_t rows, int64_t K,
                           size_t* bytes) {
  if (bytes == nullptr) return fail(AWE_ERR_INVALID_VALUE, "bytes is NULL");
  if (rows < 0 || K < 0) return fail(AWE_ERR_INVALID_VALUE, "negative size");
  if (side != AWE_SIDE_A && side != AWE_SIDE_B) return fail(AWE_ERR_INVALID_VALUE, "bad side");
  awe_status st;
  const Scheme* s = scheme_or_fail(enc, modulus, &st);
  if (!s) return st;
  *bytes = side_bytes(*s, side == AWE_SIDE_A, rows, K);
  return AWE_OK;
}

awe_status awe_encode(awe_encoding enc, int32_t modulus, awe_side side, const void* x, int64_t rows,
                      int64_t K, int64_t ld, void* planes, int32_t* d_range_flag, hipStream_t stream) {
  awe_status st;
  const Scheme* s = scheme_or_fail(enc, modulus, &st);
  if (!s) return st;
  return encode_impl(*s, side, x, rows, K, ld, planes, d_range_flag, stream);
}

awe_status awe_gemm_planes(awe_encoding enc, int32_t modulus, int64_t M, int64_t N, int64_t K,
                           const void* planes_a, const void* planes_b, void* C, int64_t ldc,
                           awe_dtype c_type, int64_t k_seg, hipStream_t stream) {
  awe_status st;
  const Scheme* s = scheme_or_fail(enc, modulus, &st);
  if (!s) return st;
  return gemm_planes_impl(*s, M, N, K, planes_a, planes_b, C, ldc, c_type, k_seg, stream);
}

awe_status awe_workspace_bytes(awe_encoding enc, int32_t modulus, int64_t M, int64_t N, int64_t K,
                               size_t* bytes) {
  if (bytes == nullptr) return fail(AWE_ERR_INVALID_VALUE, "bytes is NULL");
  if (M < 0 || N < 0 || K < 0) return fail(AWE_ERR_INVALID_VALUE, "negative size");
  awe_status st;
  const Scheme* s = scheme_or_fail(enc, modulus, &st);
  if (!s) return st;
  *bytes = (size_t)round_up((int64_t)side_bytes(*s, true, M, K), 256) + side_bytes(*s, false, N, K);
  return AWE_OK;
}

awe_status awe_gemm_exact(awe_encoding enc, int64_t M, int64_t N, int64_t K, const void* A,
                          int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc,
                          awe_dtype c_type, void* workspace, size_t ws_bytes, int32_t* d_range_flag,
                          hipStream_t stream) {
  if (enc == AWE_ENC_MOD) return fail(AWE_ERR_INVALID_VALUE, "use awe_gemm_mod for residues");
  awe_status st;
  const Scheme* s = scheme_or_fail(enc, 0, &st);
  if (!s) return st;
  return exact_impl(*s, M, N, K, A, lda, B, ldb, C, ldc, c_type, workspace, ws_bytes, d_range_flag,
                    stream);
}

awe_status awe_gemm_exact_noalloc(awe_encoding enc, int64_t M, int64_t N, int64_t K, const void* A,
                                  int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc,
                                  awe_dtype c_type, int32_t* d_range_flag, hipStream_t stream) {
  if (enc == AWE_ENC_MOD) return fail(AWE_ERR_INVALID_VALUE, "use awe_gemm_mod for residues");
  if (M < 0 || N < 0 || K < 0) return fail(AWE_ERR_INVALID_VALUE, "negative size");
  awe_status st;
  const Scheme* s = scheme_or_fail(enc, 0, &st);
  if (!s) return st;
  const size_t need = (size_t)round_up((int64_t)side_bytes(*s, true, M, K), 256) + side_bytes(*s, false, N, K);
  if (need > kNoallocBytes)
    return fail(AWE_ERR_WORKSPACE, "the planes of this product need " + std::to_string(need) +
                                       " bytes; the fixed planes array holds " + std::to_string(kNoallocBytes));
  void* ws = nullptr;
  if (M > 0 && N > 0) {
    st = noalloc_planes(&ws);
    if (st != AWE_OK) return st;
  }
  return exact_impl(*s, M, N, K, A, lda, B, ldb, C, ldc, c_type, ws, kNoallocBytes, d_range_flag, stream);
}

awe_status awe_gemm_mod(int32_t m, int64_t M, int64_t N, int64_t K, const uint8_t* A, int64_t lda,
                        const uint8_t* B, int64_t ldb, int32_t* C, int64_t ldc, void* workspace,
                        size_t ws_bytes, int32_t* d_range_flag, hipStream_t stream) {
  awe_status st;
  const Scheme* s = scheme_or_fail(AWE_ENC_MOD, m, &st);
  if (!s) return st;
  return exact_impl(*s, M, N, K, A, lda, B, ldb, C, ldc, AWE_I32, workspace, ws_bytes, d_range_flag,
                    stream);
}

awe_status awe_residues(const int64_t* x, int64_t rows, int64_t cols, int64_t ld, int64_t bound,
                        const int32_t* moduli, int32_t n, uint8_t* out, int64_t out_stride,
                        int32_t* d_range_flag, hipStream_t stream) {
  ResidueParams P;
  awe_status st = rns_setup(moduli, n, &P, nullptr, nullptr, false);
  if (st != AWE_OK) return st;
  if (rows < 0 || cols < 0) return fail(AWE_ERR_INVALID_VALUE, "negative size");
  if (rows == 0 || cols == 0) return AWE_OK;
  if (x == nullptr || out == nullptr) return fail(AWE_ERR_INVALID_VALUE, "NULL pointer");
  if (ld < cols) return fail(AWE_ERR_INVALID_VALUE, "leading dimension too small");
  if (n > 1 && out_stride < rows * cols) return fail(AWE_ERR_INVALID_VALUE, "out_stride too small");
  if (bound < 0) return fail(AWE_ERR_INVALID_VALUE, "negative bound");
  return launch_residues(x, rows, cols, ld, bound, P, out, out_stride, d_range_flag, stream);
}

awe_status awe_crt(const int32_t* residues, int64_t res_stride, int64_t rows, int64_t cols,
                   int64_t ld_res, const int32_t* moduli, int32_t n, int64_t* c128, double* c64,
                   int64_t ldc, hipStream_t stream) {
  CrtParams P;
  awe_status st = rns_setup(moduli, n, nullptr, &P, nullptr);
  if (st != AWE_OK) return st;
  if (rows < 0 || cols < 0) return fail(AWE_ERR_INVALID_VALUE, "negative size");
  if (rows == 0 || cols == 0) return AWE_OK;
  if (residues == nullptr) return fail(AWE_ERR_INVALID_VALUE, "residues are NULL");
  if (ld_res < cols || ldc < cols) return fail(AWE_ERR_INVALID_VALUE, "leading dimension too small");
  if (n > 1 && res_stride < (rows - 1) * ld_res + cols)
    return fail(AWE_ERR_INVALID_VALUE, "res_stride too small");
  if (c128 == nullptr && c64 == nullptr) return AWE_OK;
  return launch_crt(residues, res_stride, rows, cols, ld_res, P, c128, c64, ldc, stream);
}

awe_status awe_crt_workspace_bytes(const int32_t* moduli, int32_t n, int64_t M, int64_t N, int64_t K,
                                   size_t* bytes) {
  if (bytes == nullptr) return fail(AWE_ERR_INVALID_VALUE, "bytes is NULL");
  if (M < 0 || N < 0 || K < 0) return fail(AWE_ERR_INVALID_VALUE, "negative size");
  awe_status st = rns_setup(moduli, n, nullptr, nullptr, nullptr);
  if (st != AWE_OK) return st;
  const CrtLayout L = crt_layout(moduli, n, M, N, K, &st);
  if (st != AWE_OK) return st;
  *bytes = L.total;
  return AWE_OK;
}

awe_status awe_gemm_crt(int64_t M, int64_t N, int64_t K, const int64_t* A, int64_t lda,
                        const int64_t* B, int64_t ldb, int64_t bound_a, int64_t bound_b,
                        const int32_t* moduli, int32_t n, int64_t* c128, double* c64, int64_t ldc,
                        void* workspace, size_t ws_bytes, int32_t* d_range_flag,
                        hipStream_t stream) {
  ResidueParams rp;
  CrtParams cp;
  unsigned __int128 Mprod;
  awe_status st = rns_setup(moduli, n, &rp, &cp, &Mprod);
  if (st != AWE_OK) return st;
  if (M < 0 || N < 0 || K < 0) return fail(AWE_ERR_INVALID_VALUE, "negative size");
  if (bound_a < 0 || bound_b < 0) return fail(AWE_ERR_INVALID_VALUE, "negative bound");
  if (M == 0 || N == 0) return AWE_OK;
  if (K > 0 && (A == nullptr || B == nullptr)) return fail(AWE_ERR_INVALID_VALUE, "A or B is NULL");
  if (K > 0 && (lda < K || ldb < N)) return fail(AWE_ERR_INVALID_VALUE, "leading dimension too small");
  if (ldc < N) return fail(AWE_ERR_INVALID_VALUE, "ldc < N");
  // uniqueness: prod m > 2 K bound_a bound_b  <=>  bound_a bound_b <= (prod m - 1) / (2K)
  if (K > 0) {
    const unsigned __int128 ab = (unsigned __int128)(uint64_t)bound_a * (uint64_t)bound_b;
    if (ab > (Mprod - 1) / (2 * (unsigned __int128)(uint64_t)K))
      return fail(AWE_ERR_OVERFLOW, "product of the moduli must exceed 2 K bound_a bound_b");
  }
  const CrtLayout L = crt_layout(moduli, n, M, N, K, &st);
  if (st != AWE_OK) return st;
  if (L.total > 0 && (workspace == nullptr || ws_bytes < L.total))
    return fail(AWE_ERR_WORKSPACE, "workspace smaller than awe_crt_workspace_bytes");
  uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
  uint32_t* luts = reinterpret_cast<uint32_t*>(ws);
  uint8_t* pla = ws + L.luts;
  uint8_t* plb = pla + L.planes_a;
  uint8_t* rc = plb + L.planes_b;
  if (K > 0) {
    // every modulus's planes of A and of B straight from the int64 operands
    const std::vector<uint32_t>* tab = crt_tables(moduli, n, &st);
    if (!tab) return st;
    hipError_t err = hipMemcpyAsync(luts, tab->data(), tab->size() * sizeof(uint32_t),
                                    hipMemcpyHostToDevice, stream);
    if (err != hipSuccess) return fail(AWE_ERR_HIP, std::string("table upload: ") + hipGetErrorString(err));
    const int64_t kp = round_up(K, kKPad);
    for (int side = 0; side < 2; ++side) {
      const bool sideA = side == 0;
      ResidueEncodeArgs e{};
      e.x = sideA ? A : B;
      e.rows = sideA ? M : N;
      e.K = K;
      e.ld = sideA ? lda : ldb;
      e.KS = kp / kBrickK;
      e.R32 = (e.rows + kBrickRows - 1) / kBrickRows;
      e.nbricks = e.R32 * e.KS;
      e.bound = sideA ? bound_a : bound_b;
      e.luts = luts + (sideA ? 0 : (size_t)n * 256);
      e.planes = sideA ? pla : plb;
      e.plane_stride = plane_stride_bytes(e.rows, K);
      for (int j = 0; j < n; ++j) {
        const Scheme* s = scheme_or_fail(AWE_ENC_MOD, moduli[j], &st);
        if (!s) return st;
        e.off[j] = sideA ? L.off_a[j] : L.off_b[j];
        e.np[j] = sideA ? s->na : s->nb;
      }
      e.flag = d_range_flag;
      st = launch_residue_encode(e, rp, !sideA, stream);
      if (st != AWE_OK) return st;
    }
  }
  // the n mod-m GEMMs: one grouped launch when each is a single launch (AWE_GEMM_GROUPED=0
  // asks for one launch per modulus)
  std::vector<GemmLaunch> all, plan;
  bool single = true;
  for (int j = 0; j < n; ++j) {
    const Scheme* s = scheme_or_fail(AWE_ENC_MOD, moduli[j], &st);
    if (!s) return st;
    st = plan_gemm(*s, M, N, K, pla + L.off_a[j], plb + L.off_b[j], rc + (size_t)j * M * N, N, AWE_I32, 0, &plan);
    if (st != AWE_OK) return st;
    for (GemmLaunch& gl : plan) gl.c_u8 = true;  // residues below 256: bytes, a quarter of the traffic
    single = single && plan.size() == 1;
    all.insert(all.end(), plan.begin(), plan.end());
  }
  const char* ge = getenv("AWE_GEMM_GROUPED");
  if (single && !(ge && atoi(ge) == 0) && gemm_group_ok(all.data(), (int)all.size())) {
    st = launch_gemm_group(all.data(), (int)all.size(), stream);
    if (st != AWE_OK) return st;
  } else {
    for (const GemmLaunch& gl : all) {
      st = launch_gemm(gl, stream);
      if (st != AWE_OK) return st;
    }
  }
  if (c128 == nullptr && c64 == nullptr) return AWE_OK;
  return launch_crt(rc, M * N, M, N, N, cp, c128, c64, ldc, stream);
}

const char* awe_status_string(awe_status s) {
  switch (s) {
    case AWE_OK: return "success";
    case AWE_ERR_INVALID_VALUE: return "invalid argument";
    case AWE_ERR_UNSUPPORTED: return "unsupported modulus or size";
    case AWE_ERR_OVERFLOW: return "int32 output would overflow";
    case AWE_ERR_WORKSPACE: return "workspace too small";
    case AWE_ERR_HIP: return "HIP runtime error";
    case AWE_ERR_TABLE: return "encoding table failed its self-check";
  }
  return "unknown status";
}

const char* awe_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
