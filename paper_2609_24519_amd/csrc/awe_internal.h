// Internal declarations shared by the host table code, the kernels and the C ABI.
#pragma once
#include <array>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/awe.h"

namespace awe {

constexpr int kMaxLimbs = AWE_MAX_LIMBS;
constexpr int kMaxPlanes = AWE_MAX_PLANES;
constexpr int kMaxProducts = AWE_MAX_PRODUCTS;

// Plane layout constants (the MFMA fragment "brick", see include/awe.h).
constexpr int kBrickRows = 32;     // rows (A) or columns (B) per brick
constexpr int kBrickK = 64;        // reduction indices per brick
constexpr int kBrickBytes = 1024;  // 32 x 64 E2M1 codes, 2 per byte
constexpr int kKPad = AWE_K_PAD;   // the reduction length is padded to this multiple

// LUT entry flag: the input byte is outside the encoding's range.
constexpr uint32_t kLutInvalid = 0x80000000u;

// Inputs of a wide encoding are int16 in [xmin, xmax], at most this many values.
constexpr int kWideValues = 4096;

// Plane element formats and limb rules.
constexpr uint8_t kFmtE2M1 = 0, kFmtE4M3 = 1, kFmtE2M3 = 2;
constexpr int kRuleChoice = 0, kRuleBase13 = 1, kRuleFp8Fp4 = 2, kRuleBase16 = 3;

// Storage of one plane of a format, in halves of an E2M1 plane's stride.
inline int fmt_halves(uint8_t f) { return f == kFmtE4M3 ? 4 : (f == kFmtE2M3 ? 3 : 2); }

// One scheme (Definition 4.1 of the paper, or its mod-m congruence form)
// together with the encoding tables derived from it.
struct Scheme {
  awe_encoding enc = AWE_ENC_AWE6;
  int32_t modulus = 0;  // 0: exact scheme
  int p = 0, q = 0;     // limbs on the A and B side
  int32_t w[kMaxLimbs] = {}, v[kMaxLimbs] = {};
  int na = 0, nb = 0;   // stored planes per side
  int32_t alpha[kMaxPlanes][kMaxLimbs] = {};
  int32_t beta[kMaxPlanes][kMaxLimbs] = {};
  int r = 0;
  int32_t pa[kMaxProducts] = {}, pb[kMaxProducts] = {};
  int64_t ell[kMaxProducts] = {};
  int32_t group[kMaxProducts] = {};  // products with equal ell that share an accumulator
  // Launch groups: the products of group g run as one GEMM launch that folds them with
  // inner coefficients ell_k / outer_g and adds outer_g (sum) / D into C.  One group with
  // outer 1 unless the coefficients outgrow the int32 fold (the FP16 scheme).
  int n_lgroups = 1;
  int32_t lgroup[kMaxProducts] = {};
  int64_t louter[kMaxProducts] = {1};
  uint8_t lfmt[kMaxProducts] = {};    // element format of group g's operands (kFmt*)
  int64_t lkseg[kMaxProducts] = {};   // fold segment of group g (from its own plane bounds)
  // Element format of every stored plane; planes of one side are stored in this
  // order, E4M3 planes (twice the bytes) before E2M1 planes.  A side with E2M3
  // planes (1.5 times the bytes) holds only E2M3 planes.
  uint8_t fmt_a[kMaxPlanes] = {}, fmt_b[kMaxPlanes] = {};
  int limb_rule = 0;                  // kRule*: how an input's limbs are chosen
  int log2D = 0;
  int cap_a = 12, cap_b = 12;        // bound on |stored value| the tables may use
  int32_t xmin_a = 0, xmax_a = 0, xmin_b = 0, xmax_b = 0;
  bool positional13_a = false, positional13_b = false;  // base-13 digits with carries instead of the choice rule
  bool a_unsigned = false, b_unsigned = false;  // residues arrive as uint8
  bool wide = false;  // int16 inputs; tables indexed by x - xmin instead of the input byte
  // Limb weights in the block scales (Sec. 4.5): plane k of a side carries 2^sexp in its
  // E8M0 scale, every product's ell_k = 2^(sexp_a + sexp_b), and all products add into one
  // FP32 accumulator (two planes per side, one launch, fold coefficient 1).
  bool scale_weights = false;
  int sexp_a[kMaxPlanes] = {}, sexp_b[kMaxPlanes] = {};
  int planes8(bool sideA) const {  // leading E4M3 planes
    int n = 0;
    while (n < (sideA ? na : nb) && (sideA ? fmt_a : fmt_b)[n]) ++n;
    return n;
  }
  // Plane k's byte offset in halves of one E2M1 plane stride.
  int plane_halves(bool sideA, int k) const {
    int h = 0;
    for (int j = 0; j < k; ++j) h += fmt_halves((sideA ? fmt_a : fmt_b)[j]);
    return h;
  }
  // First stored plane of format f on a side (the planes of one format are adjacent).
  int first_plane(bool sideA, uint8_t f) const {
    const int n = sideA ? na : nb;
    for (int k = 0; k < n; ++k)
      if ((sideA ? fmt_a : fmt_b)[k] == f) return k;
    return n;
  }

  // derived by build_tables()
  int c_a = 0, c_b = 0, n_g = 1;
  int32_t coverage_a = 0, coverage_b = 0;
  int64_t k_star = 0, k_seg = 0;
  // Per table index (the input byte, or x - xmin for a wide encoding): the plane values
  // and the packed E2M1 codes (kLutInvalid for an input outside the range).
  std::vector<std::array<int32_t, kMaxPlanes>> val_a, val_b;
  std::vector<uint32_t> lut_a, lut_b;
  int table_size(bool sideA) const {
    return wide ? (sideA ? xmax_a - xmin_a : xmax_b - xmin_b) + 1 : 256;
  }
  // Input value of table index i.
  int table_value(bool sideA, int i) const {
    if (wide) return i + (sideA ? xmin_a : xmin_b);
    return (sideA ? a_unsigned : b_unsigned) ? i : (int)(int8_t)(uint8_t)i;
  }
  // Table index of input value x (which must lie in the range).
  int table_index(bool sideA, int x) const {
    if (wide) return x - (sideA ? xmin_a : xmin_b);
    return (sideA ? a_unsigned : b_unsigned) ? x : (int)(uint8_t)(int8_t)x;
  }
};

// Builds (once, thread-safe) and returns the scheme; nullptr with a message on failure.
const Scheme* get_scheme(awe_encoding enc, int32_t modulus, awe_status* st, std::string* msg);

// E2M1 code of a doubled integer in S (sign bit 3, magnitude code 0..7), or -1.
int e2m1_code(int s);

// E4M3 code of an integer with |v| <= 16, or -1.
int e4m3_code(int v);

// E2M3 code of v / 8 for an integer with |v| <= 16, or -1.
int e2m3_code(int v);

// Bytes of one plane of `rows` x `K`.
int64_t plane_stride_bytes(int64_t rows, int64_t K);

// ---- kernel launchers (awe_kernels.hip) ----
struct EncodeLaunch {
  const void* x;
  int64_t rows, K, ld;
  bool transposed;  // B side: x[k * ld + row]
  bool is_unsigned;
  int nplanes;
  int nplanes8;         // the first nplanes8 planes are E4M3 (8-bit codes), the rest E2M1
  bool fp6;             // every plane is E2M3 (8-bit fields of the table, 3072-byte units)
  uint8_t* planes;
  int64_t plane_stride;
  int32_t* flag;
  const uint32_t* lut;  // host memory: 256 entries (passed by value), or the wide table
  bool wide;            // int16 inputs, table over [xmin, xmin + nvalues)
  int32_t xmin, nvalues;
  int side;             // which of the two device-resident wide tables to use
  const void* table_key;  // identity of the wide table (its Scheme)
};
awe_status launch_encode(const EncodeLaunch& e, hipStream_t stream);

struct GemmLaunch {
  const uint8_t* planes_a;
  const uint8_t* planes_b;
  int64_t stride_a, stride_b;
  int64_t M, N, K;
  int r;
  int32_t pa[kMaxProducts], pb[kMaxProducts];
  int32_t fold_ell[kMaxProducts];  // coefficient applied when the accumulator is folded after product k
  int64_t outer;                   // the launch adds outer * (sum / D) into C
  uint8_t fmt;                     // element format of both operands' planes (kFmt*)
  bool shared;                     // two planes per side, every pair one product, one accumulator
  uint32_t scale_a[2], scale_b[2]; // shared: E8M0 scale byte of plane 0 / 1, replicated 4 times
  uint32_t fold_mask;              // bit k: fold after product k
  // All pairs (planes per side, 0 = off): the stream's one product stands for every pair
  // (i, j) of the first allpairs_a A planes and allpairs_b B planes, each adding into
  // accumulator group i + j, folded with fold_ell[i + j].
  int allpairs_a, allpairs_b;
  // With outer groups: pair (i, j) of the stream product's planes (stored planes k + 3 i and
  // k + 3 j) adds into group i + j, which folds with the product's coefficient into its own
  // int32 accumulator; C (+)= sum_d outer_g[d] (group d's sum / D).
  bool outer_groups;
  int32_t outer_g[3];
  int64_t k_seg;                   // fold segment length (multiple of kKPad)
  int64_t k_begin, k_end;          // reduction range of this launch (multiples of kKPad)
  void* C;
  int64_t ldc;
  awe_dtype c_type;
  bool c_u8;                       // residues (modulus set) written as bytes instead of c_type
  bool accumulate;
  int log2D;
  int32_t modulus;
};
awe_status launch_gemm(const GemmLaunch& g, hipStream_t stream);

// Several single-launch GEMMs of one shape as one launch (the residue route's moduli).  Each
// launch must pass gemm_group_ok: E2M1 planes, one product per plane pair stream of at most
// kGroupProducts products, the same M, N, K and reduction range, no accumulation into C.
constexpr int kGroupProducts = 4;
bool gemm_group_ok(const GemmLaunch* L, int n);
awe_status launch_gemm_group(const GemmLaunch* L, int n, hipStream_t stream);

// ---- residue number system (awe_rns.hip) ----
constexpr int kMaxModuli = AWE_MAX_MODULI;

struct ResidueParams {
  int32_t n;
  uint32_t m[kMaxModuli];
  float inv[kMaxModuli];      // 1/m in fp32
  double dinv[kMaxModuli];    // 1/m in fp64
  uint32_t w16[kMaxModuli];   // 2^16 mod m
  uint32_t w32[kMaxModuli];   // 2^32 mod m
  uint32_t w48[kMaxModuli];   // 2^48 mod m
  uint32_t negc[kMaxModuli];  // -2^64 mod m, in [0, m)
};
awe_status launch_residues(const int64_t* x, int64_t rows, int64_t cols, int64_t ld, int64_t bound,
                           const ResidueParams& P, uint8_t* out, int64_t out_stride, int32_t* flag,
                           hipStream_t stream);

// Residues of an int64 operand written straight as every modulus's E2M1 planes.
struct ResidueEncodeArgs {
  const int64_t* x;
  int64_t rows, K, ld;        // A side: x[row * ld + k]; B side: x[k * ld + row]
  int64_t KS, R32, nbricks;   // bricks along K per row block, row blocks, all bricks
  int64_t bound;              // |x| above it sets *flag
  const uint32_t* luts;       // device: n x 256 packed E2M1 codes, one table per modulus
  uint8_t* planes;            // modulus j's planes at planes + off[j], plane_stride apart
  int64_t plane_stride;
  int64_t off[kMaxModuli];
  int32_t np[kMaxModuli];
  int32_t* flag;
};
awe_status launch_residue_encode(const ResidueEncodeArgs& a, const ResidueParams& P, bool transposed,
                                 hipStream_t stream);

struct CrtModulus {
  uint32_t m;
  float inv;     // 1/m in fp32
  uint32_t d;    // (m_0 ... m_{j-1})^-1 mod m_j
  uint32_t off;  // multiple of m_j above any subtracted digit sum
};
struct alignas(16) CrtParams {
  uint8_t c[kMaxModuli][kMaxModuli];  // c[j][i] = (m_0 ... m_{i-1}) mod m_j, i < j (row j: digit j's)
  CrtModulus mod[kMaxModuli];
  uint64_t M_lo, M_hi;          // M = m_0 ... m_{n-1} < 2^127
  uint64_t half_lo, half_hi;    // floor(M / 2)
  int32_t n;
};
// Residues as int32 (awe_crt) or as bytes (awe_gemm_crt's own products, a quarter of the bytes).
awe_status launch_crt(const int32_t* res, int64_t res_stride, int64_t rows, int64_t cols,
                      int64_t ld_res, const CrtParams& P, int64_t* c128, double* c64, int64_t ldc,
                      hipStream_t stream);
awe_status launch_crt(const uint8_t* res, int64_t res_stride, int64_t rows, int64_t cols,
                      int64_t ld_res, const CrtParams& P, int64_t* c128, double* c64, int64_t ldc,
                      hipStream_t stream);

void set_error(const std::string& msg);

// Bytes of the fixed device array that holds the planes of awe_gemm_exact_noalloc.
constexpr size_t kNoallocBytes = AWE_NOALLOC_MAX_BYTES;
// Device address of that array on the current device (looked up once per device, with that
// device current; no allocation).
awe_status noalloc_planes(void** out);

}  // namespace awe
