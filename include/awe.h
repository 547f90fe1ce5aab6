/*
 * awe.h -- exact integer matrix products as a few FP4 (E2M1) GEMMs on MI355X.
 *
 * The method (Adaptive Weight Encoding, arXiv 2609.24519): each integer
 * operand entry is split into limbs in the storable set
 * S = {0, +-1, +-2, +-3, +-4, +-6, +-8, +-12} (the E2M1 values doubled,
 * Sec. 3.1), with integer weights w (A side) and v (B side).  Stored "planes"
 * are linear combinations of limbs (Definition 4.1).  Product k multiplies
 * plane alpha_k of A by plane beta_k of B on the FP4 matrix unit with FP32
 * accumulation, which is exact while the reduction length stays below
 * K* = 2^24 / (n_g c_A c_B) (Sec. 3.4).  The exact result is
 * C = (sum_k ell_k P_k) / D with D a power of two (Alg. 1).  Relaxed to a
 * congruence with integer coefficients, the same procedure gives C mod m for
 * the residues of Ozaki scheme II (Sec. 5.3).
 *
 * Conventions for every entry point below:
 *  - Pointers are DEVICE pointers unless marked host.  The caller allocates
 *    and owns every buffer; the library keeps only its constant tables (host
 *    memory) and allocates no device memory.
 *  - Device work is enqueued asynchronously on `stream` (0 = the null
 *    stream).  Argument errors are detected on the host before anything is
 *    enqueued and returned as a status; nothing is written then.  No C++
 *    exception crosses this interface.  awe_last_error() gives detail.
 *  - Results are bit-exact and do not depend on the launch configuration.
 *  - awe_encode, awe_gemm_planes, awe_gemm_exact and awe_gemm_mod enqueue only kernels (no
 *    memset, no copy), so they can be captured into a HIP graph once each has been called
 *    eagerly on the device (the first calls set the GEMM's LDS limit and, for the FP16
 *    scheme, upload its code table).  awe_gemm_crt also copies host tables and is not meant
 *    for capture.
 *  - Matrices are row-major: A is M x K (A[i*lda + k]), B is K x N
 *    (B[k*ldb + j]), C is M x N (C[i*ldc + j]).  Leading dimensions must be
 *    at least the row length.  Empty problems (M or N zero) succeed and write
 *    nothing; K = 0 writes zeros.
 *
 * Stored plane layout (the output of awe_encode, the input of
 * awe_gemm_planes).  One side holds P planes back to back; plane p starts at
 * byte p * stride, stride = ceil(rows/32) * (Kp/64) * 1024 with
 * Kp = K rounded up to a multiple of AWE_K_PAD (256).  A plane is a grid of 1024-byte
 * bricks, brick (rb, ks) at byte (ks * ceil(rows/32) + rb) * 1024 (k-step
 * major: the bricks of one k-step for consecutive row blocks are adjacent),
 * covering rows (A: rows of A; B: columns of B) rb*32 .. rb*32+31 and
 * reduction indices ks*64 .. ks*64+63.  Inside a brick, lane L = 32*h + t (h in {0,1},
 * t in 0..31) owns bytes L*16 .. L*16+15, which hold row rb*32 + t at
 * reduction indices ks*64 + 32*h + j, j = 0..31, element j in the low nibble
 * of byte L*16 + j/2 when j is even and in the high nibble when j is odd.
 * This is the operand order of one lane of the 32x32x64 scaled FP4 MFMA, so
 * a brick is one wave's operand fragment.  Each nibble is the E2M1 code of
 * the stored value s/2 (s in S): bit 3 the sign, bits 2..0 the magnitude
 * index of |s| in (0, 1, 2, 3, 4, 6, 8, 12).  Padding rows and reduction
 * indices hold code 0 (value 0), so they add nothing to any product.
 * E4M3 planes (the first two planes of AWE_ENC_FP8FP4) use 2048-byte bricks with
 * the same geometry: brick (rb, ks) at byte (ks * ceil(rows/32) + rb) * 2048, lane L
 * owning bytes L*32 .. L*32+31, byte j the OCP E4M3 code of element j (the integer
 * itself: every stored value has |v| <= 14).  An E4M3 plane takes two strides, and a
 * side stores its E4M3 planes before its E2M1 planes.
 * E2M3 (FP6) planes (AWE_ENC_FP6K3) take 1.5 strides each and are grouped in 3072-byte
 * units of two consecutive k-steps: unit (rb, u) at byte (u * ceil(rows/32) + rb) * 3072
 * covers rows rb*32 .. rb*32+31 and reduction indices u*128 .. u*128+127.  Lane L's 32
 * elements of k-step 2u + i (i in {0,1}, the same rows and indices as lane L of an E2M1
 * brick) form a 192-bit word, element j in bits 6j .. 6j+5; its first 16 bytes sit at
 * byte i*1024 + L*16 of the unit and its last 8 bytes at byte 2048 + i*512 + L*8.  Each
 * 6-bit field is the OCP E2M3 code of n/8 for the stored integer n (|n| <= 16):
 * bit 5 the sign, bits 4..0 the value |n| itself.
 */
#ifndef AWE_H
#define AWE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum awe_status {
  AWE_OK = 0,
  AWE_ERR_INVALID_VALUE = 1, /* bad pointer, size, leading dimension, enum or modulus */
  AWE_ERR_UNSUPPORTED = 2,   /* no scheme for this modulus, or a size past what the kernels handle */
  AWE_ERR_OVERFLOW = 3,      /* int32 C requested but max|A| max|B| K exceeds 2^31 - 1 */
  AWE_ERR_WORKSPACE = 4,     /* workspace missing or smaller than awe_workspace_bytes */
  AWE_ERR_HIP = 5,           /* a HIP runtime call failed */
  AWE_ERR_TABLE = 6          /* an encoding table failed its self-check */
} awe_status;

typedef enum awe_encoding {
  AWE_ENC_B13 = 1,     /* INT8 x INT8, base-13 positional limbs (1, 13, 169), all 9 limb pairs
                          (Sec. 3.2; Table 1 baseline).  Equal coefficients share an accumulator. */
  AWE_ENC_AWE6 = 2,    /* INT8 x INT8 in 6 products, w = v = (1, 29, 37), planes a_i and a_i + a_j,
                          stored values capped at 6 (Sec. 4.3; App. A) */
  AWE_ENC_AWE6ALT = 3, /* INT8 x INT8 in 6 products, w = v = (1, 11, 39) (Sec. 4.3; App. A) */
  AWE_ENC_AWE4 = 4,    /* INT4 x INT8 in 4 products, A = 3a0 + 5a1, B = 5b0 + 3b1 + 42b2, D = 2
                          (App. A).  The int4 operand is stored one value per int8 byte. */
  AWE_ENC_MOD = 5,     /* residues modulo m (Sec. 5.3); needs the modulus argument */
  AWE_ENC_TERNARY = 6, /* {0, +-1} x INT8 in 3 products: the ternary A entry is one limb, B takes
                          the base-13 limbs, C = sum_j 13^j P_j (Sec. 6.2).  A is int8 in [-1, 1]. */
  AWE_ENC_FP16 = 7,    /* FP16-significand integers x FP16-significand integers in 12 products,
                          w = v = (1, 9, 71, 639), D = 2 (App. A).  Both operands are int16 in
                          [-2048, 2047]; the products run as three launches, one per outer weight
                          71^(k+l) (k + l = 0, 1, 2), each adding its share into C. */
  AWE_ENC_FP8FP4 = 8,  /* INT8 x INT8 with 2 FP8 (E4M3) products and 1 FP4 product (App. A):
                          A = 13 h + 5 eps, planes h, h + eps (E4M3, 2 KiB bricks, see the
                          layout above) and eps (E2M1); AB = 104 P1 + 65 P2 - 40 P3. */
  AWE_ENC_FP6K3 = 9,   /* INT8 x INT8 in 3 E2M3 (FP6) products: A = a0 + 16 a1 with a0 in [-8, 7],
                          planes a0, a1, a0 + a1 (within [-15, 15], inside E2M3's contiguous
                          integer range, the Karatsuba condition of Sec. 3.3);
                          AB = -15 P1 + 240 P2 + 16 P3.  Not a catalogued scheme of the paper. */
  AWE_ENC_FP6P4 = 10   /* INT8 x INT8 in 4 E2M3 products with the limb weights in the block scales
                          (Sec. 4.5): the limbs of AWE_ENC_FP6K3, planes a0 and a1, every limb pair
                          a product, AB = a0 b0 + 16 (a0 b1 + a1 b0) + 256 a1 b1; plane i's E8M0
                          scale carries 16^i, so the four products add into one FP32 accumulator
                          (K* = floor(2^24 / 136^2) = 907).  Not a catalogued scheme. */
} awe_encoding;

typedef enum awe_side { AWE_SIDE_A = 0, AWE_SIDE_B = 1 } awe_side;
typedef enum awe_dtype { AWE_I32 = 0, AWE_I64 = 1 } awe_dtype;

#define AWE_MAX_LIMBS 4
#define AWE_MAX_PLANES 8
#define AWE_MAX_PRODUCTS 16
#define AWE_K_PAD 256 /* stored planes pad the reduction length to a multiple of this */

/* A configuration record (Alg. 1 input): weights, planes, reconstruction and bounds. */
typedef struct awe_encoding_info {
  int32_t r;                      /* number of FP4 products */
  int32_t limbs_a, limbs_b;       /* p and q of the cell (p, q) */
  int32_t planes_a, planes_b;     /* distinct stored planes per side */
  int32_t log2_D;                 /* reconstruction denominator D = 2^log2_D */
  int32_t c_a, c_b;               /* largest |stored value| the tables use */
  int32_t n_g;                    /* most products sharing one accumulator */
  int32_t modulus;                /* 0 for an exact scheme */
  int32_t xmin_a, xmax_a;         /* accepted input range, A side */
  int32_t xmin_b, xmax_b;         /* accepted input range, B side */
  int32_t coverage_a, coverage_b; /* contiguous half-width of w.a (v.b) over the table's tuples; exact schemes */
  int32_t w[AWE_MAX_LIMBS];       /* limb weights, A side */
  int32_t v[AWE_MAX_LIMBS];       /* limb weights, B side */
  int32_t alpha[AWE_MAX_PLANES][AWE_MAX_LIMBS]; /* A-side plane coefficient vectors */
  int32_t beta[AWE_MAX_PLANES][AWE_MAX_LIMBS];  /* B-side plane coefficient vectors */
  int32_t pair_a[AWE_MAX_PRODUCTS];             /* A plane used by product k */
  int32_t pair_b[AWE_MAX_PRODUCTS];             /* B plane used by product k */
  int64_t ell[AWE_MAX_PRODUCTS];  /* reconstruction numerators ell_k (mod m: balanced residues) */
  int32_t group[AWE_MAX_PRODUCTS];/* accumulator shared by product k (equal ell_k) */
  int64_t k_star;                 /* floor(2^24 / (n_g c_a c_b)), Sec. 3.4 */
  int64_t k_seg;                  /* default fold segment of the GEMM (<= k_star), multiple of AWE_K_PAD */
  int32_t format_a[AWE_MAX_PLANES];  /* element format of stored A plane k: 0 E2M1, 1 E4M3, 2 E2M3 */
  int32_t format_b[AWE_MAX_PLANES];
} awe_encoding_info;

/* Host.  The configuration record of an encoding (for AWE_ENC_MOD, of modulus m; the
   modulus argument is ignored otherwise).  AWE_ERR_UNSUPPORTED when no scheme exists. */
awe_status awe_get_encoding_info(awe_encoding enc, int32_t modulus, awe_encoding_info* out);

/* Host.  The encoding table (Alg. 1, "decompose each entry by table lookup"): for every
   input x in [xmin, xmax] of `side`, values[(x - xmin) * planes + p] = stored value of plane p
   (a doubled integer in S).  n_values must be at least (xmax - xmin + 1) * planes. */
awe_status awe_get_plane_table(awe_encoding enc, int32_t modulus, awe_side side,
                               int32_t* values, int64_t n_values);

/* Host.  Bytes of all stored planes of one side for `rows` x K (layout above). */
awe_status awe_plane_bytes(awe_encoding enc, int32_t modulus, awe_side side,
                           int64_t rows, int64_t K, size_t* bytes);

/* Encode one operand into its stored planes (Alg. 1, first two loops).
   side A: x is rows x K, x[i*ld + k];  side B: x is K x rows, x[k*ld + j] (rows = N).
   x holds int8 (exact encodings; int4 values for the A side of AWE_ENC_AWE4, values in
   [-1, 1] for the A side of AWE_ENC_TERNARY), int16 (AWE_ENC_FP16) or uint8
   residues (AWE_ENC_MOD).  planes receives awe_plane_bytes bytes.  A value outside the
   encoding's range is stored as 0 and, when d_range_flag is not NULL, sets *d_range_flag
   to a nonzero value (the flag is never cleared by the library). */
awe_status awe_encode(awe_encoding enc, int32_t modulus, awe_side side,
                      const void* x, int64_t rows, int64_t K, int64_t ld,
                      void* planes, int32_t* d_range_flag, hipStream_t stream);

/* The r FP4 products and the reconstruction on stored planes (Alg. 1, last two steps):
   C = (sum_k ell_k P_k) / D exactly, or (sum_k lambda_k P_k) mod m in [0, m) for
   AWE_ENC_MOD (then c_type must be AWE_I32).  planes_a / planes_b come from awe_encode
   with the same M, N, K.  k_seg: fold segment length (0 = the encoding's default;
   otherwise a positive multiple of AWE_K_PAD no larger than the default): every FP32 partial
   covers at most k_seg reduction indices and is then added to an integer accumulator. */
awe_status awe_gemm_planes(awe_encoding enc, int32_t modulus, int64_t M, int64_t N, int64_t K,
                           const void* planes_a, const void* planes_b,
                           void* C, int64_t ldc, awe_dtype c_type, int64_t k_seg,
                           hipStream_t stream);

/* Host.  Workspace awe_gemm_exact / awe_gemm_mod need (both sides' planes). */
awe_status awe_workspace_bytes(awe_encoding enc, int32_t modulus, int64_t M, int64_t N,
                               int64_t K, size_t* bytes);

/* C = A B exactly (Alg. 1 end to end): encode A, encode B, products, reconstruction.
   enc is one of the exact encodings.  A and B hold int8 (int4 values for the A side of
   AWE_ENC_AWE4, [-1, 1] for the A side of AWE_ENC_TERNARY) or int16 (AWE_ENC_FP16).
   c_type AWE_I32 requires max|A| max|B| K <= 2^31 - 1 (else AWE_ERR_OVERFLOW). */
awe_status awe_gemm_exact(awe_encoding enc, int64_t M, int64_t N, int64_t K,
                          const void* A, int64_t lda, const void* B, int64_t ldb,
                          void* C, int64_t ldc, awe_dtype c_type,
                          void* workspace, size_t ws_bytes, int32_t* d_range_flag,
                          hipStream_t stream);

/* Bytes of the fixed device array that holds the planes of awe_gemm_exact_noalloc. */
#define AWE_NOALLOC_MAX_BYTES ((size_t)64 << 20)

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
   loops, harnesses that forbid allocation): awe_gemm_exact without a workspace.  Both sides'
   stored planes go to a fixed device array of AWE_NOALLOC_MAX_BYTES bytes inside the library
   (one per GPU the library runs on, held until the process ends); the call allocates nothing
   and calls no allocating routine.  Arguments, layouts, results and errors as awe_gemm_exact,
   and AWE_ERR_WORKSPACE when awe_workspace_bytes for these sizes exceeds AWE_NOALLOC_MAX_BYTES
   (nothing is enqueued then).  Every call on a GPU uses that GPU's one array, which keeps the
   last call's planes (a call reads only planes it has written): calls that overlap on one GPU
   (other streams, other threads) race on it and give wrong results; order them on one stream.
   The first call on a device looks up the array's address (host side), and like awe_gemm_exact
   sets the GEMM's LDS limit and, for AWE_ENC_FP16, uploads its code table: make that first
   call eagerly before capturing the call into a graph. */
awe_status awe_gemm_exact_noalloc(awe_encoding enc, int64_t M, int64_t N, int64_t K,
                                  const void* A, int64_t lda, const void* B, int64_t ldb,
                                  void* C, int64_t ldc, awe_dtype c_type, int32_t* d_range_flag,
                                  hipStream_t stream);

/* C = (A B) mod m in [0, m), residue operands in [0, m) as uint8 (Sec. 5.3). */
awe_status awe_gemm_mod(int32_t m, int64_t M, int64_t N, int64_t K,
                        const uint8_t* A, int64_t lda, const uint8_t* B, int64_t ldb,
                        int32_t* C, int64_t ldc,
                        void* workspace, size_t ws_bytes, int32_t* d_range_flag,
                        hipStream_t stream);

/* ---- Residue number system (Sec. 5.3) ---------------------------------------------------
   A residue number system computes an integer product as its residues modulo pairwise
   coprime moduli m_1..m_n, one mod-m product per modulus, and recovers it by the Chinese
   remainder theorem; the result is unique when M = m_1 ... m_n > 2 K B_A B_B, B the bound
   on the entries (Sec. 5.3).  With 53-bit entries this is the integer layer of Ozaki
   scheme II (Sec. 2) for the FP64 significand.  Moduli lie in [2, 256] and n <= AWE_MAX_MODULI. */
#define AWE_MAX_MODULI 32

/* Device.  Residues of int64 entries: out + j*out_stride receives x mod moduli[j] in [0, m)
   as uint8, rows x cols row-major and dense (leading dimension cols); x is rows x cols
   row-major with leading dimension ld >= cols.  moduli is a host array.  Entries with
   |x| > bound set *d_range_flag (device, nullable) to a nonzero value; their residues are
   still exact.  The moduli need not be coprime here.  AWE_ERR_INVALID_VALUE for a modulus
   outside [2, 256], a bad n or size. */
awe_status awe_residues(const int64_t* x, int64_t rows, int64_t cols, int64_t ld, int64_t bound,
                        const int32_t* moduli, int32_t n, uint8_t* out, int64_t out_stride,
                        int32_t* d_range_flag, hipStream_t stream);

/* Device.  Chinese-remainder reconstruction.  residues + j*res_stride holds a rows x cols
   int32 matrix (leading dimension ld_res) of residues in [0, moduli[j]), as awe_gemm_mod
   writes them.  Writes the unique X in (-M/2, M/2] with X = residue (mod m_j) for all j:
   into c128 (nullable) as two int64 words per entry, c128[2*(i*ldc+j)] = low 64 bits
   (two's complement) and c128[2*(i*ldc+j)+1] = high 64 bits, so X = hi 2^64 + (unsigned) lo;
   and into c64 (nullable) rounded to the nearest double (ties to even).  The moduli must be
   pairwise coprime with M < 2^127 (AWE_ERR_INVALID_VALUE otherwise); residues outside
   [0, m_j) give an unspecified X. */
awe_status awe_crt(const int32_t* residues, int64_t res_stride, int64_t rows, int64_t cols,
                   int64_t ld_res, const int32_t* moduli, int32_t n,
                   int64_t* c128, double* c64, int64_t ldc, hipStream_t stream);

/* Host.  Workspace bytes awe_gemm_crt needs for these moduli and sizes. */
awe_status awe_crt_workspace_bytes(const int32_t* moduli, int32_t n, int64_t M, int64_t N,
                                   int64_t K, size_t* bytes);

/* Exact C = A B for int64 A (M x K, lda) and B (K x N, ldb) with |entries| <= bound_a and
   bound_b, through residues: every modulus's stored planes of both operands in one pass over
   each (the residues of awe_residues, encoded as awe_encode would), the mod-m product of
   awe_gemm_mod for every modulus (all moduli in one kernel launch where the tile configuration
   allows it), awe_crt into c128 and/or c64 (as for awe_crt, leading dimension ldc).  Requires M_prod > 2 K bound_a bound_b (AWE_ERR_OVERFLOW otherwise) and every
   modulus to have a scheme (AWE_ERR_UNSUPPORTED).  Entries beyond their bound set
   *d_range_flag.  The workspace (caller-owned device memory, awe_crt_workspace_bytes) holds the
   moduli's code tables, all their planes and the n residue products (one byte per output each:
   every modulus is at most 256); it is uploaded to and written on `stream`. */
awe_status awe_gemm_crt(int64_t M, int64_t N, int64_t K, const int64_t* A, int64_t lda,
                        const int64_t* B, int64_t ldb, int64_t bound_a, int64_t bound_b,
                        const int32_t* moduli, int32_t n, int64_t* c128, double* c64, int64_t ldc,
                        void* workspace, size_t ws_bytes, int32_t* d_range_flag,
                        hipStream_t stream);

/* Host.  Static description of a status code. */
const char* awe_status_string(awe_status s);

/* Host.  Detail of the last error returned on the calling thread ("" if none). */
const char* awe_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* AWE_H */
