/*
 * Oracle (test infrastructure only): the plain definition of the integer
 * matrix product that the FP4 method must reproduce exactly.
 *
 * The method's whole contract is that its output equals the error-free
 * integer product C = A B (Sec. 1, the definition of an error-free matrix
 * product; Alg. 1, its postcondition), or that product reduced modulo m
 * (Sec. 5.3, the congruence relaxation).  So the oracle is that definition
 * written out: a triple loop with a 64-bit integer accumulator.  It shares no
 * code, table or header with the HIP library.  Only tests/, the package's
 * smoke entry and the CPU-baseline leg of the benchmark may load it.
 *
 * Layouts: A is M x K row-major with leading dimension lda (A[i*lda + k]);
 * B is K x N row-major with leading dimension ldb (B[k*ldb + j]); C is M x N
 * row-major with leading dimension ldc.  OpenMP splits the rows of C; each
 * thread runs the same plain loop over its rows.
 */
#include <stdint.h>
#include <stdlib.h>

/* C = A B exactly, int8 inputs (an int4 operand arrives in an int8 container). */
void oracle_gemm_i8_i64(int64_t M, int64_t N, int64_t K,
                        const int8_t* A, int64_t lda,
                        const int8_t* B, int64_t ldb,
                        int64_t* C, int64_t ldc)
{
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < M; ++i) {
        int64_t* c = C + i * ldc;
        for (int64_t j = 0; j < N; ++j) c[j] = 0;
        for (int64_t k = 0; k < K; ++k) {
            const int64_t a = A[i * lda + k];
            const int8_t* b = B + k * ldb;
            for (int64_t j = 0; j < N; ++j) c[j] += a * (int64_t)b[j];
        }
    }
}

/* The same product restricted to the listed rows and columns of C:
   C[r*nc + c] = sum_k A[rows[r], k] * B[k, cols[c]].  Used to check sampled
   output tiles of products too large to form in full on the host. */
void oracle_gemm_i8_i64_sampled(int64_t nr, const int64_t* rows,
                                int64_t nc, const int64_t* cols, int64_t K,
                                const int8_t* A, int64_t lda,
                                const int8_t* B, int64_t ldb,
                                int64_t* C)
{
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < nr; ++r) {
        const int8_t* a = A + rows[r] * lda;
        for (int64_t c = 0; c < nc; ++c) {
            int64_t acc = 0;
            for (int64_t k = 0; k < K; ++k) acc += (int64_t)a[k] * (int64_t)B[k * ldb + cols[c]];
            C[r * nc + c] = acc;
        }
    }
}

/* (A B) mod m for residue operands, as the non-negative residue in [0, m).
   The exact integer row of A B is formed first (i-k-j order into an int64
   row, the same plain sum as oracle_gemm_i8_i64) and each entry is then
   reduced; the residues of Sec. 5.3 are those of the exact product, so the
   order in which the exact sum is formed does not matter. */
void oracle_gemm_u8_mod(int64_t m, int64_t M, int64_t N, int64_t K,
                        const uint8_t* A, int64_t lda,
                        const uint8_t* B, int64_t ldb,
                        int32_t* C, int64_t ldc)
{
    #pragma omp parallel
    {
        int64_t* row = (int64_t*)malloc((size_t)(N > 0 ? N : 1) * sizeof(int64_t));
        #pragma omp for schedule(static)
        for (int64_t i = 0; i < M; ++i) {
            for (int64_t j = 0; j < N; ++j) row[j] = 0;
            for (int64_t k = 0; k < K; ++k) {
                const int64_t a = A[i * lda + k];
                const uint8_t* b = B + k * ldb;
                for (int64_t j = 0; j < N; ++j) row[j] += a * (int64_t)b[j];
            }
            for (int64_t j = 0; j < N; ++j) C[i * ldc + j] = (int32_t)(((row[j] % m) + m) % m);
        }
        free(row);
    }
}

/* Sampled variant of the residue product. */
void oracle_gemm_u8_mod_sampled(int64_t m, int64_t nr, const int64_t* rows,
                                int64_t nc, const int64_t* cols, int64_t K,
                                const uint8_t* A, int64_t lda,
                                const uint8_t* B, int64_t ldb,
                                int32_t* C)
{
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < nr; ++r) {
        const uint8_t* a = A + rows[r] * lda;
        for (int64_t c = 0; c < nc; ++c) {
            int64_t acc = 0;
            for (int64_t k = 0; k < K; ++k) acc += (int64_t)a[k] * (int64_t)B[k * ldb + cols[c]];
            C[r * nc + c] = (int32_t)(((acc % m) + m) % m);
        }
    }
}

/* C = A B exactly for int64 entries, accumulated in 128 bits: the integer
   product a residue number system reconstructs (Sec. 5.3, with B the input
   bound, |C| <= K B_A B_B).  The caller keeps sum_k |A[i,k] B[k,j]| below
   2^127 (e.g. |entries| <= 2^53 - 1 with K <= 2^20).  Each entry of C is
   returned as two words, C = hi * 2^64 + lo with lo unsigned. */
void oracle_gemm_i64_i128(int64_t M, int64_t N, int64_t K,
                          const int64_t* A, int64_t lda,
                          const int64_t* B, int64_t ldb,
                          uint64_t* lo, int64_t* hi, int64_t ldc)
{
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < M; ++i) {
        for (int64_t j = 0; j < N; ++j) {
            __int128 acc = 0;
            for (int64_t k = 0; k < K; ++k) acc += (__int128)A[i * lda + k] * (__int128)B[k * ldb + j];
            lo[i * ldc + j] = (uint64_t)acc;
            hi[i * ldc + j] = (int64_t)(acc >> 64);
        }
    }
}

/* Sampled variant of the 128-bit product: rows x cols of C, row-major nr x nc. */
void oracle_gemm_i64_i128_sampled(int64_t nr, const int64_t* rows,
                                  int64_t nc, const int64_t* cols, int64_t K,
                                  const int64_t* A, int64_t lda,
                                  const int64_t* B, int64_t ldb,
                                  uint64_t* lo, int64_t* hi)
{
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < nr; ++r) {
        const int64_t* a = A + rows[r] * lda;
        for (int64_t c = 0; c < nc; ++c) {
            __int128 acc = 0;
            for (int64_t k = 0; k < K; ++k) acc += (__int128)a[k] * (__int128)B[k * ldb + cols[c]];
            lo[r * nc + c] = (uint64_t)acc;
            hi[r * nc + c] = (int64_t)(acc >> 64);
        }
    }
}

/* Number of OpenMP threads the loops above will use (reported with timings). */
int oracle_num_threads(void)
{
    int n = 1;
    #pragma omp parallel
    {
        #pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}
