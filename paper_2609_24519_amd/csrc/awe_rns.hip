// Residue number system around the mod-m products (Sec. 5.3): residues of
// int64 matrices for every modulus in one pass, and the Chinese-remainder
// reconstruction of the exact integer (Garner's mixed-radix form) with its
// correctly rounded double.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "awe_internal.h"

namespace awe {
namespace {

// x mod m for x < 2^32 and 2 <= m <= 256, with minv = floor((2^32 - 1) / m):
// q = floor(x minv / 2^32) is floor(x / m) or one less, so one correction
// step leaves r in [0, m).
__device__ __forceinline__ uint32_t mod_small(uint32_t x, uint32_t m, uint32_t minv) {
  const uint32_t q = __umulhi(x, minv);
  const uint32_t r = x - q * m;
  return r >= m ? r - m : r;
}

__global__ __launch_bounds__(256) void residues_kernel(const int64_t* __restrict__ x, int64_t rows,
                                                       int64_t cols, int64_t ld, int64_t bound,
                                                       ResidueParams P, uint8_t* __restrict__ out,
                                                       int64_t out_stride, int32_t* flag) {
  const int64_t total = rows * cols;
  bool out_of_range = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / cols, c = i - r * cols;
    const int64_t v = x[r * ld + c];
    out_of_range |= v > bound || v < -bound;
    // v = hi 2^32 + lo with hi signed; (uint32)hi = hi + 2^32 when hi < 0, so
    // v = (uint32)hi 2^32 + lo - [hi < 0] 2^64.
    const uint32_t lo = (uint32_t)v;
    const uint32_t hu = (uint32_t)((uint64_t)v >> 32);
    const bool neg = v < 0;
    for (int j = 0; j < P.n; ++j) {
      const uint32_t m = P.m[j], mi = P.minv[j];
      uint32_t t = mod_small(hu, m, mi) * P.p32[j] + mod_small(lo, m, mi);  // < 2^17
      t = mod_small(t, m, mi);
      if (neg) t = t >= P.p64[j] ? t - P.p64[j] : t + m - P.p64[j];
      out[j * out_stride + i] = (uint8_t)t;
    }
  }
  if (out_of_range && flag) *flag = 1;
}

// |X| < 2^127 (two's complement in lo/hi) -> nearest double, ties to even.
// The magnitude is shifted right until it fits in 64 bits, with every bit
// shifted out ORed into the lowest kept bit (a sticky bit), so that the one
// rounding of the 64-bit integer to 53 bits rounds as the full value would;
// the power-of-two scaling afterwards is exact.
__device__ __forceinline__ double wide_to_double(uint64_t lo, uint64_t hi) {
  const bool neg = (int64_t)hi < 0;
  if (neg) {  // negate the 128-bit value
    lo = ~lo + 1;
    hi = ~hi + (lo == 0 ? 1 : 0);
  }
  double d;
  if (hi == 0) {
    d = (double)lo;
  } else {
    const int s = 64 - __clzll((long long)hi);  // 1 .. 63: bits of hi in use
    const uint64_t sticky = (lo << (64 - s)) != 0 ? 1u : 0u;
    const uint64_t t = (hi << (64 - s)) | (lo >> s) | sticky;
    d = ldexp((double)t, s);
  }
  return neg ? -d : d;
}

template <int NMAX>
__global__ __launch_bounds__(256) void crt_kernel(const int32_t* __restrict__ res, int64_t res_stride,
                                                  int64_t rows, int64_t cols, int64_t ld_res,
                                                  CrtParams P, int64_t* __restrict__ c128,
                                                  double* __restrict__ c64, int64_t ldc) {
  const int64_t total = rows * cols;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / cols, c = i - r * cols;
    const int32_t* src = res + r * ld_res + c;
    // Mixed-radix digits: X = v_0 + v_1 P_1 + ... + v_{n-1} P_{n-1}, P_j = m_0 ... m_{j-1},
    // v_j = (r_j - sum_{i<j} v_i (P_i mod m_j)) (P_j^-1 mod m_j)  mod m_j.
    uint32_t v[NMAX];
#pragma unroll
    for (int j = 0; j < NMAX; ++j) {
      v[j] = 0;
      if (j < P.n) {
        int32_t acc = src[j * res_stride];
#pragma unroll
        for (int k = 0; k < j; ++k) acc -= (int32_t)(v[k] * P.c[k][j]);
        const uint32_t m = P.m[j], mi = P.minv[j];
        const uint32_t t = mod_small((uint32_t)(acc + P.off[j]), m, mi);  // acc + off >= 0
        v[j] = mod_small(t * P.d[j], m, mi);
      }
    }
    // Horner from the top digit, in 128 bits.
    unsigned __int128 X = 0;
#pragma unroll
    for (int j = NMAX - 1; j >= 0; --j)
      if (j < P.n) X = X * P.m[j] + v[j];
    const unsigned __int128 half = ((unsigned __int128)P.half_hi << 64) | P.half_lo;
    const unsigned __int128 Mw = ((unsigned __int128)P.M_hi << 64) | P.M_lo;
    if (X > half) X -= Mw;  // into (-M/2, M/2], two's complement
    const uint64_t lo = (uint64_t)X, hi = (uint64_t)(X >> 64);
    const int64_t o = r * ldc + c;
    if (c128) {
      c128[2 * o] = (int64_t)lo;
      c128[2 * o + 1] = (int64_t)hi;
    }
    if (c64) c64[o] = wide_to_double(lo, hi);
  }
}

unsigned grid_for(int64_t total) {
  const int64_t blocks = (total + 255) / 256;
  return (unsigned)(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096);
}

}  // namespace

awe_status launch_residues(const int64_t* x, int64_t rows, int64_t cols, int64_t ld, int64_t bound,
                           const ResidueParams& P, uint8_t* out, int64_t out_stride, int32_t* flag,
                           hipStream_t stream) {
  if (rows == 0 || cols == 0) return AWE_OK;
  hipLaunchKernelGGL(residues_kernel, dim3(grid_for(rows * cols)), dim3(256), 0, stream, x, rows, cols,
                     ld, bound, P, out, out_stride, flag);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) {
    set_error(std::string("residues launch: ") + hipGetErrorString(err));
    return AWE_ERR_HIP;
  }
  return AWE_OK;
}

awe_status launch_crt(const int32_t* res, int64_t res_stride, int64_t rows, int64_t cols,
                      int64_t ld_res, const CrtParams& P, int64_t* c128, double* c64, int64_t ldc,
                      hipStream_t stream) {
  if (rows == 0 || cols == 0) return AWE_OK;
  const dim3 grid(grid_for(rows * cols)), block(256);
  if (P.n <= 8)
    hipLaunchKernelGGL(crt_kernel<8>, grid, block, 0, stream, res, res_stride, rows, cols, ld_res, P,
                       c128, c64, ldc);
  else if (P.n <= 16)
    hipLaunchKernelGGL(crt_kernel<16>, grid, block, 0, stream, res, res_stride, rows, cols, ld_res, P,
                       c128, c64, ldc);
  else
    hipLaunchKernelGGL(crt_kernel<32>, grid, block, 0, stream, res, res_stride, rows, cols, ld_res, P,
                       c128, c64, ldc);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) {
    set_error(std::string("crt launch: ") + hipGetErrorString(err));
    return AWE_ERR_HIP;
  }
  return AWE_OK;
}

}  // namespace awe
