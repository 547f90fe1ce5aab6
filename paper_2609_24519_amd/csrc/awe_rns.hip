// Residue number system around the mod-m products (Sec. 5.3): residues of
// int64 matrices for every modulus in one pass, and the Chinese-remainder
// reconstruction of the exact integer (Garner's mixed-radix form) with its
// correctly rounded double.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <type_traits>

#include "awe_internal.h"
#include "plane_pack.h"

namespace awe {
namespace {

// x mod m for 0 <= x < 2^23 and 2 <= m <= 256, in full-rate arithmetic: x is exact
// in fp32 and x * inv (inv = 1/m in fp32) lies within 1/2 of x/m (two roundings of
// relative size 2^-24 on a quotient below 2^22), so the truncated quotient q is
// floor(x/m) - 1, floor(x/m) or floor(x/m) + 1; x + m - q m then lies in [0, 3m)
// and two unsigned-minimum steps (r - m wraps when r < m) bring it to [0, m).
__device__ __forceinline__ uint32_t mod_f(uint32_t x, uint32_t m, float inv) {
  const int32_t q = (int32_t)(uint32_t)((float)x * inv);  // below 2^22 + 1: a 24-bit operand
  uint32_t r = (uint32_t)((int32_t)(x + m) - __mul24(q, (int32_t)m));
  r = min(r, r - m);
  return min(r, r - m);
}

// Residue of one int64 value, given as its four 16-bit digits d0..d3 (two's
// complement) and its sign: u = sum_i d_i 2^(16 i) and x = u - 2^64 [x < 0], so
// x = d0 + d1 w16 + d2 w32 + d3 w48 - [x < 0] (2^64 mod m)  (mod m), with every
// product below 2^24 (24-bit multiplies) and the sum below 2^27; one more digit
// split brings it below 2^19 for mod_f.
struct ModConsts {
  uint32_t m, w16, w32, w48, negc;
  float inv;
  double dm, dinv;
};

__device__ __forceinline__ ModConsts mod_consts(const ResidueParams& P, int j) {
  return ModConsts{P.m[j], P.w16[j], P.w32[j], P.w48[j], P.negc[j], P.inv[j], (double)P.m[j], P.dinv[j]};
}

// Residue of an integer x with |x| < 2^53, held exactly as a double: q = floor(x * dinv)
// (dinv = 1/m in fp64) is within one of floor(x/m), since the product is within
// |x/m| 2^-52 <= 1 of x/m; x - q m is then an integer in [-m, 2m), computed exactly by
// one fused multiply-add, and brought to [0, m) as in mod_f.
__device__ __forceinline__ uint32_t residue_f64(double x, const ModConsts& k) {
  const double q = floor(x * k.dinv);
  uint32_t r = (uint32_t)((int32_t)fma(-q, k.dm, x) + (int32_t)k.m);
  r = min(r, r - k.m);
  return min(r, r - k.m);
}

// (neg_mask is all ones for a negative x, else zero: a select without a branch.)
__device__ __forceinline__ uint32_t residue_of(const uint32_t (&d)[4], uint32_t neg_mask, const ModConsts& k) {
  uint32_t t = d[0] + __umul24(d[1], k.w16) + __umul24(d[2], k.w32) + __umul24(d[3], k.w48) +
               (k.negc & neg_mask);
  t = __umul24(t >> 16, k.w16) + (t & 0xffffu);
  return mod_f(t, k.m, k.inv);
}

__device__ __forceinline__ void digits_of(int64_t v, uint32_t (&d)[4]) {
  const uint64_t u = (uint64_t)v;
  d[0] = (uint32_t)u & 0xffffu;
  d[1] = (uint32_t)(u >> 16) & 0xffffu;
  d[2] = (uint32_t)(u >> 32) & 0xffffu;
  d[3] = (uint32_t)(u >> 48);
}

// Residues of a rows x cols int64 matrix for every modulus: out[j * out_stride + r * cols + c].
// A thread takes 16 consecutive entries of a row.  kVec: cols and ld are multiples of 16 and
// the rows 128-byte aligned, so the entries come in as eight 16-byte loads and each modulus's
// 16 residues leave as one 16-byte store.
template <bool kVec>
__global__ __launch_bounds__(256) void residues_kernel(const int64_t* __restrict__ x, int64_t rows,
                                                       int64_t cols, int64_t ld, int64_t bound,
                                                       ResidueParams P, uint8_t* __restrict__ out,
                                                       int64_t out_stride, int32_t* flag) {
  constexpr int V = 16;
  const int64_t gpr = (cols + V - 1) / V;  // groups per row
  const int64_t total = rows * gpr;
  bool out_of_range = false;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < total;
       g += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = g / gpr, c0 = (g - r * gpr) * V;
    const int64_t* src = x + r * ld + c0;
    uint8_t* dst = out + r * cols + c0;
    if (kVec) {
      int64_t v[V];
#pragma unroll
      for (int q = 0; q < V / 2; ++q) {
        const longlong2 w = reinterpret_cast<const longlong2*>(src)[q];
        v[2 * q] = w.x;
        v[2 * q + 1] = w.y;
      }
      bool small = true;  // every entry below 2^53 in magnitude: exact as a double
#pragma unroll
      for (int e = 0; e < V; ++e) {
        out_of_range |= v[e] > bound || v[e] < -bound;
        small &= v[e] < (int64_t(1) << 53) && v[e] > -(int64_t(1) << 53);
      }
      if (small) {
        double xd[V];
#pragma unroll
        for (int e = 0; e < V; ++e) xd[e] = (double)v[e];
        for (int j = 0; j < P.n; ++j) {
          const ModConsts k = mod_consts(P, j);
          uint32_t w[V / 4] = {};
#pragma unroll
          for (int e = 0; e < V; ++e) w[e >> 2] |= residue_f64(xd[e], k) << (8 * (e & 3));
          *reinterpret_cast<uint4*>(dst + j * out_stride) = make_uint4(w[0], w[1], w[2], w[3]);
        }
      } else {
        uint32_t d[V][4], negm[V];
#pragma unroll
        for (int e = 0; e < V; ++e) {
          digits_of(v[e], d[e]);
          negm[e] = (uint32_t)(v[e] >> 63);
        }
        for (int j = 0; j < P.n; ++j) {
          const ModConsts k = mod_consts(P, j);
          uint32_t w[V / 4] = {};
#pragma unroll
          for (int e = 0; e < V; ++e) w[e >> 2] |= residue_of(d[e], negm[e], k) << (8 * (e & 3));
          *reinterpret_cast<uint4*>(dst + j * out_stride) = make_uint4(w[0], w[1], w[2], w[3]);
        }
      }
    } else {
      const int n = (int)min((int64_t)V, cols - c0);
      for (int e = 0; e < n; ++e) {
        const int64_t v = src[e];
        out_of_range |= v > bound || v < -bound;
        uint32_t d[4];
        digits_of(v, d);
        for (int j = 0; j < P.n; ++j)
          dst[j * out_stride + e] = (uint8_t)residue_of(d, (uint32_t)(v >> 63), mod_consts(P, j));
      }
    }
  }
  if (out_of_range && flag) *flag = 1;
}

// Residues of an int64 operand for every modulus, turned straight into each modulus's
// stored E2M1 planes (Alg. 1's table lookup applied to the residue), without the dense
// residue matrices in between.  One wave per brick of the plane layout, as the encoder:
// lane L = 32 h + t produces row t of the brick at reduction indices 32 h .. 32 h + 31.
// On the B side (x is K x N) lane l first loads reduction index ks*64 + l at 32 columns,
// computes their residues and stages them in LDS, then reads its column back, per modulus.
template <bool kTransposed>
__global__ __launch_bounds__(256) void residue_encode_kernel(ResidueEncodeArgs a, ResidueParams P) {
  __shared__ uint32_t slut[kMaxModuli * 256];
  __shared__ uint8_t tblk[kTransposed ? 4 : 1][kTransposed ? 64 * 32 : 1];
  const int n = P.n;
  for (int i = threadIdx.x; i < n * 256; i += blockDim.x) slut[i] = a.luts[i];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  bool out_of_range = false;
  for (int64_t brick = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); brick < a.nbricks;
       brick += (int64_t)gridDim.x * 4) {
    const int64_t rb = brick / a.KS, ks = brick - rb * a.KS;
    // this lane's 32 entries and which of them are real (the rest pad with code 0)
    int64_t v[32];
    uint32_t valid = 0;
    if (!kTransposed) {
      const int64_t row = rb * kBrickRows + (lane & 31), k0 = ks * kBrickK + (lane >> 5) * 32;
      const int64_t* src = a.x + row * a.ld + k0;
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        const bool ok = row < a.rows && k0 + e < a.K;
        v[e] = ok ? src[e] : 0;
        valid |= (ok ? 1u : 0u) << e;
      }
    } else {
      const int64_t kr = ks * kBrickK + lane, n0 = rb * kBrickRows;
      const int64_t* src = a.x + kr * a.ld + n0;
#pragma unroll
      for (int c = 0; c < 32; ++c) {
        const bool ok = kr < a.K && n0 + c < a.rows;
        v[c] = ok ? src[c] : 0;
        valid |= (ok ? 1u : 0u) << c;
      }
    }
    bool small = true;
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      out_of_range |= v[e] > a.bound || v[e] < -a.bound;
      small &= v[e] < (int64_t(1) << 53) && v[e] > -(int64_t(1) << 53);
    }
    // one route for the whole wave (a per-entry choice would run both)
    // Modulus j's planes of this brick from the lane's 32 residues r (this lane's row, or on
    // the B side its row of K x N, transposed through LDS first).
    auto emit = [&](int j, uint32_t (&r)[32]) {
      uint32_t ok = valid;
      if (kTransposed) {
        uint8_t* tw = tblk[threadIdx.x >> 6];
        uint32_t w[8] = {};
#pragma unroll
        for (int c = 0; c < 32; ++c) w[c >> 2] |= r[c] << (8 * (c & 3));
        *reinterpret_cast<uint4*>(tw + lane * 32) = make_uint4(w[0], w[1], w[2], w[3]);
        *reinterpret_cast<uint4*>(tw + lane * 32 + 16) = make_uint4(w[4], w[5], w[6], w[7]);
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
        __builtin_amdgcn_wave_barrier();
        const uint8_t* col = tw + (lane >> 5) * 32 * 32 + (lane & 31);
        const int64_t row = rb * kBrickRows + (lane & 31), k0 = ks * kBrickK + (lane >> 5) * 32;
        ok = 0;
#pragma unroll
        for (int e = 0; e < 32; ++e) {
          r[e] = col[e * 32];
          ok |= (row < a.rows && k0 + e < a.K ? 1u : 0u) << e;
        }
        __builtin_amdgcn_wave_barrier();
      }
      uint32_t code[32];
#pragma unroll
      for (int e = 0; e < 32; ++e) code[e] = ((ok >> e) & 1u) ? slut[j * 256 + r[e]] : 0u;
      uint8_t* dst = a.planes + a.off[j] + (ks * a.R32 + rb) * kBrickBytes + lane * 16;
      // the nibble transpose for exactly the planes the modulus has (1 to 3 for the mod-m
      // schemes; up to 8 fit a code word)
      auto store = [&](auto npc) {
        constexpr int NP = decltype(npc)::value;
        uint32_t d[NP][4];
        pack_e2m1_planes<NP>(code, d);
#pragma unroll
        for (int pl = 0; pl < NP; ++pl) {
          if (pl >= a.np[j]) break;
          *reinterpret_cast<uint4*>(dst + pl * a.plane_stride) = make_uint4(d[pl][0], d[pl][1], d[pl][2], d[pl][3]);
        }
      };
      const int np = a.np[j];
      if (np == 1)
        store(std::integral_constant<int, 1>{});
      else if (np == 2)
        store(std::integral_constant<int, 2>{});
      else if (np == 3)
        store(std::integral_constant<int, 3>{});
      else
        store(std::integral_constant<int, 8>{});
    };
    // one route for the whole wave (a per-entry choice would run both); the double route
    // keeps only the converted entries live across the moduli
    if (__all(small)) {
      double xd[32];
#pragma unroll
      for (int e = 0; e < 32; ++e) xd[e] = (double)v[e];
      for (int j = 0; j < n; ++j) {
        const ModConsts k = mod_consts(P, j);
        uint32_t r[32];
#pragma unroll
        for (int e = 0; e < 32; ++e) r[e] = residue_f64(xd[e], k);
        emit(j, r);
      }
    } else {
      for (int j = 0; j < n; ++j) {
        const ModConsts k = mod_consts(P, j);
        uint32_t r[32];
#pragma unroll
        for (int e = 0; e < 32; ++e) {
          uint32_t d[4];
          digits_of(v[e], d);
          r[e] = residue_of(d, (uint32_t)(v[e] >> 63), k);
        }
        emit(j, r);
      }
    }
  }
  if (out_of_range && a.flag) *a.flag = 1;
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

// The reconstruction's constants (about 1.6 KiB: the digit coefficients alone are
// n(n-1)/2 bytes) are staged once per workgroup in LDS and read there as uniform
// 16-byte words; held in scalar registers they would not fit.  Residues come as int32 or as
// bytes (RT).
template <int NMAX, class RT>
__global__ __launch_bounds__(256) void crt_kernel(const RT* __restrict__ res, int64_t res_stride,
                                                  int64_t rows, int64_t cols, int64_t ld_res,
                                                  CrtParams P, int64_t* __restrict__ c128,
                                                  double* __restrict__ c64, int64_t ldc) {
  __shared__ CrtParams sp;
  static_assert(sizeof(CrtParams) % 16 == 0 && sizeof(CrtParams) / 16 <= 256, "one 16-byte word per thread");
  if (threadIdx.x < sizeof(CrtParams) / 16)
    reinterpret_cast<uint4*>(&sp)[threadIdx.x] = reinterpret_cast<const uint4*>(&P)[threadIdx.x];
  __syncthreads();
  const int n = P.n;
  const int64_t total = rows * cols;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    asm volatile("" ::: "memory");  // read the constants from LDS where used, not hoisted into registers
    const int64_t r = i / cols, c = i - r * cols;
    const RT* src = res + r * ld_res + c;
    // Mixed-radix digits: X = v_0 + v_1 P_1 + ... + v_{n-1} P_{n-1}, P_j = m_0 ... m_{j-1},
    // v_j = (r_j - sum_{i<j} v_i (P_i mod m_j)) (P_j^-1 mod m_j)  mod m_j.  The subtracted
    // sum stays below off_j < 2^22, so both reductions are mod_f's.
    int32_t rj[NMAX];
#pragma unroll
    for (int j = 0; j < NMAX; ++j) rj[j] = j < n ? (int32_t)src[j * res_stride] : 0;
    uint32_t v[NMAX];
#pragma unroll
    for (int j = 0; j < NMAX; ++j) {
      v[j] = 0;
      if (j < n) {
        const uint4 k = *reinterpret_cast<const uint4*>(&sp.mod[j]);  // m, inv, d, off
        const uint32_t m = k.x;
        const float inv = __uint_as_float(k.y);
        int32_t acc = rj[j] + (int32_t)k.w;
#pragma unroll
        for (int q = 0; q < (j + 15) / 16; ++q) {
          const uint4 cw = *reinterpret_cast<const uint4*>(&sp.c[j][16 * q]);
          const uint32_t w[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
          for (int t = 0; t < 16 && 16 * q + t < j; ++t)
            acc -= __mul24((int32_t)v[16 * q + t], (int32_t)((w[t >> 2] >> (8 * (t & 3))) & 0xffu));
        }
        const uint32_t tj = mod_f((uint32_t)acc, m, inv);
        v[j] = mod_f(__umul24(tj, k.z), m, inv);
      }
    }
    // Horner over groups of three digits, from the top: X = D_0 + B_0 (D_1 + B_1 (D_2 + ...)),
    // D_g = v_j + m_j (v_{j+1} + m_{j+1} v_{j+2}) < B_g = m_j m_{j+1} m_{j+2} <= 2^24 (j = 3 g),
    // on four 32-bit limbs with 32 x 32 + 64-bit multiply-adds.
    constexpr int NG = (NMAX + 2) / 3;
    uint32_t X[4] = {0, 0, 0, 0};
#pragma unroll
    for (int gi = NG - 1; gi >= 0; --gi) {
      const int j = 3 * gi;
      if (j >= n) continue;
      const uint32_t m0 = sp.mod[j].m, m1 = j + 1 < n ? sp.mod[j + 1].m : 0u;
      const uint32_t v1 = j + 1 < NMAX ? v[j + 1] : 0u, v2 = j + 2 < NMAX ? v[j + 2] : 0u;
      const uint32_t D = v[j] + __umul24(m0, v1 + __umul24(m1, v2));
      if (j + 3 >= n) {  // the top group starts the Horner chain
        X[0] = D;
      } else {
        const uint32_t B = m0 * m1 * sp.mod[j + 2].m;
        uint64_t t = (uint64_t)X[0] * B + D;
        X[0] = (uint32_t)t;
#pragma unroll
        for (int q = 1; q < 4; ++q) {
          t = (uint64_t)X[q] * B + (t >> 32);
          X[q] = (uint32_t)t;
        }
      }
    }
    uint64_t lo = ((uint64_t)X[1] << 32) | X[0], hi = ((uint64_t)X[3] << 32) | X[2];
    // into (-M/2, M/2], two's complement: subtract M when X > floor(M/2)
    if (hi > P.half_hi || (hi == P.half_hi && lo > P.half_lo)) {
      const uint64_t nlo = lo - P.M_lo;
      hi = hi - P.M_hi - (lo < P.M_lo ? 1u : 0u);
      lo = nlo;
    }
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
  const bool vec = cols % 16 == 0 && ld % 16 == 0 && (reinterpret_cast<uintptr_t>(x) & 127) == 0 &&
                   (reinterpret_cast<uintptr_t>(out) & 15) == 0 && (P.n == 1 || out_stride % 16 == 0);
  const unsigned grid = grid_for(rows * ((cols + 15) / 16));
  if (vec)
    hipLaunchKernelGGL(residues_kernel<true>, dim3(grid), dim3(256), 0, stream, x, rows, cols, ld, bound,
                       P, out, out_stride, flag);
  else
    hipLaunchKernelGGL(residues_kernel<false>, dim3(grid), dim3(256), 0, stream, x, rows, cols, ld, bound,
                       P, out, out_stride, flag);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) {
    set_error(std::string("residues launch: ") + hipGetErrorString(err));
    return AWE_ERR_HIP;
  }
  return AWE_OK;
}

awe_status launch_residue_encode(const ResidueEncodeArgs& a, const ResidueParams& P, bool transposed,
                                 hipStream_t stream) {
  if (a.nbricks == 0) return AWE_OK;
  const int64_t blocks = std::min<int64_t>((a.nbricks + 3) / 4, 0x7fffffffLL);
  if (transposed)
    hipLaunchKernelGGL(residue_encode_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, a, P);
  else
    hipLaunchKernelGGL(residue_encode_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, a, P);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) {
    set_error(std::string("residue encode launch: ") + hipGetErrorString(err));
    return AWE_ERR_HIP;
  }
  return AWE_OK;
}

template <class RT>
awe_status launch_crt_t(const RT* res, int64_t res_stride, int64_t rows, int64_t cols, int64_t ld_res,
                        const CrtParams& P, int64_t* c128, double* c64, int64_t ldc, hipStream_t stream) {
  if (rows == 0 || cols == 0) return AWE_OK;
  const dim3 grid(grid_for(rows * cols)), block(256);
  if (P.n <= 8)
    hipLaunchKernelGGL((crt_kernel<8, RT>), grid, block, 0, stream, res, res_stride, rows, cols, ld_res, P,
                       c128, c64, ldc);
  else if (P.n <= 16)
    hipLaunchKernelGGL((crt_kernel<16, RT>), grid, block, 0, stream, res, res_stride, rows, cols, ld_res, P,
                       c128, c64, ldc);
  else
    hipLaunchKernelGGL((crt_kernel<32, RT>), grid, block, 0, stream, res, res_stride, rows, cols, ld_res, P,
                       c128, c64, ldc);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) {
    set_error(std::string("crt launch: ") + hipGetErrorString(err));
    return AWE_ERR_HIP;
  }
  return AWE_OK;
}

awe_status launch_crt(const int32_t* res, int64_t res_stride, int64_t rows, int64_t cols,
                      int64_t ld_res, const CrtParams& P, int64_t* c128, double* c64, int64_t ldc,
                      hipStream_t stream) {
  return launch_crt_t(res, res_stride, rows, cols, ld_res, P, c128, c64, ldc, stream);
}

awe_status launch_crt(const uint8_t* res, int64_t res_stride, int64_t rows, int64_t cols,
                      int64_t ld_res, const CrtParams& P, int64_t* c128, double* c64, int64_t ldc,
                      hipStream_t stream) {
  return launch_crt_t(res, res_stride, rows, cols, ld_res, P, c128, c64, ldc, stream);
}

}  // namespace awe
