// HIP kernels for gfx950: the plane encoder and the multi-plane FP4 GEMM with
// its fused integer reconstruction (Alg. 1 of the paper).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <map>
#include <mutex>
#include <set>
#include <string>
#include <type_traits>

#include "awe_internal.h"
#include "gemm_layout.h"
#include "plane_pack.h"

namespace awe {

// Code tables of a wide encoding (int16 inputs), one per side: too large for
// kernel arguments, so they live in device memory of the module.
__device__ uint32_t g_wide_lut[2][kWideValues];

// The planes of awe_gemm_exact_noalloc: a fixed array of the module, one per GPU the library
// runs on, held until the process ends.  Host code never passes its name to a kernel (on the
// host it is only a stand-in for the symbol): noalloc_planes() looks up its device address.
static __device__ __align__(256) uint8_t scratch[kNoallocBytes];

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));

struct LutArg {
  uint32_t v[256];
};

// ---------------------------------------------------------------------------
// Encoder (Alg. 1, table lookup and plane formation).  One wave per 1 KiB
// brick: lane L = 32 h + t turns the 32 inputs of row rb*32 + t at reduction
// indices ks*64 + 32 h + j into one 16-byte fragment per stored plane.  The
// plane values (combinations of limbs included) come from one 256-entry table
// of packed E2M1 codes, so forming a combination plane costs nothing here.
// ---------------------------------------------------------------------------
// At least four waves per SIMD (at most 128 registers): the encoder is HBM-bound and needs that
// many loads in flight (the B side took 15 % longer at three).
template <bool kTransposed>
__global__ __launch_bounds__(256, 4) void encode_kernel(const uint8_t* __restrict__ x, int64_t rows,
                                                     int64_t K, int64_t ld, int64_t KS,
                                                     int64_t R32, int64_t nbricks, int nplanes,
                                                     int nplanes8, bool fp6,
                                                     uint8_t* __restrict__ planes,
                                                     int64_t plane_stride, int32_t* flag,
                                                     LutArg lut) {
  __shared__ uint32_t slut[256];
  // B side: per-wave 64 x 32 input block stored column-major, kTileCol bytes per column (64
  // rows + 16 bytes of padding, so that the 16-byte column reads below hit distinct banks)
  constexpr int kTileCol = 80;
  __shared__ __attribute__((aligned(16))) uint8_t tblk[kTransposed ? 4 : 1][kTransposed ? 32 * kTileCol : 1];
  slut[threadIdx.x] = lut.v[threadIdx.x];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  // Each wave takes one brick, or several when the grid is capped.  A side: the four waves of
  // a workgroup take four consecutive k-steps of one row block (32 rows x 256 bytes of A).
  // B side: four adjacent column blocks of one k-step, so that a workgroup reads whole 128-byte
  // lines of B's rows (64 rows x 128 bytes); with the k-steps in a workgroup instead, each
  // line was read by four workgroups far apart in time and, when B was not in the last-level
  // cache, fetched from HBM up to four times.  Consecutive workgroups take consecutive column
  // groups of one k-step, so that the workgroups in flight read whole rows of B (measured 3-7 %
  // faster from HBM than consecutive k-steps of one column group).  Here nbricks counts
  // ceil(R32 / 4) * 4 row blocks on the B side, and the waves past R32 have no brick.
  for (int64_t brick = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); brick < nbricks;
       brick += (int64_t)gridDim.x * 4) {
  int64_t rb, ks;
  if (kTransposed) {
    const int64_t q = brick >> 2, groups = (R32 + 3) / 4;
    ks = q / groups;
    rb = (q - ks * groups) * 4 + (brick & 3);
    if (rb >= R32) continue;
  } else {
    rb = brick / KS;
    ks = brick - rb * KS;
  }
  const int64_t row = rb * kBrickRows + (lane & 31);
  const int64_t k0 = ks * kBrickK + (lane >> 5) * 32;
  const bool row_ok = row < rows;

  uint32_t e[32];
  if (!kTransposed) {
    const uint8_t* src = x + row * ld + k0;
    if (row_ok && k0 + 32 <= K && (reinterpret_cast<uintptr_t>(src) & 15) == 0) {
      const uint4 lo = *reinterpret_cast<const uint4*>(src);
      const uint4 hi = *reinterpret_cast<const uint4*>(src + 16);
      const uint32_t w[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
      for (int j = 0; j < 32; ++j) e[j] = slut[(w[j >> 2] >> (8 * (j & 3))) & 0xff];
    } else {
#pragma unroll
      for (int j = 0; j < 32; ++j) e[j] = (row_ok && k0 + j < K) ? slut[src[j]] : 0u;
    }
  } else {
    // B side, K x N row-major: the brick needs the 64 x 32 block of B at rows
    // (reduction indices) ks*64 .. +63 and columns rb*32 .. +31.  Load i of lane l takes
    // the 16 bytes at columns 16 (l & 1) .. +15 of block row 32 i + l / 2 (so each load
    // instruction covers 32 rows x 32 bytes) and writes them into those columns of this
    // wave's column-major tile; lane 32 h + t then reads rows 32 h .. 32 h + 31 of column t
    // as two 16-byte words.
    uint8_t* tw = tblk[threadIdx.x >> 6];
    const int64_t n0 = rb * kBrickRows;
    const int half = lane & 1;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = 32 * i + (lane >> 1);
      const int64_t kr = ks * kBrickK + r;
      const uint8_t* src = x + kr * ld + n0 + 16 * half;
      uint32_t w[4];
      if (kr < K && n0 + 32 <= rows && (reinterpret_cast<uintptr_t>(src) & 15) == 0) {
        const uint4 v = *reinterpret_cast<const uint4*>(src);
        w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
      } else {
#pragma unroll
        for (int d = 0; d < 4; ++d) w[d] = 0;
        for (int c = 0; c < 16; ++c)
          if (kr < K && n0 + 16 * half + c < rows) w[c >> 2] |= (uint32_t)src[c] << (8 * (c & 3));
      }
#pragma unroll
      for (int c = 0; c < 16; ++c)
        tw[(16 * half + c) * kTileCol + r] = (uint8_t)(w[c >> 2] >> (8 * (c & 3)));
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
    __builtin_amdgcn_wave_barrier();
    const uint8_t* col = tw + (lane & 31) * kTileCol + (lane >> 5) * 32;
    const uint4 c0 = *reinterpret_cast<const uint4*>(col);
    const uint4 c1 = *reinterpret_cast<const uint4*>(col + 16);
    const uint32_t cw[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
#pragma unroll
    for (int j = 0; j < 32; ++j)
      e[j] = (row_ok && k0 + j < K) ? slut[(cw[j >> 2] >> (8 * (j & 3))) & 0xff] : 0u;
  }
  uint32_t bad = 0;
#pragma unroll
  for (int j = 0; j < 32; ++j) bad |= e[j];
  if ((bad & kLutInvalid) && flag != nullptr) atomicOr(flag, 1);

  if (fp6) {
    // E2M3 planes (1.5 plane strides each) in 3 KiB units of two k-steps: lane L's 32
    // six-bit codes form 6 dwords, the first 4 at i*1024 + 16 L and the last 2 at
    // 2048 + i*512 + 8 L of the unit (i = ks & 1).
    uint8_t* unit = planes + ((ks >> 1) * R32 + rb) * (3 * kBrickBytes);
    const int i = (int)(ks & 1);
    for (int p = 0; p < nplanes; ++p) {
      uint32_t d[6] = {0, 0, 0, 0, 0, 0};
#pragma unroll
      for (int j = 0; j < 32; ++j) {
        const uint32_t c = (e[j] >> (8 * p)) & 0x3fu;
        const int bit = 6 * j;
        d[bit >> 5] |= c << (bit & 31);
        if ((bit & 31) > 26) d[(bit >> 5) + 1] |= c >> (32 - (bit & 31));
      }
      uint8_t* u = unit + p * (3 * plane_stride / 2);
      *reinterpret_cast<uint4*>(u + i * 1024 + lane * 16) = make_uint4(d[0], d[1], d[2], d[3]);
      *reinterpret_cast<uint2*>(u + 2048 + i * 512 + lane * 8) = make_uint2(d[4], d[5]);
    }
    continue;
  }

  // E4M3 planes (2 KiB bricks, 32 bytes per lane) first, then the E2M1 planes; an E4M3
  // plane occupies two plane strides.
  for (int p = 0; p < nplanes8; ++p) {
    uint32_t d[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 32; ++j) d[j >> 2] |= ((e[j] >> (8 * p)) & 0xffu) << (8 * (j & 3));
    uint8_t* dst8 = planes + 2 * p * plane_stride + (ks * R32 + rb) * (2 * kBrickBytes) + lane * 32;
    *reinterpret_cast<uint4*>(dst8) = make_uint4(d[0], d[1], d[2], d[3]);
    *reinterpret_cast<uint4*>(dst8 + 16) = make_uint4(d[4], d[5], d[6], d[7]);
  }
  uint8_t* dst = planes + 2 * nplanes8 * plane_stride + (ks * R32 + rb) * kBrickBytes + lane * 16;
  if (nplanes8 == 0) {
    // All planes E2M1: the nibble transpose of pack_e2m1_planes (about a third of the VALU work
    // of packing each plane nibble by nibble, which bounded the encoder's rate).
    uint32_t d[8][4];
    pack_e2m1_planes<8>(e, d);
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      if (p >= nplanes) break;
      *reinterpret_cast<uint4*>(dst + p * plane_stride) = make_uint4(d[p][0], d[p][1], d[p][2], d[p][3]);
    }
    continue;
  }
  for (int p = 0; p < nplanes - nplanes8; ++p) {
    const int sh = 8 * nplanes8 + 4 * p;
    uint32_t d[4] = {0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 32; ++j) d[j >> 3] |= ((e[j] >> sh) & 0xfu) << (4 * (j & 7));
    *reinterpret_cast<uint4*>(dst + p * plane_stride) = make_uint4(d[0], d[1], d[2], d[3]);
  }
  }  // bricks
}

// ---------------------------------------------------------------------------
// Encoder for a wide encoding (int16 inputs in [xmin, xmin + nvalues)): the
// same brick production from a table of up to 4096 packed codes.  The table
// is too large for kernel arguments; it lives in a device array (one per side,
// uploaded once per device) and each workgroup stages it into LDS, then walks
// several bricks per wave to spread that load.
// ---------------------------------------------------------------------------
template <bool kTransposed>
__global__ __launch_bounds__(256) void encode16_kernel(const int16_t* __restrict__ x, int64_t rows,
                                                       int64_t K, int64_t ld, int64_t KS, int64_t R32,
                                                       int64_t nbricks, int nplanes,
                                                       uint8_t* __restrict__ planes, int64_t plane_stride,
                                                       int32_t* flag, int side, int32_t xmin,
                                                       int32_t nvalues) {
  __shared__ uint32_t slut[kWideValues];
  for (int i = threadIdx.x; i < nvalues; i += blockDim.x) slut[i] = g_wide_lut[side][i];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  auto look = [&](int v) -> uint32_t {
    const uint32_t i = (uint32_t)(v - xmin);
    return i < (uint32_t)nvalues ? slut[i] : kLutInvalid;
  };
  uint32_t bad = 0;
  for (int64_t brick = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); brick < nbricks;
       brick += (int64_t)gridDim.x * 4) {
    const int64_t rb = brick / KS, ks = brick - rb * KS;
    const int64_t row = rb * kBrickRows + (lane & 31);
    const int64_t k0 = ks * kBrickK + (lane >> 5) * 32;
    const bool row_ok = row < rows;
    uint32_t e[32];
    if (!kTransposed) {
      const int16_t* src = x + row * ld + k0;
      if (row_ok && k0 + 32 <= K && (reinterpret_cast<uintptr_t>(src) & 15) == 0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint4 w = *reinterpret_cast<const uint4*>(src + 8 * q);
          const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
          for (int j = 0; j < 8; ++j) e[8 * q + j] = look((int16_t)(ws[j >> 1] >> (16 * (j & 1))));
        }
      } else {
#pragma unroll
        for (int j = 0; j < 32; ++j) e[j] = (row_ok && k0 + j < K) ? look(src[j]) : 0u;
      }
    } else {
#pragma unroll
      for (int j = 0; j < 32; ++j) e[j] = (row_ok && k0 + j < K) ? look(x[(k0 + j) * ld + row]) : 0u;
    }
#pragma unroll
    for (int j = 0; j < 32; ++j) bad |= e[j];
    uint8_t* dst = planes + (ks * R32 + rb) * kBrickBytes + lane * 16;
    for (int p = 0; p < nplanes; ++p) {
      uint32_t d[4] = {0, 0, 0, 0};
#pragma unroll
      for (int j = 0; j < 32; ++j) d[j >> 3] |= ((e[j] >> (4 * p)) & 0xfu) << (4 * (j & 7));
      *reinterpret_cast<uint4*>(dst + p * plane_stride) = make_uint4(d[0], d[1], d[2], d[3]);
    }
  }
  if ((bad & kLutInvalid) && flag != nullptr) atomicOr(flag, 1);
}

// ---------------------------------------------------------------------------
// Multi-plane FP4 GEMM (Alg. 1, the r products and the reconstruction).
//
// A workgroup of WM x WN waves computes a BM x BN tile of C; each wave owns
// (32 BMW) x (32 BNW) as BMW x BNW blocks of the 32x32x64 scaled FP4 MFMA.
// The reduction runs as one stream of k-tiles (128 indices = 2 bricks per row
// block) in the order segment -> product -> k-tile: a wave accumulates one
// product in FP32 for a whole fold segment, then folds that partial into an
// int32 accumulator with its reconstruction coefficient (cvt + 24-bit
// multiply-add) and restarts the FP32 accumulator.  Every FP32 partial is an
// exact integer of magnitude at most 2^23 - 1 by the segment length (Sec. 3.4
// with a factor 2 of margin for the 24-bit multiply), and the int32 sum is
// exact modulo 2^32; the host splits the reduction into launches so that the
// true value of each launch fits in int32.
//
// Both E8M0 block scales are 2^1 (byte 128): the stored E2M1 values are s/2
// for the doubled integers s of S, so each product of codes is s_a s_b
// exactly and the FP32 accumulators hold the integer plane products.
//
// A product-major stream needs one FP32 and one int32 accumulator per output
// (8 bytes of registers), so the register file bounds the tile; the operand
// bytes each CU must pull through its L1 per MFMA fall as the tile grows.
// ---------------------------------------------------------------------------
constexpr uint32_t kScale2 = 0x80808080u;  // E8M0 2^1 in every byte


struct GemmArgs {
  const uint8_t* pa;
  const uint8_t* pb;
  int64_t stride_a, stride_b;
  int32_t rba, rbb;  // row blocks of the A and B planes
  int32_t KS;        // bricks along K per row block
  int32_t t_begin, t_end;  // stage range of this launch (stages of KT reduction indices)
  int32_t ts;        // fold segment in stages
  int32_t r;
  uint64_t pidx_a, pidx_b;  // plane of product k in bits 4k .. 4k+3 (kept in SGPRs: no loads in the loop)
  int32_t fold_ell[kMaxProducts];
  uint32_t fold_mask;
  void* C;
  int64_t ldc;
  int32_t M, N;
  int32_t c64;  // C's elements: 0 int32, 1 int64, 2 bytes (residues only, modulus set)
  int32_t accumulate, log2D, modulus;
  int32_t tiles_m, tiles_n;
  int64_t outer;  // C (+)= outer * (sum / D)
  uint32_t sa[2], sb[2];  // two planes per side: E8M0 scale word of plane 0 / 1 of A and B
  // Tiles n_full .. tiles_m * tiles_n - 1 (the ragged last round of workgroups) are
  // each computed by `split` workgroups over consecutive parts of the reduction range,
  // which add their exact partial results into C (zeroed beforehand) with atomics.
  int32_t n_full, split;
  int32_t outer_g[4];  // outer weight of accumulator group d (all pairs with outer groups)
};

// Position in the reduction stream: product p, k-tile t, current fold segment [cs, ce).
struct Cursor {
  int p, t, cs, ce;
};

// Advance to the next stage; saturates on the last stage of the launch (the
// copies issued past the end re-read that stage into a buffer nobody reads,
// which keeps the number of copies in flight the same for every stage).
__device__ __forceinline__ void cursor_next(Cursor& c, const GemmArgs& g, int t_end) {
  const int t1 = c.t + 1;
  const bool end_t = t1 == c.ce;
  const int p1 = c.p + (end_t ? 1 : 0);
  const bool end_p = end_t && p1 == g.r;
  const bool end_all = end_p && c.ce == t_end;
  const int ncs = end_p ? c.ce : c.cs;
  const int nce = end_p ? min(c.ce + g.ts, t_end) : c.ce;
  c.t = end_all ? c.t : (end_t ? ncs : t1);
  c.p = end_all ? c.p : (end_p ? 0 : p1);
  c.cs = end_all ? c.cs : ncs;
  c.ce = end_all ? c.ce : nce;
}

// One 16-byte-per-lane global -> LDS copy: the wave's 64 lanes fill the 1 KiB
// at LDS byte address `lds` (wave-uniform, in M0).  The brick's base address
// is wave-uniform (SGPRs); every lane adds its own 16-byte offset `voff`.
// Issued as inline assembly so that the compiler does not serialise the
// copies; completion is awaited explicitly with vmcnt.
__device__ __forceinline__ void dma_brick(const uint8_t* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base), "s"(lds)
               : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most `stages` younger stages of this wave's copies are in flight.
template <class C, int STAGES>
__device__ __forceinline__ void wait_stages(int wave) {
  if (C::B_XTRA == 0 || wave < C::B_XTRA)
    wait_vmcnt<(C::A_PW + C::B_LO + (C::B_XTRA ? 1 : 0)) * C::COPIES * STAGES>();
  else
    wait_vmcnt<(C::A_PW + C::B_LO) * C::COPIES * STAGES>();
}

// Workgroup barrier that is also a compiler memory barrier: no LDS access may
// move across it.  The caller has already waited for its own copies (vmcnt)
// and LDS reads (lgkmcnt) as the protocol needs.
__device__ __forceinline__ void block_barrier() { asm volatile("s_barrier" ::: "memory"); }

__device__ __forceinline__ void wait_lgkm0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// The copies of one stage (units as copy_unit assigns them; addresses from gemm_layout.h).
template <class C>
__device__ __forceinline__ void load_stage_a(const GemmArgs& g, const Cursor& c, uint32_t stage_lds,
                                             int tm, int wave, int lane) {
  const int ka = (int)((g.pidx_a >> (4 * c.p)) & 15u);
  const uint8_t* pa = g.pa + (int64_t)ka * g.stride_a + stage_global<C>(c.t, g.rba);
  const uint32_t voff = lane * 16;
#pragma unroll
  for (int i = 0; i < C::A_PW; ++i) {
    const int id = copy_unit<C>(true, wave, i);
    const UnitPos u = unit_pos<C>(true, id);
    const int rb = min(tm * (C::BM / kBrickRows) + u.rb, g.rba - 1);
#pragma unroll
    for (int h = 0; h < C::COPIES; ++h)
      dma_brick(pa + unit_global<C>(u, rb, g.rba, g.stride_a, h), voff, stage_lds + unit_lds<C>(true, id, h));
  }
}

template <class C>
__device__ __forceinline__ void load_stage_b(const GemmArgs& g, const Cursor& c, uint32_t stage_lds,
                                             int tn, int wave, int lane) {
  const int kb = (int)((g.pidx_b >> (4 * c.p)) & 15u);
  const uint8_t* pb = g.pb + (int64_t)kb * g.stride_b + stage_global<C>(c.t, g.rbb);
  const uint32_t voff = lane * 16;
#pragma unroll
  for (int i = 0; i < C::B_LO + (C::B_XTRA ? 1 : 0); ++i) {
    const int id = copy_unit<C>(false, wave, i);
    if (id < 0) break;
    const UnitPos u = unit_pos<C>(false, id);
    const int cb = min(tn * (C::BN / kBrickRows) + u.rb, g.rbb - 1);
#pragma unroll
    for (int h = 0; h < C::COPIES; ++h)
      dma_brick(pb + unit_global<C>(u, cb, g.rbb, g.stride_b, h), voff, stage_lds + unit_lds<C>(false, id, h));
  }
}

template <class C>
__device__ __forceinline__ void load_stage(const GemmArgs& g, const Cursor& c, uint32_t stage_lds,
                                           int tm, int tn, int wave, int lane) {
  load_stage_a<C>(g, c, stage_lds, tm, wave, lane);
  load_stage_b<C>(g, c, stage_lds, tn, wave, lane);
}

// Copy q of this wave's share of a stage (one copy per unit): q < A_PW is its A unit q, then
// its B units, in the order load_stage issues them.
template <class C, int Q>
__device__ __forceinline__ void load_one(const GemmArgs& g, const Cursor& c, uint32_t stage_lds, int tm,
                                         int tn, int wave, int lane) {
  static_assert(C::COPIES == 1, "one copy per unit");
  const uint32_t voff = lane * 16;
  if constexpr (Q < C::A_PW) {
    const int ka = (int)((g.pidx_a >> (4 * c.p)) & 15u);
    const int id = copy_unit<C>(true, wave, Q);
    const UnitPos u = unit_pos<C>(true, id);
    const int rb = min(tm * (C::BM / kBrickRows) + u.rb, g.rba - 1);
    dma_brick(g.pa + (int64_t)ka * g.stride_a + stage_global<C>(c.t, g.rba) + unit_global<C>(u, rb, g.rba, g.stride_a, 0), voff,
              stage_lds + unit_lds<C>(true, id, 0));
  } else {
    const int kb = (int)((g.pidx_b >> (4 * c.p)) & 15u);
    const int id = copy_unit<C>(false, wave, Q - C::A_PW);
    const UnitPos u = unit_pos<C>(false, id);
    const int cb = min(tn * (C::BN / kBrickRows) + u.rb, g.rbb - 1);
    dma_brick(g.pb + (int64_t)kb * g.stride_b + stage_global<C>(c.t, g.rbb) + unit_global<C>(u, cb, g.rbb, g.stride_b, 0), voff,
              stage_lds + unit_lds<C>(false, id, 0));
  }
}

__device__ __forceinline__ v8i frag(const uint8_t* p) {
  const int4 x = *reinterpret_cast<const int4*>(p);
  v8i v = {x.x, x.y, x.z, x.w, 0, 0, 0, 0};
  return v;
}

// A lane's fragment of k-step i of a unit (the spans of frag_spans): E2M1 16 bytes, E4M3 32
// bytes, E2M3 24 bytes (the MFMA reads 6 of the 8 operand registers for E2M3, so the last two
// are left undefined instead of zeroed, which would cost two registers per fragment).
template <int FMT>
__device__ __forceinline__ v8i frag_fmt(const uint8_t* unit, int i, int lane) {
  constexpr Spans z = frag_spans<FMT>(0, 0);
  const Spans sp = frag_spans<FMT>(i, lane);
  if constexpr (FMT == 0) {
    return frag(unit + sp.off[0]);
  } else if constexpr (FMT == 1) {
    const int4 x = *reinterpret_cast<const int4*>(unit + sp.off[0]);
    const int4 y = *reinterpret_cast<const int4*>(unit + sp.off[0] + 16);
    v8i v = {x.x, x.y, x.z, x.w, y.x, y.y, y.z, y.w};
    return v;
  } else {
    static_assert(z.n == 2 && z.len[0] == 16 && z.len[1] == 8, "E2M3 spans");
    const v4i x = *reinterpret_cast<const v4i*>(unit + sp.off[0]);
    const v2i y = *reinterpret_cast<const v2i*>(unit + sp.off[1]);
    const v4i y4 = __builtin_shufflevector(y, y, 0, 1, -1, -1);
    return __builtin_shufflevector(x, y4, 0, 1, 2, 3, 4, 5, -1, -1);
  }
}

// The wave's operand fragments for one k-step (64 reduction indices) of a stage.
template <class C>
struct Frags {
  // plane pl's fragments at pl * BMW (pl * BNW); 16x16x128: one per 16-row block
  v8i a[C::MF == 16 ? C::AM : C::SPA * C::BMW], b[C::MF == 16 ? C::AN : C::SPB * C::BNW];
};

template <class C>
__device__ __forceinline__ void read_frags(Frags<C>& f, const uint8_t* stage, int ks, int wm,
                                           int wn, int lane) {
  if constexpr (C::MF == 16) {
    const uint32_t lo = frag16_lane_offset(lane);
#pragma unroll
    for (int ia = 0; ia < C::BMW; ++ia)
#pragma unroll
      for (int h = 0; h < 2; ++h) f.a[2 * ia + h] = frag(stage + frag16_unit<C>(true, wm * C::BMW + ia, ks, h) + lo);
#pragma unroll
    for (int j = 0; j < C::BNW; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h) f.b[2 * j + h] = frag(stage + frag16_unit<C>(false, wn * C::BNW + j, ks, h) + lo);
    return;
  }
  const int i = ks % C::UK;
#pragma unroll
  for (int pl = 0; pl < C::SPA; ++pl)
#pragma unroll
    for (int ia = 0; ia < C::BMW; ++ia)
      f.a[pl * C::BMW + ia] = frag_fmt<C::FMT>(stage + frag_unit<C>(true, pl, wm * C::BMW + ia, ks), i, lane);
#pragma unroll
  for (int pl = 0; pl < C::SPB; ++pl)
#pragma unroll
    for (int j = 0; j < C::BNW; ++j)
      f.b[pl * C::BNW + j] = frag_fmt<C::FMT>(stage + frag_unit<C>(false, pl, wn * C::BNW + j, ks), i, lane);
}

__device__ __forceinline__ void mfma_block(v16f& acc, const v8i& a, const v8i& b) {
  acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc, 4, 4, 0, kScale2, 0, kScale2);
}

// E4M3 x E4M3 (format selects 0): the stored E4M3 values are the integers
// themselves, so both block scales are 2^0 (byte 127).
constexpr uint32_t kScale1 = 0x7f7f7f7fu;
__device__ __forceinline__ void mfma_block8(v16f& acc, const v8i& a, const v8i& b) {
  acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc, 0, 0, 0, kScale1, 0, kScale1);
}

// E2M3 x E2M3 (format selects 2): a stored integer n is the E2M3 value n / 8, so
// both block scales are 2^3 (byte 130) and each product of codes is n_a n_b.
constexpr uint32_t kScale8 = 0x82828282u;
__device__ __forceinline__ void mfma_block6(v16f& acc, const v8i& a, const v8i& b) {
  acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc, 2, 2, 0, kScale8, 0, kScale8);
}

#ifndef AWE_GEMM_GROUP_M
#define AWE_GEMM_GROUP_M 4
#endif
// Workgroup -> output tile.  Workgroups are dispatched round-robin over the 8
// XCDs (each with its own L2): consecutive tiles of one XCD's share are taken
// from a band of AWE_GEMM_GROUP_M tile rows, so the workgroups an XCD runs at
// once cover a compact block of C and share their A rows and B columns in
// that XCD's L2.
__device__ __forceinline__ void tile_of_block(const GemmArgs& g, int bid, int& tm, int& tn) {
  int lin = bid;
  if (bid < g.n_full && (g.n_full & 7) == 0) lin = (bid & 7) * (g.n_full >> 3) + (bid >> 3);
  const int per_group = AWE_GEMM_GROUP_M * g.tiles_n;
  const int grp = lin / per_group;
  const int first = grp * AWE_GEMM_GROUP_M;
  const int gm = min(g.tiles_m - first, AWE_GEMM_GROUP_M);
  const int in = lin - grp * per_group;
  tm = first + in % gm;
  tn = in / gm;
}

// One output of the epilogue: the int32 accumulator holds D*C (exact schemes,
// modulo 2^32, the true value fits) or sum lambda_k P_k (residues); a launch
// group of a wider scheme contributes outer * (its sum / D).  C is written with
// non-temporal stores where it is not read back (C is not reused by the kernel,
// and all tiles of a round write at once: measured 2 % faster at 8192^3).
__device__ __forceinline__ void store_value(const GemmArgs& g, int row, int col, int64_t t) {
  if (row >= g.M || col >= g.N) return;
  const int64_t off = (int64_t)row * g.ldc + col;
  if (g.c64) {
    int64_t* Cp = reinterpret_cast<int64_t*>(g.C);
    if (g.accumulate)
      Cp[off] += t;
    else
      __builtin_nontemporal_store(t, Cp + off);
  } else {
    int32_t* Cp = reinterpret_cast<int32_t*>(g.C);
    if (g.accumulate)
      Cp[off] = (int32_t)((uint32_t)Cp[off] + (uint32_t)t);
    else
      __builtin_nontemporal_store((int32_t)t, Cp + off);
  }
}

__device__ __forceinline__ void store_output(const GemmArgs& g, int row, int col, int32_t val) {
  if (g.modulus) {
    if (row >= g.M || col >= g.N) return;
    const int64_t off = (int64_t)row * g.ldc + col;
    const int32_t m = g.modulus;
    int32_t rr = val % m;
    if (rr < 0) rr += m;
    int32_t* Cp = reinterpret_cast<int32_t*>(g.C);
    if (g.accumulate)
      Cp[off] = (Cp[off] + rr) % m;
    else
      __builtin_nontemporal_store(rr, Cp + off);
    return;
  }
  store_value(g, row, col, (int64_t)(val >> g.log2D) * g.outer);
}

// A residue written as a byte (C's elements are bytes: m <= 256).  Its own epilogue loop, so
// that the int32 / int64 one keeps its size (a larger loop body stopped its unrolling).
__device__ __forceinline__ void store_residue_u8(const GemmArgs& g, int row, int col, int32_t val) {
  if (row >= g.M || col >= g.N) return;
  const int64_t off = (int64_t)row * g.ldc + col;
  const int32_t m = g.modulus;
  int32_t rr = val % m;
  if (rr < 0) rr += m;
  uint8_t* Cb = reinterpret_cast<uint8_t*>(g.C);
  if (g.accumulate) {
    const int32_t s = Cb[off] + rr;
    Cb[off] = (uint8_t)(s >= m ? s - m : s);
  } else {
    __builtin_nontemporal_store((uint8_t)rr, Cb + off);
  }
}

// A part of a split tile: its exact partial (a whole number of reduction
// indices with all products, so a multiple of D) is added atomically into C,
// which the host zeroed (or which holds an earlier launch's sum).
__device__ __forceinline__ void add_value(const GemmArgs& g, int row, int col, int64_t t) {
  if (row >= g.M || col >= g.N) return;
  const int64_t off = (int64_t)row * g.ldc + col;
  if (g.c64)
    atomicAdd(reinterpret_cast<unsigned long long*>(g.C) + off, (unsigned long long)t);
  else
    atomicAdd(reinterpret_cast<int32_t*>(g.C) + off, (int32_t)t);
}

__device__ __forceinline__ void add_output(const GemmArgs& g, int row, int col, int32_t val) {
  add_value(g, row, col, (int64_t)(val >> g.log2D) * g.outer);
}

// Zeroes the C region of the split tiles before the parts add into it: block
// (x, y) clears rows y, y + gridDim.y, ... of split tile x, consecutive threads
// on consecutive columns.
__global__ __launch_bounds__(256) void zero_tiles_kernel(GemmArgs g, int bm, int bn, int esize) {
  int tm, tn;
  tile_of_block(g, g.n_full + blockIdx.x, tm, tn);
  const int rows = min(bm, g.M - tm * bm), cols = min(bn, g.N - tn * bn);
  for (int r = blockIdx.y; r < rows; r += gridDim.y) {
    const int64_t row = (int64_t)(tm * bm + r) * g.ldc + tn * bn;
    for (int c = threadIdx.x; c < cols; c += blockDim.x) {
      if (esize == 8)
        reinterpret_cast<int64_t*>(g.C)[row + c] = 0;
      else
        reinterpret_cast<int32_t*>(g.C)[row + c] = 0;
    }
  }
}

// f(integral_constant<int, Q>) for Q = I .. N - 1, unrolled at compile time.
template <int I, int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// One workgroup's output tile over reduction stages t_beg .. t_end - 1 (part >= 0: one
// part of a split tile, added into C).  fold_coef(p): the fold coefficient of product p.
// The arguments come by value: through a reference the compiler keeps more of them live
// (the 256 x 192 tiles then spill).
template <class C, bool ROWS16, class FoldCoef>
__device__ __forceinline__ void gemm_tile(GemmArgs g, FoldCoef fold_coef, int tile, int part, int t_beg,
                                          int t_end) {
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int tm, tn;
  tile_of_block(g, tile, tm, tn);
  const int wm = wave / C::WN, wn = wave % C::WN;
  const uint32_t lds0 = (uint32_t)(uintptr_t)smem;

  using AccT = std::conditional_t<C::MF == 16, v4f, v16f>;
  AccT acc[C::AM][C::AN];
  AccT accg[C::AP ? C::NG : 1][C::AM][C::AN];  // all pairs: one accumulator per group i + j
  int32_t iaccg[C::NOUT][C::AM][C::AN][C::AV];   // outer groups: one int32 accumulator per group
  // Blocks b = i * AN + j < NREG keep their int32 fold accumulators in iacc; the others in this
  // wave's LDS fold area (int32 v of lane L of block b - NREG at ((b - NREG) * AV + v) * 64 + L).
  constexpr int NREG = C::AM * C::AN - C::NLB;
  int32_t iacc[C::AM][C::AN][C::AV];
  // int32 v of this lane in LDS fold block lb is fold_lds[(lb * AV + v) * 64] (fold_lds_offset)
  int32_t* const fold_lds = reinterpret_cast<int32_t*>(smem + C::FOLD_LDS_OFFSET) +
                            (fold_lds_offset<C>(wave, 0, 0, lane) - C::FOLD_LDS_OFFSET) / 4;
  // (register blocks and LDS blocks in separate loops: an expression that chooses between
  // iacc and the LDS area would keep iacc out of registers)
#pragma unroll
  for (int i = 0; i < C::AM; ++i)
#pragma unroll
    for (int j = 0; j < C::AN; ++j)
#pragma unroll
      for (int v = 0; v < C::AV; ++v) acc[i][j][v] = 0.0f;
  if constexpr (C::AP) {
#pragma unroll
    for (int d = 0; d < C::NG; ++d)
#pragma unroll
      for (int i = 0; i < C::AM; ++i)
#pragma unroll
        for (int j = 0; j < C::AN; ++j)
#pragma unroll
          for (int v = 0; v < C::AV; ++v) {
            accg[d][i][j][v] = 0.0f;
            if constexpr (C::OUTG) iaccg[d][i][j][v] = 0;
          }
  }
#pragma unroll
  for (int b = 0; b < NREG; ++b)
#pragma unroll
    for (int v = 0; v < C::AV; ++v) iacc[b / C::AN][b % C::AN][v] = 0;
#pragma unroll
  for (int b = NREG; b < C::AM * C::AN; ++b)
#pragma unroll
    for (int v = 0; v < C::AV; ++v) fold_lds[((b - NREG) * C::AV + v) * 64] = 0;

  // After product p's last stage of a fold segment: fold its FP32 partials into the int32
  // accumulators with the product's coefficient and restart them.
  auto fold_product = [&](int p) {
    if constexpr (C::OUTG) {
      // outer groups: every group's partial with the stream product's coefficient, into the
      // group's own int32 accumulator
      if ((g.fold_mask >> p) & 1u) {
        const int32_t l = fold_coef(p);
#pragma unroll
        for (int d = 0; d < C::NG; ++d) {
#pragma unroll
          for (int i = 0; i < C::AM; ++i)
#pragma unroll
            for (int j = 0; j < C::AN; ++j)
#pragma unroll
              for (int v = 0; v < C::AV; ++v) {
                iaccg[d][i][j][v] += __mul24(l, (int32_t)accg[d][i][j][v]);
                accg[d][i][j][v] = 0.0f;
              }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      return;
    } else if constexpr (C::AP) {
      // all pairs: every group's partial with its coefficient (fold_coef of the group index)
#pragma unroll
      for (int d = 0; d < C::NG; ++d) {
        const int32_t l = fold_coef(d);
#pragma unroll
        for (int b = 0; b < NREG; ++b) {
          const int i = b / C::AN, j = b % C::AN;
#pragma unroll
          for (int v = 0; v < C::AV; ++v) {
            iacc[i][j][v] += __mul24(l, (int32_t)accg[d][i][j][v]);
            accg[d][i][j][v] = 0.0f;
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      return;
    }
    if ((g.fold_mask >> p) & 1u) {
      const int32_t l = fold_coef(p);
      // one 32x32 block at a time keeps the temporaries of the fold small
#pragma unroll
      for (int b = 0; b < NREG; ++b) {
        const int i = b / C::AN, j = b % C::AN;
#pragma unroll
        for (int v = 0; v < C::AV; ++v) {
          // (two planes per side: the weights are in the scales, the partial may use
          // all 24 bits, and it is added unmultiplied)
          if constexpr (C::NPL == 2)
            iacc[i][j][v] += (int32_t)acc[i][j][v];
          else
            iacc[i][j][v] += __mul24(l, (int32_t)acc[i][j][v]);
          acc[i][j][v] = 0.0f;
        }
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int b = NREG; b < C::AM * C::AN; ++b) {
        const int i = b / C::AN, j = b % C::AN;
#pragma unroll
        for (int v = 0; v < C::AV; ++v) {
          fold_lds[((b - NREG) * C::AV + v) * 64] += __mul24(l, (int32_t)acc[i][j][v]);
          acc[i][j][v] = 0.0f;
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  constexpr int NSTAGE = C::NSTAGE;
  if constexpr (C::SCHED == 3) {
    // Stream stage u sits in buffer u % 3; its barrier sits inside its second k-step, after the
    // MFMAs of the first row of fragments (BAR of them).  A k-step's MFMAs run over the NR x NC
    // pairs of the wave's A and B fragments, row by row (all pairs: row pi * BMW + i is block i
    // of the stage's A plane pi, column pj * BNW + j block j of B plane pj, into accumulator
    // group pi + pj).
    //  k-step 0: MFMAs on fragments read before; the fragments of k-step 1 are read from
    //    buffer u into each register set as soon as its last k-step-0 MFMA has issued; stage
    //    u + 2's copies go to buffer (u + 2) % 3 (freed by the barrier of stage u - 1), one after
    //    every other MFMA (after the odd ones: 1-2 % faster than right after that barrier, where
    //    they meet every wave's reads of the next fragments, or after the even MFMAs).
    //  k-step 1, first BAR MFMAs; then wait until stage u + 1 has landed (stage u + 2's copies
    //    may still be in flight) and this wave's reads of buffer u are done (they have had the
    //    first BAR MFMAs to land); barrier: every wave is done with buffer u, stage u + 1 is
    //    complete.
    //  k-step 1, the other MFMAs: stage u + 1's k-step-0 fragments are read from buffer
    //    (u + 1) % 3 into the registers already free and then as more free up.
    constexpr int PER_STAGE = C::A_PW + C::B_LO;  // copies per wave and stage
    constexpr int NR = C::SPA * C::BMW, NC = C::SPB * C::BNW;  // fragment rows and columns
    constexpr int NQ = NR * NC, BAR = NC;
    constexpr int GAP = NQ / PER_STAGE;  // MFMAs per copy in k-step 0
    Frags<C> f;
    // MFMA q of a k-step, and the reads of fragment row r / column c of k-step ks from a buffer
    auto mfma_q = [&](auto qc) {
      constexpr int q = decltype(qc)::value, r = q / NC, c = q % NC;
      if constexpr (C::AP)
        mfma_block(accg[r / C::BMW + c / C::BNW][r % C::BMW][c % C::BNW], f.a[r], f.b[c]);
      else
        mfma_block(acc[r][c], f.a[r], f.b[c]);
    };
    auto read_a = [&](auto rc, uint32_t off, int ks) {
      constexpr int r = decltype(rc)::value;
      f.a[r] = frag(smem + off + frag_unit<C>(true, r / C::BMW, wm * C::BMW + r % C::BMW, ks) + lane * 16);
    };
    auto read_b = [&](auto cc, uint32_t off, int ks) {
      constexpr int c = decltype(cc)::value;
      f.b[c] = frag(smem + off + frag_unit<C>(false, c / C::BNW, wn * C::BNW + c % C::BNW, ks) + lane * 16);
    };
    static_assert(C::KSTEPS == 2 && NSTAGE == 3 && NQ % PER_STAGE == 0, "schedule 3");
    Cursor nxt{0, t_beg, t_beg, min(t_beg + g.ts, t_end)};
    load_stage<C>(g, nxt, lds0, tm, tn, wave, lane);
    cursor_next(nxt, g, t_end);
    load_stage<C>(g, nxt, lds0 + C::STAGE_BYTES, tm, tn, wave, lane);
    cursor_next(nxt, g, t_end);
    wait_vmcnt<PER_STAGE>();
    block_barrier();
    read_frags<C>(f, smem, 0, wm, wn, lane);
    int buf = 0;
    for (int cs = t_beg; cs < t_end; cs += g.ts) {
      const int ce = min(cs + g.ts, t_end);
      for (int p = 0; p < g.r; ++p) {
        for (int t = cs; t < ce; ++t) {
          const int b1 = buf == 2 ? 0 : buf + 1, b2 = b1 == 2 ? 0 : b1 + 1;
          const uint32_t cur_off = buf * C::STAGE_BYTES, next_off = b1 * C::STAGE_BYTES;
          static_for<0, NQ>([&](auto qc) {
            constexpr int q = decltype(qc)::value, r = q / NC, c = q % NC;
            mfma_q(qc);
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (q % GAP == GAP / 2)
              load_one<C, q / GAP>(g, nxt, lds0 + b2 * C::STAGE_BYTES, tm, tn, wave, lane);
            if constexpr (c == NC - 1) read_a(std::integral_constant<int, r>{}, cur_off, 1);
            if constexpr (r == NR - 1) read_b(std::integral_constant<int, c>{}, cur_off, 1);
            __builtin_amdgcn_sched_barrier(0);
          });
          cursor_next(nxt, g, t_end);
          static_for<0, NQ>([&](auto qc) {
            constexpr int q = decltype(qc)::value;
            mfma_q(qc);
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (q == BAR - 1) {
              wait_vmcnt<PER_STAGE>();
              wait_lgkm0();
              block_barrier();
            }
            if constexpr (q >= BAR - 1) {
              // registers whose last use is MFMA q (at the barrier: MFMA BAR - 1 or earlier)
              static_for<0, NR>([&](auto rc) {
                constexpr int last = decltype(rc)::value * NC + NC - 1;
                if constexpr (last == q || (q == BAR - 1 && last < q)) read_a(rc, next_off, 0);
              });
              static_for<0, NC>([&](auto cc) {
                constexpr int last = (NR - 1) * NC + decltype(cc)::value;
                if constexpr (last == q || (q == BAR - 1 && last < q)) read_b(cc, next_off, 0);
              });
            }
            __builtin_amdgcn_sched_barrier(0);
          });
          buf = b1;
        }
        fold_product(p);
      }
    }
  } else if constexpr (C::SCHED >= 1) {
    // Stream stage u sits in buffer u % NSTAGE.  During stage u each wave issues its copies of
    // stage u + NSTAGE - 1 into the buffer of stage u - 1 (freed by the barrier at the end of
    // stage u - 1), spread over the stage, one after every GAP-th MFMA: the eight waves' copies
    // then do not queue at the address unit together, and a wave that waits for one has matrix
    // work in flight.  Schedule 2 also reads a later k-step's fragments during the k-step before
    // it, each into its register set as soon as the last MFMA that uses the old value has
    // issued.  Before the barrier at the end of stage u each wave waits until stage u + 1 has
    // landed (its copies of the NSTAGE - 2 stages after u + 1 may still be in flight) and its
    // reads of stage u are done.
    constexpr int PER_STAGE = C::A_PW + C::B_LO;  // copies per wave and stage
    constexpr int CPK = PER_STAGE / C::KSTEPS, GAP = C::BMW * C::BNW / CPK;
    Cursor nxt{0, t_beg, t_beg, min(t_beg + g.ts, t_end)};
#pragma unroll
    for (int i = 0; i < NSTAGE - 1; ++i) {
      load_stage<C>(g, nxt, lds0 + i * C::STAGE_BYTES, tm, tn, wave, lane);
      cursor_next(nxt, g, t_end);
    }
    wait_vmcnt<(NSTAGE - 2) * PER_STAGE>();
    block_barrier();
    Frags<C> f;
    int buf = 0, cbuf = NSTAGE - 1;
    for (int cs = t_beg; cs < t_end; cs += g.ts) {
      const int ce = min(cs + g.ts, t_end);
      for (int p = 0; p < g.r; ++p) {
        for (int t = cs; t < ce; ++t) {
          const uint32_t cur_off = buf * C::STAGE_BYTES, cp_lds = lds0 + cbuf * C::STAGE_BYTES;
          static_for<0, C::KSTEPS>([&](auto kc) {
            constexpr int ks = decltype(kc)::value;
            if constexpr (C::SCHED == 1 || ks == 0) {
              read_frags<C>(f, smem + cur_off, ks, wm, wn, lane);
              __builtin_amdgcn_sched_barrier(0);
            }
            static_for<0, C::BMW * C::BNW>([&](auto qc) {
              constexpr int q = decltype(qc)::value, i = q / C::BNW, j = q % C::BNW;
              mfma_block(acc[i][j], f.a[i], f.b[j]);
              if constexpr (q % GAP == 0) {
                __builtin_amdgcn_sched_barrier(0);
                load_one<C, ks * CPK + q / GAP>(g, nxt, cp_lds, tm, tn, wave, lane);
                __builtin_amdgcn_sched_barrier(0);
              }
              if constexpr (C::SCHED == 2 && ks + 1 < C::KSTEPS) {
                __builtin_amdgcn_sched_barrier(0);
                if constexpr (j == C::BNW - 1)
                  f.a[i] = frag(smem + cur_off + frag_unit<C>(true, 0, wm * C::BMW + i, ks + 1) + lane * 16);
                if constexpr (i == C::BMW - 1)
                  f.b[j] = frag(smem + cur_off + frag_unit<C>(false, 0, wn * C::BNW + j, ks + 1) + lane * 16);
                __builtin_amdgcn_sched_barrier(0);
              }
            });
            __builtin_amdgcn_sched_barrier(0);
          });
          cursor_next(nxt, g, t_end);
          wait_vmcnt<(NSTAGE - 2) * PER_STAGE>();
          wait_lgkm0();
          block_barrier();
          buf = buf + 1 == NSTAGE ? 0 : buf + 1;
          cbuf = cbuf + 1 == NSTAGE ? 0 : cbuf + 1;
        }
        fold_product(p);
      }
    }
  } else {
    Cursor nxt{0, t_beg, t_beg, min(t_beg + g.ts, t_end)};
    // Prologue: stages 0 .. NSTAGE-1 fill the whole ring.
#pragma unroll
    for (int i = 0; i < NSTAGE; ++i) {
      load_stage<C>(g, nxt, lds0 + i * C::STAGE_BYTES, tm, tn, wave, lane);
      cursor_next(nxt, g, t_end);
    }
    wait_stages<C, NSTAGE - 1>(wave);
    block_barrier();
    constexpr int PD = C::PD, NSETS = C::NSETS;
    Frags<C> f[NSETS];
#pragma unroll
    for (int ks = 0; ks < PD; ++ks) read_frags<C>(f[ks], smem, ks, wm, wn, lane);

    // Stage s, k-steps 0 .. KST-1: the MFMAs of k-step ks run on fragment set
    // ks % NSETS while the reads of k-step ks + PD go into another set.  At k-step
    // KST - PD, before the first read that crosses into stage s+1: wait until
    // stage s+1 has landed and this wave's reads of stage s are done (all of them
    // were issued by then), barrier, refill stage s's buffer with stage s+NSTAGE.
    // The barrier sits between two groups of MFMAs.
    int buf = 0;
    for (int cs = t_beg; cs < t_end; cs += g.ts) {
      const int ce = min(cs + g.ts, t_end);
      for (int p = 0; p < g.r; ++p) {
        for (int t = cs; t < ce; ++t) {
          const uint32_t cur_off = buf * C::STAGE_BYTES;
          const int nbuf = buf + 1 == NSTAGE ? 0 : buf + 1;
#pragma unroll
          for (int ks = 0; ks < C::KSTEPS; ++ks) {
            if (ks == C::KSTEPS - PD) {
              wait_stages<C, NSTAGE - 2>(wave);
              wait_lgkm0();
              block_barrier();
              load_stage<C>(g, nxt, lds0 + cur_off, tm, tn, wave, lane);
              cursor_next(nxt, g, t_end);
            }
            const int kr = ks + PD;  // k-step whose fragments are read now
            if (kr < C::KSTEPS)
              read_frags<C>(f[kr % NSETS], smem + cur_off, kr, wm, wn, lane);
            else
              read_frags<C>(f[kr % NSETS], smem + nbuf * C::STAGE_BYTES, kr - C::KSTEPS, wm, wn, lane);
            // in place (PD = 0) the MFMAs wait for these reads; read ahead, the reads are
            // spread between the MFMAs below
            if constexpr (PD == 0) __builtin_amdgcn_sched_barrier(0);
            const Frags<C>& cur = f[ks % NSETS];
            if constexpr (C::MF == 16) {
#pragma unroll
              for (int i = 0; i < C::AM; ++i)
#pragma unroll
                for (int j = 0; j < C::AN; ++j)
                  acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(cur.a[i], cur.b[j], acc[i][j], 4, 4,
                                                                               0, kScale2, 0, kScale2);
            } else if constexpr (C::AP) {
              // every pair (pi, pj) of the stage's planes into accumulator group pi + pj
#pragma unroll
              for (int pi = 0; pi < C::NPA; ++pi)
#pragma unroll
                for (int pj = 0; pj < C::NPB; ++pj)
#pragma unroll
                  for (int i = 0; i < C::BMW; ++i)
#pragma unroll
                    for (int j = 0; j < C::BNW; ++j)
                      mfma_block(accg[pi + pj][i][j], cur.a[pi * C::BMW + i], cur.b[pj * C::BNW + j]);
            } else if constexpr (C::NPL == 2) {
              // the four plane pairs, each block's MFMAs four apart in issue order
#pragma unroll
              for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int i = 0; i < C::BMW; ++i)
#pragma unroll
                  for (int j = 0; j < C::BNW; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                        cur.a[(q >> 1) * C::BMW + i], cur.b[(q & 1) * C::BNW + j], acc[i][j], 2, 2, 0,
                        (int)g.sa[q >> 1], 0, (int)g.sb[q & 1]);
            } else {
#pragma unroll
              for (int i = 0; i < C::BMW; ++i)
#pragma unroll
                for (int j = 0; j < C::BNW; ++j) {
                  if constexpr (C::FMT == 0)
                    mfma_block(acc[i][j], cur.a[i], cur.b[j]);
                  else if constexpr (C::FMT == 1)
                    mfma_block8(acc[i][j], cur.a[i], cur.b[j]);
                  else
                    mfma_block6(acc[i][j], cur.a[i], cur.b[j]);
                }
            }
            if constexpr (PD > 0) {
              // issue order: one MFMA, then one fragment read of a later k-step (measured
              // 1-3 % faster than all reads ahead of the MFMAs)
#pragma unroll
              for (int q = 0; q < (C::AP ? C::NPA * C::NPB : C::NPL * C::NPL) * C::AM * C::AN; ++q) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // an MFMA
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // an LDS read
              }
            }
            __builtin_amdgcn_sched_barrier(0);
          }
          if constexpr (PD == 0) {
            // every read of stage s has been consumed: refill its buffer after the barrier
            wait_stages<C, NSTAGE - 2>(wave);
            block_barrier();
            load_stage<C>(g, nxt, lds0 + cur_off, tm, tn, wave, lane);
            cursor_next(nxt, g, t_end);
          }
          buf = nbuf;
        }
        fold_product(p);
      }
    }
  }
  wait_vmcnt<0>();  // the saturated copies past the end must land before the wave exits

  // Epilogue: exact shift by log2 D, or the non-negative residue mod m.  Output layout of
  // the MFMA: 32x32 blocks, lane L holds rows 8 (v / 4) + 4 (L / 32) + v % 4 of column L % 32;
  // 16x16 blocks, rows 4 (L / 16) + v of column L % 16.
  constexpr int BS = C::MF;  // rows and columns of an accumulator block
  const int row0 = tm * C::BM + wm * (32 * C::BMW) + (BS == 16 ? 4 * (lane >> 4) : 4 * (lane >> 5));
  const int col0 = tn * C::BN + wn * (32 * C::BNW) + (lane & (BS - 1));
  auto emit = [&](int i, int j, int v, int32_t val) {
    const int row = row0 + i * BS + (BS == 16 ? v : 8 * (v >> 2) + (v & 3)), col = col0 + j * BS;
    if (part < 0)
      store_output(g, row, col, val);
    else
      add_output(g, row, col, val);
  };
  if constexpr (ROWS16 && C::MF == 32 && !C::OUTG && C::FMT == 0 && C::NPL == 1) {
    // Whole tiles written (not added) as int32 or int64: each 32 x 32 block goes through a
    // per-wave LDS slot (rows of 36 words, 16-byte aligned) so that a lane stores 16 bytes of
    // one row (4 outputs) instead of 16 single outputs of one column: a quarter of the store
    // instructions.  Uniform per workgroup.
    static_assert(C::NW * 32 * 36 * 4 <= C::NSTAGE * C::STAGE_BYTES, "row slots inside the ring");
    const bool rows16 = part < 0 && !g.modulus && !g.accumulate && (tm + 1) * C::BM <= g.M &&
                        (tn + 1) * C::BN <= g.N && (g.ldc & 3) == 0 &&
                        (reinterpret_cast<uintptr_t>(g.C) & 15) == 0;
    if (rows16) {
      block_barrier();  // every wave is past its last ring read, and its last copies have landed
      int32_t* const slot = reinterpret_cast<int32_t*>(smem) + wave * (32 * 36);
      const int rr = lane >> 3, cc = (lane & 7) * 4;  // read: rows rr + 8 q, columns cc .. cc + 3
      auto put_block = [&](int i, int j, auto value) {
#pragma unroll
        for (int v = 0; v < 16; ++v) slot[(8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)) * 36 + (lane & 31)] = value(v);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const v4i w = *reinterpret_cast<const v4i*>(slot + (rr + 8 * q) * 36 + cc);
          const int64_t off =
              (int64_t)(tm * C::BM + wm * (32 * C::BMW) + i * 32 + rr + 8 * q) * g.ldc + tn * C::BN +
              wn * (32 * C::BNW) + j * 32 + cc;
          if (g.c64) {
            typedef long long v2l __attribute__((ext_vector_type(2)));
            v2l lo, hi;
            lo[0] = (long long)(w[0] >> g.log2D) * g.outer;
            lo[1] = (long long)(w[1] >> g.log2D) * g.outer;
            hi[0] = (long long)(w[2] >> g.log2D) * g.outer;
            hi[1] = (long long)(w[3] >> g.log2D) * g.outer;
            v2l* Cp = reinterpret_cast<v2l*>(reinterpret_cast<int64_t*>(g.C) + off);
            __builtin_nontemporal_store(lo, Cp);
            __builtin_nontemporal_store(hi, Cp + 1);
          } else {
            v4i t;
#pragma unroll
            for (int e = 0; e < 4; ++e) t[e] = (int32_t)((int64_t)(w[e] >> g.log2D) * g.outer);
            __builtin_nontemporal_store(t, reinterpret_cast<v4i*>(reinterpret_cast<int32_t*>(g.C) + off));
          }
        }
      };
#pragma unroll
      for (int b = 0; b < NREG; ++b)
        put_block(b / C::AN, b % C::AN, [&](int v) { return iacc[b / C::AN][b % C::AN][v]; });
#pragma unroll
      for (int b = NREG; b < C::AM * C::AN; ++b)
        put_block(b / C::AN, b % C::AN, [&](int v) { return fold_lds[((b - NREG) * C::AV + v) * 64]; });
      return;
    }
  }
  if constexpr (C::OUTG) {
    // sum_d outer_d (group d's sum / D), exact in int64 (each group's sum is a multiple of D)
#pragma unroll
    for (int i = 0; i < C::AM; ++i)
#pragma unroll
      for (int j = 0; j < C::AN; ++j)
#pragma unroll
        for (int v = 0; v < C::AV; ++v) {
          int64_t t = 0;
#pragma unroll
          for (int d = 0; d < C::NG; ++d) t += (int64_t)(iaccg[d][i][j][v] >> g.log2D) * g.outer_g[d];
          const int row = row0 + i * BS + 8 * (v >> 2) + (v & 3), col = col0 + j * BS;
          if (part < 0)
            store_value(g, row, col, t);
          else
            add_value(g, row, col, t);
        }
    return;
  }
  if (g.c64 == 2) {  // residues as bytes (only with a modulus, whose tiles are never split)
    auto emit8 = [&](int i, int j, int v, int32_t val) {
      store_residue_u8(g, row0 + i * BS + (BS == 16 ? v : 8 * (v >> 2) + (v & 3)), col0 + j * BS, val);
    };
#pragma unroll
    for (int b = 0; b < NREG; ++b)
#pragma unroll
      for (int v = 0; v < C::AV; ++v) emit8(b / C::AN, b % C::AN, v, iacc[b / C::AN][b % C::AN][v]);
#pragma unroll
    for (int b = NREG; b < C::AM * C::AN; ++b)
#pragma unroll
      for (int v = 0; v < C::AV; ++v) emit8(b / C::AN, b % C::AN, v, fold_lds[((b - NREG) * C::AV + v) * 64]);
    return;
  }
#pragma unroll
  for (int b = 0; b < NREG; ++b)
#pragma unroll
    for (int v = 0; v < C::AV; ++v) emit(b / C::AN, b % C::AN, v, iacc[b / C::AN][b % C::AN][v]);
#pragma unroll
  for (int b = NREG; b < C::AM * C::AN; ++b)
#pragma unroll
    for (int v = 0; v < C::AV; ++v) emit(b / C::AN, b % C::AN, v, fold_lds[((b - NREG) * C::AV + v) * 64]);
}

template <class C>
__global__ __launch_bounds__(C::THREADS, 1) void gemm_kernel(GemmArgs g) {
  // Which tile, and which part of the reduction range: the workgroups past n_full
  // share the ragged last round's tiles, `split` to a tile.
  int tile = blockIdx.x, part = -1;
  int t_beg = g.t_begin, t_end = g.t_end;
  if (tile >= g.n_full) {
    const int rel = tile - g.n_full;
    tile = g.n_full + rel / g.split;
    part = rel % g.split;
    const int per = (g.t_end - g.t_begin + g.split - 1) / g.split;
    t_beg = g.t_begin + part * per;
    t_end = min(g.t_end, t_beg + per);
    if (t_beg >= t_end) return;  // the host splits only ranges of at least 2 stages per part
  }
  gemm_tile<C, true>(g, [&](int p) { return g.fold_ell[p]; }, tile, part, t_beg, t_end);
}

// Several GEMMs of one shape in one launch (the residue route's moduli): job j's tiles are
// workgroups j * tiles .. j * tiles + tiles - 1, the jobs ordered by the host (most products
// first, so that the short jobs fill the last rounds).  Every job covers the launch's whole
// reduction range; nothing is split.
struct GroupJob {
  const uint8_t* pa;
  const uint8_t* pb;
  void* C;
  uint64_t pidx_a, pidx_b;
  int32_t fold_ell[kGroupProducts];
  uint32_t fold_mask;
  int32_t r, modulus, ts;
};
struct GroupArgs {
  GemmArgs g;  // the fields all jobs share (shape, strides, reduction range, tiling)
  GroupJob job[kMaxModuli];
  int32_t tiles;
};

// A wave-uniform value in scalar registers.
__device__ __forceinline__ uint32_t uniform(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ int32_t uniform(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint64_t uniform(uint64_t v) {
  return ((uint64_t)uniform((uint32_t)(v >> 32)) << 32) | uniform((uint32_t)v);
}
template <class T>
__device__ __forceinline__ T* uniform(T* p) {
  return reinterpret_cast<T*>(uniform(reinterpret_cast<uint64_t>(p)));
}

template <class C>
__global__ __launch_bounds__(C::THREADS, 1) void gemm_group_kernel(GroupArgs ga) {
  // wave-uniform job index, so that the job's fields load into scalar registers
  const int j = __builtin_amdgcn_readfirstlane((int)(blockIdx.x / ga.tiles));
  const int tile = blockIdx.x - j * ga.tiles;
  const GroupJob& jb = ga.job[j];
  GemmArgs g = ga.g;
  g.pa = uniform(jb.pa);
  g.pb = uniform(jb.pb);
  g.C = uniform(jb.C);
  g.pidx_a = uniform(jb.pidx_a);
  g.pidx_b = uniform(jb.pidx_b);
  g.fold_mask = uniform(jb.fold_mask);
  g.r = uniform(jb.r);
  g.modulus = uniform(jb.modulus);
  g.ts = uniform(jb.ts);
  static_assert(kGroupProducts == 4, "the fold coefficients below");
  const int32_t f0 = uniform(jb.fold_ell[0]), f1 = uniform(jb.fold_ell[1]), f2 = uniform(jb.fold_ell[2]),
                f3 = uniform(jb.fold_ell[3]);
  gemm_tile<C, false>(g, [=](int p) { return p == 0 ? f0 : p == 1 ? f1 : p == 2 ? f2 : f3; }, tile, -1, g.t_begin,
               g.t_end);
}

__global__ void fill_zero_kernel(uint8_t* C, int64_t rows, int64_t row_bytes, int64_t ld_bytes) {
  const int64_t total = rows * row_bytes;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / row_bytes, c = i - r * row_bytes;
    C[r * ld_bytes + c] = 0;
  }
}

// Compute units of the current device (AWE_GEMM_CUS overrides the count used
// for planning the rounds of workgroups; it changes no result).
int compute_units() {
  const char* e = getenv("AWE_GEMM_CUS");
  if (e && atoi(e) > 0) return atoi(e);
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
      cus = v;
  }
  return cus;
}

// Rounds of workgroups for `tiles` tiles on `cus` CUs, with the ragged last
// round split as launch_tile does.
double rounds(int64_t tiles, int cus) {
  const int64_t full = tiles / cus, rem = tiles % cus;
  if (rem == 0) return (double)full;
  const int64_t S = std::min<int64_t>(cus / rem, 4);
  return (double)full + (full > 0 && S >= 2 ? 1.0 / S : 1.0);
}

// Whether n names one of the E2M1 tile configurations (AWE_GEMM_CFG): 1: 256x128 with 8
// waves, 2: 256x192 with 8 waves, 4: as 1 with 4 k-steps per stage, 5: as 4 with fragments
// read three k-steps ahead, 6: 256x192 with 4 k-steps per stage in 2 stages, 7: 256x192 with 2
// k-steps per stage in 5 stages, 8: as 6 with fragments read in place, 9: as 4 on the
// 16x16x128 MFMA, 10: as 9 with fragments read in place, 12: 256x256 with the int32 fold
// accumulators of 3 blocks per wave in LDS and a 2-stage ring, 13: as 12 with 2 blocks per wave
// in LDS and a 3-stage ring, 15: as 13 with the copies that refill a freed buffer spread over
// the next stage's MFMAs, 16: as 15 with the second k-step's fragments read during the first,
// 17: as 16 with the barrier inside the second k-step and the next stage's first fragments read
// during the rest of it.
bool e2m1_cfg(int n) { return n == 1 || n == 2 || (n >= 4 && n <= 17 && n != 11 && n != 14); }

// Tile configuration for a problem: AWE_GEMM_CFG if it names one, else the configuration whose
// rounds of workgroups finish first: 5, 6 (a round about 1.48 times as long as a round of 5;
// only when clearly sooner) or 17.  A round takes about 2.05 k + 1090 time units (10 ns) for 5
// and 3.76 k + 1800 for 17, k = r K / 6 reduction indices at r products: a fit of the kernel
// times measured on one MI355X for 8192^2 outputs at K = 2048 .. 8192 (r = 6); it also orders
// 4096^2 outputs at K = 4096 .. 16384 with 1 to 6 products, 6144^3 and 2048^2 x 8192 as
// measured.  The larger tile moves fewer bytes per MAC but fills the chip only with enough
// tiles: at 2048^2 x 8192 its 64 tiles leave most CUs idle and 5 wins.
int choose_cfg(int64_t M, int64_t N, int r, int64_t K) {
  const char* e = getenv("AWE_GEMM_CFG");
  const int forced = e ? atoi(e) : -1;
  if (e2m1_cfg(forced)) return forced;
  const int cus = compute_units();
  const int64_t tm = (M + 255) / 256;
  const double k = (double)r * (double)K / 6.0;
  const double r128 = 2.05 * k + 1090.0, r256 = 3.76 * k + 1800.0;
  const double t128 = rounds(tm * ((N + 127) / 128), cus) * r128;
  const double t192 = rounds(tm * ((N + 191) / 192), cus) * 1.48 * r128;
  const double t256 = rounds(tm * ((N + 255) / 256), cus) * r256;
  if (t256 < t128 && t256 < t192) return 17;
  return t192 < 0.97 * t128 ? 6 : 5;
}

// Tile configuration of a grouped launch of n jobs of one shape: AWE_GEMM_CFG if set, else 5
// or 16 (256 x 128 or 256 x 256, the latter on config 16's schedule), whichever a per-round model
// fitted to configs 5 and 13 gives less time summed over the jobs' tiles (many jobs fill the
// rounds, so the rounds are not quantised); config 16 runs the residue route's grouped GEMM at
// 4096 x 4096 x 16384 about 4 % faster than 13.
int choose_group_cfg(const GemmLaunch* L, int n) {
  const char* e = getenv("AWE_GEMM_CFG");
  const int forced = e ? atoi(e) : -1;
  if (forced >= 0) return forced;
  const double tm = (double)((L[0].M + 255) / 256);
  const double t128 = tm * (double)((L[0].N + 127) / 128), t256 = tm * (double)((L[0].N + 255) / 256);
  double s128 = 0.0, s256 = 0.0;
  for (int j = 0; j < n; ++j) {
    const double k = (double)L[j].r * (double)(L[j].k_end - L[j].k_begin) / 6.0;
    s128 += t128 * (2.2 * k + 1700.0);
    s256 += t256 * (3.9 * k + 6000.0);
  }
  return s256 < s128 ? 16 : 5;
}

// Tile configuration for E2M3 operands: AWE_GEMM_CFG_E2M3 (0: 256x128 with 8 waves in
// 3 stages, 1: as 0 in 4 stages, 3: as 0 with 4 k-steps per stage in 2 stages, 5: 256x192 with
// 8 waves reading fragments in place and the int32 fold accumulators of 1 of each wave's 6
// blocks in LDS, 6: as 5 with 2 blocks in LDS and 2 stages) overrides the default 5, the
// fastest measured at 8192^3 (in one process: 3: 1.16-1.18 ms, 5: 1.07-1.10 ms, 6: 1.24-1.26 ms).
int choose_cfg_e2m3() {
  const char* e = getenv("AWE_GEMM_CFG_E2M3");
  const int forced = e ? atoi(e) : -1;
  return forced == 0 || forced == 1 || forced == 3 || forced == 6 ? forced : 5;
}

// The kernel arguments of one launch.
void fill_args(const GemmLaunch& L, GemmArgs& g) {
  g.pa = L.planes_a;
  g.pb = L.planes_b;
  g.stride_a = L.stride_a;
  g.stride_b = L.stride_b;
  g.rba = (int32_t)((L.M + kBrickRows - 1) / kBrickRows);
  g.rbb = (int32_t)((L.N + kBrickRows - 1) / kBrickRows);
  const int64_t kp = (L.K + kKPad - 1) / kKPad * kKPad;
  g.KS = (int32_t)(kp / kBrickK);
  g.r = L.r;
  g.pidx_a = g.pidx_b = 0;
  for (int k = 0; k < L.r; ++k) {
    g.pidx_a |= (uint64_t)(L.pa[k] & 15) << (4 * k);
    g.pidx_b |= (uint64_t)(L.pb[k] & 15) << (4 * k);
  }
  // (all pairs: one stream product, one coefficient per accumulator group)
  for (int k = 0; k < kMaxProducts; ++k) g.fold_ell[k] = L.fold_ell[k];
  g.fold_mask = L.fold_mask;
  g.C = L.C;
  g.ldc = L.ldc;
  g.M = (int32_t)L.M;
  g.N = (int32_t)L.N;
  g.c64 = L.c_u8 && L.modulus ? 2 : (L.c_type == AWE_I64 ? 1 : 0);
  g.accumulate = L.accumulate;
  g.log2D = L.log2D;
  g.modulus = L.modulus;
  g.outer = L.outer;
}

// Raises a kernel's dynamic LDS limit to `bytes` once per device (the GEMM's ring exceeds
// the default).
awe_status set_lds_limit(const void* fn, int bytes, std::mutex& mu, std::set<int>& done) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  std::lock_guard<std::mutex> lk(mu);
  if (e == hipSuccess && !done.count(dev)) {
    e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e == hipSuccess) done.insert(dev);
  }
  if (e != hipSuccess) {
    set_error(std::string("gemm LDS attribute: ") + hipGetErrorString(e));
    return AWE_ERR_HIP;
  }
  return AWE_OK;
}

template <class C>
awe_status launch_tile(GemmArgs& g, const GemmLaunch& L, hipStream_t stream) {
  const int64_t tiles_m = (L.M + C::BM - 1) / C::BM, tiles_n = (L.N + C::BN - 1) / C::BN;
  g.t_begin = (int32_t)(L.k_begin / C::KT);
  g.t_end = (int32_t)(L.k_end / C::KT);
  g.ts = (int32_t)(L.k_seg / C::KT);
  g.tiles_m = (int32_t)tiles_m;
  g.tiles_n = (int32_t)tiles_n;
  const int64_t tiles = tiles_m * tiles_n;
  if (tiles > 0x3fffffffLL) return AWE_ERR_UNSUPPORTED;
  // A ragged last round of workgroups (rem tiles on cus CUs) is split along the
  // reduction: each of its tiles is computed by S = min(cus / rem, 4) workgroups
  // over consecutive parts of the range, so that round takes about 1/S of a
  // tile's time.  Residues need the whole sum before their reduction mod m and
  // are never split.
  const int cus = compute_units();
  const int stages = g.t_end - g.t_begin;
  g.n_full = (int32_t)tiles;
  g.split = 1;
  if (!L.modulus && tiles > cus && tiles % cus != 0) {
    const int64_t rem = tiles % cus;
    const int S = (int)std::min<int64_t>(cus / rem, 4);
    if (S >= 2 && stages >= 2 * S) {
      g.n_full = (int32_t)(tiles - rem);
      g.split = S;
    }
  }
  const int64_t blocks = g.n_full + (tiles - g.n_full) * g.split;
  if (g.split > 1 && !L.accumulate) {
    hipLaunchKernelGGL(zero_tiles_kernel, dim3((unsigned)(tiles - g.n_full), 32), dim3(256), 0, stream, g,
                       C::BM, C::BN, g.c64 ? 8 : 4);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
      set_error(std::string("zero launch: ") + hipGetErrorString(err));
      return AWE_ERR_HIP;
    }
  }
  {
    static std::mutex mu;
    static std::set<int> done;
    const awe_status st = set_lds_limit(reinterpret_cast<const void*>(&gemm_kernel<C>), C::LDS_BYTES, mu, done);
    if (st != AWE_OK) return st;
  }
  hipLaunchKernelGGL(gemm_kernel<C>, dim3((unsigned)blocks), dim3(C::THREADS), C::LDS_BYTES, stream, g);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) {
    set_error(std::string("gemm launch: ") + hipGetErrorString(err));
    return AWE_ERR_HIP;
  }
  return AWE_OK;
}

// One launch for n jobs (launch_gemm_group): the shared arguments from the first, each job's
// planes, C, products and coefficients from its own launch.
template <class C>
awe_status launch_group_tile(const GemmLaunch* L, const int* order, int n, hipStream_t stream) {
  GroupArgs ga{};
  GemmArgs& g = ga.g;
  fill_args(L[order[0]], g);
  const int64_t tiles_m = (L[0].M + C::BM - 1) / C::BM, tiles_n = (L[0].N + C::BN - 1) / C::BN;
  const int64_t tiles = tiles_m * tiles_n;
  if (tiles * n > 0x7fffffffLL) {
    set_error("too many workgroups for one grouped launch");
    return AWE_ERR_UNSUPPORTED;
  }
  g.t_begin = (int32_t)(L[0].k_begin / C::KT);
  g.t_end = (int32_t)(L[0].k_end / C::KT);
  g.tiles_m = (int32_t)tiles_m;
  g.tiles_n = (int32_t)tiles_n;
  g.n_full = (int32_t)tiles;
  g.split = 1;
  ga.tiles = (int32_t)tiles;
  for (int j = 0; j < n; ++j) {
    const GemmLaunch& Lj = L[order[j]];
    GroupJob& jb = ga.job[j];
    jb.pa = Lj.planes_a;
    jb.pb = Lj.planes_b;
    jb.C = Lj.C;
    jb.pidx_a = jb.pidx_b = 0;
    for (int k = 0; k < Lj.r; ++k) {
      jb.pidx_a |= (uint64_t)(Lj.pa[k] & 15) << (4 * k);
      jb.pidx_b |= (uint64_t)(Lj.pb[k] & 15) << (4 * k);
      jb.fold_ell[k] = Lj.fold_ell[k];
    }
    jb.fold_mask = Lj.fold_mask;
    jb.r = Lj.r;
    jb.modulus = Lj.modulus;
    jb.ts = (int32_t)(Lj.k_seg / C::KT);
  }
  {
    static std::mutex mu;
    static std::set<int> done;
    const awe_status st =
        set_lds_limit(reinterpret_cast<const void*>(&gemm_group_kernel<C>), C::LDS_BYTES, mu, done);
    if (st != AWE_OK) return st;
  }
  hipLaunchKernelGGL(gemm_group_kernel<C>, dim3((unsigned)(tiles * n)), dim3(C::THREADS), C::LDS_BYTES, stream,
                     ga);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) {
    set_error(std::string("grouped gemm launch: ") + hipGetErrorString(err));
    return AWE_ERR_HIP;
  }
  return AWE_OK;
}

}  // namespace

// Uploads a wide encoding's code table into g_wide_lut on the current device,
// once per device and side (the table never changes afterwards: one wide
// encoding per side is supported).
awe_status ensure_wide_table(const EncodeLaunch& e) {
  static std::mutex mu;
  static std::map<std::pair<int, int>, const void*> loaded;
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) {
    set_error(std::string("wide table: ") + hipGetErrorString(err));
    return AWE_ERR_HIP;
  }
  std::lock_guard<std::mutex> lk(mu);
  auto it = loaded.find({dev, e.side});
  if (it != loaded.end()) {
    if (it->second == e.table_key) return AWE_OK;
    set_error("only one wide encoding table per side is supported");
    return AWE_ERR_UNSUPPORTED;
  }
  if (e.nvalues > kWideValues) {
    set_error("wide encoding table too large");
    return AWE_ERR_UNSUPPORTED;
  }
  err = hipMemcpyToSymbol(HIP_SYMBOL(g_wide_lut), e.lut, sizeof(uint32_t) * e.nvalues,
                          sizeof(uint32_t) * kWideValues * e.side, hipMemcpyHostToDevice);
  if (err != hipSuccess) {
    set_error(std::string("wide table upload: ") + hipGetErrorString(err));
    return AWE_ERR_HIP;
  }
  loaded[{dev, e.side}] = e.table_key;
  return AWE_OK;
}

awe_status noalloc_planes(void** out) {
  static std::mutex mu;
  static std::map<int, void*> ptrs;
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) {
    set_error(std::string("planes array: ") + hipGetErrorString(err));
    return AWE_ERR_HIP;
  }
  std::lock_guard<std::mutex> lk(mu);
  auto it = ptrs.find(dev);
  if (it == ptrs.end()) {
    void* p = nullptr;
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess || p == nullptr) {
      set_error(std::string("planes array address: ") + hipGetErrorString(err));
      return AWE_ERR_HIP;
    }
    it = ptrs.emplace(dev, p).first;
  }
  *out = it->second;
  return AWE_OK;
}

awe_status launch_encode(const EncodeLaunch& e, hipStream_t stream) {
  const int64_t rb = (e.rows + kBrickRows - 1) / kBrickRows;
  const int64_t kp = (e.K + kKPad - 1) / kKPad * kKPad;
  const int64_t KS = kp / kBrickK;
  const int64_t nbricks = rb * KS;
  if (nbricks == 0) return AWE_OK;
  if (e.wide) {
    awe_status st = ensure_wide_table(e);
    if (st != AWE_OK) return st;
    const int64_t blocks = std::min<int64_t>((nbricks + 15) / 16, 4096);
    const int16_t* x = reinterpret_cast<const int16_t*>(e.x);
    if (e.transposed)
      hipLaunchKernelGGL(encode16_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, x, e.rows,
                         e.K, e.ld, KS, rb, nbricks, e.nplanes, e.planes, e.plane_stride, e.flag, e.side,
                         e.xmin, e.nvalues);
    else
      hipLaunchKernelGGL(encode16_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, x, e.rows,
                         e.K, e.ld, KS, rb, nbricks, e.nplanes, e.planes, e.plane_stride, e.flag, e.side,
                         e.xmin, e.nvalues);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
      set_error(std::string("encode launch: ") + hipGetErrorString(err));
      return AWE_ERR_HIP;
    }
    return AWE_OK;
  }
  LutArg lut;
  for (int i = 0; i < 256; ++i) lut.v[i] = e.lut[i];
  // one brick per wave; past 2^31 - 1 workgroups the waves walk several bricks each (the B
  // side in groups of four column blocks, the last group padded)
  const int64_t nb = e.transposed ? (rb + 3) / 4 * 4 * KS : nbricks;
  const int64_t blocks = std::min<int64_t>((nb + 3) / 4, 0x7fffffffLL);
  if (e.transposed)
    hipLaunchKernelGGL(encode_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream,
                       reinterpret_cast<const uint8_t*>(e.x), e.rows, e.K, e.ld, KS, rb, nb,
                       e.nplanes, e.nplanes8, e.fp6, e.planes, e.plane_stride, e.flag, lut);
  else
    hipLaunchKernelGGL(encode_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream,
                       reinterpret_cast<const uint8_t*>(e.x), e.rows, e.K, e.ld, KS, rb, nbricks,
                       e.nplanes, e.nplanes8, e.fp6, e.planes, e.plane_stride, e.flag, lut);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) {
    set_error(std::string("encode launch: ") + hipGetErrorString(err));
    return AWE_ERR_HIP;
  }
  return AWE_OK;
}

awe_status launch_gemm(const GemmLaunch& L, hipStream_t stream) {
  if (L.M == 0 || L.N == 0) return AWE_OK;
  const int64_t esize = L.c_u8 && L.modulus ? 1 : (L.c_type == AWE_I64 ? 8 : 4);
  if (L.k_end <= L.k_begin) {
    if (L.accumulate) return AWE_OK;
    hipLaunchKernelGGL(fill_zero_kernel, dim3(1024), dim3(256), 0, stream,
                       reinterpret_cast<uint8_t*>(L.C), L.M, L.N * esize, L.ldc * esize);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
      set_error(std::string("fill launch: ") + hipGetErrorString(err));
      return AWE_ERR_HIP;
    }
    return AWE_OK;
  }
  GemmArgs g{};
  fill_args(L, g);
  if (L.fmt == kFmtE4M3) return launch_tile<Cfg8w64x64e4m3>(g, L, stream);
  if (L.allpairs_a == 3 && L.allpairs_b == 3 && !L.outer_groups) return launch_tile<Cfg8w32x64ap33>(g, L, stream);
  if (L.allpairs_a == 2 && L.allpairs_b == 2 && L.outer_groups) {
    for (int d = 0; d < 3; ++d) g.outer_g[d] = L.outer_g[d];
    return launch_tile<Cfg8w32x64ap22o>(g, L, stream);
  }
  if (L.shared) {
    for (int k = 0; k < 2; ++k) {
      g.sa[k] = L.scale_a[k];
      g.sb[k] = L.scale_b[k];
    }
    // AWE_GEMM_CFG_SHARED: 1 reads each k-step's fragments in place
    const char* e = getenv("AWE_GEMM_CFG_SHARED");
    if (e && atoi(e) == 1) return launch_tile<Cfg8w64x64shp0>(g, L, stream);
    return launch_tile<Cfg8w64x64sh>(g, L, stream);
  }
  if (L.fmt == kFmtE2M3) {
    switch (choose_cfg_e2m3()) {
      case 1: return launch_tile<Cfg8w64x64s4e2m3>(g, L, stream);
      case 3: return launch_tile<Cfg8w64x64k4e2m3>(g, L, stream);
      case 5: return launch_tile<Cfg8w64x96p0lfe2m3>(g, L, stream);
      case 6: return launch_tile<Cfg8w64x96p0lf2e2m3>(g, L, stream);
      default: return launch_tile<Cfg8w64x64e2m3>(g, L, stream);
    }
  }
  switch (choose_cfg(L.M, L.N, L.r, L.k_end - L.k_begin)) {
    case 2: return launch_tile<Cfg8w64x96>(g, L, stream);
    case 4: return launch_tile<Cfg8w64x64k4>(g, L, stream);
    case 5: return launch_tile<Cfg8w64x64k4p3>(g, L, stream);
    case 6: return launch_tile<Cfg8w64x96k4>(g, L, stream);
    case 7: return launch_tile<Cfg8w64x96s5>(g, L, stream);
    case 8: return launch_tile<Cfg8w64x96k4p0>(g, L, stream);
    case 9: return launch_tile<Cfg8w64x64k4m16>(g, L, stream);
    case 10: return launch_tile<Cfg8w64x64k4p0m16>(g, L, stream);
    case 12: return launch_tile<Cfg8w64x128lf>(g, L, stream);
    case 13: return launch_tile<Cfg8w64x128lf3>(g, L, stream);
    case 15: return launch_tile<Cfg8w64x128cs>(g, L, stream);
    case 16: return launch_tile<Cfg8w64x128cr>(g, L, stream);
    case 17: return launch_tile<Cfg8w64x128cm>(g, L, stream);
    default: return launch_tile<Cfg8w64x64>(g, L, stream);
  }
}

// The grouped kernel is built for the 256 x 128 tiles on 8 waves (configurations 1, 4
// and 5) and the 256 x 256 tiles of configurations 13 and 16 (with config 17's schedule it
// spills 23 registers); the 256 x 192 ones leave no registers for the jobs' fields.
bool group_cfg(int cfg) { return cfg == 1 || cfg == 4 || cfg == 5 || cfg == 13 || cfg == 16; }

bool gemm_group_ok(const GemmLaunch* L, int n) {
  if (n < 1 || n > kMaxModuli) return false;
  if (!group_cfg(choose_group_cfg(L, n))) return false;
  for (int j = 0; j < n; ++j) {
    const GemmLaunch& a = L[j];
    if (a.fmt != kFmtE2M1 || a.shared || a.allpairs_a || a.accumulate || a.r < 1 || a.r > kGroupProducts)
      return false;
    if (a.M != L[0].M || a.N != L[0].N || a.K != L[0].K || a.k_begin != L[0].k_begin ||
        a.k_end != L[0].k_end || a.k_end <= a.k_begin)
      return false;
    if (a.c_type != L[0].c_type || a.c_u8 != L[0].c_u8 || (a.c_u8 && !a.modulus) || a.log2D != L[0].log2D ||
        a.outer != L[0].outer || a.ldc != L[0].ldc || a.stride_a != L[0].stride_a || a.stride_b != L[0].stride_b)
      return false;
  }
  return true;
}

awe_status launch_gemm_group(const GemmLaunch* L, int n, hipStream_t stream) {
  if (!gemm_group_ok(L, n)) {
    set_error("these GEMMs cannot share one launch");
    return AWE_ERR_UNSUPPORTED;
  }
  if (L[0].M == 0 || L[0].N == 0) return AWE_OK;
  // the jobs with the most products first: the short ones fill the last rounds
  int order[kMaxModuli];
  for (int j = 0; j < n; ++j) order[j] = j;
  std::stable_sort(order, order + n, [&](int a, int b) { return L[a].r > L[b].r; });
  switch (choose_group_cfg(L, n)) {
    case 4: return launch_group_tile<Cfg8w64x64k4>(L, order, n, stream);
    case 5: return launch_group_tile<Cfg8w64x64k4p3>(L, order, n, stream);
    case 13: return launch_group_tile<Cfg8w64x128lf3>(L, order, n, stream);
    case 16: return launch_group_tile<Cfg8w64x128cr>(L, order, n, stream);
    default: return launch_group_tile<Cfg8w64x64>(L, order, n, stream);
  }
}

}  // namespace awe
