// Tile configurations of the multi-plane FP4 GEMM and the addresses of its global -> LDS
// copies, LDS ring, operand fragments and LDS fold blocks.  The kernels compute every such
// address with the helpers below, and a host program checks them against the bounds of the
// planes, the stage buffers and the LDS of a CU for every configuration (no GPU needed).
#pragma once

#include <hip/hip_runtime.h>

#include "awe_internal.h"

namespace awe {

template <int WM_, int WN_, int BMW_, int BNW_, int KST_, int NSTAGE_, int PD_ = 1, int FMT_ = 0,
          int NPL_ = 1, int MF_ = 32, int NLB_ = 0, int SCHED_ = 0, int NPA_ = 0, int NPB_ = 0, int PSTEP_ = 1,
          int OUTG_ = 0>
struct Cfg {
  static constexpr int WM = WM_, WN = WN_, BMW = BMW_, BNW = BNW_;
  static constexpr int KST = KST_;        // bricks (64 reduction indices each) per row block and stage
  static constexpr int KT = 64 * KST;     // reduction indices per stage
  static constexpr int NSTAGE = NSTAGE_;  // LDS ring depth
  // MFMA shape: 32 (32x32x64: one k-step is one brick) or 16 (16x16x128: one k-step is two
  // bricks; a wave's 32x32 block is four 16x16 MFMA blocks).  Both read the same operand
  // bytes from LDS per MAC for a given wave tile; on changing operands the 16x16x128 form
  // sustains a higher rate at the board's power limit, but the GEMM, bound by its data path,
  // runs no faster on it.
  static constexpr int MF = MF_;
  static_assert(MF == 32 || (MF == 16 && FMT_ == 0 && NPL_ == 1 && KST % 2 == 0), "MFMA shape");
  static constexpr int KSTEPS = MF == 16 ? KST / 2 : KST;  // MFMA k-steps per stage
  // Fragments are read PD k-steps before their MFMAs, into NSETS register sets
  // (k-step ks of every stage uses set ks % NSETS, so NSETS divides KSTEPS).  PD = 0
  // reads each k-step's fragments right before its MFMAs into a single set (the
  // other wave of the SIMD covers the wait), which saves one set of registers.
  static constexpr int PD = PD_;
  static constexpr int NSETS = PD == 0 ? 1 : (PD == 1 ? 2 : KSTEPS);
  static_assert(PD == 0 || (PD < NSETS && KSTEPS % NSETS == 0), "fragment prefetch distance");
  // Accumulator blocks per wave (M x N) and FP32 values per lane and block.
  static constexpr int AM = MF == 16 ? 2 * BMW : BMW, AN = MF == 16 ? 2 * BNW : BNW;
  static constexpr int AV = MF == 16 ? 4 : 16;
  // Operand element format and its storage unit: 0 E2M1, one k-step in 1 KiB (16 bytes
  // per lane); 1 E4M3, one k-step in 2 KiB (32 bytes per lane); 2 E2M3, two k-steps in
  // 3 KiB (24 bytes per lane and k-step).  Units move as 1 KiB copies.
  static constexpr int FMT = FMT_;
  static constexpr int UK = FMT == 2 ? 2 : 1;  // k-steps per unit
  static constexpr int UNIT_BYTES = FMT == 0 ? kBrickBytes : (FMT == 1 ? 2 * kBrickBytes : 3 * kBrickBytes);
  static constexpr int COPIES = UNIT_BYTES / kBrickBytes;
  static constexpr int KU = KST / UK;          // units per row block and stage
  static_assert(KST % UK == 0, "a stage holds whole units");
  static constexpr int NW = WM * WN;
  static constexpr int THREADS = 64 * NW;
  static constexpr int BM = WM * BMW * 32, BN = WN * BNW * 32;
  // Planes per side in a stage: 1 (one product's planes, product-major stream), or 2 (both
  // planes of each side; every pair is a product, its weight in the E8M0 scales, all four
  // into one accumulator).
  static constexpr int NPL = NPL_;
  static_assert(NPL == 1 || (NPL == 2 && FMT == 2), "two planes per side: E2M3 with weights in the scales");
  // All pairs (NPA > 0): a stage brings NPA planes of A and NPB planes of B, and every pair
  // (i, j) is a product whose coefficient depends on i + j only, so its MFMAs add into
  // accumulator group i + j (NG groups), folded once per segment with the group's coefficient
  // (products with equal coefficients share an accumulator, Alg. 1): each plane is copied once
  // per stage for all the products that use it.
  static constexpr int NPA = NPA_, NPB = NPB_;
  static constexpr bool AP = NPA_ > 0;
  static constexpr int NG = AP ? NPA + NPB - 1 : 1;
  // A stage's plane pl is stored plane (first plane of the stream product) + pl * PSTEP.
  static constexpr int PSTEP = PSTEP_;
  // Outer groups (OUTG = 1, all pairs only): each group i + j has its own int32 accumulator,
  // into which the stream product's coefficient folds it; the epilogue adds the groups with
  // their outer weights (GemmArgs::outer_g) in int64.  Otherwise all groups fold into one int32
  // accumulator with the group's coefficient.
  static constexpr int OUTG = OUTG_;
  static constexpr int NOUT = OUTG ? NG : 1;
  static_assert(!OUTG || AP, "outer groups belong to the all-pairs stream");
  static_assert(!AP || (NPB > 0 && FMT == 0 && NPL == 1 && MF == 32 && NLB_ == 0 && (SCHED_ == 0 || SCHED_ == 3)),
                "all pairs: E2M1, 32x32x64 MFMAs, int32 accumulators in registers, schedule 0 or 3");
  static constexpr int PA_UNITS = (BM / kBrickRows) * KU;  // per plane and stage: row blocks x units
  static constexpr int PB_UNITS = (BN / kBrickRows) * KU;
  static constexpr int SPA = AP ? NPA : NPL, SPB = AP ? NPB : NPL;  // planes per side in a stage
  static constexpr int A_UNITS = SPA * PA_UNITS;
  static constexpr int B_UNITS = SPB * PB_UNITS;
  static constexpr int STAGE_BYTES = (A_UNITS + B_UNITS) * UNIT_BYTES;
  // The int32 fold accumulators of the last NLB accumulator blocks of every wave live in LDS
  // after the ring (each wave its own 4 KiB per block, lane-major), so that a tile whose
  // registers hold only its FP32 accumulators and part of its int32 ones still fits.
  static constexpr int NLB = NLB_;
  static_assert(NLB >= 0 && NLB < AM * AN && (NLB == 0 || (MF == 32 && NPL_ == 1)), "LDS fold blocks");
  static constexpr int FOLD_LDS_OFFSET = NSTAGE * STAGE_BYTES;
  static constexpr int LDS_BYTES = NSTAGE * STAGE_BYTES + NW * NLB * AV * 64 * 4;
  static_assert(LDS_BYTES <= 160 * 1024, "LDS of one CU");
  // copies per wave and stage: A units evenly, B units round-robin (the first
  // B_UNITS % NW waves take one more)
  static constexpr int A_PW = A_UNITS / NW;
  static constexpr int B_LO = B_UNITS / NW, B_XTRA = B_UNITS % NW;
  static_assert(A_UNITS % NW == 0, "A units must split evenly over the waves");
  static_assert(kKPad % KT == 0, "a stage must divide the reduction padding");
  // Schedule of the stage loop.  0: after the barrier that frees a buffer every wave issues
  // its copies of the stage that refills it, then runs the stage's k-steps.  1: the copies that
  // refill the freed buffer are spread over the next stage's MFMAs instead, one after every few,
  // so that the eight waves' copies do not queue at the address unit at once and a wave waiting
  // for one has matrix work in flight.  2: as 1, and a later k-step's fragments are read during
  // the k-step before it, each as soon as the last MFMA that uses the register's old value has
  // issued.  3: as 2, with the barrier inside the second k-step after its first row of MFMAs,
  // so that the next stage's first fragments are read during the rest of that k-step, and each
  // refill issued during the first k-step of the stage after its buffer was freed.
  static constexpr int SCHED = SCHED_;
  static_assert(SCHED == 0 ||
                    (NPL == 1 && MF == 32 && B_XTRA == 0 && COPIES == 1 && PD == 0 && NSTAGE >= 3 &&
                     (A_PW + B_LO) % KSTEPS == 0 && (SPA * BMW * SPB * BNW) % ((A_PW + B_LO) / KSTEPS) == 0),
                "copies between the MFMAs: E2M1, one plane per side, 32x32x64 MFMAs, fragments in place, "
                "the copies spread evenly over the k-steps");
};

// ---------------------------------------------------------------------------
// Addresses.  A stage holds A units 0 .. A_UNITS - 1, then B units; unit id of side X
// covers plane pl = id / PX_UNITS of the stage, row block rb = (id % PX_UNITS) / KU of the
// tile (rows or columns of B) and unit ku = id % KU of the stage's reduction range.
// ---------------------------------------------------------------------------
struct UnitPos {
  int pl, rb, ku;
};

template <class C>
__host__ __device__ constexpr UnitPos unit_pos(bool sideA, int id) {
  const int per = sideA ? C::PA_UNITS : C::PB_UNITS;
  return UnitPos{id / per, (id % per) / C::KU, (id % per) % C::KU};
}

// Unit of copy i of a wave: A units wave * A_PW .. wave * A_PW + A_PW - 1; B units wave,
// wave + NW, ... (the first B_XTRA waves take one more); -1 past the wave's share.
template <class C>
__host__ __device__ constexpr int copy_unit(bool sideA, int wave, int i) {
  if (sideA) return i < C::A_PW ? wave * C::A_PW + i : -1;
  return (i < C::B_LO || (i == C::B_LO && wave < C::B_XTRA)) ? wave + i * C::NW : -1;
}

// LDS byte offset of 1 KiB copy h of a unit, from the start of its stage buffer.
template <class C>
__host__ __device__ constexpr uint32_t unit_lds(bool sideA, int id, int h) {
  return (uint32_t)((sideA ? id : C::A_UNITS + id) * C::UNIT_BYTES + h * kBrickBytes);
}

// Global byte offset of stage t's units from the first plane of the stream product (a side with
// rbs row blocks), and of copy h of a unit from there (plane u.pl of the stage, the planes
// `stride` bytes apart; row block rb of the planes: the tile's, clamped to rbs - 1).
template <class C>
__host__ __device__ constexpr int64_t stage_global(int64_t t, int rbs) {
  return t * C::KU * rbs * C::UNIT_BYTES;
}
template <class C>
__host__ __device__ constexpr int64_t unit_global(UnitPos u, int rb, int rbs, int64_t stride, int h) {
  return (int64_t)u.pl * C::PSTEP * stride + (int64_t)(u.ku * rbs + rb) * C::UNIT_BYTES + h * kBrickBytes;
}

// LDS offset, from the start of a stage buffer, of the unit holding k-step ks of fragment
// (plane pl, block row/column q of the tile) of side A or B.
template <class C>
__host__ __device__ constexpr uint32_t frag_unit(bool sideA, int pl, int q, int ks) {
  return (uint32_t)(((sideA ? 0 : C::A_UNITS) + pl * (sideA ? C::PA_UNITS : C::PB_UNITS) + q * C::KU + ks / C::UK) *
                    C::UNIT_BYTES);
}

// The bytes lane reads of k-step i of a unit of format FMT: `n` spans (offset from the unit,
// length): E2M1 16 bytes at 16 lane; E4M3 32 bytes at 32 lane; E2M3 16 bytes at
// i 1024 + 16 lane and 8 bytes at 2048 + i 512 + 8 lane.
struct Spans {
  int n;
  uint32_t off[2], len[2];
};
template <int FMT>
__host__ __device__ constexpr Spans frag_spans(int i, int lane) {
  if (FMT == 0) return Spans{1, {(uint32_t)lane * 16u, 0u}, {16u, 0u}};
  if (FMT == 1) return Spans{1, {(uint32_t)lane * 32u, 0u}, {32u, 0u}};
  return Spans{2, {(uint32_t)(i * 1024 + lane * 16), (uint32_t)(2048 + i * 512 + lane * 8)}, {16u, 8u}};
}

// 16x16x128 operand fragment: lane L holds row (column) L % 16 of its 16-row block at
// reduction indices 32 (L / 16) .. 32 (L / 16) + 31 of the k-step's 128, i.e. the 16
// bytes that lane (L / 16 % 2) * 32 + row of brick L / 32 holds in the stored layout.
__host__ __device__ constexpr uint32_t frag16_lane_offset(int lane) {
  return (uint32_t)(((lane >> 4) >> 1) * kBrickBytes + (((lane >> 4) & 1) * 32 + (lane & 15)) * 16);
}
// Offset, from the start of a stage buffer, of half h (16 rows) of block q of side A or B at
// 16x16x128 k-step ks (two bricks).
template <class C>
__host__ __device__ constexpr uint32_t frag16_unit(bool sideA, int q, int ks, int h) {
  return (uint32_t)(((sideA ? 0 : C::A_UNITS) + q * C::KU + 2 * ks) * C::UNIT_BYTES + h * 256);
}

// Byte offset in LDS of int32 v of lane `lane` of LDS fold block lb of a wave.
template <class C>
__host__ __device__ constexpr uint32_t fold_lds_offset(int wave, int lb, int v, int lane) {
  return (uint32_t)(C::FOLD_LDS_OFFSET + 4 * (((wave * C::NLB + lb) * C::AV + v) * 64 + lane));
}

// The tile configurations the launcher chooses from: waves (M x N), 32x32
// blocks per wave (M x N), k-steps per stage, LDS ring depth.
using Cfg8w64x64 = Cfg<4, 2, 2, 2, 2, 4>;    // 256 x 128, 8 waves (2 per SIMD)
using Cfg8w64x96 = Cfg<4, 2, 2, 3, 2, 4>;    // 256 x 192, 8 waves (2 per SIMD)
using Cfg8w64x64k4 = Cfg<4, 2, 2, 2, 4, 3>;  // 256 x 128, 8 waves, 4 k-steps per stage
using Cfg8w64x64k4p3 = Cfg<4, 2, 2, 2, 4, 3, 3>;  // as above, fragments read 3 k-steps ahead
using Cfg8w64x64e4m3 = Cfg<4, 2, 2, 2, 2, 3, 1, 1>;  // 256 x 128, 8 waves, E4M3 operands
using Cfg8w64x96k4 = Cfg<4, 2, 2, 3, 4, 2>;         // 256 x 192, 8 waves, 4 k-steps, 2 stages
using Cfg8w64x96s5 = Cfg<4, 2, 2, 3, 2, 5>;         // 256 x 192, 8 waves, 2 k-steps, 5 stages
using Cfg8w64x96k4p0 = Cfg<4, 2, 2, 3, 4, 2, 0>;    // as 6, fragments read in place
// 16x16x128 MFMAs (one k-step = two bricks)
using Cfg8w64x64k4m16 = Cfg<4, 2, 2, 2, 4, 3, 1, 0, 1, 16>;   // 256 x 128, 8 waves, 2 k-steps of 128 per stage
using Cfg8w64x64k4p0m16 = Cfg<4, 2, 2, 2, 4, 3, 0, 0, 1, 16>; // as above, fragments read in place
// 256 x 256 on 8 waves of 2 x 4 blocks, 2 k-steps per stage in 2 stages, fragments read in place;
// the int32 fold accumulators of 3 of each wave's 8 blocks in LDS (96 KiB + a 64 KiB ring)
using Cfg8w64x128lf = Cfg<4, 2, 2, 4, 2, 2, 0, 0, 1, 32, 3>;
// as above with the fold accumulators of 2 blocks per wave in LDS (64 KiB) and a 3-stage ring
using Cfg8w64x128lf3 = Cfg<4, 2, 2, 4, 2, 3, 0, 0, 1, 32, 2>;
// config 13 with the copies that refill a freed buffer spread over the next stage's MFMAs (15),
// and with the second k-step's fragments read during the first (16)
using Cfg8w64x128cs = Cfg<4, 2, 2, 4, 2, 3, 0, 0, 1, 32, 2, 1>;
using Cfg8w64x128cr = Cfg<4, 2, 2, 4, 2, 3, 0, 0, 1, 32, 2, 2>;
// as 16 with the barrier inside the second k-step, after its first row of MFMAs (17)
using Cfg8w64x128cm = Cfg<4, 2, 2, 4, 2, 3, 0, 0, 1, 32, 2, 3>;
// all pairs of 3 planes per side (9 products, 5 accumulator groups): 128 x 128 on 8 waves of
// 1 x 2 blocks, 2 k-steps per stage (48 KiB) in 3 stages, fragments read in place
using Cfg8w32x64ap33 = Cfg<4, 2, 1, 2, 2, 3, 0, 0, 1, 32, 0, 0, 3, 3>;
// all pairs of 2 planes per side, 3 apart (the two halves of a 12-bit significand), each group
// i + j with its own int32 accumulator and outer weight: 128 x 128 on 8 waves of 1 x 2 blocks,
// 2 k-steps per stage (32 KiB) in 3 stages, on schedule 3 (fragments read in place during the
// k-step before, the barrier inside the second k-step)
using Cfg8w32x64ap22o = Cfg<4, 2, 1, 2, 2, 3, 0, 0, 1, 32, 0, 3, 2, 2, 3, 1>;
// E2M3 operands (3 KiB units of two k-steps)
using Cfg8w64x64e2m3 = Cfg<4, 2, 2, 2, 2, 3, 1, 2>;   // 256 x 128, 8 waves, 2 k-steps, 3 stages
using Cfg8w64x64s4e2m3 = Cfg<4, 2, 2, 2, 2, 4, 1, 2>; // 256 x 128, 8 waves, 2 k-steps, 4 stages
using Cfg8w64x64k4e2m3 = Cfg<4, 2, 2, 2, 4, 2, 1, 2>; // 256 x 128, 8 waves, 4 k-steps, 2 stages
// 256 x 192, 8 waves, fragments read in place, the int32 fold accumulators of 1 of each wave's 6
// blocks in LDS
using Cfg8w64x96p0lfe2m3 = Cfg<4, 2, 2, 3, 2, 3, 0, 2, 1, 32, 1>;
// 2 of each wave's 6 blocks in LDS, 2 stages
using Cfg8w64x96p0lf2e2m3 = Cfg<4, 2, 2, 3, 2, 2, 0, 2, 1, 32, 2>;
// E2M3, two planes per side with the weights in the scales (4 products, one accumulator)
using Cfg8w64x64sh = Cfg<4, 2, 2, 2, 2, 2, 1, 2, 2>;    // 256 x 128, 8 waves, 2 k-steps, 2 stages
using Cfg8w64x64shp0 = Cfg<4, 2, 2, 2, 2, 2, 0, 2, 2>;  // as above, fragments read in place


}  // namespace awe
