// Packing of E2M1 codes into the stored plane layout (Alg. 1, plane formation), shared by the
// byte encoder and the residue encoder.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace awe {

// One lane's 32 elements of a brick: e[j] holds element j's 4-bit E2M1 code of plane p in bits
// 4p .. 4p + 3 (up to 8 planes).  The stored layout wants, for each plane, 16 bytes with the 32
// elements in order, two per byte (element 2i in the low nibble): d[p][w] receives dword w of
// plane p (elements 8w .. 8w + 7) for p < NP.
//
// A nibble transpose: byte q of x[i] (y[i]) holds the byte of plane 2q (2q + 1) for elements
// 2i and 2i + 1, and a 4 x 4 byte transpose of x[4w .. 4w + 3] (three v_perm_b32 per output
// dword, shared between pairs of outputs) gives dword w of planes 0, 2, 4, 6.  About 100 + 12 NP
// instructions for NP planes, where packing each plane nibble by nibble takes about 128 per
// plane.  Outputs past NP are never formed (the compiler drops their work).
template <int NP>
__device__ __forceinline__ void pack_e2m1_planes(const uint32_t (&e)[32], uint32_t (&d)[NP][4]) {
  static_assert(NP >= 1 && NP <= 8, "planes per code word");
  uint32_t x[16], y[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const uint32_t lo = e[2 * i], hi = e[2 * i + 1];
    x[i] = (lo & 0x0f0f0f0fu) | ((hi & 0x0f0f0f0fu) << 4);
    y[i] = ((lo >> 4) & 0x0f0f0f0fu) | (hi & 0xf0f0f0f0u);
  }
  // v_perm_b32(a, b, sel): result byte k = byte sel_k of {a : b}, b being bytes 0..3
  auto transpose4 = [](const uint32_t* v, uint32_t* out) {
    const uint32_t t0 = __builtin_amdgcn_perm(v[1], v[0], 0x05010400u);
    const uint32_t t1 = __builtin_amdgcn_perm(v[1], v[0], 0x07030602u);
    const uint32_t t2 = __builtin_amdgcn_perm(v[3], v[2], 0x05010400u);
    const uint32_t t3 = __builtin_amdgcn_perm(v[3], v[2], 0x07030602u);
    out[0] = __builtin_amdgcn_perm(t2, t0, 0x05040100u);
    out[1] = __builtin_amdgcn_perm(t2, t0, 0x07060302u);
    out[2] = __builtin_amdgcn_perm(t3, t1, 0x05040100u);
    out[3] = __builtin_amdgcn_perm(t3, t1, 0x07060302u);
  };
  uint32_t px[4][4], py[4][4];  // [dword w][plane pair q]
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    transpose4(x + 4 * w, px[w]);
    transpose4(y + 4 * w, py[w]);
  }
#pragma unroll
  for (int p = 0; p < NP; ++p)
#pragma unroll
    for (int w = 0; w < 4; ++w) d[p][w] = (p & 1) ? py[w][p >> 1] : px[w][p >> 1];
}

}  // namespace awe
