// Host check of the multi-plane GEMM's addressing for every tile configuration the library
// builds (gemm_layout.h, the same helpers the kernels call): no GPU is touched.  For each
// configuration it checks that
//  * the copies of one stage, over all waves, write every byte of the stage buffer exactly once
//    and nothing else, each unit's copies landing inside the unit;
//  * every copy's source lies inside its plane for ragged and full shapes (the tile's row block
//    clamped to the plane's last one), and a unit's copies come from the stage's reduction range;
//  * every fragment a lane reads at every k-step lies inside the unit that holds its plane, row
//    block and reduction indices (for the 16x16x128 form, the two units of its k-step);
//  * the LDS fold blocks lie after the ring, inside the CU's LDS, one int32 per (wave, block,
//    value, lane) and no two alike;
//  * the LDS in use fits the 160 KiB of a CU.
// Prints one line per configuration and exits nonzero at the first violation.
#include <cstdio>
#include <cstdlib>
#include <set>
#include <string>
#include <vector>

#include "gemm_layout.h"

using namespace awe;

static int fails = 0;
#define CHECK(cond, ...)                           \
  do {                                             \
    if (!(cond)) {                                 \
      std::printf("FAIL %s: ", name);              \
      std::printf(__VA_ARGS__);                    \
      std::printf("\n");                           \
      ++fails;                                     \
      return;                                      \
    }                                              \
  } while (0)

template <class C>
static void check(const char* name) {
  CHECK(C::LDS_BYTES <= 160 * 1024, "LDS %d bytes", C::LDS_BYTES);
  CHECK(C::NSTAGE * C::STAGE_BYTES <= C::FOLD_LDS_OFFSET, "ring past the fold blocks");
  // copies of one stage
  std::vector<int> written(C::STAGE_BYTES, 0);
  for (int side = 0; side < 2; ++side) {
    const bool A = side == 0;
    const int units = A ? C::A_UNITS : C::B_UNITS;
    std::vector<int> unit_seen(units, 0);
    for (int wave = 0; wave < C::NW; ++wave)
      for (int i = 0; i < 16; ++i) {
        const int id = copy_unit<C>(A, wave, i);
        if (id < 0) continue;
        CHECK(id < units, "side %d wave %d copy %d: unit %d of %d", side, wave, i, id, units);
        ++unit_seen[id];
        const UnitPos u = unit_pos<C>(A, id);
        CHECK(u.pl >= 0 && u.pl < (A ? C::SPA : C::SPB) && u.rb >= 0 &&
                  u.rb < (A ? C::BM : C::BN) / kBrickRows && u.ku >= 0 && u.ku < C::KU,
              "unit %d decodes to plane %d row block %d unit %d", id, u.pl, u.rb, u.ku);
        for (int h = 0; h < C::COPIES; ++h) {
          const uint32_t off = unit_lds<C>(A, id, h);
          const uint32_t base = unit_lds<C>(A, id, 0);
          CHECK(off >= base && off + kBrickBytes <= base + C::UNIT_BYTES, "copy %d of unit %d outside it", h, id);
          CHECK(off + kBrickBytes <= (uint32_t)C::STAGE_BYTES, "copy past the stage buffer");
          for (uint32_t b = off; b < off + kBrickBytes; ++b) ++written[b];
        }
      }
    for (int id = 0; id < units; ++id) CHECK(unit_seen[id] == 1, "side %d unit %d copied %d times", side, id, unit_seen[id]);
  }
  for (int b = 0; b < C::STAGE_BYTES; ++b) CHECK(written[b] == 1, "stage byte %d written %d times", b, written[b]);

  // copy sources: every stage of ragged and full shapes (rows, reduction length)
  const int shapes[][2] = {{1, 256}, {31, 256}, {33, 512}, {300, 1100}, {513, 2048}, {4096, 4096}};
  for (const auto& sh : shapes) {
    const int rows = sh[0];
    const int64_t kp = (sh[1] + kKPad - 1) / kKPad * kKPad;
    const int rbs = (rows + kBrickRows - 1) / kBrickRows;
    const int64_t stride = (int64_t)rbs * (kp / kBrickK) * kBrickBytes;  // one E2M1 plane
    const int64_t ustride = stride * C::UNIT_BYTES / kBrickBytes / C::UK;  // a plane of this format
    const int64_t stages = kp / C::KT;
    for (int side = 0; side < 2; ++side) {
      const bool A = side == 0;
      const int tile_rb = (A ? C::BM : C::BN) / kBrickRows;
      const int tiles = (rbs + tile_rb - 1) / tile_rb;
      for (int tile = 0; tile < tiles; ++tile)
        for (int64_t t = 0; t < stages; ++t)
          for (int wave = 0; wave < C::NW; ++wave)
            for (int i = 0; i < 16; ++i) {
              const int id = copy_unit<C>(A, wave, i);
              if (id < 0) continue;
              const UnitPos u = unit_pos<C>(A, id);
              const int rb = tile * tile_rb + u.rb < rbs - 1 ? tile * tile_rb + u.rb : rbs - 1;
              for (int h = 0; h < C::COPIES; ++h) {
                const int64_t g = stage_global<C>(t, rbs) + unit_global<C>(u, rb, rbs, ustride, h);
                const int64_t in_plane = g - (int64_t)u.pl * C::PSTEP * ustride;
                CHECK(in_plane >= 0 && in_plane + kBrickBytes <= ustride,
                      "rows %d K %lld side %d tile %d stage %lld unit %d: source %lld of plane %lld", rows,
                      (long long)kp, side, tile, (long long)t, id, (long long)in_plane, (long long)ustride);
                // the unit holds reduction indices [(t KU + ku) UK 64, + UK 64) of row block rb
                const int64_t unit_index = in_plane / C::UNIT_BYTES;
                CHECK(unit_index == (t * C::KU + u.ku) * rbs + rb, "unit order");
              }
            }
    }
  }

  // fragments
  for (int ks = 0; ks < C::KSTEPS; ++ks)
    for (int lane = 0; lane < 64; ++lane)
      for (int side = 0; side < 2; ++side) {
        const bool A = side == 0;
        const int blocks = A ? C::BMW : C::BNW, waves = A ? C::WM : C::WN;
        for (int w = 0; w < waves; ++w)
          for (int q = 0; q < blocks; ++q) {
            const int rb = w * blocks + q;  // the tile's row block of the fragment
            if (C::MF == 16) {
              for (int h = 0; h < 2; ++h) {
                const uint32_t off = frag16_unit<C>(A, rb, ks, h) + frag16_lane_offset(lane);
                const uint32_t u0 = unit_lds<C>(A, rb * C::KU + 2 * ks, 0);
                CHECK(off >= u0 && off + 16 <= u0 + 2 * kBrickBytes, "16x16x128 fragment outside its two units");
              }
              continue;
            }
            for (int pl = 0; pl < (A ? C::SPA : C::SPB); ++pl) {
              const uint32_t unit = frag_unit<C>(A, pl, rb, ks);
              const int id = pl * (A ? C::PA_UNITS : C::PB_UNITS) + rb * C::KU + ks / C::UK;
              CHECK(unit == unit_lds<C>(A, id, 0), "fragment of plane %d row block %d k-step %d reads unit %u", pl, rb,
                    ks, unit);
              const UnitPos u = unit_pos<C>(A, id);
              CHECK(u.pl == pl && u.rb == rb && u.ku == ks / C::UK, "fragment unit decodes elsewhere");
              const Spans sp = frag_spans<C::FMT>(ks % C::UK, lane);
              for (int k = 0; k < sp.n; ++k)
                CHECK(sp.off[k] + sp.len[k] <= (uint32_t)C::UNIT_BYTES, "lane %d span %d outside its unit", lane, k);
            }
          }
      }
  // spans of one k-step: the 64 lanes' bytes are disjoint and fill the k-step's part of a unit
  {
    for (int i = 0; i < C::UK; ++i) {
      std::vector<int> hit(C::UNIT_BYTES, 0);
      for (int lane = 0; lane < 64; ++lane) {
        const Spans sp = frag_spans<C::FMT>(i, lane);
        for (int k = 0; k < sp.n; ++k) {
          CHECK(sp.off[k] + sp.len[k] <= (uint32_t)C::UNIT_BYTES, "lane %d span %d outside its unit", lane, k);
          for (uint32_t b = sp.off[k]; b < sp.off[k] + sp.len[k]; ++b) ++hit[b];
        }
      }
      int total = 0;
      for (int b = 0; b < C::UNIT_BYTES; ++b) {
        CHECK(hit[b] <= 1, "k-step %d: unit byte %d read by %d lanes", i, b, hit[b]);
        total += hit[b];
      }
      CHECK(total * C::UK == C::UNIT_BYTES, "k-step %d reads %d of %d bytes", i, total, C::UNIT_BYTES / C::UK);
    }
  }

  // LDS fold blocks
  std::set<uint32_t> seen;
  for (int wave = 0; wave < C::NW; ++wave)
    for (int lb = 0; lb < C::NLB; ++lb)
      for (int v = 0; v < C::AV; ++v)
        for (int lane = 0; lane < 64; ++lane) {
          const uint32_t off = fold_lds_offset<C>(wave, lb, v, lane);
          CHECK(off >= (uint32_t)C::FOLD_LDS_OFFSET && off + 4 <= (uint32_t)C::LDS_BYTES, "fold word outside its area");
          CHECK(seen.insert(off).second, "fold word %u used twice", off);
        }
  std::printf("ok %s: %d waves, tile %dx%d, stage %d bytes x %d, LDS %d bytes\n", name, C::NW, C::BM, C::BN,
              C::STAGE_BYTES, C::NSTAGE, C::LDS_BYTES);
}

int main() {
#define CFG(T) check<T>(#T)
  CFG(Cfg8w64x64);
  CFG(Cfg8w64x96);
  CFG(Cfg8w64x64k4);
  CFG(Cfg8w64x64k4p3);
  CFG(Cfg8w64x64e4m3);
  CFG(Cfg8w64x96k4);
  CFG(Cfg8w64x96s5);
  CFG(Cfg8w64x96k4p0);
  CFG(Cfg8w64x64k4m16);
  CFG(Cfg8w64x64k4p0m16);
  CFG(Cfg8w64x128lf);
  CFG(Cfg8w64x128lf3);
  CFG(Cfg8w64x128cs);
  CFG(Cfg8w64x128cr);
  CFG(Cfg8w64x128cm);
  CFG(Cfg8w32x64ap33);
  CFG(Cfg8w32x64ap22o);
  CFG(Cfg8w64x64e2m3);
  CFG(Cfg8w64x64s4e2m3);
  CFG(Cfg8w64x64k4e2m3);
  CFG(Cfg8w64x96p0lfe2m3);
  CFG(Cfg8w64x96p0lf2e2m3);
  CFG(Cfg8w64x64sh);
  CFG(Cfg8w64x64shp0);
  return fails ? 1 : 0;
}
