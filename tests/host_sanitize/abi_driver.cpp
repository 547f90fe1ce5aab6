// Drives the host side of the C ABI (every encoding's tables and self-checks, plane and workspace
// sizes, argument checks, the residue set's constants) with the device launchers stubbed out.
// Built with -fsanitize=address,undefined by tests/test_host_sanitizers.py; any sanitizer report
// aborts, and every status this program expects is checked.
#include <atomic>
#include <cstdio>
#include <vector>

#include "awe.h"

namespace awe {
extern std::atomic<int> g_launches;
}

static int failures = 0;
static void expect(awe_status got, awe_status want, const char* what) {
  if (got != want) {
    std::printf("FAIL %s: status %d, expected %d (%s)\n", what, (int)got, (int)want, awe_last_error());
    ++failures;
  }
}

int main() {
  void* fake = reinterpret_cast<void*>(0x100000);  // never dereferenced: the launchers are stubs
  int schemes = 0;
  for (int enc = 0; enc <= 12; ++enc) {
    for (int m = 0; m <= 260; ++m) {
      if ((enc == AWE_ENC_MOD) != (m != 0)) continue;
      awe_encoding_info info;
      if (awe_get_encoding_info((awe_encoding)enc, m, &info) != AWE_OK) continue;
      ++schemes;
      for (int side = 0; side < 2; ++side) {
        const int lo = side ? info.xmin_b : info.xmin_a, hi = side ? info.xmax_b : info.xmax_a;
        const int np = side ? info.planes_b : info.planes_a;
        std::vector<int32_t> vals((size_t)(hi - lo + 1) * np);
        expect(awe_get_plane_table((awe_encoding)enc, m, (awe_side)side, vals.data(), (int64_t)vals.size()),
               AWE_OK, "plane table");
        size_t b = 0;
        for (int64_t rows : {0, 1, 31, 33, 300})
          for (int64_t K : {0, 1, 255, 257, 1100})
            expect(awe_plane_bytes((awe_encoding)enc, m, (awe_side)side, rows, K, &b), AWE_OK, "plane bytes");
        expect(awe_encode((awe_encoding)enc, m, (awe_side)side, fake, 300, 1100, side ? 300 : 1100, fake, nullptr,
                          nullptr),
               AWE_OK, "encode");
        expect(awe_encode((awe_encoding)enc, m, (awe_side)side, fake, -1, 1100, 1100, fake, nullptr, nullptr),
               AWE_ERR_INVALID_VALUE, "encode, negative rows");
        expect(awe_encode((awe_encoding)enc, m, (awe_side)side, nullptr, 3, 3, 3, fake, nullptr, nullptr),
               AWE_ERR_INVALID_VALUE, "encode, NULL input");
      }
      size_t ws = 0;
      for (int64_t K : {0, 1, 256, 100000, 70000000})
        expect(awe_workspace_bytes((awe_encoding)enc, m, 300, 200, K, &ws), AWE_OK, "workspace bytes");
      for (int64_t K : {0, 64, 1100, 200000, 3000000}) {
        awe_gemm_planes((awe_encoding)enc, m, 300, 200, K, fake, fake, fake, 200, AWE_I32, 0, nullptr);
        if (m == 0)
          expect(awe_gemm_planes((awe_encoding)enc, m, 300, 200, K, fake, fake, fake, 200, AWE_I64, 0, nullptr),
                 AWE_OK, "gemm_planes, int64 C");
      }
      expect(awe_gemm_planes((awe_encoding)enc, m, -1, 200, 5, fake, fake, fake, 200, AWE_I32, 0, nullptr),
             AWE_ERR_INVALID_VALUE, "gemm_planes, negative M");
      expect(awe_gemm_planes((awe_encoding)enc, m, 300, 200, 5, fake, fake, fake, 100, AWE_I32, 0, nullptr),
             AWE_ERR_INVALID_VALUE, "gemm_planes, ldc < N");
      expect(awe_gemm_planes((awe_encoding)enc, m, 300, 200, 5, fake, fake, fake, 200, (awe_dtype)7, 0, nullptr),
             AWE_ERR_INVALID_VALUE, "gemm_planes, bad C type");
      const awe_dtype ct = m ? AWE_I32 : AWE_I64;  // residues are int32; int64 never overflows here
      expect(awe_gemm_planes((awe_encoding)enc, m, 300, 200, 512, fake, fake, fake, 200, ct, 100, nullptr),
             AWE_ERR_INVALID_VALUE, "gemm_planes, k_seg not a multiple of the padding");
      expect(awe_gemm_planes((awe_encoding)enc, m, (int64_t)1 << 40, 200, 512, fake, fake, fake, 200, ct, 0, nullptr),
             AWE_ERR_UNSUPPORTED, "gemm_planes, M too large");
      if (m != 0)
        expect(awe_gemm_mod(m, 300, 200, 1100, (const uint8_t*)fake, 1100, (const uint8_t*)fake, 200,
                            (int32_t*)fake, 200, fake, (size_t)1 << 40, nullptr, nullptr),
               AWE_OK, "gemm_mod");
      if (m == 0) {
        // the allocation-free variant: small sizes run, sizes whose planes exceed the fixed array
        // and negative sizes are refused
        expect(awe_gemm_exact_noalloc((awe_encoding)enc, 300, 200, 1100, fake, 1100, fake, 200, fake, 200, AWE_I64,
                                      nullptr, nullptr),
               AWE_OK, "gemm_exact_noalloc");
        expect(awe_gemm_exact_noalloc((awe_encoding)enc, 8192, 8192, 8192, fake, 8192, fake, 8192, fake, 8192,
                                      AWE_I64, nullptr, nullptr),
               AWE_ERR_WORKSPACE, "gemm_exact_noalloc, planes past the array");
        expect(awe_gemm_exact_noalloc((awe_encoding)enc, -1, 200, 1100, fake, 1100, fake, 200, fake, 200, AWE_I64,
                                      nullptr, nullptr),
               AWE_ERR_INVALID_VALUE, "gemm_exact_noalloc, negative M");
      } else {
        expect(awe_gemm_exact_noalloc((awe_encoding)enc, 300, 200, 1100, fake, 1100, fake, 200, fake, 200, AWE_I32,
                                      nullptr, nullptr),
               AWE_ERR_INVALID_VALUE, "gemm_exact_noalloc, residues");
      }
    }
  }
  // the FP64-significand residue set
  const int32_t set[] = {5, 7, 8, 9, 11, 13, 31, 37, 41, 43, 47, 53, 59, 61, 67, 71, 73, 79, 83, 89, 149, 151, 157};
  const int n = (int)(sizeof(set) / sizeof(set[0]));
  for (int k : {1, 5, n}) {
    size_t ws = 0;
    expect(awe_crt_workspace_bytes(set, k, 300, 200, 1100, &ws), AWE_OK, "crt workspace bytes");
    expect(awe_residues((const int64_t*)fake, 300, 200, 200, 1000, set, k, (uint8_t*)fake, 60000, nullptr, nullptr),
           AWE_OK, "residues");
    expect(awe_crt((const int32_t*)fake, 60000, 300, 200, 200, set, k, (int64_t*)fake, (double*)fake, 200, nullptr),
           AWE_OK, "crt");
    expect(awe_gemm_crt(300, 200, 0, (const int64_t*)fake, 1100, (const int64_t*)fake, 200, 1000, 1000, set, k,
                        (int64_t*)fake, (double*)fake, 200, fake, ws, nullptr, nullptr),
           AWE_OK, "gemm_crt, K = 0");
  }
  expect(awe_gemm_crt(300, 200, 1100, (const int64_t*)fake, 1100, (const int64_t*)fake, 200, (int64_t)1 << 52,
                      (int64_t)1 << 52, set, 5, (int64_t*)fake, (double*)fake, 200, fake, (size_t)1 << 40, nullptr,
                      nullptr),
         AWE_ERR_OVERFLOW, "gemm_crt, moduli too few for the bounds");
  const int32_t not_coprime[] = {6, 4};
  expect(awe_crt((const int32_t*)fake, 60000, 300, 200, 200, not_coprime, 2, (int64_t*)fake, nullptr, 200, nullptr),
         AWE_ERR_INVALID_VALUE, "crt, moduli not coprime");
  expect(awe_residues((const int64_t*)fake, 300, 200, 200, 1000, set, 33, (uint8_t*)fake, 60000, nullptr, nullptr),
         AWE_ERR_INVALID_VALUE, "residues, too many moduli");
  std::printf("schemes %d launches %d failures %d\n", schemes, awe::g_launches.load(), failures);
  return failures ? 1 : 0;
}
