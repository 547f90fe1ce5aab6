// Several host threads call the C ABI at once (first use of every scheme, the residue tables'
// cache, argument checks), with the device launchers stubbed out.  Built with
// -fsanitize=thread by tests/test_host_sanitizers.py: a data race in the library's caches is
// reported and fails the run.
#include <cstdio>
#include <thread>
#include <vector>

#include "awe.h"

int main() {
  void* fake = reinterpret_cast<void*>(0x100000);  // never dereferenced: the launchers are stubs
  const int32_t set[] = {5, 7, 8, 9, 11, 13, 31, 37, 41, 43, 47, 53, 59, 61, 67, 71, 73, 79, 83, 89, 149, 151, 157};
  const int n = (int)(sizeof(set) / sizeof(set[0]));
  std::vector<int> bad(8, 0);
  std::vector<std::thread> th;
  for (int t = 0; t < 8; ++t)
    th.emplace_back([&, t]() {
      // each thread walks the encodings and moduli from a different starting point
      for (int i = 0; i < 10 + 257; ++i) {
        const int k = (i + 37 * t) % (10 + 257);
        const int enc = k < 10 ? k + 1 : AWE_ENC_MOD;
        const int m = k < 10 ? 0 : k - 10;
        awe_encoding_info info;
        if (awe_get_encoding_info((awe_encoding)enc, m, &info) != AWE_OK) continue;
        size_t b = 0;
        if (awe_plane_bytes((awe_encoding)enc, m, AWE_SIDE_A, 300, 1100, &b) != AWE_OK) ++bad[t];
        const awe_dtype ct = m ? AWE_I32 : AWE_I64;
        if (awe_gemm_planes((awe_encoding)enc, m, 300, 200, 1100, fake, fake, fake, 200, ct, 0, nullptr) != AWE_OK)
          ++bad[t];
      }
      size_t ws = 0;
      if (awe_crt_workspace_bytes(set, n, 300, 200, 1100, &ws) != AWE_OK) ++bad[t];
      if (awe_gemm_crt(300, 200, 0, (const int64_t*)fake, 1100, (const int64_t*)fake, 200, 1000, 1000, set, n,
                       (int64_t*)fake, (double*)fake, 200, fake, ws, nullptr, nullptr) != AWE_OK)
        ++bad[t];
    });
  for (auto& x : th) x.join();
  int failures = 0;
  for (int v : bad) failures += v;
  std::printf("threads 8 failures %d\n", failures);
  return failures ? 1 : 0;
}
