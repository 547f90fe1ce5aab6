// Host-only stand-ins for the device launchers of libawe: with these, the table builder and the
// C ABI's argument checks link and run without a GPU (and under the host sanitizers).  Each stub
// only counts its calls.
#include <atomic>

#include "awe_internal.h"

namespace awe {
std::atomic<int> g_launches{0};  // atomic: the thread test calls the ABI from several threads
awe_status launch_encode(const EncodeLaunch&, hipStream_t) { ++g_launches; return AWE_OK; }
awe_status launch_gemm(const GemmLaunch&, hipStream_t) { ++g_launches; return AWE_OK; }
bool gemm_group_ok(const GemmLaunch*, int n) { return n >= 1 && n <= kMaxModuli; }
awe_status launch_gemm_group(const GemmLaunch*, int, hipStream_t) { ++g_launches; return AWE_OK; }
awe_status launch_residues(const int64_t*, int64_t, int64_t, int64_t, int64_t, const ResidueParams&, uint8_t*,
                           int64_t, int32_t*, hipStream_t) {
  ++g_launches;
  return AWE_OK;
}
awe_status launch_residue_encode(const ResidueEncodeArgs&, const ResidueParams&, bool, hipStream_t) {
  ++g_launches;
  return AWE_OK;
}
awe_status launch_crt(const int32_t*, int64_t, int64_t, int64_t, int64_t, const CrtParams&, int64_t*, double*,
                      int64_t, hipStream_t) {
  ++g_launches;
  return AWE_OK;
}
awe_status launch_crt(const uint8_t*, int64_t, int64_t, int64_t, int64_t, const CrtParams&, int64_t*, double*,
                      int64_t, hipStream_t) {
  ++g_launches;
  return AWE_OK;
}
// a host buffer stands in for the device planes array (the stubbed launchers never touch it)
awe_status noalloc_planes(void** out) {
  static unsigned char planes[256];
  *out = planes;
  return AWE_OK;
}
}  // namespace awe
