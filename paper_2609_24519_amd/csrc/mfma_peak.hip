// Sustained rate of the GEMM's instruction, the scaled 32x32x64 MFMA with E2M1
// (or E2M3, E4M3) operands and FP32 accumulation, when every wave issues independent MFMAs
// from registers and touches no memory in the loop.  It gives the practical
// ceiling the GEMM kernel is compared with next to the data-sheet peak (which
// assumes the peak engine clock under full MFMA load).  Benchmark helper only:
// not part of the product path.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kMfmaPerIter = 16;
constexpr double kFlopPerMfma = 2.0 * 32 * 32 * 64;

// Operand formats as the MFMA's format selects: 4 E2M1 (scale 2^1), 2 E2M3 (2^3), 0 E4M3 (2^0).
template <int FMT>
__global__ __launch_bounds__(512) void mfma_peak_kernel(int iters, float* sink) {
  constexpr uint32_t kScale = FMT == 4 ? 0x80808080u : (FMT == 2 ? 0x82828282u : 0x7f7f7f7fu);
  v16f c[4] = {};
  const v8i a = {(int)threadIdx.x, 0x11111111, 0x22222222, 0x33333333, 0x04040404, 0x05050505, 0, 0};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int m = 0; m < kMfmaPerIter; ++m)
      c[m & 3] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, a, c[m & 3], FMT, FMT, 0, kScale,
                                                                0, kScale);
  }
  const float s = c[0][0] + c[1][0] + c[2][0] + c[3][0];
  if (s == 0.125f) sink[blockIdx.x] = s;  // never true in practice; keeps the MFMAs live
}

// MFMAs whose operands change from one MFMA to the next (four A and four B
// register sets of per-lane pseudo-random codes, cycled), so the matrix unit
// switches as it does on real data; the constant operands above switch far less and
// draw less power, which lets the clock stay higher.
template <int FMT>
__global__ __launch_bounds__(512) void mfma_varied_kernel(int iters, float* sink) {
  constexpr uint32_t kScale = FMT == 4 ? 0x80808080u : (FMT == 2 ? 0x82828282u : 0x7f7f7f7fu);
  v16f c[4] = {};
  v8i a[4], b[4];
  uint32_t h = 0x9e3779b9u * (threadIdx.x + 1) + 0x85ebca6bu * blockIdx.x;
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      h ^= h << 13; h ^= h >> 17; h ^= h << 5;  // xorshift32
      a[s][j] = (int)h;
      h ^= h << 13; h ^= h >> 17; h ^= h << 5;
      b[s][j] = (int)h;
    }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int m = 0; m < kMfmaPerIter; ++m)
      c[m & 3] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[m & 3], b[(m >> 2) & 3], c[m & 3], FMT,
                                                                FMT, 0, kScale, 0, kScale);
  }
  const float s = c[0][0] + c[1][0] + c[2][0] + c[3][0];
  if (s == 0.125f) sink[blockIdx.x] = s;  // keeps the MFMAs live
}

// As mfma_varied_kernel with E2M1 operands on the 16x16x128 form of the scaled MFMA (the
// same operand registers, half the FLOP per instruction): 32 MFMAs per iteration, the same
// FLOP per iteration as 16 of the 32x32x64 form.
__global__ __launch_bounds__(512) void mfma_varied16_kernel(int iters, float* sink) {
  constexpr uint32_t kScale = 0x80808080u;
  v4f c[8] = {};
  v8i a[4], b[4];
  uint32_t h = 0x9e3779b9u * (threadIdx.x + 1) + 0x85ebca6bu * blockIdx.x;
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      h ^= h << 13; h ^= h >> 17; h ^= h << 5;
      a[s][j] = (int)h;
      h ^= h << 13; h ^= h >> 17; h ^= h << 5;
      b[s][j] = (int)h;
    }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int m = 0; m < 2 * kMfmaPerIter; ++m)
      c[m & 7] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a[m & 3], b[(m >> 2) & 3], c[m & 7], 4, 4, 0,
                                                                 kScale, 0, kScale);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) s += c[i][0];
  if (s == 0.125f) sink[blockIdx.x] = s;  // keeps the MFMAs live
}

}  // namespace

namespace {

template <int FMT, bool kVaried = false, bool k16 = false>
int run_peak(int waves_per_cu, int iters, double* tflops) {
  if (waves_per_cu < 1 || waves_per_cu > 8 || iters < 1 || tflops == nullptr) return (int)hipErrorInvalidValue;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return (int)e;
  float* sink = nullptr;
  if ((e = hipMalloc(&sink, sizeof(float) * cus)) != hipSuccess) return (int)e;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  float ms = 0.f;
  const dim3 grid(cus), block(64 * waves_per_cu);
  if ((e = hipEventCreate(&e0)) == hipSuccess && (e = hipEventCreate(&e1)) == hipSuccess) {
    auto launch = [&]() {
      if (k16)
        hipLaunchKernelGGL(mfma_varied16_kernel, grid, block, 0, nullptr, iters, sink);
      else if (kVaried)
        hipLaunchKernelGGL(mfma_varied_kernel<FMT>, grid, block, 0, nullptr, iters, sink);
      else
        hipLaunchKernelGGL(mfma_peak_kernel<FMT>, grid, block, 0, nullptr, iters, sink);
      return hipGetLastError();
    };
    e = launch();
    if (e == hipSuccess) e = hipEventRecord(e0, nullptr);
    if (e == hipSuccess) e = launch();
    if (e == hipSuccess) e = hipEventRecord(e1, nullptr);
    if (e == hipSuccess) e = hipEventSynchronize(e1);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  }
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  (void)hipFree(sink);
  if (e != hipSuccess) return (int)e;
  const double flop = (double)cus * waves_per_cu * iters * kMfmaPerIter * kFlopPerMfma;
  *tflops = flop / ((double)ms * 1e-3) / 1e12;
  return 0;
}

}  // namespace

// Runs one workgroup of `waves_per_cu` waves (1..8) per compute unit for
// `iters` iterations of 16 MFMAs per wave after one warm-up launch, and
// writes the achieved dense FP4 rate in TFLOP/s.  Returns 0, or a HIP error code.
extern "C" int awe_mfma_peak(int waves_per_cu, int iters, double* tflops) {
  return run_peak<4>(waves_per_cu, iters, tflops);
}

// As awe_mfma_peak with E2M1 operands that change between MFMAs (realistic switching).
extern "C" int awe_mfma_peak_varied(int waves_per_cu, int iters, double* tflops) {
  return run_peak<4, true>(waves_per_cu, iters, tflops);
}

// As awe_mfma_peak_varied for operand format `fmt` (4 E2M1, 2 E2M3, 0 E4M3).
extern "C" int awe_mfma_peak_varied_fmt(int fmt, int waves_per_cu, int iters, double* tflops) {
  switch (fmt) {
    case 4: return run_peak<4, true>(waves_per_cu, iters, tflops);
    case 2: return run_peak<2, true>(waves_per_cu, iters, tflops);
    case 0: return run_peak<0, true>(waves_per_cu, iters, tflops);
    default: return (int)hipErrorInvalidValue;
  }
}

// As awe_mfma_peak for operand format `fmt` (4 E2M1, 2 E2M3, 0 E4M3).
extern "C" int awe_mfma_peak_fmt(int fmt, int waves_per_cu, int iters, double* tflops) {
  switch (fmt) {
    case 4: return run_peak<4>(waves_per_cu, iters, tflops);
    case 2: return run_peak<2>(waves_per_cu, iters, tflops);
    case 0: return run_peak<0>(waves_per_cu, iters, tflops);
    default: return (int)hipErrorInvalidValue;
  }
}

// As awe_mfma_peak_varied on the 16x16x128 form of the MFMA (E2M1 operands that change
// between MFMAs).
extern "C" int awe_mfma_peak_varied16(int waves_per_cu, int iters, double* tflops) {
  return run_peak<4, true, true>(waves_per_cu, iters, tflops);
}
