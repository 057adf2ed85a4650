// diag.hip -- device diagnostics: measured matrix-core ceilings and device facts.
//
// The roofline of the NTK kernels is the fp32 matrix-core peak (and fp64 for the forward
// pass).  Beside the published figures, ntk_mfma_peak measures what a kernel made of nothing
// but independent MFMA chains reaches on this device, which is the ceiling a real kernel can
// approach.
#include <hip/hip_runtime.h>

#include "ntk.h"

namespace ntk {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef double f64x4 __attribute__((ext_vector_type(4)));

constexpr int kChains = 4;        // independent accumulators per wave
constexpr int kBlocksPerCu = 4;   // 4 workgroups of 4 waves: 4 waves per SIMD
constexpr int kThreads = 256;
constexpr int kUnroll = 8;        // MFMA rounds per loop iteration (iters is a multiple)

__global__ void __launch_bounds__(kThreads) k_mfma_f32_chains(int iters, float* __restrict__ out) {
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[c][v] = 0.f;
  const float a = (float)(threadIdx.x & 63) * 1e-3f, b = 1e-3f;
  for (int i = 0; i < iters; i += kUnroll) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
#pragma unroll
      for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[c][v];
  out[blockIdx.x * kThreads + threadIdx.x] = s;
}

__global__ void __launch_bounds__(kThreads) k_mfma_f64_chains(int iters, float* __restrict__ out) {
  f64x4 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[c][v] = 0.0;
  const double a = (double)(threadIdx.x & 63) * 1e-3, b = 1e-3;
  for (int i = 0; i < iters; i += kUnroll) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
#pragma unroll
      for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc[c], 0, 0, 0);
  }
  double s = 0.0;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int v = 0; v < 4; ++v) s += acc[c][v];
  out[blockIdx.x * kThreads + threadIdx.x] = (float)s;
}

}  // namespace
}  // namespace ntk

extern "C" int ntk_device_info(int* num_cu, int* clock_khz) {
  if (!num_cu || !clock_khz) return NTK_E_ARG;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return NTK_E_HIP;
  if (hipDeviceGetAttribute(num_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipDeviceGetAttribute(clock_khz, hipDeviceAttributeClockRate, dev) != hipSuccess)
    return NTK_E_HIP;
  return NTK_OK;
}

extern "C" int ntk_mfma_peak(int which, double* tflops) {
  if (!tflops || (which != 0 && which != 1)) return NTK_E_ARG;
  int num_cu = 0, clock = 0;
  int rc = ntk_device_info(&num_cu, &clock);
  if (rc != NTK_OK) return rc;
  const int blocks = num_cu * ntk::kBlocksPerCu;
  // fp32: 2*32*32*2 FLOPs per MFMA; fp64: 2*16*16*4
  const double flop_per_mfma = which == 0 ? 4096.0 : 2048.0;
  const int iters = 20000;  // a multiple of kUnroll
  float* out = nullptr;
  hipStream_t s = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  rc = NTK_E_HIP;
  if (hipMalloc(&out, (size_t)blocks * ntk::kThreads * sizeof(float)) != hipSuccess) return NTK_E_OOM;
  if (hipStreamCreateWithFlags(&s, hipStreamNonBlocking) == hipSuccess && hipEventCreate(&e0) == hipSuccess &&
      hipEventCreate(&e1) == hipSuccess) {
    auto launch = [&]() {
      if (which == 0)
        ntk::k_mfma_f32_chains<<<dim3(blocks), dim3(ntk::kThreads), 0, s>>>(iters, out);
      else
        ntk::k_mfma_f64_chains<<<dim3(blocks), dim3(ntk::kThreads), 0, s>>>(iters, out);
    };
    launch();  // warm-up
    (void)hipEventRecord(e0, s);
    launch();
    (void)hipEventRecord(e1, s);
    float ms = 0.f;
    if (hipGetLastError() == hipSuccess && hipEventSynchronize(e1) == hipSuccess &&
        hipEventElapsedTime(&ms, e0, e1) == hipSuccess && ms > 0.f) {
      const double waves = (double)blocks * (ntk::kThreads / 64);
      *tflops = waves * iters * ntk::kChains * flop_per_mfma / (ms * 1e-3) / 1e12;
      rc = NTK_OK;
    }
  }
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (s) (void)hipStreamDestroy(s);
  (void)hipFree(out);
  return rc;
}
