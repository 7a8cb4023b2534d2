// Matrix-core rate probe (measurement only, not a step of the method): the bf16 rate the
// matrix cores sustain and the shader clock they hold while doing it, the figures the
// rooflines of the GEMM and attention kernels are read against beside the published peak.
//
// One workgroup of four waves per CU (one wave per SIMD); every wave issues `iters`
// rounds of eight independent 32x32x16 bf16 MFMAs (no operand traffic after the start),
// then writes its accumulator sum (so that nothing is removed) and its cycle and
// constant-counter (100 MHz) tick counts.
#include <vector>

#include "kernels.h"

namespace dn {
namespace {

constexpr int kProbeAcc = 8;

__global__ __launch_bounds__(256) void mfma_rate_kernel(float* out, long long* ticks, int iters, float seed) {
  f32x16 acc[kProbeAcc];
#pragma unroll
  for (int i = 0; i < kProbeAcc; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = static_cast<bf16>(seed * static_cast<float>(threadIdx.x + e));
    b[e] = static_cast<bf16>(seed * static_cast<float>(e + 1));
  }
  const long long c0 = clock64(), w0 = wall_clock64();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kProbeAcc; ++i) acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[i], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kProbeAcc; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[i][r];
  const long long c1 = clock64(), w1 = wall_clock64();
  out[blockIdx.x * 256 + threadIdx.x] = s;
  if ((threadIdx.x & 63) == 0) {
    long long* d = ticks + (blockIdx.x * 4 + (threadIdx.x >> 6)) * 2;
    d[0] = c1 - c0;
    d[1] = w1 - w0;
  }
}

}  // namespace

void mfma_rate(int iters, double* tflops, double* clock_ghz) {
  DN_CHECK(iters >= 1 && iters <= (1 << 20), "mfma_rate: iters must be in [1, 2^20]");
  int dev = 0;
  DN_HIP(hipGetDevice(&dev));
  hipDeviceProp_t prop;
  DN_HIP(hipGetDeviceProperties(&prop, dev));
  const int wgs = prop.multiProcessorCount;
  float* out = nullptr;
  long long* ticks = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  auto release = [&]() {
    if (out) (void)hipFree(out);
    if (ticks) (void)hipFree(ticks);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
  };
  try {
    DN_HIP(hipMalloc(&out, (size_t)wgs * 256 * sizeof(float)));
    DN_HIP(hipMalloc(&ticks, (size_t)wgs * 4 * 2 * sizeof(long long)));
    DN_HIP(hipEventCreate(&e0));
    DN_HIP(hipEventCreate(&e1));
    // one launch to bring the clock up, then the timed one
    hipLaunchKernelGGL(mfma_rate_kernel, dim3(wgs), dim3(256), 0, nullptr, out, ticks, iters, 1e-3f);
    DN_HIP(hipGetLastError());
    DN_HIP(hipEventRecord(e0, nullptr));
    hipLaunchKernelGGL(mfma_rate_kernel, dim3(wgs), dim3(256), 0, nullptr, out, ticks, iters, 1e-3f);
    DN_HIP(hipGetLastError());
    DN_HIP(hipEventRecord(e1, nullptr));
    DN_HIP(hipEventSynchronize(e1));
    float ms = 0.f;
    DN_HIP(hipEventElapsedTime(&ms, e0, e1));
    std::vector<long long> h((size_t)wgs * 8);
    DN_HIP(hipMemcpy(h.data(), ticks, h.size() * sizeof(long long), hipMemcpyDeviceToHost));
    double cyc = 0.0, tick = 0.0;
    for (int i = 0; i < wgs * 4; ++i) {
      cyc += static_cast<double>(h[2 * i]);
      tick += static_cast<double>(h[2 * i + 1]);
    }
    const double flop = 2.0 * 32 * 32 * 16 * kProbeAcc * static_cast<double>(iters) * wgs * 4;
    *tflops = flop / (static_cast<double>(ms) * 1e-3) / 1e12;
    *clock_ghz = tick > 0.0 ? cyc / tick * 0.1 : 0.0;  // the constant counter ticks at 100 MHz
  } catch (...) {
    release();
    throw;
  }
  release();
}

}  // namespace dn
