// Benchmark support: a kernel that issues nothing but bf16
// v_mfma_f32_32x32x16 instructions, to measure the matrix-core rate the
// attention kernels are compared against on the same device.
#include "kernels.h"

namespace hstu {

namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeChains = 8;  // independent accumulators per wave

__global__ __launch_bounds__(kProbeThreads) void mfma_probe_kernel(int32_t iters, float* sink) {
  // Small operands keep the accumulators finite for any iteration count.
  const uint32_t w = 0x3b803b80u + (threadIdx.x & 1);  // bf16 pair ~ 2^-8
  const u32x4 a{w, w, w, w}, b{w ^ 1u, w, w, w ^ 1u};
  f32x16 c[kProbeChains];
#pragma unroll
  for (int k = 0; k < kProbeChains; k++) c[k] = f32x16{};
  for (int32_t i = 0; i < iters; i++) {
#pragma unroll
    for (int k = 0; k < kProbeChains; k++) c[k] = mfma32x32x16(as_bf16x8(a), as_bf16x8(b), c[k]);
  }
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < kProbeChains; k++)
#pragma unroll
    for (int q = 0; q < 16; q++) s += c[k][q];
  if (s == -1.0f) sink[threadIdx.x] = s;  // never true; keeps the contractions live
}

}  // namespace

hipError_t launch_mfma_probe(int32_t iters, int32_t waves_per_simd, float* sink, double* flop,
                             hipStream_t s) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int64_t blocks = (int64_t)cus * waves_per_simd;  // 4 waves each: one per SIMD
  *flop = (double)blocks * (kProbeThreads / 64) * (double)iters * kProbeChains * 32.0 * 32.0 *
          16.0 * 2.0;
  hipLaunchKernelGGL(mfma_probe_kernel, dim3((unsigned)blocks), dim3(kProbeThreads), 0, s, iters,
                     sink);
  return hipGetLastError();
}

}  // namespace hstu
