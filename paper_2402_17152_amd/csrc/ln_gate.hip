// Epilogue of the HSTU layer (Eq. 3): Y_pre = LayerNorm(A V) (.) U.
// Layer norm over the D = h * d_v features of each token with biased
// variance and optional affine weight/bias; the result gates U
// elementwise.  Saves per-token mean and 1/sqrt(var + eps) for a backward.
//
// HBM-bound: one wave per token, each lane holds its 8-element chunks in
// registers (16-byte loads for bf16), two-pass mean/variance in fp32 with
// wave reductions, one pass of stores.
#include "kernels.h"

namespace hstu {

namespace {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

template <bool BF16>
__device__ __forceinline__ void load8(const void* base, int64_t idx, float* out) {
  if constexpr (BF16) {
    u32x4 r = *reinterpret_cast<const u32x4*>((const uint16_t*)base + idx);
#pragma unroll
    for (int e = 0; e < 4; e++) {
      out[2 * e] = __uint_as_float(r[e] << 16);
      out[2 * e + 1] = __uint_as_float(r[e] & 0xffff0000u);
    }
  } else {
    const f32x4* p = reinterpret_cast<const f32x4*>((const float*)base + idx);
    f32x4 a = p[0], b = p[1];
#pragma unroll
    for (int e = 0; e < 4; e++) {
      out[e] = a[e];
      out[4 + e] = b[e];
    }
  }
}

template <bool BF16>
__device__ __forceinline__ void store8(void* base, int64_t idx, const float* v) {
  if constexpr (BF16) {
    u32x4 r;
#pragma unroll
    for (int e = 0; e < 4; e++) r[e] = pack_bf16x2(v[2 * e], v[2 * e + 1]);
    *reinterpret_cast<u32x4*>((uint16_t*)base + idx) = r;
  } else {
    f32x4 a, b;
#pragma unroll
    for (int e = 0; e < 4; e++) {
      a[e] = v[e];
      b[e] = v[4 + e];
    }
    f32x4* p = reinterpret_cast<f32x4*>((float*)base + idx);
    p[0] = a;
    p[1] = b;
  }
}

// CH = chunks of 8 elements per lane (D <= 512 * CH).
template <bool BF16, int CH>
__global__ __launch_bounds__(256) void ln_gate_kernel(int64_t T, int D, const void* __restrict__ x,
                                                      const void* __restrict__ u, int64_t u_stride,
                                                      const float* __restrict__ w,
                                                      const float* __restrict__ b, float eps,
                                                      void* __restrict__ y, float* __restrict__ mean,
                                                      float* __restrict__ rstd) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + wave;
  if (t >= T) return;
  float v[CH][8];
  float sum = 0.0f;
#pragma unroll
  for (int c = 0; c < CH; c++) {
    const int idx = (c * 64 + lane) * 8;
    if (idx < D) {
      load8<BF16>(x, t * D + idx, v[c]);
#pragma unroll
      for (int e = 0; e < 8; e++) sum += v[c][e];
    }
  }
  const float mu = wave_sum(sum) / (float)D;
  float sq = 0.0f;
#pragma unroll
  for (int c = 0; c < CH; c++) {
    const int idx = (c * 64 + lane) * 8;
    if (idx < D) {
#pragma unroll
      for (int e = 0; e < 8; e++) {
        const float d = v[c][e] - mu;
        sq += d * d;
      }
    }
  }
  const float var = wave_sum(sq) / (float)D;
  const float rs = 1.0f / sqrtf(var + eps);
#pragma unroll
  for (int c = 0; c < CH; c++) {
    const int idx = (c * 64 + lane) * 8;
    if (idx < D) {
      float g[8], out[8];
      load8<BF16>(u, t * u_stride + idx, g);
#pragma unroll
      for (int e = 0; e < 8; e++) {
        float z = (v[c][e] - mu) * rs;
        if (w) z *= w[idx + e];
        if (b) z += b[idx + e];
        out[e] = z * g[e];
      }
      store8<BF16>(y, t * D + idx, out);
    }
  }
  if (lane == 0) {
    if (mean) mean[t] = mu;
    if (rstd) rstd[t] = rs;
  }
}

template <bool BF16>
hipError_t ln_case(int64_t T, int32_t D, const void* x, const void* u, int64_t u_stride,
                   const float* w, const float* b, float eps, void* y, float* mean, float* rstd,
                   hipStream_t s) {
  dim3 grid((unsigned)((T + 3) / 4));
  const int ch = (D + 511) / 512;
#define LN_CALL(C)                                                                          \
  hipLaunchKernelGGL((ln_gate_kernel<BF16, C>), grid, dim3(256), 0, s, T, D, x, u, u_stride, \
                     w, b, eps, y, mean, rstd);                                             \
  return hipGetLastError();
  if (ch <= 1) { LN_CALL(1) }
  if (ch <= 2) { LN_CALL(2) }
  if (ch <= 4) { LN_CALL(4) }
  if (ch <= 8) { LN_CALL(8) }
#undef LN_CALL
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_ln_gate(int is_bf16, int64_t T, int32_t D, const void* x, const void* u,
                          int64_t u_stride, const float* w, const float* b, float eps, void* y,
                          float* mean, float* rstd, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (is_bf16) return ln_case<true>(T, D, x, u, u_stride, w, b, eps, y, mean, rstd, s);
  return ln_case<false>(T, D, x, u, u_stride, w, b, eps, y, mean, rstd, s);
}

}  // namespace hstu
