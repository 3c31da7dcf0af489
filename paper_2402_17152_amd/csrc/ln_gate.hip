// Epilogue of the HSTU layer (Eq. 3): Y_pre = LayerNorm(A V) (.) U, and
// its backward.
// Layer norm over the D = h * d_v features of each token with biased
// variance and optional affine weight/bias; the result gates U
// elementwise.  Saves per-token mean and 1/sqrt(var + eps) for a backward.
//
// HBM-bound: one wave per token, each lane holds its 8-element chunks in
// registers (16-byte loads for bf16), two-pass mean/variance in fp32 with
// wave reductions, one pass of stores.  The attention output x is read in
// fp32 for both dtypes: normalising divides by the row's spread, which can
// be far smaller than its magnitude, so a bf16-rounded x would carry
// errors of several percent into Y.
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
                                                      void* __restrict__ y,
                                                      float* __restrict__ mean,
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
      load8<false>(x, t * D + idx, v[c]);
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

// Backward of the epilogue, per token: with z = (x - mean) * rstd (the
// forward's saved statistics) and zn = z * w + b,
//   du = zn (.) dy,  dzn = dy (.) u,  dw += dzn z,  db += dzn,
//   dz = dzn (.) w,  dx = rstd (dz - mean(dz) - z mean(dz z)).
// One wave per token in a grid-stride loop; dw / db partials stay in
// registers across the wave's tokens and reach HBM with one float atomic
// per feature and wave.
template <bool BF16, int CH>
__global__ __launch_bounds__(256) void ln_gate_bwd_kernel(
    int64_t T, int D, const void* __restrict__ x, const void* __restrict__ u, int64_t u_stride,
    const void* __restrict__ dy, const float* __restrict__ w, const float* __restrict__ b,
    const float* __restrict__ mean, const float* __restrict__ rstd, void* __restrict__ du,
    void* __restrict__ dx, void* __restrict__ dx_lo, float* __restrict__ dw,
    float* __restrict__ db) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float pw[CH][8], pb[CH][8];
#pragma unroll
  for (int c = 0; c < CH; c++)
#pragma unroll
    for (int e = 0; e < 8; e++) pw[c][e] = pb[c][e] = 0.0f;
  for (int64_t t = (int64_t)blockIdx.x * 4 + wave; t < T; t += (int64_t)gridDim.x * 4) {
    const float mu = mean[t], rs = rstd[t];
    float z[CH][8], dz[CH][8];
    float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
    for (int c = 0; c < CH; c++) {
      const int idx = (c * 64 + lane) * 8;
      if (idx < D) {
        float xv[8], uv[8], gv[8], o[8];
        load8<false>(x, t * D + idx, xv);
        load8<BF16>(u, t * u_stride + idx, uv);
        load8<BF16>(dy, t * D + idx, gv);
#pragma unroll
        for (int e = 0; e < 8; e++) {
          const float zz = (xv[e] - mu) * rs;
          const float ww = w ? w[idx + e] : 1.0f, bb = b ? b[idx + e] : 0.0f;
          const float dzn = gv[e] * uv[e];
          z[c][e] = zz;
          o[e] = (zz * ww + bb) * gv[e];
          pw[c][e] += dzn * zz;
          pb[c][e] += dzn;
          dz[c][e] = dzn * ww;
          s1 += dz[c][e];
          s2 += dz[c][e] * zz;
        }
        store8<BF16>(du, t * D + idx, o);
      }
    }
    const float m1 = wave_sum(s1) / (float)D, m2 = wave_sum(s2) / (float)D;
#pragma unroll
    for (int c = 0; c < CH; c++) {
      const int idx = (c * 64 + lane) * 8;
      if (idx < D) {
        float o[8];
#pragma unroll
        for (int e = 0; e < 8; e++) o[e] = rs * (dz[c][e] - m1 - z[c][e] * m2);
        store8<BF16>(dx, t * D + idx, o);
        if (BF16 && dx_lo) {
          // low terms: o - bf16(o), exact in fp32
          float r[8];
#pragma unroll
          for (int e = 0; e < 8; e++) r[e] = o[e] - bf16_bits_to_f32(f32_to_bf16_bits(o[e]));
          store8<BF16>(dx_lo, t * D + idx, r);
        }
      }
    }
  }
#pragma unroll
  for (int c = 0; c < CH; c++) {
    const int idx = (c * 64 + lane) * 8;
    if (idx < D) {
#pragma unroll
      for (int e = 0; e < 8; e++) {
        if (dw) unsafeAtomicAdd(&dw[idx + e], pw[c][e]);
        if (db) unsafeAtomicAdd(&db[idx + e], pb[c][e]);
      }
    }
  }
}

template <bool BF16>
hipError_t ln_bwd_case(int64_t T, int32_t D, const void* x, const void* u, int64_t u_stride,
                       const void* dy, const float* w, const float* b, const float* mean,
                       const float* rstd, void* du, void* dx, void* dx_lo, float* dw,
                       float* db, hipStream_t s) {
  // Enough waves to fill the device; each walks several tokens so the
  // per-feature atomics stay few.
  const int64_t blocks = min((T + 3) / 4, (int64_t)1024);
  dim3 grid((unsigned)blocks);
  const int ch = (D + 511) / 512;
#define LN_BWD_CALL(C)                                                                        \
  hipLaunchKernelGGL((ln_gate_bwd_kernel<BF16, C>), grid, dim3(256), 0, s, T, D, x, u,         \
                     u_stride, dy, w, b, mean, rstd, du, dx, dx_lo, dw, db);                  \
  return hipGetLastError();
  if (ch <= 1) { LN_BWD_CALL(1) }
  if (ch <= 2) { LN_BWD_CALL(2) }
  if (ch <= 4) { LN_BWD_CALL(4) }
  if (ch <= 8) { LN_BWD_CALL(8) }
#undef LN_BWD_CALL
  return hipErrorInvalidValue;
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

hipError_t launch_ln_gate_bwd(int is_bf16, int64_t T, int32_t D, const void* x, const void* u,
                              int64_t u_stride, const void* dy, const float* w, const float* b,
                              const float* mean, const float* rstd, void* du, void* dx,
                              void* dx_lo, float* dw, float* db, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (is_bf16)
    return ln_bwd_case<true>(T, D, x, u, u_stride, dy, w, b, mean, rstd, du, dx, dx_lo, dw, db,
                             s);
  return ln_bwd_case<false>(T, D, x, u, u_stride, dy, w, b, mean, rstd, du, dx, nullptr, dw, db,
                            s);
}

hipError_t launch_ln_gate(int is_bf16, int64_t T, int32_t D, const void* x, const void* u,
                          int64_t u_stride, const float* w, const float* b, float eps, void* y,
                          float* mean, float* rstd, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (is_bf16) return ln_case<true>(T, D, x, u, u_stride, w, b, eps, y, mean, rstd, s);
  return ln_case<false>(T, D, x, u, u_stride, w, b, eps, y, mean, rstd, s);
}

}  // namespace hstu
