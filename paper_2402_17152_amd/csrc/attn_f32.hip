// fp32 jagged pointwise attention, forward and backward, plain SIMT
// arithmetic (no matrix cores): the HSTU_F32 variant of the library,
// meant for small problems where fp32 throughout is wanted.
//
// Same definitions as the bf16 kernels (Eq. 2 with the pointwise 1/N
// normaliser, rab^{p,t} from the two tables, Algorithm 1 mask), one
// thread per (token, head):
//   forward       thread = query row i: O_i = (1/N) sum_j SiLU(s_ij) v_j;
//   backward (a)  thread = query row i: dQ_i = (1/N) sum_j dS_ij k_j and
//                 the bias gradients, summed in fp64 (one atomic per pair
//                 for the position table; for the time table a running
//                 sum per thread, added when the bucket changes, so that a
//                 bucket's millions of terms do not pile up fp32 rounding);
//   backward (b)  thread = key row j:   dK_j = (1/N) sum_i dS_ij q_i,
//                                       dV_j = (1/N) sum_i SiLU(s_ij) dO_i.
#include "kernels.h"

namespace hstu {

namespace {

struct Row {
  int64_t o;
  int L, n_h, idx;
};

// Sequence holding global token r: last b with seq_offsets[b] <= r.
__device__ __forceinline__ Row locate(const JaggedArgs& ja, int64_t r) {
  int lo = 0, hi = ja.num_seqs;  // seq_offsets[lo] <= r < seq_offsets[hi]
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (ja.seq_offsets[mid] <= r) lo = mid; else hi = mid;
  }
  Row w;
  w.o = ja.seq_offsets[lo];
  w.L = (int)(ja.seq_offsets[lo + 1] - w.o);
  w.n_h = w.L - (ja.num_targets ? (int)ja.num_targets[lo] : 0);
  w.idx = (int)(r - w.o);
  return w;
}

__device__ __forceinline__ float bias_of(const JaggedArgs& ja, const Row& w, int i, int j,
                                         int64_t ti, int64_t tj) {
  const int idx = (ja.max_seq_len - 1) + bias_pos(j, w.n_h) - bias_pos(i, w.n_h);
  return ja.rab_pos[idx] + ja.rab_time[time_bucket64(ti - tj, ja.num_buckets)];
}

template <int DQK, int DV>
__global__ __launch_bounds__(64) void fwd_f32_kernel(JaggedArgs ja, Tensors t, float* out) {
  const int64_t r = (int64_t)blockIdx.x * 64 + threadIdx.x;
  if (r >= ja.total_tokens) return;
  const int head = blockIdx.y, H = ja.num_heads;
  const Row w = locate(ja, r);
  const int i = w.idx;
  const float* qg = (const float*)t.q + r * t.q_stride + head * DQK;
  float q[DQK], acc[DV];
  for (int c = 0; c < DQK; c++) q[c] = qg[c];
  for (int c = 0; c < DV; c++) acc[c] = 0.0f;
  const int64_t ti = ja.timestamps[r];
  for (int j = 0; j <= i; j++) {
    if (!pair_valid(i, j, w.n_h)) continue;
    const float* kj = (const float*)t.k + (w.o + j) * t.k_stride + head * DQK;
    const float* vj = (const float*)t.v + (w.o + j) * t.v_stride + head * DV;
    float s = bias_of(ja, w, i, j, ti, ja.timestamps[w.o + j]);
    for (int c = 0; c < DQK; c++) s += q[c] * kj[c];
    const float p = s * sigmoid_fast(s);
    for (int c = 0; c < DV; c++) acc[c] += p * vj[c];
  }
  const float invN = 1.0f / (float)ja.max_seq_len;
  float* og = out + (r * H + head) * DV;
  for (int c = 0; c < DV; c++) og[c] = acc[c] * invN;
}

template <int DQK, int DV>
__global__ __launch_bounds__(64) void bwd_dq_f32_kernel(JaggedArgs ja, Tensors t, const float* dO,
                                                        float* dq, double* rab_pos_acc,
                                                        double* rab_time_acc) {
  const int64_t r = (int64_t)blockIdx.x * 64 + threadIdx.x;
  if (r >= ja.total_tokens) return;
  const int head = blockIdx.y, H = ja.num_heads, N = ja.max_seq_len;
  const Row w = locate(ja, r);
  const int i = w.idx;
  const float invN = 1.0f / (float)N;
  const float* qg = (const float*)t.q + r * t.q_stride + head * DQK;
  const float* dog = dO + (r * H + head) * DV;
  float q[DQK], g[DV], acc[DQK];
  for (int c = 0; c < DQK; c++) {
    q[c] = qg[c];
    acc[c] = 0.0f;
  }
  for (int c = 0; c < DV; c++) g[c] = dog[c];
  const int64_t ti = ja.timestamps[r];
  int run_b = -1;
  double run = 0.0;
  for (int j = 0; j <= i; j++) {
    if (!pair_valid(i, j, w.n_h)) continue;
    const float* kj = (const float*)t.k + (w.o + j) * t.k_stride + head * DQK;
    const float* vj = (const float*)t.v + (w.o + j) * t.v_stride + head * DV;
    const int64_t tj = ja.timestamps[w.o + j];
    float s = bias_of(ja, w, i, j, ti, tj);
    for (int c = 0; c < DQK; c++) s += q[c] * kj[c];
    float dp = 0.0f;
    for (int c = 0; c < DV; c++) dp += g[c] * vj[c];
    const float sg = sigmoid_fast(s);
    const float ds = dp * (sg + s * sg * (1.0f - sg));
    for (int c = 0; c < DQK; c++) acc[c] += ds * kj[c];
    const int kpos = bias_pos(i, w.n_h) - bias_pos(j, w.n_h);
    unsafeAtomicAdd(&rab_pos_acc[(N - 1) - kpos], (double)ds);
    const int b = time_bucket64(ti - tj, ja.num_buckets);
    if (b != run_b) {
      if (run_b >= 0) unsafeAtomicAdd(&rab_time_acc[run_b], run);
      run_b = b;
      run = 0.0;
    }
    run += (double)ds;
  }
  if (run_b >= 0) unsafeAtomicAdd(&rab_time_acc[run_b], run);
  float* out = dq + (r * H + head) * DQK;
  for (int c = 0; c < DQK; c++) out[c] = acc[c] * invN;
}

template <int DQK, int DV>
__global__ __launch_bounds__(64) void bwd_dkv_f32_kernel(JaggedArgs ja, Tensors t, const float* dO,
                                                         float* dk, float* dv) {
  const int64_t r = (int64_t)blockIdx.x * 64 + threadIdx.x;
  if (r >= ja.total_tokens) return;
  const int head = blockIdx.y, H = ja.num_heads;
  const Row w = locate(ja, r);
  const int j = w.idx;
  const float* kg = (const float*)t.k + r * t.k_stride + head * DQK;
  const float* vg = (const float*)t.v + r * t.v_stride + head * DV;
  float k[DQK], v[DV], ak[DQK], av[DV];
  for (int c = 0; c < DQK; c++) {
    k[c] = kg[c];
    ak[c] = 0.0f;
  }
  for (int c = 0; c < DV; c++) {
    v[c] = vg[c];
    av[c] = 0.0f;
  }
  const int64_t tj = ja.timestamps[r];
  const int i_end = j >= w.n_h ? j + 1 : w.L;  // a candidate key is seen by itself only
  for (int i = j; i < i_end; i++) {
    if (!pair_valid(i, j, w.n_h)) continue;
    const float* qi = (const float*)t.q + (w.o + i) * t.q_stride + head * DQK;
    const float* gi = dO + ((w.o + i) * H + head) * DV;
    float s = bias_of(ja, w, i, j, ja.timestamps[w.o + i], tj);
    for (int c = 0; c < DQK; c++) s += qi[c] * k[c];
    float dp = 0.0f;
    for (int c = 0; c < DV; c++) dp += gi[c] * v[c];
    const float sg = sigmoid_fast(s);
    const float p = s * sg;
    const float ds = dp * (sg + p * (1.0f - sg));
    for (int c = 0; c < DQK; c++) ak[c] += ds * qi[c];
    for (int c = 0; c < DV; c++) av[c] += p * gi[c];
  }
  const float invN = 1.0f / (float)ja.max_seq_len;
  float* ok = dk + (r * H + head) * DQK;
  float* ov = dv + (r * H + head) * DV;
  for (int c = 0; c < DQK; c++) ok[c] = ak[c] * invN;
  for (int c = 0; c < DV; c++) ov[c] = av[c] * invN;
}

template <int DQK, int DV>
hipError_t fwd_case(const JaggedArgs& ja, const Tensors& t, void* out, hipStream_t s) {
  dim3 grid((unsigned)((ja.total_tokens + 63) / 64), (unsigned)ja.num_heads);
  hipLaunchKernelGGL((fwd_f32_kernel<DQK, DV>), grid, dim3(64), 0, s, ja, t, (float*)out);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void f64_to_f32_kernel(const double* in, float* out, int64_t n,
                                                        double scale) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    out[i] = (float)(in[i] * scale);
}

template <int DQK, int DV>
hipError_t bwd_case(const JaggedArgs& ja, const Tensors& t, const void* d_out, void* dq, void* dk,
                    void* dv, double* drp, double* drt, hipStream_t s) {
  dim3 grid((unsigned)((ja.total_tokens + 63) / 64), (unsigned)ja.num_heads);
  hipLaunchKernelGGL((bwd_dq_f32_kernel<DQK, DV>), grid, dim3(64), 0, s, ja, t,
                     (const float*)d_out, (float*)dq, drp, drt);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((bwd_dkv_f32_kernel<DQK, DV>), grid, dim3(64), 0, s, ja, t,
                     (const float*)d_out, (float*)dk, (float*)dv);
  return hipGetLastError();
}

}  // namespace

#define HSTU_F32_DISPATCH(CALL)      \
  if (dqk == 32 && dv == 32) CALL(32, 32)   \
  if (dqk == 32 && dv == 64) CALL(32, 64)   \
  if (dqk == 32 && dv == 128) CALL(32, 128) \
  if (dqk == 64 && dv == 32) CALL(64, 32)   \
  if (dqk == 64 && dv == 64) CALL(64, 64)   \
  if (dqk == 64 && dv == 128) CALL(64, 128) \
  if (dqk == 128 && dv == 32) CALL(128, 32) \
  if (dqk == 128 && dv == 64) CALL(128, 64) \
  if (dqk == 128 && dv == 128) CALL(128, 128)

hipError_t launch_attn_fwd_f32(const JaggedArgs& ja, const Tensors& t, int dqk, int dv, void* out,
                               hipStream_t s) {
  if (ja.total_tokens <= 0) return hipSuccess;
#define CALL(A, B) return fwd_case<A, B>(ja, t, out, s);
  HSTU_F32_DISPATCH(CALL)
#undef CALL
  return hipErrorInvalidValue;
}

hipError_t launch_f64_to_f32_scaled(const double* in, float* out, int64_t n, double scale,
                                    hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(f64_to_f32_kernel, dim3((unsigned)(blocks < 1024 ? blocks : 1024)), dim3(256),
                     0, s, in, out, n, scale);
  return hipGetLastError();
}

hipError_t launch_attn_bwd_f32(const JaggedArgs& ja, const Tensors& t, int dqk, int dv,
                               const void* d_out, void* dq, void* dk, void* dv_out,
                               double* rab_pos_acc, double* rab_time_acc, hipStream_t s) {
  if (ja.total_tokens <= 0) return hipSuccess;
#define CALL(A, B) \
  return bwd_case<A, B>(ja, t, d_out, dq, dk, dv_out, rab_pos_acc, rab_time_acc, s);
  HSTU_F32_DISPATCH(CALL)
#undef CALL
  return hipErrorInvalidValue;
}

}  // namespace hstu
