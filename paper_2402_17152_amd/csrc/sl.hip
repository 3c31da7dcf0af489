// Stochastic Length (Eq. 4 and the subsequence selection appendix): shrinks
// a jagged batch before attention.  A sequence whose history (the tokens
// before its candidates) has n_h > L tokens keeps it whole with
// probability N_c^alpha / n_h^2 (the draw u_keep[b] and the numerator
// N_c^alpha are inputs) and otherwise
// keeps exactly L history tokens: those with the L smallest selection keys
// (equal keys: the later token first), in their original order.  The
// candidates always follow.  The result is a gather list of original
// token indices and the new offsets.
//
// Keys (the random draws e_rand are Exp(1) variates supplied by the
// caller): greedy = t_max - t_i (elapsed time, an integer); random = e_i;
// feature-weighted = e_i / (F - f_i), F = sum of f = t_max - t_i over the
// history, which orders the items as the exponential-race keys e_i / w_i
// of weighted sampling without replacement with w_i = 1 - f_i / F.  Keys
// are non-negative, so their bit patterns order like their values, and
// one workgroup per sequence finds the L-th smallest by an 8-pass radix
// select over the 64-bit patterns (LDS histograms of 8-bit digits), then
// writes the chosen indices in order with block prefix sums.
#include "kernels.h"

namespace hstu {

namespace {

constexpr int kSlThreads = 256;

__global__ __launch_bounds__(256) void sl_lengths_kernel(int32_t B,
                                                         const int64_t* __restrict__ offs,
                                                         const int64_t* __restrict__ nt, int32_t L,
                                                         double keep_num,
                                                         const double* __restrict__ u_keep,
                                                         int64_t* __restrict__ new_len,
                                                         int32_t* __restrict__ whole) {
  for (int b = blockIdx.x * 256 + threadIdx.x; b < B; b += gridDim.x * 256) {
    const int64_t n = offs[b + 1] - offs[b];
    const int64_t t = nt ? nt[b] : 0;
    const int64_t nh = n - t;
    const bool w = nh <= L || u_keep[b] < keep_num / ((double)nh * (double)nh);
    new_len[b] = w ? n : (int64_t)L + t;
    whole[b] = w ? 1 : 0;
  }
}

__device__ __forceinline__ uint64_t dbits(double x) { return (uint64_t)__double_as_longlong(x); }

struct SlKey {
  const int64_t* ts;
  const double* e;
  int64_t tmax, F;
  int mode;
  __device__ __forceinline__ uint64_t operator()(int i) const {
    const int64_t f = tmax - ts[i];
    if (mode == kSlGreedy) return (uint64_t)f;
    const double ei = e[i] > 0.0 ? e[i] : 0.0;
    if (mode == kSlRandom) return dbits(ei);
    if (F == 0) return dbits(ei);
    const int64_t den = F - f;
    if (den == 0) return dbits(__builtin_inf());
    return dbits(ei / (double)den);
  }
};

// Exclusive prefix count of `flag` over the 256 threads in thread order;
// *total receives the block's count.  Uses sc[0..3].
__device__ __forceinline__ int block_excl_count(bool flag, int* sc, int* total) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t m = __ballot(flag);
  const int below = __popcll(m & ((lane ? (~0ull >> (64 - lane)) : 0ull)));
  if (lane == 0) sc[wave] = __popcll(m);
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < 4; w++) {
    before += w < wave ? sc[w] : 0;
    tot += sc[w];
  }
  __syncthreads();
  *total = tot;
  return before + below;
}

__global__ __launch_bounds__(kSlThreads) void sl_select_kernel(
    int32_t B, const int64_t* __restrict__ offs, const int64_t* __restrict__ ts,
    const int64_t* __restrict__ nt, int32_t L, int32_t mode, const double* __restrict__ e_rand,
    const int32_t* __restrict__ whole, const int64_t* __restrict__ new_offs,
    int64_t* __restrict__ gather) {
  __shared__ int hist[256];
  __shared__ int sc[4];
  __shared__ int64_t red[2][4];
  __shared__ uint64_t s_prefix;
  __shared__ int s_k, s_eq;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int b = blockIdx.x; b < B; b += gridDim.x) {
    const int64_t o = offs[b];
    const int n = (int)(offs[b + 1] - o);
    const int t = nt ? (int)nt[b] : 0;
    const int nh = n - t;
    int64_t* out = gather + new_offs[b];
    if (whole[b]) {
      for (int i = tid; i < n; i += kSlThreads) out[i] = o + i;
      continue;
    }
    // Candidates follow the L chosen history tokens.
    for (int c = tid; c < t; c += kSlThreads) out[L + c] = o + nh + c;

    // t_max and (feature-weighted) F = sum of t_max - t_i over the history.
    const int64_t* th = ts + o;
    int64_t mx = (int64_t)(~0ull >> 1) * -1 - 1;
    for (int i = tid; i < nh; i += kSlThreads) mx = th[i] > mx ? th[i] : mx;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const int64_t x = __shfl_xor(mx, off, 64);
      mx = x > mx ? x : mx;
    }
    if (lane == 0) red[0][wave] = mx;
    __syncthreads();
    const int64_t tmax = max(max(red[0][0], red[0][1]), max(red[0][2], red[0][3]));
    int64_t F = 0;
    if (mode == kSlWeighted) {
      int64_t sum = 0;
      for (int i = tid; i < nh; i += kSlThreads) sum += tmax - th[i];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off, 64);
      if (lane == 0) red[1][wave] = sum;
      __syncthreads();
      F = red[1][0] + red[1][1] + red[1][2] + red[1][3];
    }
    const SlKey key{th, e_rand ? e_rand + o : nullptr, tmax, F, mode};

    // Radix select: after pass p the top 8(p+1) bits of the L-th smallest
    // key are known; k is its rank among the keys sharing those bits.
    uint64_t prefix = 0;
    int k = L, eq = 0;
    for (int p = 0; p < 8; p++) {
      const int shift = 56 - 8 * p;
      const uint64_t hi_mask = p == 0 ? 0ull : ~((1ull << (shift + 8)) - 1ull);
      hist[tid] = 0;
      __syncthreads();
      for (int i = tid; i < nh; i += kSlThreads) {
        const uint64_t kv = key(i);
        if ((kv & hi_mask) == prefix) atomicAdd(&hist[(kv >> shift) & 255], 1);
      }
      __syncthreads();
      if (tid == 0) {
        int before = 0, d = 0;
        while (d < 255 && before + hist[d] < k) before += hist[d++];
        s_prefix = prefix | ((uint64_t)d << shift);
        s_k = k - before;
        s_eq = hist[d];
      }
      __syncthreads();
      prefix = s_prefix;
      k = s_k;
      eq = s_eq;
      __syncthreads();
    }
    // prefix = the L-th smallest key; eq tokens carry it, of which the k
    // with the largest indices are chosen (with every smaller key).
    const int skip_eq = eq - k;
    int seen_eq = 0, written = 0;
    for (int c0 = 0; c0 < nh; c0 += kSlThreads) {
      const int i = c0 + tid;
      const uint64_t kv = i < nh ? key(i) : ~0ull;
      const bool is_eq = i < nh && kv == prefix;
      int tot_eq, tot_sel;
      const int eq_before = seen_eq + block_excl_count(is_eq, sc, &tot_eq);
      const bool sel = i < nh && (kv < prefix || (is_eq && eq_before >= skip_eq));
      const int pos = written + block_excl_count(sel, sc, &tot_sel);
      if (sel && pos < L) out[pos] = o + i;
      seen_eq += tot_eq;
      written += tot_sel;
    }
    __syncthreads();
  }
}

// dst row r = src row index[r] for r < *count (count read on the device).
__global__ __launch_bounds__(256) void gather_rows_kernel(const char* __restrict__ src,
                                                          int64_t src_stride, int64_t words,
                                                          int wbytes,
                                                          const int64_t* __restrict__ index,
                                                          const int64_t* __restrict__ count,
                                                          int64_t max_rows, char* __restrict__ dst,
                                                          int64_t dst_stride) {
  const int64_t rows = min(*count, max_rows);
  const int64_t total = rows * words;
  for (int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x; x < total;
       x += (int64_t)gridDim.x * 256) {
    const int64_t r = x / words, w = x - r * words;
    const char* s = src + index[r] * src_stride + w * wbytes;
    char* d = dst + r * dst_stride + w * wbytes;
    if (wbytes == 16)
      *reinterpret_cast<u32x4*>(d) = *reinterpret_cast<const u32x4*>(s);
    else
      *reinterpret_cast<uint32_t*>(d) = *reinterpret_cast<const uint32_t*>(s);
  }
}

}  // namespace

hipError_t launch_sl_lengths(int32_t B, const int64_t* offs, const int64_t* nt, int32_t L,
                             double keep_num, const double* u_keep, int64_t* new_len,
                             int32_t* whole, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  const int blocks = (B + 255) / 256 < 1024 ? (B + 255) / 256 : 1024;
  hipLaunchKernelGGL(sl_lengths_kernel, dim3(blocks), dim3(256), 0, s, B, offs, nt, L, keep_num,
                     u_keep,
                     new_len, whole);
  return hipGetLastError();
}

hipError_t launch_sl_select(int32_t B, const int64_t* offs, const int64_t* ts, const int64_t* nt,
                            int32_t L, int32_t mode, const double* e_rand, const int32_t* whole,
                            const int64_t* new_offs, int64_t* gather, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(sl_select_kernel, dim3((unsigned)(B < 65535 ? B : 65535)), dim3(kSlThreads), 0,
                     s, B, offs, ts, nt, L, mode, e_rand, whole, new_offs, gather);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const void* src, int64_t src_stride, int64_t row_bytes,
                              const int64_t* index, const int64_t* count, int64_t max_rows,
                              void* dst, int64_t dst_stride, hipStream_t s) {
  if (max_rows <= 0 || row_bytes <= 0) return hipSuccess;
  const bool v16 = row_bytes % 16 == 0 && src_stride % 16 == 0 && dst_stride % 16 == 0 &&
                   (uintptr_t)src % 16 == 0 && (uintptr_t)dst % 16 == 0;
  const int wb = v16 ? 16 : 4;
  const int64_t words = row_bytes / wb;
  const int64_t total = max_rows * words;
  const int64_t blocks = (total + 255) / 256;
  hipLaunchKernelGGL(gather_rows_kernel, dim3((unsigned)(blocks < 8192 ? blocks : 8192)),
                     dim3(256), 0, s, (const char*)src, src_stride, words, wb, index, count,
                     max_rows, (char*)dst, dst_stride);
  return hipGetLastError();
}

}  // namespace hstu
