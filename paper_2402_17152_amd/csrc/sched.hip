// Jagged tile scheduler and small utility kernels.
//
// The scheduler turns the jagged batch into a list of (sequence, block)
// work items for the attention kernels -- the grouped computation over
// unpadded sequences of the paper (Sec. 3.2; appendix on the fused kernels):
// no padding, causally empty tiles never become work.  Items are written
// longest-first (counting sort by tile count) so that the hardware
// dispatcher, which hands out workgroups in index order, starts the
// longest items first.
#include "kernels.h"

namespace hstu {

namespace {

constexpr int kSchedThreads = 1024;

__device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Forward item (q-block qb): number of key tiles of kFwdBN the forward
// kernel visits.  Key tiles made only of candidates that lie before the
// block's first row are fully masked and skipped.
__device__ __forceinline__ int fwd_weight(int L, int n_h, int qb) {
  int i0 = qb * kFwdBM;
  int rows_end = min(i0 + kFwdBM, L);
  int kend = ceil_div(rows_end, kFwdBN);
  int skipped = max(0, i0 / kFwdBN - ceil_div(n_h, kFwdBN));
  return kend - skipped;
}

// Cross-mode forward item: key chunk c of a candidate block visits keys
// [c kCrossChunk, min(n_h, (c + 1) kCrossChunk)) of the cached prefix.
__device__ __forceinline__ int cross_weight(int n_h, int c) {
  return ceil_div(min(kCrossChunk, n_h - c * kCrossChunk), kFwdBN);
}

// Backward item (k-block kb): number of query steps of kBwdBM rows.
__device__ __forceinline__ int bwd_weight(int L, int n_h, int kb) {
  int j0 = kb * kBwdBN;
  int i_end = j0 >= n_h ? min(j0 + kBwdBN, L) : L;
  return ceil_div(i_end - j0, kBwdBM);
}

// One workgroup of kSchedThreads builds the whole list; s_bins holds
// maxw + 1 ints (dynamic LDS), s_scan kSchedThreads.
__device__ void schedule_block(const JaggedArgs& ja, int mode, WorkItem* items, int32_t* count,
                               int* s_bins, int* s_scan) {
  const int tid = threadIdx.x;
  const int blk = mode == 0 ? kFwdBM : kBwdBN;
  const int maxw = mode == 0 ? ceil_div(ja.max_seq_len, kFwdBN) : ceil_div(ja.max_seq_len, kBwdBM);
  // (cross mode: a chunk's weight is at most kCrossChunk / kFwdBN <= maxw)
  const int nbins = maxw + 1;
  for (int i = tid; i < nbins; i += kSchedThreads) s_bins[i] = 0;
  __syncthreads();

  // Sequences are handed to groups of G lanes (G a power of two up to a
  // wave, larger for fewer sequences); a group's lanes share its items.
  int G = 1;
  while (G < 64 && G * ja.num_seqs < kSchedThreads) G <<= 1;
  const int group = tid / G, sub = tid % G, ngroups = kSchedThreads / G;
  // Calls f(seq, block, weight) for every item.
  auto for_items = [&](auto&& f) {
    for (int b = group; b < ja.num_seqs; b += ngroups) {
      const int L = (int)(ja.seq_offsets[b + 1] - ja.seq_offsets[b]);
      int n_h = L - (ja.num_targets ? (int)ja.num_targets[b] : 0);
      const bool cross = mode == 0 && ja.key_offsets;
      if (cross) n_h = (int)(ja.key_offsets[b + 1] - ja.key_offsets[b]);
      const int nblk = ceil_div(L, blk);
      // (chunks past key_chunks exist only if n_h >= N: they are not scheduled)
      const int nch = cross ? min(ceil_div(n_h, kCrossChunk), ja.key_chunks) : 1;
      for (int e = sub; e < nblk * nch; e += G) {
        const int x = e / nch, c = e - x * nch;
        int w = cross       ? cross_weight(n_h, c)
                : mode == 0 ? fwd_weight(L, n_h, x)
                            : bwd_weight(L, n_h, x);
        w = min(max(w, 0), maxw);
        f(b, cross ? x * ja.key_chunks + c : x, w);
      }
    }
  };

  // Pass 1: histogram of item weights (bin index = maxw - weight, so that
  // an ascending scan orders items by descending weight).
  for_items([&](int, int, int w) { atomicAdd(&s_bins[maxw - w], 1); });
  __syncthreads();

  // Exclusive scan of the bins: each thread owns a contiguous run.
  const int per = ceil_div(nbins, kSchedThreads);
  const int lo = tid * per, hi = min(lo + per, nbins);
  int local = 0;
  for (int i = lo; i < hi; i++) local += s_bins[i];
  s_scan[tid] = local;
  __syncthreads();
  for (int off = 1; off < kSchedThreads; off <<= 1) {
    int v = tid >= off ? s_scan[tid - off] : 0;
    __syncthreads();
    s_scan[tid] += v;
    __syncthreads();
  }
  int run = s_scan[tid] - local;
  for (int i = lo; i < hi; i++) {
    int c = s_bins[i];
    s_bins[i] = run;
    run += c;
  }
  if (tid == kSchedThreads - 1) *count = s_scan[tid];
  __syncthreads();

  // Pass 2: scatter the items to their sorted positions.
  for_items([&](int b, int x, int w) {
    const int pos = atomicAdd(&s_bins[maxw - w], 1);
    WorkItem it;
    it.seq = b;
    it.blk = x;
    items[pos] = it;
  });
}

__global__ void fill_f32_kernel(float* p, int64_t n, float value) {
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = value;
}

// out[0] = 0, out[i+1] = out[i] + x_i; x_i = in[i], or (in[i+1]-in[i])^2
// when square_of_diff (pair offsets of the bucket matrices).
__global__ __launch_bounds__(kSchedThreads) void cumsum_kernel(int32_t n, const int64_t* in,
                                                               int64_t* out, int square_of_diff) {
  __shared__ int64_t s[kSchedThreads];
  const int tid = threadIdx.x;
  int64_t carry = 0;
  if (tid == 0) out[0] = 0;
  for (int32_t base = 0; base < n; base += kSchedThreads) {
    int32_t i = base + tid;
    int64_t x = 0;
    if (i < n) {
      if (square_of_diff) {
        int64_t d = in[i + 1] - in[i];
        x = d * d;
      } else {
        x = in[i];
      }
    }
    s[tid] = x;
    __syncthreads();
    for (int off = 1; off < kSchedThreads; off <<= 1) {
      int64_t v = tid >= off ? s[tid - off] : 0;
      __syncthreads();
      s[tid] += v;
      __syncthreads();
    }
    if (i < n) out[i + 1] = carry + s[tid];
    int64_t total = s[kSchedThreads - 1];
    __syncthreads();
    carry += total;
  }
}

// acc is head-major [h][T][d] (fp32), dq token-major [T][h][d] (bf16);
// one thread per 4 features.
__global__ void dq_convert_kernel(const float* __restrict__ acc, uint16_t* __restrict__ dq,
                                  int64_t T, int32_t H, int32_t d4, float scale) {
  const int64_t n4 = T * H * d4;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    const int64_t row = i / d4;  // t * H + h
    const int64_t c = i - row * d4;
    const int64_t t = row / H, h = row - t * H;
    f32x4 a = reinterpret_cast<const f32x4*>(acc)[(h * T + t) * d4 + c];
    uint32_t lo = pack_bf16x2(a[0] * scale, a[1] * scale);
    uint32_t hi = pack_bf16x2(a[2] * scale, a[3] * scale);
    reinterpret_cast<uint2*>(dq)[i] = make_uint2(lo, hi);
  }
}

int grid_for(int64_t n, int threads) {
  int64_t g = (n + threads - 1) / threads;
  if (g > 65536) g = 65536;
  return (int)(g < 1 ? 1 : g);
}

// Per-sequence timestamp extremes (one workgroup per sequence; eight
// independent loads in flight per thread).  The attention kernels use them
// to pick 32-bit rebased time arithmetic when a sequence spans < 2^31.
__device__ void time_range_block(const JaggedArgs& ja, int b, int64_t* out,
                                 int64_t (*red)[kSchedThreads / 64]) {
  const int tid = threadIdx.x;
  const int64_t o = ja.seq_offsets[b];
  const int L = (int)(ja.seq_offsets[b + 1] - o);
  const int64_t* ts = ja.timestamps + o;
  int64_t lo = 0x7fffffffffffffffll, hi = -0x7fffffffffffffffll - 1;
  for (int x0 = 0; x0 < L; x0 += 8 * kSchedThreads) {
    int64_t v[8];
#pragma unroll
    for (int k = 0; k < 8; k++) v[k] = ts[min(x0 + k * kSchedThreads + tid, L - 1)];
#pragma unroll
    for (int k = 0; k < 8; k++) {
      lo = v[k] < lo ? v[k] : lo;
      hi = v[k] > hi ? v[k] : hi;
    }
  }
  // Cross mode: the cached prefix's timestamps count too.
  int Lk = 0;
  if (ja.key_offsets) {
    const int64_t ok = ja.key_offsets[b];
    Lk = (int)(ja.key_offsets[b + 1] - ok);
    const int64_t* tk = ja.key_timestamps + ok;
    for (int x = tid; x < Lk; x += kSchedThreads) {
      const int64_t v = tk[x];
      lo = v < lo ? v : lo;
      hi = v > hi ? v : hi;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const int64_t a = __shfl_xor(lo, off, 64), c = __shfl_xor(hi, off, 64);
    lo = a < lo ? a : lo;
    hi = c > hi ? c : hi;
  }
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = lo;
    red[1][tid >> 6] = hi;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kSchedThreads / 64; w++) {
      lo = red[0][w] < lo ? red[0][w] : lo;
      hi = red[1][w] > hi ? red[1][w] : hi;
    }
    out[2 * b] = L + Lk > 0 ? lo : 0;
    out[2 * b + 1] = L + Lk > 0 ? hi : 0;
  }
}

// Zero fills: fill block f of nf covers a grid-stride share of every job.
__device__ void fill_blocks(const PrepFills& fills, int f, int nf) {
  const int64_t stride = (int64_t)nf * kSchedThreads;
  for (int k = 0; k < fills.n; k++) {
    float* p = fills.ptr[k];
    const int64_t n = fills.count[k];
    int64_t done = 0;
    if (((uintptr_t)p & 15) == 0) {
      const int64_t n4 = n / 4;
      const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
      for (int64_t i = (int64_t)f * kSchedThreads + threadIdx.x; i < n4; i += stride)
        reinterpret_cast<f32x4*>(p)[i] = z;
      done = 4 * n4;
    }
    for (int64_t i = done + (int64_t)f * kSchedThreads + threadIdx.x; i < n; i += stride)
      p[i] = 0.0f;
  }
}

// Slot tables of the two-role backward's partial dQ blocks: bases[b] =
// sum over b' < b of ceil(L/32) (row blocks), bases[B + 1 + b] = sum over
// b' < b of K S - 2 K (K - 1) with K = ceil(L/128), S = ceil(L/32) (the
// 32-row steps of all 128-key blocks of a sequence).
__device__ void bases_block(const JaggedArgs& ja, int64_t* bases, int64_t (*s)[kSchedThreads]) {
  const int tid = threadIdx.x, B = ja.num_seqs;
  int64_t* rbase = bases;
  int64_t* pbase = bases + B + 1;
  if (tid == 0) {
    rbase[0] = 0;
    pbase[0] = 0;
  }
  int64_t carry_r = 0, carry_p = 0;
  for (int base = 0; base < B; base += kSchedThreads) {
    const int b = base + tid;
    int64_t r = 0, q = 0;
    if (b < B) {
      const int64_t L = ja.seq_offsets[b + 1] - ja.seq_offsets[b];
      const int64_t S = (L + kBwdBM - 1) / kBwdBM, K = (L + kBwdBN - 1) / kBwdBN;
      r = S;
      q = K * S - 2 * K * (K - 1);
    }
    s[0][tid] = r;
    s[1][tid] = q;
    __syncthreads();
    for (int off = 1; off < kSchedThreads; off <<= 1) {
      const int64_t a = tid >= off ? s[0][tid - off] : 0;
      const int64_t c = tid >= off ? s[1][tid - off] : 0;
      __syncthreads();
      s[0][tid] += a;
      s[1][tid] += c;
      __syncthreads();
    }
    if (b < B) {
      rbase[b + 1] = carry_r + s[0][tid];
      pbase[b + 1] = carry_p + s[1][tid];
    }
    carry_r += s[0][kSchedThreads - 1];
    carry_p += s[1][kSchedThreads - 1];
    __syncthreads();
  }
}

// Everything an attention call needs before its main kernel, in one
// launch: workgroup 0 builds the work list, workgroups 1..B take one
// sequence's timestamp range each, the next ones zero the fills, and (if
// `bases` is set) the last one writes the backward's slot tables.
__global__ __launch_bounds__(kSchedThreads) void prep_kernel(JaggedArgs ja, int mode,
                                                             WorkItem* items, int32_t* count,
                                                             int64_t* trange, PrepFills fills,
                                                             int nfill_blocks, int64_t* bases) {
  extern __shared__ int s_bins[];  // [maxw + 1]
  __shared__ int s_scan[kSchedThreads];
  __shared__ int64_t red[2][kSchedThreads / 64];
  __shared__ int64_t s_bases[2][kSchedThreads];
  const int g = (int)blockIdx.x;
  if (g == 0) {
    schedule_block(ja, mode, items, count, s_bins, s_scan);
  } else if (g <= ja.num_seqs) {
    time_range_block(ja, g - 1, trange, red);
  } else if (g <= ja.num_seqs + nfill_blocks) {
    fill_blocks(fills, g - 1 - ja.num_seqs, nfill_blocks);
  } else {
    bases_block(ja, bases, s_bases);
  }
}

}  // namespace

hipError_t launch_prep(const JaggedArgs& ja, int mode, WorkItem* items, int32_t* count,
                       int64_t* trange, const PrepFills& fills, int64_t* bases, hipStream_t s) {
  const int maxw = mode == 0 ? (ja.max_seq_len + kFwdBN - 1) / kFwdBN
                             : (ja.max_seq_len + kBwdBM - 1) / kBwdBM;
  const size_t lds = sizeof(int) * (size_t)(maxw + 1);
  int64_t work4 = 0;
  for (int k = 0; k < fills.n; k++) work4 += (fills.count[k] + 3) / 4;
  // About four float4 stores per thread for large fills, at most 1024 blocks.
  int64_t nf = (work4 + 4 * kSchedThreads - 1) / (4 * kSchedThreads);
  nf = nf > 1024 ? 1024 : nf;
  if (work4 > 0 && nf < 1) nf = 1;
  const int64_t grid = 1 + (int64_t)ja.num_seqs + nf + (bases ? 1 : 0);
  hipLaunchKernelGGL(prep_kernel, dim3((unsigned)grid), dim3(kSchedThreads), lds, s, ja, mode,
                     items, count, trange, fills, (int)nf, bases);
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, int64_t n, float value, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_f32_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, p, n, value);
  return hipGetLastError();
}

hipError_t launch_complete_cumsum(int32_t n, const int64_t* in, int64_t* out, int square_of_diff,
                                  hipStream_t s) {
  hipLaunchKernelGGL(cumsum_kernel, dim3(1), dim3(kSchedThreads), 0, s, n, in, out,
                     square_of_diff);
  return hipGetLastError();
}

hipError_t launch_dq_convert_bf16(const float* acc, void* dq, int64_t T, int32_t H, int32_t d,
                                  float scale, hipStream_t s) {
  const int64_t n4 = T * H * (d / 4);  // d is a multiple of 32
  if (n4 <= 0) return hipSuccess;
  hipLaunchKernelGGL(dq_convert_kernel, dim3(grid_for(n4, 256)), dim3(256), 0, s, acc,
                     (uint16_t*)dq, T, H, d / 4, scale);
  return hipGetLastError();
}

}  // namespace hstu
