// Standalone timestamp bucketisation: materialises, for every sequence,
// the L x L matrix of time buckets bkt(t_i - t_j) (notation table, entry
// rab^{p,t}) as uint8, row-major, sequences concatenated at pair_offsets.
//
// HBM-write bound.  A workgroup owns 16 rows of one sequence and walks the
// columns in slabs of 2048 whose timestamps it stages in LDS.  When the
// timestamps of its rows and of the slab lie within 2^30 of the sequence's
// first one (always, for real event times), they are rebased to 32 bits
// and a pair costs one v_sad_u32 and one v_ffbh_u32; otherwise the exact
// 64-bit form runs.
// A wave writes one row segment at a time, each lane aligned dwords (4
// buckets) of the flat output, so a wave store covers 256 contiguous
// bytes; only the two end dwords of a segment use byte stores.  Rows start
// at any byte, so the slab is staged four times, shifted by 0..3 words:
// the copy matching the row's alignment gives every lane its 4 column
// timestamps in one aligned, bank-conflict-free 16-byte LDS read.
#include "bias.h"
#include "kernels.h"

namespace hstu {

namespace {

constexpr int kBktThreads = 256;
constexpr int kBktRows = 16;    // rows per workgroup
constexpr int kBktCols = 2048;  // columns staged per slab
constexpr int kBktLd = kBktCols + 4;

struct BktShared {
  union {
    uint32_t t32[4][kBktLd];  // copy k holds column x at index x + k
    int64_t t64[kBktCols];
  };
};

// |dt| < 2^31, so floor(log2) <= 30: the clamp matters only for B_t <= 31.
template <bool CLAMP>
__device__ __forceinline__ uint32_t bkt32(uint32_t ti, uint32_t tj, int nb) {
  uint32_t d;
  asm("v_sad_u32 %0, %1, %2, 0" : "=v"(d) : "v"(ti), "v"(tj));
  const int b = 31 - __clz((int)(d | 1u));
  return (uint32_t)(CLAMP ? min(b, nb - 1) : b);
}

template <bool CLAMP>
__device__ __forceinline__ void row_segment32(const BktShared& sm, uint32_t ti, int nb, int64_t P,
                                              int ncols, uint8_t* __restrict__ out, int lane) {
  // Flat bytes [P, P + ncols) hold columns 0 .. ncols-1 of the slab; dword
  // dw covers columns 4 dw - P .. +3.  Four dwords per lane and pass, 64
  // apart, keep every LDS read and store contiguous across the wave.
  const int64_t first = P >> 2, last = (P + ncols - 1) >> 2;
  const int k = (int)(P & 3);  // column 4 dw - P of copy k sits at 4 (dw - P / 4)
  const uint32_t* tk = sm.t32[k];
  // The two end dwords may hold bytes of neighbouring rows: byte stores.
  if (lane < 2 && (lane == 0 || last != first)) {
    const int64_t dw = lane ? last : first;
    const int j0 = (int)((dw << 2) - P);
    for (int e = 0; e < 4; e++) {
      const int j = j0 + e;
      if (j >= 0 && j < ncols) out[(dw << 2) + e] = (uint8_t)bkt32<CLAMP>(ti, tk[j + k], nb);
    }
  }
  // Interior dwords first+1 .. last-1, four per lane and pass; lanes past
  // the end redo the last one (same value to the same address), so the
  // pass has no branches and its four LDS reads are in flight together.
  // Interior dword a (from 0) starts at column 4a + c1, c1 = 4(first+1) - P
  // in [1, 4], and c1 + k = 4: its columns sit at tk[4a + 4 ..].
  const int n_int = (int)(last - first - 1);
  uint32_t* const seg = reinterpret_cast<uint32_t*>(out + ((first + 1) << 2));
  const uint32_t* const tc = tk + 4;
  for (int d0 = 0; d0 < n_int; d0 += 256) {
    int a[4];
    uint32_t v[4];
#pragma unroll
    for (int q = 0; q < 4; q++) {
      a[q] = min(d0 + lane + 64 * q, n_int - 1);
      const u32x4 tj = *reinterpret_cast<const u32x4*>(tc + 4 * a[q]);
      v[q] = bkt32<CLAMP>(ti, tj[0], nb) | bkt32<CLAMP>(ti, tj[1], nb) << 8 |
             bkt32<CLAMP>(ti, tj[2], nb) << 16 | bkt32<CLAMP>(ti, tj[3], nb) << 24;
    }
#pragma unroll
    for (int q = 0; q < 4; q++) seg[a[q]] = v[q];
  }
}

__device__ __forceinline__ void row_segment64(const BktShared& sm, int64_t ti, int nb, int64_t P,
                                              int ncols, uint8_t* __restrict__ out, int lane) {
  for (int j = lane; j < ncols; j += 64) out[P + j] = (uint8_t)time_bucket64(ti - sm.t64[j], nb);
}

__global__ __launch_bounds__(kBktThreads) void bucketize_kernel(
    int32_t num_seqs, int32_t nb, const int64_t* __restrict__ offs, const int64_t* __restrict__ ts,
    const int64_t* __restrict__ pair_offs, uint8_t* __restrict__ out) {
  __shared__ BktShared sm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int b = blockIdx.y; b < num_seqs; b += gridDim.y) {
    const int64_t o = offs[b];
    const int L = (int)(offs[b + 1] - o);
    const int r0 = blockIdx.x * kBktRows;
    if (r0 >= L) continue;  // uniform over the workgroup
    const int rows = min(kBktRows, L - r0);
    const int64_t* __restrict__ t = ts + o;
    const int64_t base = pair_offs[b];

    // 32-bit form: timestamps as offsets from t[0] + 2^30; it applies when
    // every offset the workgroup touches lies in [0, 2^31), so that two of
    // them differ by less than 2^31.  The next slab's timestamps are
    // loaded while the current one is bucketed.
    const int64_t t0 = t[0] - ((int64_t)1 << 30);
    auto in32 = [](int64_t d) { return d >= 0 && d < ((int64_t)1 << 31); };
    bool rows_ok = true;
    if (tid < rows) rows_ok = in32(t[r0 + tid] - t0);
    constexpr int kPer = kBktCols / kBktThreads;
    int64_t nxt[kPer];
#pragma unroll
    for (int e = 0; e < kPer; e++) nxt[e] = tid + e * kBktThreads < L ? t[tid + e * kBktThreads] : t0;
    for (int c0 = 0; c0 < L; c0 += kBktCols) {
      const int ncols = min(kBktCols, L - c0);
      int64_t cur[kPer];
      bool ok = rows_ok;
#pragma unroll
      for (int e = 0; e < kPer; e++) {
        cur[e] = nxt[e];
        ok = ok && in32(cur[e] - t0);
      }
      const bool fast = __syncthreads_and(ok);  // also: previous slab fully consumed
      if (fast) {
#pragma unroll
        for (int e = 0; e < kPer; e++) {
          const int x = tid + e * kBktThreads;
          const uint32_t v = (uint32_t)(cur[e] - t0);
#pragma unroll
          for (int k = 0; k < 4; k++) sm.t32[k][x + k] = v;
        }
      } else {
#pragma unroll
        for (int e = 0; e < kPer; e++) sm.t64[tid + e * kBktThreads] = cur[e];
      }
      __syncthreads();
      const int c1 = c0 + kBktCols;
#pragma unroll
      for (int e = 0; e < kPer; e++) {
        const int x = c1 + tid + e * kBktThreads;
        nxt[e] = x < L ? t[x] : t0;
      }
      for (int r = wave; r < rows; r += kBktThreads / 64) {
        const int i = r0 + r;
        const int64_t ti = t[i];
        const int64_t P = base + (int64_t)i * L + c0;
        if (!fast)
          row_segment64(sm, ti, nb, P, ncols, out, lane);
        else if (nb <= 31)
          row_segment32<true>(sm, (uint32_t)(ti - t0), nb, P, ncols, out, lane);
        else
          row_segment32<false>(sm, (uint32_t)(ti - t0), nb, P, ncols, out, lane);
      }
    }
    __syncthreads();  // the next sequence restages the slab
  }
}

}  // namespace

hipError_t launch_bucketize(int32_t num_seqs, int64_t total_tokens, int32_t num_buckets,
                            const int64_t* seq_offsets, const int64_t* timestamps,
                            const int64_t* pair_offsets, int64_t total_pairs, uint8_t* out,
                            hipStream_t s) {
  if (total_pairs <= 0 || num_seqs <= 0) return hipSuccess;
  // The longest sequence has L^2 <= total_pairs and L <= total_tokens;
  // workgroups past a sequence's rows return at once.
  int64_t lmax = (int64_t)sqrt((double)total_pairs);
  while (lmax * lmax > total_pairs) lmax--;
  while ((lmax + 1) * (lmax + 1) <= total_pairs) lmax++;
  lmax = min(lmax, total_tokens);
  const dim3 grid((unsigned)((lmax + kBktRows - 1) / kBktRows), (unsigned)min(num_seqs, 65535));
  hipLaunchKernelGGL(bucketize_kernel, grid, dim3(kBktThreads), 0, s, num_seqs, num_buckets,
                     seq_offsets, timestamps, pair_offsets, out);
  return hipGetLastError();
}

}  // namespace hstu
