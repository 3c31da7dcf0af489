// Standalone timestamp bucketisation: materialises, for every sequence,
// the L x L matrix of time buckets bkt(t_i - t_j) (notation table, entry
// rab^{p,t}) as uint8, row-major, sequences concatenated at pair_offsets.
//
// HBM-write bound.  Each thread owns one 16-byte aligned chunk of the
// flat output, so every store is a full aligned 16-byte store no matter
// how rows and sequences fall; the (sequence, row, column) of the chunk's
// first byte comes from one binary search and one division, and the
// remaining bytes advance incrementally.
#include "kernels.h"

namespace hstu {

namespace {

__global__ __launch_bounds__(256) void bucketize_kernel(int32_t num_seqs, int32_t nb,
                                                        const int64_t* __restrict__ offs,
                                                        const int64_t* __restrict__ ts,
                                                        const int64_t* __restrict__ pair_offs,
                                                        int64_t total, uint8_t* __restrict__ out) {
  const int64_t nchunks = (total + 15) / 16;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < nchunks; c += stride) {
    const int64_t p = c * 16;
    // last b with pair_offs[b] <= p  (skips empty sequences)
    int lo = 0, hi = num_seqs;  // invariant: pair_offs[lo] <= p < pair_offs[hi]
    while (hi - lo > 1) {
      int mid = (lo + hi) >> 1;
      if (pair_offs[mid] <= p) lo = mid; else hi = mid;
    }
    int b = lo;
    int64_t o = offs[b];
    int64_t L = offs[b + 1] - o;
    int64_t local = p - pair_offs[b];
    int64_t i = local / L, j = local - i * L;
    int64_t ti = ts[o + i];
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    const int nbytes = (int)min((int64_t)16, total - p);
    for (int e = 0; e < nbytes; e++) {
      uint32_t bk = (uint32_t)time_bucket64(ti - ts[o + j], nb);
      w[e >> 2] |= bk << (8 * (e & 3));
      if (e + 1 == nbytes) break;  // advance only while bytes remain
      if (++j == L) {
        j = 0;
        if (++i == L) {
          // Bytes remain, so a later non-empty sequence exists: take the
          // first one (its pair offset is exactly p + e + 1).
          do {
            ++b;
          } while (offs[b + 1] == offs[b]);
          o = offs[b];
          L = offs[b + 1] - o;
          i = 0;
        }
        ti = ts[o + i];
      }
    }
    if (nbytes == 16) {
      uint4 v = make_uint4(w[0], w[1], w[2], w[3]);
      *reinterpret_cast<uint4*>(out + p) = v;
    } else {
      for (int e = 0; e < nbytes; e++) out[p + e] = (uint8_t)(w[e >> 2] >> (8 * (e & 3)));
    }
  }
}

}  // namespace

hipError_t launch_bucketize(int32_t num_seqs, int32_t num_buckets, const int64_t* seq_offsets,
                            const int64_t* timestamps, const int64_t* pair_offsets,
                            int64_t total_pairs, uint8_t* out, hipStream_t s) {
  if (total_pairs <= 0) return hipSuccess;
  int64_t nchunks = (total_pairs + 15) / 16;
  int64_t g = (nchunks + 255) / 256;
  if (g > 1 << 20) g = 1 << 20;
  hipLaunchKernelGGL(bucketize_kernel, dim3((unsigned)g), dim3(256), 0, s, num_seqs, num_buckets,
                     seq_offsets, timestamps, pair_offsets, total_pairs, out);
  return hipGetLastError();
}

}  // namespace hstu
