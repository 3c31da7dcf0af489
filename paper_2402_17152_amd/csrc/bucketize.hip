// Standalone timestamp bucketisation: materialises, for every sequence,
// the L x L matrix of time buckets bkt(t_i - t_j) (notation table, entry
// rab^{p,t}) as uint8, row-major, sequences concatenated at pair_offsets.
//
// HBM-write bound.  A workgroup owns 48 consecutive tokens of the batch,
// i.e. 48 rows of one sequence (or the rows of two or more sequences that
// meet inside the block), and walks the columns in slabs of 8192 (whole
// rows, for sequences up to that length) whose timestamps it stages in
// LDS.  When the
// timestamps of its rows and of the slab lie within 2^30 of the sequence's
// first one (always, for real event times), they are rebased to 32 bits
// and a pair costs v_sad_u32, v_ffbh_u32 and one saturating subtract that
// writes the bucket straight into its byte of the output dword (SDWA);
// otherwise the exact 64-bit form runs.
// A row segment is written as aligned 16-byte chunks, one per lane (a wave
// store covers 1 KB), plus at most 15 bytes at each end, written one byte
// per lane.  A chunk needs the timestamps of 16 consecutive columns: the
// slab is staged twice, shifted by 0 and 1 words, so that the copy
// matching the row's alignment holds them as four aligned 16-byte words
// (or, for half of the alignments, eight 8-byte words), and each copy
// inserts one padding word-quad every 64 entries, so that the lanes of a
// read (64 bytes apart) spread over the LDS banks.
#include "bias.h"
#include "kernels.h"

namespace hstu {

namespace {

constexpr int kBktThreads = 256;
constexpr int kBktRows = 48;    // rows per workgroup
constexpr int kBktCols = 8192;  // columns staged per slab
// Entry y of a copy sits at y + 4 (y >> kPadShift); y <= kBktCols.
constexpr int kPadShift = 6;
__device__ __forceinline__ int bkt_pidx(int y) { return y + 4 * (y >> kPadShift); }
constexpr int kBktLd = ((kBktCols + 2) + 4 * ((kBktCols + 2) / (1 << kPadShift) + 1) + 3) / 4 * 4;
// Entries 1024 further on (64 chunks of 16) sit this many words further.
constexpr int kChunkStep = 1024 + 4 * (1024 >> kPadShift);

struct __align__(16) BktShared {
  union {
    uint32_t t32[2][kBktLd];  // copy s holds column x at bkt_pidx(x + s)
    int64_t t64[kBktCols];
  };
  int64_t rowt[kBktRows];     // the workgroup's row timestamps
};

// Leading-zero count of |ti - tj| < 2^31 (0xffffffff for 0), raised to
// zmin = 32 - nb when CLAMP (nb <= 31), so that the saturating 31 - z
// below is min(floor(log2 |dt|), nb - 1), and 0 for |dt| <= 1.
template <bool CLAMP>
__device__ __forceinline__ uint32_t lz32(uint32_t ti, uint32_t tj, uint32_t zmin) {
  uint32_t d, z;
  asm("v_sad_u32 %0, %1, %2, 0" : "=v"(d) : "v"(ti), "v"(tj));
  asm("v_ffbh_u32 %0, %1" : "=v"(z) : "v"(d));
  if constexpr (CLAMP) z = z > zmin ? z : zmin;  // 0xffffffff stays
  return z;
}

// Four buckets packed little-endian into one dword: byte 0 by a saturating
// subtract, bytes 1-3 by the same subtract writing its byte in place (SDWA).
template <bool CLAMP>
__device__ __forceinline__ uint32_t bkt4(uint32_t ti, uint32_t a, uint32_t b, uint32_t c,
                                         uint32_t d, uint32_t zmin, uint32_t c31) {
  const uint32_t z0 = lz32<CLAMP>(ti, a, zmin), z1 = lz32<CLAMP>(ti, b, zmin);
  const uint32_t z2 = lz32<CLAMP>(ti, c, zmin), z3 = lz32<CLAMP>(ti, d, zmin);
  uint32_t r;
  asm("v_sub_u32_e64 %0, 31, %1 clamp" : "=v"(r) : "v"(z0));
  asm("v_sub_u32_sdwa %0, %1, %2 clamp dst_sel:BYTE_1 dst_unused:UNUSED_PRESERVE "
      "src0_sel:DWORD src1_sel:DWORD"
      : "+v"(r) : "v"(c31), "v"(z1));
  asm("v_sub_u32_sdwa %0, %1, %2 clamp dst_sel:BYTE_2 dst_unused:UNUSED_PRESERVE "
      "src0_sel:DWORD src1_sel:DWORD"
      : "+v"(r) : "v"(c31), "v"(z2));
  asm("v_sub_u32_sdwa %0, %1, %2 clamp dst_sel:BYTE_3 dst_unused:UNUSED_PRESERVE "
      "src0_sel:DWORD src1_sel:DWORD"
      : "+v"(r) : "v"(c31), "v"(z3));
  return r;
}

template <bool CLAMP>
__device__ __forceinline__ void row_segment32(const BktShared& sm, uint32_t ti, int nb, int64_t P,
                                              int ncols, uint8_t* __restrict__ out, int lane) {
  // Flat bytes [P, P + ncols) hold columns 0 .. ncols-1 of the slab;
  // relative to P: the head [0, hend), nch aligned 16-byte chunks from h =
  // (16 - P) mod 16, and the tail [tstart, ncols) (at most 15 bytes each).
  const uint32_t zmin = CLAMP ? (uint32_t)(32 - nb) : 0u;
  const uint32_t c31 = 31u;
  const int64_t cfirst = (P + 15) >> 4;
  const int h = (int)((cfirst << 4) - P);
  const int nch = max(0, (int)(((P + ncols) >> 4) - cfirst));
  const int hend = min(h, ncols), tstart = max(hend, h + 16 * nch);
  uint8_t* const row = out + P;
  // End bytes: lanes 0-15 the head, lanes 32-47 the tail (copy 0).
  {
    const int r = lane < 32 ? lane : tstart + (lane - 32);
    const bool on = lane < 32 ? lane < hend : (lane < 48 && r < ncols);
    if (on) {
      const uint32_t z = lz32<CLAMP>(ti, sm.t32[0][bkt_pidx(r)], zmin);
      uint32_t b;
      asm("v_sub_u32_e64 %0, 31, %1 clamp" : "=v"(b) : "v"(z));
      row[r] = (uint8_t)b;
    }
  }
  if (lane >= nch) return;
  // Chunk a covers columns h + 16 a .. +15, entries y .. y + 15 of copy
  // s = P mod 2 with y = h + 16 a + s: a multiple of 4 when P mod 4 < 2
  // (16-byte reads), else 2 mod 4 (8-byte reads).  Moving 64 chunks on
  // adds 1024 entries, 16 whole pad periods: the offsets of the reads
  // from the first stay fixed and the first moves by 1088.
  const int k = (int)(P & 3), sc = k & 1;
  const int y = h + sc + 16 * lane;
  const int p0 = bkt_pidx(y);
  const uint32_t* src = sm.t32[sc] + p0;
  u32x4* dst = reinterpret_cast<u32x4*>(row + h + 16 * lane);
  if (k < 2) {
    const int d1 = bkt_pidx(y + 4) - p0, d2 = bkt_pidx(y + 8) - p0, d3 = bkt_pidx(y + 12) - p0;
    for (int a = lane; a < nch; a += 64) {
      const u32x4 t0 = *reinterpret_cast<const u32x4*>(src);
      const u32x4 t1 = *reinterpret_cast<const u32x4*>(src + d1);
      const u32x4 t2 = *reinterpret_cast<const u32x4*>(src + d2);
      const u32x4 t3 = *reinterpret_cast<const u32x4*>(src + d3);
      u32x4 v;
      v[0] = bkt4<CLAMP>(ti, t0[0], t0[1], t0[2], t0[3], zmin, c31);
      v[1] = bkt4<CLAMP>(ti, t1[0], t1[1], t1[2], t1[3], zmin, c31);
      v[2] = bkt4<CLAMP>(ti, t2[0], t2[1], t2[2], t2[3], zmin, c31);
      v[3] = bkt4<CLAMP>(ti, t3[0], t3[1], t3[2], t3[3], zmin, c31);
      *dst = v;
      src += kChunkStep;
      dst += 64;
    }
  } else {
    int dd[8];
#pragma unroll
    for (int m = 0; m < 8; m++) dd[m] = bkt_pidx(y + 2 * m) - p0;
    for (int a = lane; a < nch; a += 64) {
      uint2 t[8];
#pragma unroll
      for (int m = 0; m < 8; m++) t[m] = *reinterpret_cast<const uint2*>(src + dd[m]);
      u32x4 v;
#pragma unroll
      for (int q = 0; q < 4; q++)
        v[q] = bkt4<CLAMP>(ti, t[2 * q].x, t[2 * q].y, t[2 * q + 1].x, t[2 * q + 1].y, zmin, c31);
      *dst = v;
      src += kChunkStep;
      dst += 64;
    }
  }
}

__device__ __forceinline__ void row_segment64(const BktShared& sm, int64_t ti, int nb, int64_t P,
                                              int ncols, uint8_t* __restrict__ out, int lane) {
  for (int j = lane; j < ncols; j += 64) out[P + j] = (uint8_t)time_bucket64(ti - sm.t64[j], nb);
}

// Rows r0 .. r0 + rows - 1 of one sequence (timestamps t, length L, pairs
// from base), every column.
__device__ __forceinline__ void bucketize_rows(BktShared& sm, int nb, const int64_t* __restrict__ t,
                                               int L, int64_t base, int r0, int rows,
                                               uint8_t* __restrict__ out, int tid, int wave,
                                               int lane) {
  // 32-bit form: timestamps as offsets from t[0] - 2^30; it applies when
  // every offset the workgroup touches lies in [0, 2^31), so that two of
  // them differ by less than 2^31.  A slab's timestamps are loaded before
  // any output of that slab is stored: loads and stores share the wave's
  // memory counter, so a load issued after stores would wait for them.
  const int64_t t0 = t[0] - ((int64_t)1 << 30);
  auto in32 = [](int64_t d) { return d >= 0 && d < ((int64_t)1 << 31); };
  bool rows_ok = true;
  if (tid < rows) {
    const int64_t tr = t[r0 + tid];
    sm.rowt[tid] = tr;
    rows_ok = in32(tr - t0);
  }
  constexpr int kPer = kBktCols / kBktThreads;
  for (int c0 = 0; c0 < L; c0 += kBktCols) {
    const int ncols = min(kBktCols, L - c0);
    // Rebased low words, kept only if the whole workgroup passes (the
    // 64-bit form reloads the values).
    uint32_t cur[kPer];
    bool ok = rows_ok;
#pragma unroll
    for (int e = 0; e < kPer; e++) {
      const int x = tid + e * kBktThreads;
      const int64_t d = (x < ncols ? t[c0 + x] : t0) - t0;
      ok = ok && in32(d);
      cur[e] = (uint32_t)d;
    }
    const bool fast = __syncthreads_and(ok);  // also: previous slab fully consumed
    if (fast) {
#pragma unroll
      for (int e = 0; e < kPer; e++) {
        const int x = tid + e * kBktThreads;
        sm.t32[0][bkt_pidx(x)] = cur[e];
        sm.t32[1][bkt_pidx(x + 1)] = cur[e];
      }
    } else {
      for (int e = 0; e < kPer; e++) {
        const int x = tid + e * kBktThreads;
        sm.t64[x] = x < ncols ? t[c0 + x] : t0;
      }
    }
    __syncthreads();
    // Row set-up is wave-uniform (scalar unit).
    for (int r = wave; r < rows; r += kBktThreads / 64) {
      const int64_t ti = ((int64_t)__builtin_amdgcn_readfirstlane((int)(sm.rowt[r] >> 32)) << 32) |
                         (uint32_t)__builtin_amdgcn_readfirstlane((int)sm.rowt[r]);
      const int64_t P = base + (int64_t)(r0 + r) * L + c0;
      if (!fast)
        row_segment64(sm, ti, nb, P, ncols, out, lane);
      else if (nb <= 31)
        row_segment32<true>(sm, (uint32_t)(ti - t0), nb, P, ncols, out, lane);
      else
        row_segment32<false>(sm, (uint32_t)(ti - t0), nb, P, ncols, out, lane);
    }
    __syncthreads();  // the slab (or the row timestamps) is restaged next
  }
}

// Workgroup g covers tokens [48 g, 48 g + 48) of the concatenated batch:
// the rows of the sequence(s) those tokens belong to, every column.
__global__ __launch_bounds__(kBktThreads) void bucketize_kernel(
    int32_t num_seqs, int64_t total_tokens, int32_t nb, const int64_t* __restrict__ offs,
    const int64_t* __restrict__ ts, const int64_t* __restrict__ pair_offs,
    uint8_t* __restrict__ out) {
  __shared__ BktShared sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  for (int64_t g = blockIdx.x; g * kBktRows < total_tokens; g += gridDim.x) {
    int64_t R0 = g * kBktRows;
    const int64_t R1 = min(R0 + kBktRows, total_tokens);
    // b = the last sequence with offs[b] <= R0 (offsets are non-decreasing).
    int lo = 0, hi = num_seqs - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (offs[mid] <= R0) lo = mid; else hi = mid - 1;
    }
    for (int b = lo; b < num_seqs && R0 < R1; b++) {
      const int64_t o = offs[b], e = offs[b + 1];
      if (e <= R0) continue;  // empty sequence
      const int rows = (int)(min(e, R1) - R0);
      bucketize_rows(sm, nb, ts + o, (int)(e - o), pair_offs[b], (int)(R0 - o), rows, out, tid,
                     wave, lane);
      R0 += rows;
    }
  }
}

}  // namespace

hipError_t launch_bucketize(int32_t num_seqs, int64_t total_tokens, int32_t num_buckets,
                            const int64_t* seq_offsets, const int64_t* timestamps,
                            const int64_t* pair_offsets, int64_t total_pairs, uint8_t* out,
                            hipStream_t s) {
  if (total_pairs <= 0 || num_seqs <= 0 || total_tokens <= 0) return hipSuccess;
  const int64_t blocks = (total_tokens + kBktRows - 1) / kBktRows;
  const unsigned grid = (unsigned)min(blocks, (int64_t)1 << 30);
  hipLaunchKernelGGL(bucketize_kernel, dim3(grid), dim3(kBktThreads), 0, s, num_seqs, total_tokens,
                     num_buckets, seq_offsets, timestamps, pair_offsets, out);
  return hipGetLastError();
}

}  // namespace hstu
