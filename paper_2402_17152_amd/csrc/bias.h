// Relative-bias helpers shared by the bf16 attention kernels.
//
// rab(i,j) = rab_pos[(N-1) + p(j) - p(i)] + rab_time[bkt(t_i - t_j)]
// (notation table, entry rab^{p,t}).  The time bucket
// bkt(x) = min(B_t - 1, floor(log2(max(|x|, 1)))) is handled through its
// "slot" s = 63 - floor(log2(max(|x|, 1))) = clz64(|x| | 1) in [0, 63]:
// the rab_time lookup becomes a 64-entry table indexed by slot
// (tab[s] = rab_time[min(63 - s, B_t - 1)]) and the gradient is summed
// per slot and folded onto buckets when it is flushed.
//
// Fast path: when every timestamp a workgroup touches lies within 2^31 of
// the smallest one, timestamps are rebased to 32-bit offsets and
// |t_i - t_j| is one v_sad_u32; clz of a 32-bit value plus 32 is the
// 64-bit clz.  Otherwise the exact 64-bit form is used.
#pragma once

#include "common.h"

namespace hstu {

__device__ __forceinline__ int slot64(int64_t dt) {
  uint64_t a = dt < 0 ? (uint64_t)0 - (uint64_t)dt : (uint64_t)dt;
  return __clzll((long long)(a | 1ull));
}

// |a - b| < 2^31 for rebased 32-bit timestamps.
__device__ __forceinline__ int slot32(uint32_t a, uint32_t b) {
  return 32 + __clz((int)(__usad(a, b, 0u) | 1u));
}

// Slot range [s_lo, s_hi] covering every |t_i - t_j| with t_i in
// [rlo, rhi] and t_j in [klo, khi].
__device__ __forceinline__ void slot_range(int64_t rlo, int64_t rhi, int64_t klo, int64_t khi,
                                           int& s_lo, int& s_hi) {
  int64_t dmin, dmax;
  if (rlo >= khi) {
    dmin = rlo - khi;
    dmax = rhi - klo;
  } else if (klo >= rhi) {
    dmin = klo - rhi;
    dmax = khi - rlo;
  } else {
    dmin = 0;
    dmax = max(rhi - klo, khi - rlo);
  }
  s_lo = slot64(dmax);
  s_hi = slot64(dmin);
}

// Whole-wave reductions on DPP (no LDS round trip): butterflies within
// rows of 16 lanes, then row_bcast:15 / row_bcast:31 fold the four rows
// into lane 63, which is read back as a scalar.
template <int CTRL, int ROW_MASK, typename T>
__device__ __forceinline__ T dpp_mov(T identity, T x) {
  return __builtin_bit_cast(T, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, identity),
                                                           __builtin_bit_cast(int, x), CTRL,
                                                           ROW_MASK, 0xf, false));
}

template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce_dpp(T x, T identity, Op op) {
  static_assert(sizeof(T) == 4, "32-bit values");
  x = op(x, dpp_mov<0xb1, 0xf>(identity, x));   // quad_perm [1,0,3,2]
  x = op(x, dpp_mov<0x4e, 0xf>(identity, x));   // quad_perm [2,3,0,1]
  x = op(x, dpp_mov<0x141, 0xf>(identity, x));  // row_half_mirror
  x = op(x, dpp_mov<0x140, 0xf>(identity, x));  // row_mirror
  x = op(x, dpp_mov<0x142, 0xa>(identity, x));  // row_bcast:15 into rows 1 and 3
  x = op(x, dpp_mov<0x143, 0xc>(identity, x));  // row_bcast:31 into rows 2 and 3
  return __builtin_bit_cast(T, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 63));
}

__device__ __forceinline__ float wave_sum_dpp(float v) {
  return wave_reduce_dpp(v, 0.0f, [](float a, float b) { return a + b; });
}
__device__ __forceinline__ uint32_t wave_min_dpp(uint32_t v) {
  return wave_reduce_dpp(v, 0xffffffffu, [](uint32_t a, uint32_t b) { return a < b ? a : b; });
}
__device__ __forceinline__ uint32_t wave_max_dpp(uint32_t v) {
  return wave_reduce_dpp(v, 0u, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
}

__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ int64_t wave_min_i64(int64_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    int64_t o = __shfl_xor(v, off, 64);
    v = o < v ? o : v;
  }
  return v;
}

__device__ __forceinline__ int64_t wave_max_i64(int64_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    int64_t o = __shfl_xor(v, off, 64);
    v = o > v ? o : v;
  }
  return v;
}

// Transposing LDS read (ds_read_b64_tr_b16): in each group of 16 lanes,
// lane 16g + k receives element k % 4 of the 4-element rows addressed by
// lanes 16g + k/4 + 4e, e = 0..3.  Used to fetch an MFMA operand whose
// contraction index runs down the rows of a row-major LDS tile.
__device__ __forceinline__ uint2 lds_read_tr16(const uint16_t* p) {
  typedef short v4i16 __attribute__((ext_vector_type(4)));
  v4i16 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)p);
  return __builtin_bit_cast(uint2, r);
}

}  // namespace hstu
