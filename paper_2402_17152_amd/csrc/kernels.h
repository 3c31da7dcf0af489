// Host-side launchers of the libhstu kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.h"

namespace hstu {

// Everything an attention kernel needs to know about the jagged batch.
struct JaggedArgs {
  const int64_t* seq_offsets;
  const int64_t* timestamps;
  const int64_t* num_targets;  // may be null
  const float* rab_pos;
  const float* rab_time;
  // [2B] per-sequence timestamp min / max (workspace, filled by
  // launch_seq_time_range before the attention kernels run).
  const int64_t* seq_trange;
  // Cross mode (the cached candidate pass of M-FALCON): the rows of
  // sequence b are its candidates, all at position n_h, and the keys its
  // cached prefix, a jagged batch of its own (key_offsets [B+1],
  // key_timestamps); null for self-attention over seq_offsets.
  const int64_t* key_offsets;
  const int64_t* key_timestamps;
  int32_t num_seqs;
  int32_t max_seq_len;  // N
  int32_t num_heads;
  int32_t num_buckets;
  int64_t total_tokens;
};

struct Tensors {
  const void* q;
  int64_t q_stride;
  const void* k;
  int64_t k_stride;
  const void* v;
  int64_t v_stride;
};

// Tile sizes of the bf16 MFMA kernels.
constexpr int kFwdBM = 128;  // query rows per forward workgroup
constexpr int kFwdBN = 32;   // keys per forward step
constexpr int kBwdBN = 128;  // keys owned by a backward workgroup (4 waves x 32)
constexpr int kBwdBM = 32;   // query rows per backward step
constexpr size_t kLdsBytes = 160 * 1024;  // LDS a gfx950 workgroup may allocate

// Upper bound on the number of (sequence, block) work items for blocks of
// `blk` tokens: sum_b ceil(L_b / blk) <= ceil(T / blk) + B.
inline int64_t max_work_items(int64_t T, int32_t B, int blk) {
  return (T + blk - 1) / blk + B;
}

// Scheduler: builds the work list (longest first) into `items` and
// its length into `count`.  mode 0: forward (seq, q-block of kFwdBM rows;
// in cross mode the candidate rows in blocks of kFwdBM); mode 1: backward
// (seq, k-block of kBwdBN keys).
hipError_t launch_schedule(const JaggedArgs& ja, int mode, WorkItem* items, int32_t* count,
                           hipStream_t s);

hipError_t launch_fill_f32(float* p, int64_t n, float value, hipStream_t s);
// Per-sequence timestamp min / max into out[2b], out[2b+1] (0, 0 for an
// empty sequence).
hipError_t launch_seq_time_range(const JaggedArgs& ja, int64_t* out, hipStream_t s);
hipError_t launch_complete_cumsum(int32_t n, const int64_t* in, int64_t* out, int square_of_diff,
                                  hipStream_t s);
hipError_t launch_bucketize(int32_t num_seqs, int64_t total_tokens, int32_t num_buckets,
                            const int64_t* seq_offsets, const int64_t* timestamps,
                            const int64_t* pair_offsets, int64_t total_pairs, uint8_t* out,
                            hipStream_t s);

// bf16 MFMA attention.  The forward stores O as bf16, or as fp32 when
// out_f32; with split, P enters P V as two bf16 terms (the layer path).
// In cross mode (ja.key_offsets) the rows are candidates and the keys the
// cached prefix, without the candidates' own keys.
hipError_t launch_attn_fwd_bf16(const JaggedArgs& ja, const Tensors& t, int dqk, int dv, void* out,
                                int out_f32, int split, const WorkItem* items,
                                const int32_t* count, int64_t max_items, hipStream_t s);
// The self term of the cached candidate pass: out = o32 + SiLU(q.k +
// rab_pos[N-1] + rab_time[0]) v / N per (row, head), in bf16 or fp32.
hipError_t launch_cached_self(int is_bf16, int64_t T, int32_t H, int32_t dqk, int32_t dv,
                              const Tensors& t, const float* rab_pos, const float* rab_time,
                              int32_t N, const float* o32, void* out, hipStream_t s);
// d_out_lo: null, or the low bf16 terms of dO (d_out holding the high
// ones), for a dO that is the fp32 output of the layer's LayerNorm backward.
hipError_t launch_attn_bwd_bf16(const JaggedArgs& ja, const Tensors& t, int dqk, int dv,
                                const void* d_out, const void* d_out_lo, float* dq_acc, void* dk,
                                void* dv_out, float* d_rab_pos, float* d_rab_time,
                                const WorkItem* items, const int32_t* count, int64_t max_items,
                                hipStream_t s);
// fp32 head-major dQ accumulator [h][T][d] -> bf16 token-major [T][h][d], scaled.
hipError_t launch_dq_convert_bf16(const float* acc, void* dq, int64_t T, int32_t H, int32_t d,
                                  float scale, hipStream_t s);

// fp32 SIMT attention.
hipError_t launch_attn_fwd_f32(const JaggedArgs& ja, const Tensors& t, int dqk, int dv, void* out,
                               hipStream_t s);
hipError_t launch_attn_bwd_f32(const JaggedArgs& ja, const Tensors& t, int dqk, int dv,
                               const void* d_out, void* dq, void* dk, void* dv_out,
                               float* d_rab_pos, float* d_rab_time, hipStream_t s);

// Matrix-core rate probe (benchmark support): `waves_per_simd` waves per
// SIMD on every CU, each issuing iters x 8 independent bf16 32x32x16 MFMAs.
hipError_t launch_mfma_probe(int32_t iters, int32_t waves_per_simd, float* sink, double* flop,
                             hipStream_t s);

// Backward of LayerNorm(x) (.) u: du, dx (dense [T][D]) and, when non-null,
// dw / db accumulated into fp32 [D] (zeroed by the caller).  x is fp32;
// u, dy, du, dx are bf16 when is_bf16, else fp32; with is_bf16 and a
// non-null dx_lo, dx = bf16(v) and dx_lo = bf16(v - dx) hold the fp32 v
// as two terms.
hipError_t launch_ln_gate_bwd(int is_bf16, int64_t T, int32_t D, const void* x, const void* u,
                              int64_t u_stride, const void* dy, const float* w, const float* b,
                              const float* mean, const float* rstd, void* du, void* dx,
                              void* dx_lo, float* dw, float* db, hipStream_t s);

// LayerNorm(x) (.) u per token over D features; x fp32, u and y bf16 when
// is_bf16, else fp32.
hipError_t launch_ln_gate(int is_bf16, int64_t T, int32_t D, const void* x, const void* u,
                          int64_t u_stride, const float* w, const float* b, float eps, void* y,
                          float* mean, float* rstd, hipStream_t s);

}  // namespace hstu
