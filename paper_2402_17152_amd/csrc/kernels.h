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
  // launch_prep before the attention kernels run).
  const int64_t* seq_trange;
  // Cross mode (the cached candidate pass of M-FALCON): the rows of
  // sequence b are its candidates, all at position n_h, and the keys its
  // cached prefix, a jagged batch of its own (key_offsets [B+1],
  // key_timestamps); null for self-attention over seq_offsets.
  const int64_t* key_offsets;
  const int64_t* key_timestamps;
  // Cross mode: the prefix keys of a candidate block are split into chunks
  // of kCrossChunk keys, one work item each (blk = q-block * key_chunks +
  // chunk); chunk c writes its fp32 partial output at out + c * chunk_stride.
  int32_t key_chunks;
  int64_t chunk_stride;
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
constexpr int kCrossChunk = 512;  // prefix keys per cross-mode work item (16 steps)
constexpr int kBwdBN = 128;  // keys owned by a backward workgroup (4 waves x 32)
constexpr int kBwdBM = 32;   // query rows per backward step
constexpr size_t kLdsBytes = 160 * 1024;  // LDS a gfx950 workgroup may allocate

// Upper bound on the number of (sequence, block) work items for blocks of
// `blk` tokens: sum_b ceil(L_b / blk) <= ceil(T / blk) + B.
inline int64_t max_work_items(int64_t T, int32_t B, int blk) {
  return (T + blk - 1) / blk + B;
}

// Up to three float arrays an attention call zeroes before its main kernel.
struct PrepFills {
  float* ptr[3];
  int64_t count[3];
  int n;
};

// The work an attention call does before its main kernel, in one launch:
//  - the scheduler: the work list (longest first) into `items` and its
//    length into `count`; mode 0: forward (seq, q-block of kFwdBM rows;
//    in cross mode the candidate rows in blocks of kFwdBM), mode 1:
//    backward (seq, k-block of kBwdBN keys);
//  - per-sequence timestamp min / max into trange[2b], trange[2b+1] (0, 0
//    for an empty sequence);
//  - zeroing the arrays in `fills`;
//  - if `bases` is set, the slot tables of the two-role backward's partial
//    dQ blocks (int64 [2 (B + 1)]: row-block and partial-slot prefixes).
hipError_t launch_prep(const JaggedArgs& ja, int mode, WorkItem* items, int32_t* count,
                       int64_t* trange, const PrepFills& fills, int64_t* bases, hipStream_t s);

hipError_t launch_fill_f32(float* p, int64_t n, float value, hipStream_t s);
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
// The self term of the cached candidate pass: out = (sum over the row's
// key chunks, in order, of the fp32 partials at o32 + c * ja.chunk_stride)
// + SiLU(q.k + rab_pos[N-1] + rab_time[0]) v / N per (row, head), in bf16
// (at most 64 heads).  ja: the cross-mode arguments (seq_offsets of the
// candidates, key_offsets, key_chunks, chunk_stride, num_seqs, max_seq_len,
// rab tables).
hipError_t launch_cached_self(const JaggedArgs& ja, int32_t dqk, int32_t dv, const Tensors& t,
                              const float* o32, void* out, hipStream_t s);
// Whether the two-term (d_out_lo) backward of these head sizes runs the
// two-role kernel (its LDS holds the low terms for d_qk, d_v <= 64) or
// the single-role one.
constexpr bool bwd_split_two_role(int dqk, int dv) { return dqk <= 64 && dv <= 64; }

// d_out_lo: null, or the low bf16 terms of dO (d_out holding the high
// ones), for a dO that is the fp32 output of the layer's LayerNorm backward.
// The two-role kernel (d_out_lo null, or bwd_split_two_role) stores dQ as
// scaled f16 partial blocks in dq_part / dq_scale (slots from `bases`;
// launch_dq_reduce_bf16 sums them); the single-role kernel adds dQ to the
// zeroed fp32 dq_acc [h][T][d_qk] with atomics (launch_dq_convert_bf16 then).
hipError_t launch_attn_bwd_bf16(const JaggedArgs& ja, const Tensors& t, int dqk, int dv,
                                const void* d_out, const void* d_out_lo, float* dq_acc,
                                uint16_t* dq_part, float* dq_scale, int64_t dq_slots,
                                const int64_t* bases, void* dk, void* dv_out, float* d_rab_pos,
                                float* d_rab_time, const WorkItem* items, const int32_t* count,
                                int64_t max_items, hipStream_t s);
// dQ of the two-role backward (d_out_lo null): sums the f16 partial
// blocks in dq_part times their scales in dq_scale (slots laid out by the
// bases launch_prep writes) into bf16 dq [T][h][d_qk], scaled by 1/N.
// dq_slots: the slots the buffer holds; both kernels skip slots past it,
// which only sequences longer than N (a data error) can reach.
hipError_t launch_dq_reduce_bf16(const JaggedArgs& ja, int dqk, const uint16_t* dq_part,
                                 const float* dq_scale, int64_t dq_slots, const int64_t* bases,
                                 void* dq, hipStream_t s);
// Partial-slot count bound of the two-role backward (32-row steps of every
// 128-key block): sum over sequences of K S - 2 K (K - 1), K = ceil(L/128),
// S = ceil(L/32), bounded from T, B and N alone.
inline int64_t dq_part_slots_bound(int64_t T, int32_t B, int32_t N) {
  return (N * T + 254 * T + 16129 * (int64_t)B + 8191) / 8192 + (T + 127 * (int64_t)B + 63) / 64 +
         B;
}
// fp32 head-major dQ accumulator [h][T][d] -> bf16 token-major [T][h][d], scaled.
hipError_t launch_dq_convert_bf16(const float* acc, void* dq, int64_t T, int32_t H, int32_t d,
                                  float scale, hipStream_t s);

// fp32 SIMT attention.
hipError_t launch_attn_fwd_f32(const JaggedArgs& ja, const Tensors& t, int dqk, int dv, void* out,
                               hipStream_t s);
// The bias gradients are added, unscaled (sums of dS), to fp64
// accumulators that the caller zeroes and converts.
hipError_t launch_attn_bwd_f32(const JaggedArgs& ja, const Tensors& t, int dqk, int dv,
                               const void* d_out, void* dq, void* dk, void* dv_out,
                               double* rab_pos_acc, double* rab_time_acc, hipStream_t s);
// out[i] = (float)(in[i] * scale), i < n.
hipError_t launch_f64_to_f32_scaled(const double* in, float* out, int64_t n, double scale,
                                    hipStream_t s);

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

// ---- dense products of the linear maps f_1 (Eq. 1) and f_2 (Eq. 3) ----
// C[m][n] = sum_k A(m, k) B(n, k).  Epilogues: kEpiSilu stores
// SiLU(acc + bias) to c and, if c2, the pre-activation acc + bias to c2;
// kEpiAdd stores acc (+ bias) (+ res); kEpiSlab stores the fp32 partial of
// contraction split blockIdx.y to slab[split][M][N].
enum { kEpiSilu = 1, kEpiAdd = 2, kEpiSlab = 3 };

// bf16 operands.  A k-contiguous: element (m, k) at a[m * lda + k]; k-major:
// a[k * lda + m] (likewise B with n).  Requirements (checked by the
// callers): K a multiple of 64 for a k-contiguous operand and a single
// split; the contiguous dimension of a k-major operand a multiple of 8;
// N a multiple of 8; every byte offset of an operand below 2^31; the
// output row strides multiples of 8 elements.
struct GemmArgs {
  const uint16_t* a;
  int64_t lda;
  const uint16_t* b;
  int64_t ldb;
  int32_t M, N, K;
  int32_t k_split;  // contraction rows per split (multiple of 64)
  const float* bias;
  const uint16_t* res;
  int64_t ldr;
  uint16_t* c;
  int64_t ldc;
  uint16_t* c2;
  int64_t ldc2;
  float* slab;
};
hipError_t launch_gemm_bf16(const GemmArgs& g, int a_kmajor, int b_kmajor, int epi, int splits,
                            hipStream_t s);
// Contraction splits for a k-major x k-major product of M x N outputs over
// K rows: about 512 workgroups, at least 256 rows per split.
int gemm_num_splits(int M, int N, int64_t K, int* k_split);

// fp32 operands with arbitrary element strides (A(m, k) = a[m sam + k sak],
// B(n, k) = b[n sbn + k sbk]); kEpiSlab stores the plain product to c.
struct GemmArgsF32 {
  const float* a;
  int64_t sam, sak;
  const float* b;
  int64_t sbn, sbk;
  int32_t M, N, K;
  const float* bias;
  const float* res;
  int64_t ldr;
  float* c;
  int64_t ldc;
  float* c2;
  int64_t ldc2;
};
hipError_t launch_gemm_f32(const GemmArgsF32& g, int epi, hipStream_t s);

// dpre = [dU|dV|dQ|dK] * SiLU'(pre) ([T][F], dtype of the problem; the
// gradients dense [T][h][d], hv = h d_v, hq = h d_qk) and partial column
// sums of dpre, [colsum_blocks(T)][F] fp32.
int64_t colsum_blocks(int64_t T);
hipError_t launch_silu_bwd(int is_bf16, int64_t T, int F, int hv, int hq, const void* pre,
                           const void* du, const void* dv, const void* dq, const void* dk,
                           void* dpre, float* partial, hipStream_t s);
// Partial column sums of x [T][N] (row stride ld; N and ld multiples of
// 8): [colsum_blocks(T)][N].  Activations 16-byte aligned.
hipError_t launch_colsum(int is_bf16, int64_t T, int N, int64_t ld, const void* x, float* partial,
                         hipStream_t s);
// out[i] = sum_s part[s][i] (s = 0 .. S-1 in order), i < n.
hipError_t launch_reduce_slabs(int64_t n, int S, const float* part, float* out, hipStream_t s);
// The same fixed-order-per-group sum for many rows S and few columns n
// (bias partials): 16 row groups per column, then the groups in order.
hipError_t launch_reduce_cols(int n, int S, const float* part, float* out, hipStream_t s);

// ---- Stochastic Length (Eq. 4) ----
enum { kSlGreedy = 0, kSlRandom = 1, kSlWeighted = 2 };
// new_len[b] and whole[b] (1: the sequence stays whole) per sequence.
hipError_t launch_sl_lengths(int32_t B, const int64_t* offs, const int64_t* nt, int32_t L,
                             double keep_num, const double* u_keep, int64_t* new_len,
                             int32_t* whole, hipStream_t s);
// gather[new_offs[b] ..] = the original indices a sequence keeps.
hipError_t launch_sl_select(int32_t B, const int64_t* offs, const int64_t* ts, const int64_t* nt,
                            int32_t L, int32_t mode, const double* e_rand, const int32_t* whole,
                            const int64_t* new_offs, int64_t* gather, hipStream_t s);
// dst row r = src row index[r], r < min(*count, max_rows); strides in bytes.
hipError_t launch_gather_rows(const void* src, int64_t src_stride, int64_t row_bytes,
                              const int64_t* index, const int64_t* count, int64_t max_rows,
                              void* dst, int64_t dst_stride, hipStream_t s);

}  // namespace hstu
