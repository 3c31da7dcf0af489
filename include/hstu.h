/*
 * hstu.h -- C ABI of libhstu: the HSTU layer's jagged pointwise attention
 * for AMD Instinct MI355X (gfx950).
 *
 * Operation (Zhai et al., "Actions Speak Louder than Words", ICML 2024):
 *   Eq. 2  A(X)V(X) = SiLU(Q K^T + rab^{p,t}) V, with the pointwise
 *          aggregation of Sec. 3.1 normalised by the constant N
 *          (= max_seq_len) instead of a softmax, no 1/sqrt(d) scaling;
 *   rab^{p,t} (notation table) is shared by all heads:
 *          rab(i,j) = rab_pos[(N-1) + p(j) - p(i)] + rab_time[bkt(t_i - t_j)],
 *          bkt(x) = min(B_t - 1, floor(log2(max(|x|, 1))));
 *   mask   causal with the diagonal; with n_t = num_targets[b] > 0 the
 *          last n_t tokens of a sequence are candidates that see the
 *          n_h = L_b - n_t history tokens and themselves only, and all sit
 *          at position p = n_h (Algorithm 1, M-FALCON mask);
 *   Eq. 3  Y_pre = LayerNorm(A V) (.) U, layer norm over the h*d_v
 *          features of a token, biased variance, optional affine;
 *   backward: recomputes attention and bias (appendix on the fused
 *          kernels) and produces dQ, dK, dV and the gradients of both
 *          bias tables, summed over heads and sequences.
 *
 * Conventions
 *   Memory   every pointer is DEVICE memory owned by the caller unless a
 *            comment says "host".  The library keeps no pointer after a
 *            call returns and allocates no device memory; scratch space
 *            comes from the caller's workspace (hstu_workspace_bytes).
 *            Outputs must not alias inputs.
 *   Layout   jagged, token-major: sequence b owns tokens
 *            [seq_offsets[b], seq_offsets[b+1]).  Q/K/V/U rows: row r of X
 *            starts at X + r * x_stride (in elements); inside a row the
 *            layout is [h][d] contiguous, so Q/K/V/U may be strided views
 *            of one fused projection output [U | V | Q | K] (notation
 *            table, entry Split).  Outputs are dense [T][h][d].
 *            Every Q/K/V/U/O/dO pointer is 16-byte aligned and every
 *            stride a multiple of 16 bytes; max_seq_len rows of any
 *            input span at most 2 GiB (max_seq_len * stride * element
 *            size <= 2^31, else HSTU_ERR_UNSUPPORTED).
 *   Streams  all work is enqueued on hip_stream (a hipStream_t, NULL =
 *            the null stream) and the call returns before it completes.
 *            Only hstu_validate synchronises.
 *   Errors   host-side argument checks run before any launch; on failure
 *            the call returns a non-zero hstu_status_t, sets
 *            hstu_last_error() and enqueues nothing.  A failed launch
 *            returns HSTU_ERR_HIP.  Device-data preconditions
 *            (offsets monotone from 0 to T, L_b <= N, 0 <= n_t <= L_b,
 *            timestamps in [0, 2^62)) are not checked by the hot calls;
 *            breaking them is undefined.  hstu_validate checks them.
 *   Precision HSTU_F32: fp32 storage and arithmetic (the bias-table
 *            gradients are summed in fp64 and stored as fp32).  Its
 *            kernels are plain SIMT loops, one thread per (token, head),
 *            meant for small problems and as an fp32 reference: every shape
 *            the ABI accepts runs, but long sequences are slow (the matrix
 *            cores serve HSTU_BF16 only).  HSTU_BF16: bf16 storage, fp32
 *            accumulation; in hstu_attn_fwd / hstu_attn_bwd the attention
 *            weights and dS are rounded to bf16 (nearest-even) where they
 *            enter the matrix cores; hstu_layer_fwd / hstu_layer_bwd carry
 *            them, and the layer's dO, as two bf16 terms (hi + lo, about
 *            2^-17 relative instead of 2^-9).  Bias tables and their
 *            gradients are fp32; offsets and timestamps int64.
 *   Determinism  hstu_attn_fwd, hstu_layer_fwd, hstu_time_bucketize and
 *            hstu_complete_cumsum are bitwise deterministic, and so are
 *            dQ, dK and dV of hstu_attn_bwd for HSTU_BF16 (dQ is summed
 *            from per-key-block partials in a fixed order), and of
 *            hstu_layer_bwd for HSTU_BF16 with d_qk, d_v <= 64.  The bias
 *            gradients, the layer-norm parameter gradients, and dQ of
 *            hstu_layer_bwd at d_qk or d_v = 128 are accumulated with
 *            atomics, so their last bits may vary between runs.
 */
#ifndef HSTU_H_
#define HSTU_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HSTU_ABI_VERSION 1

typedef enum {
  HSTU_OK = 0,
  HSTU_ERR_INVALID_ARGUMENT = 1, /* null pointer, bad size or stride      */
  HSTU_ERR_UNSUPPORTED = 2,      /* a shape the library has no kernel for */
  HSTU_ERR_WORKSPACE = 3,        /* workspace missing or too small        */
  HSTU_ERR_HIP = 4,              /* a HIP runtime call failed             */
  HSTU_ERR_DATA = 5              /* hstu_validate found bad device data   */
} hstu_status_t;

typedef enum { HSTU_F32 = 0, HSTU_BF16 = 1 } hstu_dtype_t;

/* Host-side shape of one jagged batch; nothing is read back from the
 * device to fill it. */
typedef struct {
  int32_t num_seqs;         /* B >= 1                                           */
  int64_t total_tokens;     /* T == seq_offsets[B] (0 allowed)                  */
  int32_t max_seq_len;      /* N >= 1: normaliser 1/N; rab_pos has 2N-1 entries;
                               every L_b <= N.  Supported: N <= 65536          */
  int32_t num_heads;        /* h in [1, 64]                                     */
  int32_t d_qk, d_v;        /* head sizes, each in {32, 64, 128}                */
  int32_t num_time_buckets; /* B_t in [1, 256]                                  */
  hstu_dtype_t dtype;       /* storage of Q, K, V, U, O, Y, dO, dQ, dK, dV      */
} hstu_problem_t;

/* Device arrays describing the jagged structure and the bias tables. */
typedef struct {
  const int64_t* seq_offsets; /* [B+1]: 0 = o_0 <= o_1 <= ... <= o_B = T        */
  const int64_t* timestamps;  /* [T]: each in [0, 2^62)                         */
  const int64_t* num_targets; /* [B] or NULL (all 0): 0 <= n_t,b <= L_b         */
  const float* rab_pos;       /* [2N-1]: entry (N-1)+p(j)-p(i)                  */
  const float* rab_time;      /* [B_t]: entry bkt(t_i - t_j)                    */
} hstu_jagged_t;

/* Bytes of device workspace the attention calls need for problem p (host
 * pointer).  0 only if p is invalid.  One workspace of this size serves
 * every call below for the same shape; it may be reused between calls
 * on one stream but not by calls that overlap.  For HSTU_BF16 it holds
 * the backward's partial dQ blocks: about (N T / 8192 + T / 20) h d_qk
 * 64 bytes at most (bounded from T, B and N alone), after the layer
 * backward's dO terms (4 T h d_v bytes): 1.7 GB for T = 48118, N = 8192,
 * h = 4, d_qk = d_v = 128. */
size_t hstu_workspace_bytes(const hstu_problem_t* p);

/* Eq. 2 forward: out[t][a][:] = (1/N) sum_{j kept} SiLU(q.k + rab) v_j.
 * q, k: rows of h*d_qk elements at q_stride / k_stride; v: h*d_v at
 * v_stride; out: dense [T][h][d_v], overwritten (rows of empty sequences
 * do not exist; every token row is written). */
hstu_status_t hstu_attn_fwd(const hstu_problem_t* p, const hstu_jagged_t* j,
                            const void* q, int64_t q_stride,
                            const void* k, int64_t k_stride,
                            const void* v, int64_t v_stride,
                            void* out, void* ws, size_t ws_bytes,
                            void* hip_stream);

/* hstu_attn_fwd without a workspace, for callers that cannot allocate
 * device memory (code under stream capture, serving loops that forbid
 * allocation).  Same arguments, result and determinism as hstu_attn_fwd
 * minus ws / ws_bytes; the call itself allocates nothing.  The forward's
 * scratch (work list, its length, per-sequence timestamp ranges) lives in
 * one static device array of HSTU_NOALLOC_SCRATCH_BYTES per GPU, held from
 * the library's first call on that GPU until the process ends; the prep
 * launch rewrites all of it on every call, so nothing carries over between
 * calls.  Limit: the bf16 path needs 256 + 8 (ceil(T / 128) + B) + 16 B
 * bytes (each term rounded up to 256) within that size, about 6.6 * 10^7
 * tokens for B = 1024; a larger problem returns HSTU_ERR_UNSUPPORTED
 * without launching anything (the fp32 path uses no scratch).  All calls on
 * one GPU share the array: two calls that overlap in time on that GPU (on
 * different streams, or from different host threads without ordering)
 * race and may return wrong results. */
#define HSTU_NOALLOC_SCRATCH_BYTES (4u << 20)
hstu_status_t hstu_attn_fwd_noalloc(const hstu_problem_t* p, const hstu_jagged_t* j,
                                    const void* q, int64_t q_stride,
                                    const void* k, int64_t k_stride,
                                    const void* v, int64_t v_stride,
                                    void* out, void* hip_stream);

/* M-FALCON cached candidate pass (Algorithm 1, one microbatch; the
 * encoder-level cache of the appendix on M-FALCON): the attention output
 * of a microbatch of ranking candidates against the cached keys and
 * values of their users' histories, without recomputing the histories.
 * j describes the candidates: sequence b owns candidate rows
 * [seq_offsets[b], seq_offsets[b+1]) of q, k, v (as in hstu_attn_fwd) and
 * their timestamps; j->num_targets is ignored.  The histories form a
 * jagged batch of their own: cache_offsets [B+1] (device), history b having
 * n_b = cache_offsets[b+1] - cache_offsets[b] tokens, cache_timestamps
 * [cache_tokens], and the history K and V rows k_cache, v_cache (h*d_qk
 * and h*d_v elements at kc_stride / vc_stride), e.g. the k and v of an
 * hstu_attn_fwd call over the histories.  Every candidate sits at
 * position n_b and sees all n_b history keys and itself, no other
 * candidate: out (dense [T][h][d_v], T = candidate rows) equals the
 * candidate rows of hstu_attn_fwd over history ++ candidates with
 * num_targets = the candidate count (the target-aware mask), for any
 * split of a user's candidates into microbatches.  p: num_seqs = B,
 * total_tokens = T, max_seq_len = N, the normaliser (n_b + candidates of
 * b <= N, not checked); bf16 problems only (HSTU_ERR_UNSUPPORTED for fp32).
 * The prefix keys are processed in chunks of 512 (one work item per
 * candidate block and chunk, so small microbatches still fill the device)
 * whose fp32 partial outputs are added in chunk order: a candidate's
 * output does not depend on the other candidates of the call, bit for bit.
 * ws: hstu_attn_fwd_cached_workspace_bytes(p) bytes (not the
 * hstu_workspace_bytes of the uncached calls), 256-byte aligned. */
size_t hstu_attn_fwd_cached_workspace_bytes(const hstu_problem_t* p);

hstu_status_t hstu_attn_fwd_cached(const hstu_problem_t* p, const hstu_jagged_t* j,
                                   const void* q, int64_t q_stride,
                                   const void* k, int64_t k_stride,
                                   const void* v, int64_t v_stride,
                                   const int64_t* cache_offsets,
                                   const int64_t* cache_timestamps,
                                   int64_t cache_tokens,
                                   const void* k_cache, int64_t kc_stride,
                                   const void* v_cache, int64_t vc_stride,
                                   void* out, void* ws, size_t ws_bytes,
                                   void* hip_stream);

/* Backward of hstu_attn_fwd for the loss <out, d_out>.
 * d_out: dense [T][h][d_v].  dq, dk: dense [T][h][d_qk]; dv: dense
 * [T][h][d_v]; d_rab_pos [2N-1] and d_rab_time [B_t] (fp32, summed over
 * heads and sequences).  Every output is overwritten; the bias
 * gradients are cleared on the stream first. */
hstu_status_t hstu_attn_bwd(const hstu_problem_t* p, const hstu_jagged_t* j,
                            const void* q, int64_t q_stride,
                            const void* k, int64_t k_stride,
                            const void* v, int64_t v_stride,
                            const void* d_out,
                            void* dq, void* dk, void* dv,
                            float* d_rab_pos, float* d_rab_time,
                            void* ws, size_t ws_bytes, void* hip_stream);

/* Eq. 2 then the Eq. 3 gate: attn_out = the attention output of
 * hstu_attn_fwd, written dense [T][D] with D = h*d_v in fp32 for both
 * dtypes (the layer norm divides by a row's spread, which can be far
 * smaller than its magnitude, so it reads the output before any bf16
 * rounding; kept for the backward), then per token
 * y = ((x - mean) * rstd * ln_weight + ln_bias) (.) u with
 * rstd = 1/sqrt(var + ln_eps), biased variance over the D features.
 * ln_weight, ln_bias: fp32 [D] or NULL (identity).  u: rows of D elements
 * at u_stride; y: dense [T][D], both in the problem's dtype.  ln_mean,
 * ln_rstd: fp32 [T] or NULL.  D <= 4096. */
hstu_status_t hstu_layer_fwd(const hstu_problem_t* p, const hstu_jagged_t* j,
                             const void* q, int64_t q_stride,
                             const void* k, int64_t k_stride,
                             const void* v, int64_t v_stride,
                             const void* u, int64_t u_stride,
                             const float* ln_weight, const float* ln_bias,
                             float ln_eps, void* attn_out, void* y,
                             float* ln_mean, float* ln_rstd,
                             void* ws, size_t ws_bytes, void* hip_stream);

/* Backward of the whole layer (Eq. 2 and Eq. 3) from dY, the gradient of
 * Y = LayerNorm(attn_out) (.) U: du = LN(attn_out) (.) dY, the layer-norm
 * backward to dO = d attn_out (into the workspace: two bf16 terms for
 * HSTU_BF16, fp32 for HSTU_F32), then the attention backward of
 * hstu_attn_bwd with that dO (for HSTU_BF16 with P and dS as two bf16
 * terms in every contraction).  attn_out (fp32), ln_weight,
 * ln_bias, ln_mean and ln_rstd are the output, parameters and saved
 * statistics of the hstu_layer_fwd call (ln_mean, ln_rstd required;
 * weight / bias NULL for the identity affine).  d_y, du: dense [T][h*d_v]
 * in the problem's dtype
 * (du overwritten).  d_ln_weight, d_ln_bias: fp32 [h*d_v], overwritten
 * with the gradients (summed over tokens by float atomics, so their last
 * bits may vary between runs), or NULL to skip them.  Other arguments and
 * outputs as hstu_attn_bwd.  h*d_v <= 4096. */
hstu_status_t hstu_layer_bwd(const hstu_problem_t* p, const hstu_jagged_t* j,
                             const void* q, int64_t q_stride,
                             const void* k, int64_t k_stride,
                             const void* v, int64_t v_stride,
                             const void* u, int64_t u_stride,
                             const void* attn_out, const float* ln_weight,
                             const float* ln_bias, const float* ln_mean,
                             const float* ln_rstd, const void* d_y,
                             void* dq, void* dk, void* dv, void* du,
                             float* d_ln_weight, float* d_ln_bias,
                             float* d_rab_pos, float* d_rab_time,
                             void* ws, size_t ws_bytes, void* hip_stream);

/* Standalone timestamp bucketisation (notation table, rab^{p,t}): for
 * each sequence b writes its L_b x L_b matrix of bkt(t_i - t_j),
 * row-major (entry (i, j) at pair_offsets[b] + i*L_b + j), as uint8.
 * pair_offsets [B+1] is the exclusive prefix sum of L_b^2
 * (hstu_pair_offsets computes it); total_pairs = pair_offsets[B] (host
 * value).  num_time_buckets in [1, 256]. */
hstu_status_t hstu_time_bucketize(int32_t num_seqs, int64_t total_tokens,
                                  int32_t num_time_buckets,
                                  const int64_t* seq_offsets,
                                  const int64_t* timestamps,
                                  const int64_t* pair_offsets,
                                  int64_t total_pairs, uint8_t* buckets,
                                  void* hip_stream);

/* out[0] = 0, out[i+1] = out[i] + in[i] for i < n (int64, exact): turns
 * per-sequence lengths into the offsets of the jagged layout. */
hstu_status_t hstu_complete_cumsum(int32_t n, const int64_t* in, int64_t* out,
                                   void* hip_stream);

/* pair_offsets[0] = 0, pair_offsets[b+1] = pair_offsets[b] + L_b^2 with
 * L_b = seq_offsets[b+1] - seq_offsets[b]: the layout of
 * hstu_time_bucketize's output. */
hstu_status_t hstu_pair_offsets(int32_t num_seqs, const int64_t* seq_offsets,
                                int64_t* pair_offsets, void* hip_stream);

/* Synchronously copies the jagged metadata to the host and checks the
 * device-data preconditions listed above; HSTU_ERR_DATA on a violation. */
hstu_status_t hstu_validate(const hstu_problem_t* p, const hstu_jagged_t* j,
                            void* hip_stream);

/* Message of the last failed call on this thread (host string, valid
 * until the next call on this thread); "" after a success. */
const char* hstu_last_error(void);

int32_t hstu_abi_version(void);

/* Kernel timing for measurement: while enabled, every main kernel launch
 * is bracketed by HIP events on its stream.  hstu_timing_read
 * synchronises those events and returns, for the kernel family `name`
 * ("attn_fwd", "attn_bwd", "ln_gate", "bucketize"), the summed
 * milliseconds and launch count since the last reset. */
hstu_status_t hstu_timing_enable(int32_t on);
hstu_status_t hstu_timing_read(const char* name, double* total_ms,
                               int64_t* launches);
hstu_status_t hstu_timing_reset(void);

/* ---- The layer's linear maps: f_1 with phi_1 (Eq. 1) and f_2 (Eq. 3) ----
 * f_1 and f_2 are single linear layers with bias (Sec. 3.1, after Eq. 3).
 * Weights are stored [out][in] row-major in the problem's dtype, biases
 * are fp32 (NULL: none).  With D = d_model, hv = h*d_v, hq = h*d_qk and
 * F = 2 hv + 2 hq (the width of the fused projection, notation table entry
 * for Split), a token row of Z holds U (hv), V (hv), Q (hq), K (hq) in that
 * order, each [h][d]: pass z, z + hv, z + 2hv, z + 2hv + hq with row stride
 * F as u, v, q, k to the attention entry points.  Activations are dense
 * rows (x, g: given row strides) of p->total_tokens tokens; p's sequence
 * fields are not used.  All pointers are device memory, 16-byte aligned.
 * D must be a multiple of 8.  bf16 problems run on the matrix cores with
 * fp32 accumulation and need D and hv to be multiples of 64 and
 * T * max(F, D) * 2 below 2^31;
 * fp32 problems run a plain vector-ALU product (meant for small shapes).
 * Weight and bias gradients are written (not accumulated) in fp32; their
 * sums over tokens run in a fixed order, so results are reproducible.
 * Errors: HSTU_ERR_INVALID_ARGUMENT (NULL, misaligned, stride below the
 * row), HSTU_ERR_UNSUPPORTED (shapes above), HSTU_ERR_WORKSPACE. */

/* Workspace bytes needed by hstu_proj_in_bwd and hstu_proj_out_bwd for
 * problem p and model width d_model (0 if the arguments are invalid). */
size_t hstu_proj_workspace_bytes(const hstu_problem_t* p, int32_t d_model);

/* Eq. 1: z = SiLU(x W1^T + b1), x [T][D] (row stride x_stride), w1 [F][D],
 * b1 [F]; z [T][F] dense.  z_pre (NULL or [T][F] dense) receives the
 * pre-activation x W1^T + b1, which hstu_proj_in_bwd needs. */
hstu_status_t hstu_proj_in_fwd(const hstu_problem_t* p, int32_t d_model,
                               const void* x, int64_t x_stride,
                               const void* w1, const float* b1,
                               void* z, void* z_pre, void* hip_stream);

/* Eq. 3's f_2 and the residual connection between layers (Sec. 3.1):
 * y = g W2^T + b2 + residual, g [T][hv] (row stride g_stride; the y output
 * of hstu_layer_fwd), w2 [D][hv], b2 [D], residual NULL or [T][D] dense
 * (the layer's input x), y [T][D] dense. */
hstu_status_t hstu_proj_out_fwd(const hstu_problem_t* p, int32_t d_model,
                                const void* g, int64_t g_stride,
                                const void* w2, const float* b2,
                                const void* residual, void* y, void* hip_stream);

/* Backward of hstu_proj_out_fwd for the loss <y, dy>: dg = dy W2 ([T][hv]
 * dense, the d_y of hstu_layer_bwd), dw2 = dy^T g (fp32 [D][hv]), db2 =
 * column sums of dy (fp32 [D], skipped if NULL).  The residual's gradient
 * is dy itself. */
hstu_status_t hstu_proj_out_bwd(const hstu_problem_t* p, int32_t d_model,
                                const void* g, int64_t g_stride, const void* w2,
                                const void* dy, void* dg, float* dw2, float* db2,
                                void* ws, size_t ws_bytes, void* hip_stream);

/* Backward of hstu_proj_in_fwd for the loss <z, dZ>, dZ = [du|dv|dq|dk]
 * given as four dense [T][h][d] tensors (the gradients of hstu_layer_bwd):
 * with dpre = dZ * SiLU'(z_pre), dx = dpre W1 (+ dx_add, NULL or [T][D]
 * dense, e.g. the residual's gradient), dw1 = dpre^T x (fp32 [F][D]),
 * db1 = column sums of dpre (fp32 [F], skipped if NULL).  bf16 problems
 * round dpre to bf16 before the two products. */
hstu_status_t hstu_proj_in_bwd(const hstu_problem_t* p, int32_t d_model,
                               const void* x, int64_t x_stride, const void* w1,
                               const void* z_pre, const void* du, const void* dv,
                               const void* dq, const void* dk, const void* dx_add,
                               void* dx, float* dw1, float* db1,
                               void* ws, size_t ws_bytes, void* hip_stream);

/* ---- Stochastic Length (Eq. 4; subsequence selection and sparsity in
 * the appendix on Stochastic Length) ----
 * Shrinks a jagged batch before attention.  With L = subseq_len
 * (floor(N_c^(alpha/2)) of Eq. 4, see hstu_sl_subseq_len), keep_numerator
 * = N_c^alpha (see hstu_sl_keep_numerator; finite, >= 0) and n_h the number
 * of history tokens of sequence b (its tokens before the num_targets[b]
 * candidates; num_targets NULL: no candidates), the sequence is kept whole
 * if n_h <= L or u_keep[b] < keep_numerator / n_h^2 (fp64: the keep
 * probability of Eq. 4), else it keeps exactly L
 * history tokens, chosen by `selection`, in their original order, and then
 * all its candidates.  Selection keys (the L smallest win; equal keys: the
 * later token first), with f_i = t_max - t_i over the history:
 *   HSTU_SL_GREEDY    f_i: the most recent tokens;
 *   HSTU_SL_RANDOM    e_rand[i]: a uniformly random subset;
 *   HSTU_SL_WEIGHTED  e_rand[i] / (F - f_i), F = sum f_i: weighted sampling
 *                     without replacement with weights 1 - f_i / F (the
 *                     exponential-race form; +inf when F - f_i = 0, e_rand
 *                     alone when F = 0).  Needs F < 2^53 to be exact.
 * The random draws are inputs (device memory): u_keep [B] uniform in
 * [0, 1); e_rand [T] Exp(1) draws (values <= 0 count as 0; unused and may
 * be NULL for greedy).  Outputs (device): new_offsets [B+1] of the new
 * batch, gather [T] of which the first new_offsets[B] entries are the
 * original indices of the kept tokens in order (new num_targets equal the
 * old).  Results are exact and deterministic.  ws: hstu_sl_workspace_bytes
 * (num_seqs) bytes, 256-byte aligned.  Apply the selection to any per-token
 * tensor with hstu_gather_rows. */
enum { HSTU_SL_GREEDY = 0, HSTU_SL_RANDOM = 1, HSTU_SL_WEIGHTED = 2 };

/* L = floor(max_seq_len^(alpha/2)) for alpha in (0, 2]; 0 if invalid. */
int32_t hstu_sl_subseq_len(int32_t max_seq_len, double alpha);

/* max_seq_len^alpha (fp64 pow) for alpha in (0, 2]: the numerator of Eq. 4's
 * keep probability; 0 if invalid. */
double hstu_sl_keep_numerator(int32_t max_seq_len, double alpha);

size_t hstu_sl_workspace_bytes(int32_t num_seqs);

hstu_status_t hstu_stochastic_length(int32_t num_seqs, const int64_t* seq_offsets,
                                     const int64_t* timestamps, const int64_t* num_targets,
                                     int32_t subseq_len, double keep_numerator, int32_t selection,
                                     const double* u_keep, const double* e_rand,
                                     int64_t* new_offsets, int64_t* gather,
                                     void* ws, size_t ws_bytes, void* hip_stream);

/* dst row r = src row index[r] for r < min(*count, max_rows) (count and
 * index in device memory, e.g. new_offsets + B and gather of
 * hstu_stochastic_length); rows of row_bytes bytes at byte strides
 * src_stride / dst_stride; all multiples of 4 (16-byte rows move as
 * 16-byte words when everything is 16-byte aligned). */
hstu_status_t hstu_gather_rows(const void* src, int64_t src_stride, int64_t row_bytes,
                               const int64_t* index, const int64_t* count, int64_t max_rows,
                               void* dst, int64_t dst_stride, void* hip_stream);

/* Sparsity metrics of a batch (appendix on the impact of Stochastic Length
 * on sequence sparsity; host memory offsets): sparsity = 1 - mean length /
 * max_seq_len; s2, the same measure over the B padded attention matrices,
 * = 1 - sum_b L_b^2 / (B max_seq_len^2).  That form is the one the
 * appendix's printed tables admit (s2 >= sparsity in every cell). */
hstu_status_t hstu_sl_sparsity(int32_t num_seqs, const int64_t* seq_offsets, int32_t max_seq_len,
                               double* sparsity, double* s2);

/* Matrix-core rate probe for measurement: launches on `stream` a kernel
 * that issues only bf16 v_mfma_f32_32x32x16 instructions, `iters` x 8
 * independent ones per wave, with `waves_per_simd` (1 or 2) waves on every
 * SIMD of the device.  *flop receives the launch's flop count (2 per
 * multiply-add); time the launch with events on the same stream (it is
 * also recorded as kernel family "mfma_probe").  `sink` is device memory
 * of at least 256 floats that the kernel may write.  iters in [1, 2^24]. */
hstu_status_t hstu_probe_mfma_bf16(int32_t iters, int32_t waves_per_simd, float* sink,
                                   double* flop, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* HSTU_H_ */
