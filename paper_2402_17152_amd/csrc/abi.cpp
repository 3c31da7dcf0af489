// libhstu C ABI: argument validation, workspace layout, kernel dispatch.
// See include/hstu.h for the contract of every entry point.
#include "hstu.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"

namespace {

using namespace hstu;

thread_local std::string g_err;

hstu_status_t fail(hstu_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

hstu_status_t ok() {
  g_err.clear();
  return HSTU_OK;
}

hstu_status_t hip_fail(hipError_t e, const char* what) {
  return fail(HSTU_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// ---- kernel timing ----------------------------------------------------

struct Pending {
  std::string name;
  hipEvent_t start, stop;
};
std::mutex g_tmu;
bool g_timing = false;
std::vector<Pending> g_pending;
std::map<std::string, std::pair<double, int64_t>> g_acc;

struct TimedScope {
  bool on = false;
  Pending p;
  hipStream_t s;
  TimedScope(const char* name, hipStream_t stream) : s(stream) {
    if (!name) return;
    std::lock_guard<std::mutex> lk(g_tmu);
    if (!g_timing) return;
    p.name = name;
    if (hipEventCreate(&p.start) != hipSuccess) return;
    if (hipEventCreate(&p.stop) != hipSuccess) {
      (void)hipEventDestroy(p.start);
      return;
    }
    on = hipEventRecord(p.start, s) == hipSuccess;
  }
  ~TimedScope() {
    if (!on) return;
    (void)hipEventRecord(p.stop, s);
    std::lock_guard<std::mutex> lk(g_tmu);
    g_pending.push_back(p);
  }
};

// ---- validation helpers -------------------------------------------------

bool is_head_dim(int d) { return d == 32 || d == 64 || d == 128; }

hstu_status_t check_problem(const hstu_problem_t* p) {
  if (!p) return fail(HSTU_ERR_INVALID_ARGUMENT, "problem is NULL");
  if (p->num_seqs < 1)
    return fail(HSTU_ERR_INVALID_ARGUMENT, "num_seqs must be >= 1 (got %d)", p->num_seqs);
  if (p->total_tokens < 0) return fail(HSTU_ERR_INVALID_ARGUMENT, "total_tokens must be >= 0");
  if (p->total_tokens > (int64_t)1 << 40)
    return fail(HSTU_ERR_UNSUPPORTED, "total_tokens above 2^40 is not supported");
  if (p->max_seq_len < 1 || p->max_seq_len > 65536)
    return fail(HSTU_ERR_UNSUPPORTED, "max_seq_len must be in [1, 65536] (got %d)", p->max_seq_len);
  if (p->num_heads < 1 || p->num_heads > 64)
    return fail(HSTU_ERR_UNSUPPORTED, "num_heads must be in [1, 64] (got %d)", p->num_heads);
  if (!is_head_dim(p->d_qk) || !is_head_dim(p->d_v))
    return fail(HSTU_ERR_UNSUPPORTED, "d_qk and d_v must be 32, 64 or 128 (got %d, %d)", p->d_qk,
                p->d_v);
  if (p->num_time_buckets < 1 || p->num_time_buckets > 256)
    return fail(HSTU_ERR_UNSUPPORTED, "num_time_buckets must be in [1, 256] (got %d)",
                p->num_time_buckets);
  if (p->dtype != HSTU_F32 && p->dtype != HSTU_BF16)
    return fail(HSTU_ERR_INVALID_ARGUMENT, "unknown dtype %d", (int)p->dtype);
  return HSTU_OK;
}

hstu_status_t check_jagged(const hstu_jagged_t* j) {
  if (!j) return fail(HSTU_ERR_INVALID_ARGUMENT, "jagged descriptor is NULL");
  if (!j->seq_offsets) return fail(HSTU_ERR_INVALID_ARGUMENT, "seq_offsets is NULL");
  if (!j->timestamps) return fail(HSTU_ERR_INVALID_ARGUMENT, "timestamps is NULL");
  if (!j->rab_pos) return fail(HSTU_ERR_INVALID_ARGUMENT, "rab_pos is NULL");
  if (!j->rab_time) return fail(HSTU_ERR_INVALID_ARGUMENT, "rab_time is NULL");
  return HSTU_OK;
}

size_t elem_size(const hstu_problem_t* p) { return p->dtype == HSTU_BF16 ? 2 : 4; }

hstu_status_t check_rows(const hstu_problem_t* p, const char* name, const void* ptr,
                         int64_t stride, int64_t width) {
  if (!ptr) return fail(HSTU_ERR_INVALID_ARGUMENT, "%s is NULL", name);
  if ((uintptr_t)ptr % 16)
    return fail(HSTU_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", name);
  if (stride < width)
    return fail(HSTU_ERR_INVALID_ARGUMENT, "%s_stride %lld is smaller than a row (%lld)", name,
                (long long)stride, (long long)width);
  if ((stride * (int64_t)elem_size(p)) % 16)
    return fail(HSTU_ERR_INVALID_ARGUMENT, "%s_stride must be a multiple of 16 bytes", name);
  // The kernels address one sequence of a tensor with 32-bit byte offsets.
  if ((int64_t)p->max_seq_len * stride * (int64_t)elem_size(p) > ((int64_t)1 << 31))
    return fail(HSTU_ERR_UNSUPPORTED, "max_seq_len rows of %s span more than 2 GiB", name);
  return HSTU_OK;
}

hstu_status_t check_dense(const char* name, const void* ptr, size_t align) {
  if (!ptr) return fail(HSTU_ERR_INVALID_ARGUMENT, "%s is NULL", name);
  if ((uintptr_t)ptr % align)
    return fail(HSTU_ERR_INVALID_ARGUMENT, "%s is not %zu-byte aligned", name, align);
  return HSTU_OK;
}

// ---- workspace layout ---------------------------------------------------

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Layout {
  size_t counts;    // int32 [2]: forward and backward item counts
  size_t fwd_items;
  size_t bwd_items;
  size_t trange;    // int64 [2B]: per-sequence timestamp min / max
  size_t bases;     // int64 [2 (B + 1)]: slot tables of the partial dQ blocks
  size_t dout;      // [T][h*d_v] fp32, or bf16 high then low terms: dO of hstu_layer_bwd
  size_t dq_acc;    // fp32 [h][T][d_qk]: dQ of the single-role kernel (bf16 problems)
  size_t dq_part;   // f16 partial dQ blocks of the two-role kernel (bf16 problems), then
  size_t dq_scale;  // their fp32 block scales; both share the space of dq_acc, which a
                    // call using them does not use
  size_t rab64;     // fp64 [2N-1 + B_t]: bias-gradient sums of the fp32 backward
  size_t total;
  int64_t max_fwd, max_bwd;
};

Layout layout(const hstu_problem_t* p) {
  Layout l;
  l.max_fwd = max_work_items(p->total_tokens, p->num_seqs, kFwdBM);
  l.max_bwd = max_work_items(p->total_tokens, p->num_seqs, kBwdBN);
  size_t off = 0;
  l.counts = off;
  off = align_up(off + 2 * sizeof(int32_t));
  l.fwd_items = off;
  off = align_up(off + sizeof(WorkItem) * (size_t)l.max_fwd);
  l.bwd_items = off;
  off = align_up(off + sizeof(WorkItem) * (size_t)l.max_bwd);
  l.trange = off;
  off = align_up(off + 2 * sizeof(int64_t) * (size_t)p->num_seqs);
  l.bases = off;
  off = align_up(off + 2 * sizeof(int64_t) * ((size_t)p->num_seqs + 1));
  l.dout = off;
  off = align_up(off + 4 * (size_t)p->total_tokens * p->num_heads * p->d_v);
  const size_t shared = off;
  l.dq_acc = off;
  if (p->dtype == HSTU_BF16)
    off = align_up(off + sizeof(float) * (size_t)p->total_tokens * p->num_heads * p->d_qk);
  l.dq_part = shared;
  l.dq_scale = shared;
  if (p->dtype == HSTU_BF16) {
    // Per slot and head, d_qk / 32 blocks of 32 x 32 f16 and one fp32 scale each.
    const size_t slots =
        (size_t)dq_part_slots_bound(p->total_tokens, p->num_seqs, p->max_seq_len) *
        (size_t)p->num_heads;
    l.dq_scale = align_up(shared + slots * (size_t)p->d_qk * 64);
    off = std::max(off, align_up(l.dq_scale + slots * (size_t)(p->d_qk / 32) * 4));
  }
  l.rab64 = off;
  if (p->dtype == HSTU_F32)
    off = align_up(off + sizeof(double) *
                             ((size_t)(2 * p->max_seq_len - 1) + (size_t)p->num_time_buckets));
  l.total = off;
  return l;
}

hstu_status_t check_ws(const hstu_problem_t* p, void* ws, size_t ws_bytes, Layout* l) {
  *l = layout(p);
  if (!ws) return fail(HSTU_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", l->total);
  if ((uintptr_t)ws % kAlign) return fail(HSTU_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < l->total)
    return fail(HSTU_ERR_WORKSPACE, "workspace too small: %zu < %zu bytes", ws_bytes, l->total);
  return HSTU_OK;
}

// Workspace of the cached candidate pass: its own work list (one item per
// candidate block and prefix-key chunk) and the fp32 partial outputs, one
// slot of [T][h][d_v] per chunk.
struct CachedLayout {
  size_t counts, items, trange, partial, total;
  int64_t max_items;
  int32_t chunks;
};

CachedLayout cached_layout(const hstu_problem_t* p) {
  CachedLayout l;
  l.chunks = (p->max_seq_len + kCrossChunk - 1) / kCrossChunk;
  l.max_items = max_work_items(p->total_tokens, p->num_seqs, kFwdBM) * l.chunks;
  size_t off = 0;
  l.counts = off;
  off = align_up(off + 2 * sizeof(int32_t));
  l.items = off;
  off = align_up(off + sizeof(WorkItem) * (size_t)l.max_items);
  l.trange = off;
  off = align_up(off + 2 * sizeof(int64_t) * (size_t)p->num_seqs);
  l.partial = off;
  off = align_up(off + sizeof(float) * (size_t)l.chunks * p->total_tokens * p->num_heads * p->d_v);
  l.total = off;
  return l;
}

JaggedArgs make_args(const hstu_problem_t* p, const hstu_jagged_t* j) {
  JaggedArgs a;
  a.seq_offsets = j->seq_offsets;
  a.timestamps = j->timestamps;
  a.num_targets = j->num_targets;
  a.rab_pos = j->rab_pos;
  a.rab_time = j->rab_time;
  a.seq_trange = nullptr;
  a.key_offsets = nullptr;
  a.key_timestamps = nullptr;
  a.key_chunks = 0;
  a.chunk_stride = 0;
  a.num_seqs = p->num_seqs;
  a.max_seq_len = p->max_seq_len;
  a.num_heads = p->num_heads;
  a.num_buckets = p->num_time_buckets;
  a.total_tokens = p->total_tokens;
  return a;
}

#define HSTU_TRY(expr)                 \
  do {                                 \
    hstu_status_t st_ = (expr);        \
    if (st_ != HSTU_OK) return st_;    \
  } while (0)

#define HSTU_HIP(expr, what)                  \
  do {                                        \
    hipError_t e_ = (expr);                   \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

hstu_status_t check_fwd_args(const hstu_problem_t* p, const hstu_jagged_t* j, const Tensors& t,
                             void* out) {
  HSTU_TRY(check_problem(p));
  HSTU_TRY(check_jagged(j));
  const int H = p->num_heads;
  HSTU_TRY(check_rows(p, "q", t.q, t.q_stride, (int64_t)H * p->d_qk));
  HSTU_TRY(check_rows(p, "k", t.k, t.k_stride, (int64_t)H * p->d_qk));
  HSTU_TRY(check_rows(p, "v", t.v, t.v_stride, (int64_t)H * p->d_v));
  HSTU_TRY(check_dense("out", out, 16));
  return HSTU_OK;
}

// The forward's launches once its scratch is placed: the item count, the
// work list (max_items entries) and the per-sequence timestamp ranges, all
// written by the prep launch before the attention kernel reads them.
hstu_status_t attn_fwd_run(const hstu_problem_t* p, const hstu_jagged_t* j, const Tensors& t,
                           void* out, int out_f32, int32_t* counts, WorkItem* items,
                           int64_t* trange, int64_t max_items, bool timed, hipStream_t s) {
  JaggedArgs ja = make_args(p, j);
  if (p->dtype == HSTU_F32) {
    TimedScope ts(timed ? "attn_fwd" : nullptr, s);
    HSTU_HIP(launch_attn_fwd_f32(ja, t, p->d_qk, p->d_v, out, s), "attn_fwd_f32 launch");
    return ok();
  }
  ja.seq_trange = trange;
  HSTU_HIP(launch_prep(ja, 0, items, counts, trange, PrepFills{}, nullptr, s), "prep launch");
  TimedScope ts(timed ? "attn_fwd" : nullptr, s);
  HSTU_HIP(launch_attn_fwd_bf16(ja, t, p->d_qk, p->d_v, out, out_f32, out_f32, items, counts,
                                max_items, s),
           "attn_fwd launch");
  return ok();
}

hstu_status_t attn_fwd_impl(const hstu_problem_t* p, const hstu_jagged_t* j, const Tensors& t,
                            void* out, int out_f32, void* ws, size_t ws_bytes, hipStream_t s) {
  HSTU_TRY(check_fwd_args(p, j, t, out));
  Layout l;
  HSTU_TRY(check_ws(p, ws, ws_bytes, &l));
  if (p->total_tokens == 0) return ok();
  char* w = (char*)ws;
  return attn_fwd_run(p, j, t, out, out_f32, (int32_t*)(w + l.counts),
                      (WorkItem*)(w + l.fwd_items), (int64_t*)(w + l.trange), l.max_fwd, true, s);
}

// ---- forward without a workspace ------------------------------------------
// hstu_attn_fwd_noalloc keeps the forward's scratch in one static device
// array per GPU instead of a caller workspace.  Host code never passes the
// array's name to a kernel: its device address is looked up once per
// device with hipGetSymbolAddress and kept in g_scratch_dev.

constexpr size_t kNoAllocScratch = HSTU_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratch];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// Device address of the current device's scratch array, or an error.
hstu_status_t scratch_for_current_device(char** out) {
  int dev = -1;
  HSTU_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(HSTU_ERR_UNSUPPORTED, "device index %d is above %d", dev, kMaxDevices - 1);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* ptr = nullptr;
    HSTU_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (!ptr) return fail(HSTU_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_dev[dev] = ptr;
  }
  *out = (char*)g_scratch_dev[dev];
  return HSTU_OK;
}

// Offsets of the forward's scratch inside the static array.
struct NoAllocLayout {
  size_t counts, items, trange, total;
  int64_t max_items;
};

NoAllocLayout noalloc_layout(const hstu_problem_t* p) {
  NoAllocLayout l;
  l.max_items = max_work_items(p->total_tokens, p->num_seqs, kFwdBM);
  size_t off = 0;
  l.counts = off;
  off = align_up(off + 2 * sizeof(int32_t));
  l.items = off;
  off = align_up(off + sizeof(WorkItem) * (size_t)l.max_items);
  l.trange = off;
  off = align_up(off + 2 * sizeof(int64_t) * (size_t)p->num_seqs);
  l.total = off;
  return l;
}

// ---- linear maps f_1 (Eq. 1) and f_2 (Eq. 3) -----------------------------

struct ProjDims {
  int64_t T;
  int D, hv, hq, F;
  bool bf16;
  size_t e;
};

hstu_status_t proj_dims(const hstu_problem_t* p, int32_t d_model, ProjDims* d) {
  HSTU_TRY(check_problem(p));
  d->T = p->total_tokens;
  d->D = d_model;
  d->hv = p->num_heads * p->d_v;
  d->hq = p->num_heads * p->d_qk;
  d->F = 2 * d->hv + 2 * d->hq;
  d->bf16 = p->dtype == HSTU_BF16;
  d->e = elem_size(p);
  if (d_model < 8 || d_model > 65536 || d_model % 8)
    return fail(HSTU_ERR_UNSUPPORTED, "d_model must be a multiple of 8 in [8, 65536] (got %d)",
                d_model);
  if (d->bf16) {
    // The matrix-core kernels take contraction lengths in steps of 64.
    if (d_model % 64 || d->hv % 64)
      return fail(HSTU_ERR_UNSUPPORTED,
                  "bf16 projections need d_model and h*d_v to be multiples of 64 (got %d, %d)",
                  d_model, d->hv);
    const int64_t widest = d->F > d_model ? d->F : d_model;
    if (d->T * widest * 2 >= ((int64_t)1 << 31))
      return fail(HSTU_ERR_UNSUPPORTED, "T * max(F, d_model) * 2 bytes must stay below 2 GiB");
  }
  return HSTU_OK;
}

// A [rows][width] matrix with row stride `stride` (NULL allowed when it has no rows).
hstu_status_t check_mat(const char* name, const void* ptr, int64_t stride, int64_t width,
                        size_t e, int64_t rows) {
  if (!ptr && rows == 0) return HSTU_OK;
  if (!ptr) return fail(HSTU_ERR_INVALID_ARGUMENT, "%s is NULL", name);
  if ((uintptr_t)ptr % 16)
    return fail(HSTU_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", name);
  if (stride < width)
    return fail(HSTU_ERR_INVALID_ARGUMENT, "%s_stride %lld is smaller than a row (%lld)", name,
                (long long)stride, (long long)width);
  if ((stride * (int64_t)e) % 16)
    return fail(HSTU_ERR_INVALID_ARGUMENT, "%s_stride must be a multiple of 16 bytes", name);
  return HSTU_OK;
}

hstu_status_t check_opt(const char* name, const void* ptr) {
  if (ptr && (uintptr_t)ptr % 16)
    return fail(HSTU_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", name);
  return HSTU_OK;
}

struct ProjLayout {
  size_t dpre, partial, slab, total;
  int splits_in, ksplit_in, splits_out, ksplit_out;
};

ProjLayout proj_layout(const ProjDims& d) {
  ProjLayout l{};
  const size_t cb = (size_t)colsum_blocks(d.T);
  l.splits_in = gemm_num_splits(d.F, d.D, d.T, &l.ksplit_in);
  l.splits_out = gemm_num_splits(d.D, d.hv, d.T, &l.ksplit_out);
  size_t off = 0;
  l.dpre = off;
  off = align_up(off + d.e * (size_t)d.T * d.F);
  l.partial = off;
  const size_t wide = (size_t)(d.F > d.D ? d.F : d.D);
  off = align_up(off + sizeof(float) * cb * wide);
  l.slab = off;
  if (d.bf16) {
    const size_t a = (size_t)l.splits_in * d.F * d.D, b = (size_t)l.splits_out * d.D * d.hv;
    off = align_up(off + sizeof(float) * (a > b ? a : b));
  }
  l.total = off > kAlign ? off : kAlign;  // never 0, which means "invalid"
  return l;
}

hstu_status_t check_proj_ws(const ProjDims& d, void* ws, size_t ws_bytes, ProjLayout* l) {
  *l = proj_layout(d);
  if (!ws) return fail(HSTU_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", l->total);
  if ((uintptr_t)ws % kAlign) return fail(HSTU_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < l->total)
    return fail(HSTU_ERR_WORKSPACE, "workspace too small: %zu < %zu bytes", ws_bytes, l->total);
  return HSTU_OK;
}

// C = A(m, k) B(n, k) in either dtype; a_km / b_km: operand stored k-major.
// For fp32 operands the same layouts become element strides.
hipError_t proj_gemm(const ProjDims& d, int epi, const void* a, int64_t lda, int a_km,
                     const void* b, int64_t ldb, int b_km, int M, int N, int64_t K,
                     const float* bias, const void* res, int64_t ldr, void* c, int64_t ldc,
                     void* c2, float* slab, int splits, int ksplit, hipStream_t s) {
  if (d.bf16) {
    GemmArgs g{};
    g.a = (const uint16_t*)a;
    g.lda = lda;
    g.b = (const uint16_t*)b;
    g.ldb = ldb;
    g.M = M;
    g.N = N;
    g.K = (int32_t)K;
    g.k_split = ksplit;
    g.bias = bias;
    g.res = (const uint16_t*)res;
    g.ldr = ldr;
    g.c = (uint16_t*)c;
    g.ldc = ldc;
    g.c2 = (uint16_t*)c2;
    g.ldc2 = ldc;
    g.slab = slab;
    return launch_gemm_bf16(g, a_km, b_km, epi, splits, s);
  }
  GemmArgsF32 g{};
  g.a = (const float*)a;
  g.sam = a_km ? 1 : lda;
  g.sak = a_km ? lda : 1;
  g.b = (const float*)b;
  g.sbn = b_km ? 1 : ldb;
  g.sbk = b_km ? ldb : 1;
  g.M = M;
  g.N = N;
  g.K = (int32_t)K;
  g.bias = bias;
  g.res = (const float*)res;
  g.ldr = ldr;
  g.c = (float*)c;
  g.ldc = ldc;
  g.c2 = (float*)c2;
  g.ldc2 = ldc;
  return launch_gemm_f32(g, epi, s);
}

// Weight gradient dW [M][N] = sum_t A(m, t) B(n, t) over all tokens, both
// operands k-major: fp32 slabs per token split, then their ordered sum
// (bf16), or one direct product (fp32).
hipError_t weight_grad(const ProjDims& d, const void* a, int64_t lda, const void* b,
                       int64_t ldb, int M, int N, float* dw, float* slab, int splits,
                       int ksplit, hipStream_t s) {
  if (d.T == 0) return launch_reduce_slabs((int64_t)M * N, 0, nullptr, dw, s);
  if (!d.bf16)
    return proj_gemm(d, kEpiSlab, a, lda, 1, b, ldb, 1, M, N, d.T, nullptr, nullptr, 0, dw, N,
                     nullptr, nullptr, 1, 0, s);
  hipError_t e = proj_gemm(d, kEpiSlab, a, lda, 1, b, ldb, 1, M, N, d.T, nullptr, nullptr, 0,
                           nullptr, 0, nullptr, slab, splits, ksplit, s);
  if (e != hipSuccess) return e;
  return launch_reduce_slabs((int64_t)M * N, splits, slab, dw, s);
}

}  // namespace

extern "C" {

// ---- Stochastic Length (Eq. 4) ----------------------------------------

int32_t hstu_sl_subseq_len(int32_t max_seq_len, double alpha) {
  if (max_seq_len < 1 || !(alpha > 0.0) || alpha > 2.0) return 0;
  return (int32_t)std::floor(std::pow((double)max_seq_len, alpha / 2.0) + 1e-9);
}

double hstu_sl_keep_numerator(int32_t max_seq_len, double alpha) {
  if (max_seq_len < 1 || !(alpha > 0.0) || alpha > 2.0) return 0.0;
  return std::pow((double)max_seq_len, alpha);
}

size_t hstu_sl_workspace_bytes(int32_t num_seqs) {
  if (num_seqs < 1) return 0;
  return align_up(sizeof(int64_t) * (size_t)num_seqs) +
         align_up(sizeof(int32_t) * (size_t)num_seqs);
}

hstu_status_t hstu_stochastic_length(int32_t num_seqs, const int64_t* seq_offsets,
                                     const int64_t* timestamps, const int64_t* num_targets,
                                     int32_t subseq_len, double keep_numerator, int32_t selection,
                                     const double* u_keep, const double* e_rand,
                                     int64_t* new_offsets, int64_t* gather, void* ws,
                                     size_t ws_bytes, void* hip_stream) {
  try {
    hipStream_t s = (hipStream_t)hip_stream;
    if (num_seqs < 1) return fail(HSTU_ERR_INVALID_ARGUMENT, "num_seqs must be >= 1");
    if (subseq_len < 1) return fail(HSTU_ERR_INVALID_ARGUMENT, "subseq_len must be >= 1");
    if (!(keep_numerator >= 0.0) || std::isinf(keep_numerator))
      return fail(HSTU_ERR_INVALID_ARGUMENT, "keep_numerator must be finite and >= 0");
    if (selection < HSTU_SL_GREEDY || selection > HSTU_SL_WEIGHTED)
      return fail(HSTU_ERR_INVALID_ARGUMENT, "unknown selection %d", selection);
    if (!seq_offsets || !timestamps || !u_keep || !new_offsets || !gather)
      return fail(HSTU_ERR_INVALID_ARGUMENT, "NULL pointer");
    if (selection != HSTU_SL_GREEDY && !e_rand)
      return fail(HSTU_ERR_INVALID_ARGUMENT, "e_rand is NULL (needed by this selection)");
    const size_t need = hstu_sl_workspace_bytes(num_seqs);
    if (!ws || ws_bytes < need)
      return fail(HSTU_ERR_WORKSPACE, "workspace too small: %zu < %zu bytes", ws_bytes, need);
    if ((uintptr_t)ws % kAlign)
      return fail(HSTU_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    char* w = (char*)ws;
    int64_t* new_len = (int64_t*)w;
    int32_t* whole = (int32_t*)(w + align_up(sizeof(int64_t) * (size_t)num_seqs));
    TimedScope ts("stochastic_length", s);
    HSTU_HIP(launch_sl_lengths(num_seqs, seq_offsets, num_targets, subseq_len, keep_numerator,
                               u_keep, new_len, whole, s),
             "sl lengths launch");
    HSTU_HIP(launch_complete_cumsum(num_seqs, new_len, new_offsets, 0, s), "sl offsets launch");
    HSTU_HIP(launch_sl_select(num_seqs, seq_offsets, timestamps, num_targets, subseq_len,
                              selection, e_rand, whole, new_offsets, gather, s),
             "sl select launch");
    return ok();
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_gather_rows(const void* src, int64_t src_stride, int64_t row_bytes,
                               const int64_t* index, const int64_t* count, int64_t max_rows,
                               void* dst, int64_t dst_stride, void* hip_stream) {
  try {
    if (max_rows < 0 || row_bytes < 0) return fail(HSTU_ERR_INVALID_ARGUMENT, "negative size");
    if (max_rows == 0 || row_bytes == 0) return ok();
    if (!src || !index || !count || !dst) return fail(HSTU_ERR_INVALID_ARGUMENT, "NULL pointer");
    if (row_bytes % 4 || src_stride % 4 || dst_stride % 4 || (uintptr_t)src % 4 ||
        (uintptr_t)dst % 4)
      return fail(HSTU_ERR_INVALID_ARGUMENT, "rows, strides and pointers must be 4-byte aligned");
    if (src_stride < row_bytes || dst_stride < row_bytes)
      return fail(HSTU_ERR_INVALID_ARGUMENT, "stride smaller than a row");
    HSTU_HIP(launch_gather_rows(src, src_stride, row_bytes, index, count, max_rows, dst,
                                dst_stride, (hipStream_t)hip_stream),
             "gather launch");
    return ok();
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_sl_sparsity(int32_t num_seqs, const int64_t* seq_offsets, int32_t max_seq_len,
                               double* sparsity, double* s2) {
  if (num_seqs < 1 || max_seq_len < 1) return fail(HSTU_ERR_INVALID_ARGUMENT, "bad sizes");
  if (!seq_offsets || !sparsity || !s2) return fail(HSTU_ERR_INVALID_ARGUMENT, "NULL pointer");
  double sum = 0.0, sq = 0.0;
  for (int32_t b = 0; b < num_seqs; b++) {
    const double n = (double)(seq_offsets[b + 1] - seq_offsets[b]);
    sum += n;
    sq += n * n;
  }
  const double N = (double)max_seq_len;
  *sparsity = 1.0 - sum / num_seqs / N;
  *s2 = 1.0 - sq / ((double)num_seqs * N * N);
  return ok();
}

size_t hstu_proj_workspace_bytes(const hstu_problem_t* p, int32_t d_model) {
  try {
    ProjDims d;
    if (proj_dims(p, d_model, &d) != HSTU_OK) return 0;
    return proj_layout(d).total;
  } catch (...) {
    return 0;
  }
}

hstu_status_t hstu_proj_in_fwd(const hstu_problem_t* p, int32_t d_model, const void* x,
                               int64_t x_stride, const void* w1, const float* b1, void* z,
                               void* z_pre, void* hip_stream) {
  try {
    hipStream_t s = (hipStream_t)hip_stream;
    ProjDims d;
    HSTU_TRY(proj_dims(p, d_model, &d));
    HSTU_TRY(check_mat("x", x, x_stride, d.D, d.e, d.T));
    HSTU_TRY(check_mat("w1", w1, d.D, d.D, d.e, d.F));
    HSTU_TRY(check_opt("b1", b1));
    HSTU_TRY(check_mat("z", z, d.F, d.F, d.e, d.T));
    HSTU_TRY(check_opt("z_pre", z_pre));
    if (d.T == 0) return ok();
    TimedScope ts("proj_in_fwd", s);
    HSTU_HIP(proj_gemm(d, kEpiSilu, x, x_stride, 0, w1, d.D, 0, (int)d.T, d.F, d.D, b1, nullptr,
                       0, z, d.F, z_pre, nullptr, 1, d.D, s),
             "proj_in_fwd launch");
    return ok();
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_proj_out_fwd(const hstu_problem_t* p, int32_t d_model, const void* g,
                                int64_t g_stride, const void* w2, const float* b2,
                                const void* residual, void* y, void* hip_stream) {
  try {
    hipStream_t s = (hipStream_t)hip_stream;
    ProjDims d;
    HSTU_TRY(proj_dims(p, d_model, &d));
    HSTU_TRY(check_mat("g", g, g_stride, d.hv, d.e, d.T));
    HSTU_TRY(check_mat("w2", w2, d.hv, d.hv, d.e, d.D));
    HSTU_TRY(check_opt("b2", b2));
    HSTU_TRY(check_opt("residual", residual));
    HSTU_TRY(check_mat("y", y, d.D, d.D, d.e, d.T));
    if (d.T == 0) return ok();
    TimedScope ts("proj_out_fwd", s);
    HSTU_HIP(proj_gemm(d, kEpiAdd, g, g_stride, 0, w2, d.hv, 0, (int)d.T, d.D, d.hv, b2, residual,
                       d.D, y, d.D, nullptr, nullptr, 1, d.hv, s),
             "proj_out_fwd launch");
    return ok();
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_proj_out_bwd(const hstu_problem_t* p, int32_t d_model, const void* g,
                                int64_t g_stride, const void* w2, const void* dy, void* dg,
                                float* dw2, float* db2, void* ws, size_t ws_bytes,
                                void* hip_stream) {
  try {
    hipStream_t s = (hipStream_t)hip_stream;
    ProjDims d;
    HSTU_TRY(proj_dims(p, d_model, &d));
    HSTU_TRY(check_mat("g", g, g_stride, d.hv, d.e, d.T));
    HSTU_TRY(check_mat("w2", w2, d.hv, d.hv, d.e, d.D));
    HSTU_TRY(check_mat("dy", dy, d.D, d.D, d.e, d.T));
    HSTU_TRY(check_mat("dg", dg, d.hv, d.hv, d.e, d.T));
    HSTU_TRY(check_dense("dw2", dw2, 16));
    HSTU_TRY(check_opt("db2", db2));
    ProjLayout l;
    HSTU_TRY(check_proj_ws(d, ws, ws_bytes, &l));
    char* w = (char*)ws;
    float* partial = (float*)(w + l.partial);
    float* slab = (float*)(w + l.slab);
    TimedScope ts("proj_out_bwd", s);
    // dG = dY W2 (W2 [D][h d_v] read k-major).
    if (d.T > 0)
      HSTU_HIP(proj_gemm(d, kEpiAdd, dy, d.D, 0, w2, d.hv, 1, (int)d.T, d.hv, d.D, nullptr,
                         nullptr, 0, dg, d.hv, nullptr, nullptr, 1, d.D, s),
               "proj_out_bwd dgrad launch");
    // dW2 = dY^T G over the tokens.
    HSTU_HIP(weight_grad(d, dy, d.D, g, g_stride, d.D, d.hv, dw2, slab, l.splits_out,
                         l.ksplit_out, s),
             "proj_out_bwd wgrad launch");
    if (db2) {
      HSTU_HIP(launch_colsum(d.bf16, d.T, d.D, d.D, dy, partial, s), "colsum launch");
      HSTU_HIP(launch_reduce_cols(d.D, (int)colsum_blocks(d.T), partial, db2, s),
               "bias reduce launch");
    }
    return ok();
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_proj_in_bwd(const hstu_problem_t* p, int32_t d_model, const void* x,
                               int64_t x_stride, const void* w1, const void* z_pre,
                               const void* du, const void* dv, const void* dq, const void* dk,
                               const void* dx_add, void* dx, float* dw1, float* db1, void* ws,
                               size_t ws_bytes, void* hip_stream) {
  try {
    hipStream_t s = (hipStream_t)hip_stream;
    ProjDims d;
    HSTU_TRY(proj_dims(p, d_model, &d));
    HSTU_TRY(check_mat("x", x, x_stride, d.D, d.e, d.T));
    HSTU_TRY(check_mat("w1", w1, d.D, d.D, d.e, d.F));
    HSTU_TRY(check_mat("z_pre", z_pre, d.F, d.F, d.e, d.T));
    HSTU_TRY(check_mat("du", du, d.hv, d.hv, d.e, d.T));
    HSTU_TRY(check_mat("dv", dv, d.hv, d.hv, d.e, d.T));
    HSTU_TRY(check_mat("dq", dq, d.hq, d.hq, d.e, d.T));
    HSTU_TRY(check_mat("dk", dk, d.hq, d.hq, d.e, d.T));
    HSTU_TRY(check_opt("dx_add", dx_add));
    HSTU_TRY(check_mat("dx", dx, d.D, d.D, d.e, d.T));
    HSTU_TRY(check_dense("dw1", dw1, 16));
    HSTU_TRY(check_opt("db1", db1));
    ProjLayout l;
    HSTU_TRY(check_proj_ws(d, ws, ws_bytes, &l));
    char* w = (char*)ws;
    void* dpre = w + l.dpre;
    float* partial = (float*)(w + l.partial);
    float* slab = (float*)(w + l.slab);
    TimedScope ts("proj_in_bwd", s);
    HSTU_HIP(launch_silu_bwd(d.bf16, d.T, d.F, d.hv, d.hq, z_pre, du, dv, dq, dk, dpre, partial,
                             s),
             "silu backward launch");
    // dX = dpre W1 (+ dx_add), W1 [F][D] read k-major.
    if (d.T > 0)
      HSTU_HIP(proj_gemm(d, kEpiAdd, dpre, d.F, 0, w1, d.D, 1, (int)d.T, d.D, d.F, nullptr,
                         dx_add, d.D, dx, d.D, nullptr, nullptr, 1, d.F, s),
               "proj_in_bwd dgrad launch");
    // dW1 = dpre^T X over the tokens.
    HSTU_HIP(weight_grad(d, dpre, d.F, x, x_stride, d.F, d.D, dw1, slab, l.splits_in,
                         l.ksplit_in, s),
             "proj_in_bwd wgrad launch");
    if (db1)
      HSTU_HIP(launch_reduce_cols(d.F, (int)colsum_blocks(d.T), partial, db1, s),
               "bias reduce launch");
    return ok();
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

int32_t hstu_abi_version(void) { return HSTU_ABI_VERSION; }

const char* hstu_last_error(void) { return g_err.c_str(); }

size_t hstu_workspace_bytes(const hstu_problem_t* p) {
  try {
    if (check_problem(p) != HSTU_OK) return 0;
    return layout(p).total;
  } catch (...) {
    return 0;
  }
}

hstu_status_t hstu_attn_fwd(const hstu_problem_t* p, const hstu_jagged_t* j, const void* q,
                            int64_t q_stride, const void* k, int64_t k_stride, const void* v,
                            int64_t v_stride, void* out, void* ws, size_t ws_bytes,
                            void* hip_stream) {
  try {
    Tensors t{q, q_stride, k, k_stride, v, v_stride};
    return attn_fwd_impl(p, j, t, out, 0, ws, ws_bytes, (hipStream_t)hip_stream);
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_attn_fwd_noalloc(const hstu_problem_t* p, const hstu_jagged_t* j,
                                    const void* q, int64_t q_stride, const void* k,
                                    int64_t k_stride, const void* v, int64_t v_stride, void* out,
                                    void* hip_stream) {
  try {
    hipStream_t s = (hipStream_t)hip_stream;
    Tensors t{q, q_stride, k, k_stride, v, v_stride};
    HSTU_TRY(check_fwd_args(p, j, t, out));
    const NoAllocLayout l = noalloc_layout(p);
    if (p->dtype == HSTU_BF16 && l.total > kNoAllocScratch)
      return fail(HSTU_ERR_UNSUPPORTED,
                  "hstu_attn_fwd_noalloc: %zu bytes of scratch needed (num_seqs %d, total_tokens "
                  "%lld), above its static %zu bytes; use hstu_attn_fwd with a workspace",
                  l.total, p->num_seqs, (long long)p->total_tokens, kNoAllocScratch);
    if (p->total_tokens == 0) return ok();
    char* w = nullptr;
    HSTU_TRY(scratch_for_current_device(&w));
    return attn_fwd_run(p, j, t, out, 0, (int32_t*)(w + l.counts), (WorkItem*)(w + l.items),
                        (int64_t*)(w + l.trange), l.max_items, false, s);
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

size_t hstu_attn_fwd_cached_workspace_bytes(const hstu_problem_t* p) {
  try {
    if (check_problem(p) != HSTU_OK) return 0;
    return cached_layout(p).total;
  } catch (...) {
    return 0;
  }
}

hstu_status_t hstu_attn_fwd_cached(const hstu_problem_t* p, const hstu_jagged_t* j, const void* q,
                                   int64_t q_stride, const void* k, int64_t k_stride,
                                   const void* v, int64_t v_stride, const int64_t* cache_offsets,
                                   const int64_t* cache_timestamps, int64_t cache_tokens,
                                   const void* k_cache, int64_t kc_stride, const void* v_cache,
                                   int64_t vc_stride, void* out, void* ws, size_t ws_bytes,
                                   void* hip_stream) {
  try {
    hipStream_t s = (hipStream_t)hip_stream;
    HSTU_TRY(check_problem(p));
    HSTU_TRY(check_jagged(j));
    if (p->dtype != HSTU_BF16)
      return fail(HSTU_ERR_UNSUPPORTED, "hstu_attn_fwd_cached supports bf16 problems only");
    const int H = p->num_heads;
    HSTU_TRY(check_rows(p, "q", q, q_stride, (int64_t)H * p->d_qk));
    HSTU_TRY(check_rows(p, "k", k, k_stride, (int64_t)H * p->d_qk));
    HSTU_TRY(check_rows(p, "v", v, v_stride, (int64_t)H * p->d_v));
    HSTU_TRY(check_dense("out", out, 16));
    if (!cache_offsets) return fail(HSTU_ERR_INVALID_ARGUMENT, "cache_offsets is NULL");
    if (cache_tokens < 0) return fail(HSTU_ERR_INVALID_ARGUMENT, "cache_tokens must be >= 0");
    if (cache_tokens > 0) {
      if (!cache_timestamps) return fail(HSTU_ERR_INVALID_ARGUMENT, "cache_timestamps is NULL");
      HSTU_TRY(check_rows(p, "k_cache", k_cache, kc_stride, (int64_t)H * p->d_qk));
      HSTU_TRY(check_rows(p, "v_cache", v_cache, vc_stride, (int64_t)H * p->d_v));
    }
    const CachedLayout l = cached_layout(p);
    if (!ws) return fail(HSTU_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", l.total);
    if ((uintptr_t)ws % kAlign)
      return fail(HSTU_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    if (ws_bytes < l.total)
      return fail(HSTU_ERR_WORKSPACE, "workspace too small: %zu < %zu bytes", ws_bytes, l.total);
    const int64_t T = p->total_tokens;
    if (T == 0) return ok();
    JaggedArgs ja = make_args(p, j);
    ja.num_targets = nullptr;
    ja.key_offsets = cache_offsets;
    ja.key_timestamps = cache_timestamps;
    ja.key_chunks = l.chunks;
    ja.chunk_stride = T * H * p->d_v;
    char* w = (char*)ws;
    int32_t* counts = (int32_t*)(w + l.counts);
    WorkItem* items = (WorkItem*)(w + l.items);
    float* o32 = (float*)(w + l.partial);  // fp32 partial outputs, one slot per key chunk
    ja.seq_trange = (const int64_t*)(w + l.trange);
    HSTU_HIP(launch_prep(ja, 0, items, counts, (int64_t*)(w + l.trange), PrepFills{}, nullptr,
                         s),
             "prep launch");
    TimedScope ts("attn_fwd_cached", s);
    const Tensors keys{q, q_stride, k_cache, kc_stride, v_cache, vc_stride};
    HSTU_HIP(launch_attn_fwd_bf16(ja, keys, p->d_qk, p->d_v, o32, 1, 0, items, counts, l.max_items,
                                  s),
             "attn_fwd_cached launch");
    const Tensors cand{q, q_stride, k, k_stride, v, v_stride};
    HSTU_HIP(launch_cached_self(ja, p->d_qk, p->d_v, cand, o32, out, s),
             "cached self-term launch");
    return ok();
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

// Argument checks of the attention backward (shared by hstu_layer_bwd,
// which runs them before launching anything).
hstu_status_t attn_bwd_check(const hstu_problem_t* p, const hstu_jagged_t* j, const Tensors& t,
                             const void* d_out, void* dq, void* dk, void* dv, float* d_rab_pos,
                             float* d_rab_time, void* ws, size_t ws_bytes, Layout* l) {
  HSTU_TRY(check_problem(p));
  HSTU_TRY(check_jagged(j));
  const int H = p->num_heads;
  HSTU_TRY(check_rows(p, "q", t.q, t.q_stride, (int64_t)H * p->d_qk));
  HSTU_TRY(check_rows(p, "k", t.k, t.k_stride, (int64_t)H * p->d_qk));
  HSTU_TRY(check_rows(p, "v", t.v, t.v_stride, (int64_t)H * p->d_v));
  HSTU_TRY(check_dense("d_out", d_out, 16));
  HSTU_TRY(check_dense("dq", dq, 16));
  HSTU_TRY(check_dense("dk", dk, 16));
  HSTU_TRY(check_dense("dv", dv, 16));
  HSTU_TRY(check_dense("d_rab_pos", d_rab_pos, 4));
  HSTU_TRY(check_dense("d_rab_time", d_rab_time, 4));
  return check_ws(p, ws, ws_bytes, l);
}

// d_out_lo: null, or the low bf16 terms of a dO given as two terms (bf16
// problems only).
hstu_status_t attn_bwd_impl(const hstu_problem_t* p, const hstu_jagged_t* j, const Tensors& t,
                            const void* d_out, const void* d_out_lo, void* dq, void* dk,
                            void* dv, float* d_rab_pos, float* d_rab_time, void* ws,
                            size_t ws_bytes, hipStream_t s) {
  Layout l;
  HSTU_TRY(attn_bwd_check(p, j, t, d_out, dq, dk, dv, d_rab_pos, d_rab_time, ws, ws_bytes, &l));
  const int64_t T = p->total_tokens;
  const int H = p->num_heads;
  const int N = p->max_seq_len;
  if (T == 0 || p->dtype == HSTU_F32) {
    HSTU_HIP(launch_fill_f32(d_rab_pos, 2 * (int64_t)N - 1, 0.0f, s), "fill launch");
    HSTU_HIP(launch_fill_f32(d_rab_time, p->num_time_buckets, 0.0f, s), "fill launch");
  }
  if (T == 0) return ok();
  JaggedArgs ja = make_args(p, j);
  char* w = (char*)ws;
  if (p->dtype == HSTU_F32) {
    // Bias gradients summed in fp64 in the workspace, then stored as fp32.
    double* rab64 = (double*)(w + l.rab64);
    const int64_t nrab = 2 * (int64_t)N - 1 + p->num_time_buckets;
    HSTU_HIP(launch_fill_f32((float*)rab64, 2 * nrab, 0.0f, s), "fill launch");
    TimedScope ts("attn_bwd", s);
    HSTU_HIP(launch_attn_bwd_f32(ja, t, p->d_qk, p->d_v, d_out, dq, dk, dv, rab64,
                                 rab64 + (2 * (int64_t)N - 1), s),
             "attn_bwd_f32 launch");
    HSTU_HIP(launch_f64_to_f32_scaled(rab64, d_rab_pos, 2 * (int64_t)N - 1, 1.0 / N, s),
             "convert launch");
    HSTU_HIP(launch_f64_to_f32_scaled(rab64 + (2 * (int64_t)N - 1), d_rab_time,
                                      p->num_time_buckets, 1.0 / N, s),
             "convert launch");
    return ok();
  }
  int32_t* counts = (int32_t*)(w + l.counts);
  WorkItem* items = (WorkItem*)(w + l.bwd_items);
  float* dq_acc = (float*)(w + l.dq_acc);
  uint16_t* dq_part = (uint16_t*)(w + l.dq_part);
  float* dq_scale = (float*)(w + l.dq_scale);
  const int64_t dq_slots = dq_part_slots_bound(T, p->num_seqs, N);
  int64_t* bases = (int64_t*)(w + l.bases);
  const int64_t ndq = T * H * p->d_qk;
  ja.seq_trange = (const int64_t*)(w + l.trange);
  // Both bias-gradient tables start at zero, and so does the fp32 dQ
  // accumulator of the single-role kernel (two-term dO at d > 64); the
  // two-role kernel needs the slot tables of its partial dQ blocks instead.
  const bool single = d_out_lo != nullptr && !bwd_split_two_role(p->d_qk, p->d_v);
  const PrepFills fills =
      single ? PrepFills{{dq_acc, d_rab_pos, d_rab_time},
                         {ndq, 2 * (int64_t)N - 1, (int64_t)p->num_time_buckets}, 3}
             : PrepFills{{d_rab_pos, d_rab_time, nullptr},
                         {2 * (int64_t)N - 1, (int64_t)p->num_time_buckets, 0}, 2};
  HSTU_HIP(launch_prep(ja, 1, items, counts + 1, (int64_t*)(w + l.trange), fills,
                       single ? nullptr : bases, s),
           "prep launch");
  {
    TimedScope ts("attn_bwd", s);
    HSTU_HIP(launch_attn_bwd_bf16(ja, t, p->d_qk, p->d_v, d_out, d_out_lo, dq_acc, dq_part,
                                  dq_scale, dq_slots, bases, dk, dv, d_rab_pos, d_rab_time,
                                  items, counts + 1, l.max_bwd, s),
             "attn_bwd launch");
  }
  if (single)
    HSTU_HIP(launch_dq_convert_bf16(dq_acc, dq, T, H, p->d_qk, 1.0f / (float)N, s),
             "dq convert launch");
  else {
    TimedScope ts("dq_reduce", s);
    HSTU_HIP(launch_dq_reduce_bf16(ja, p->d_qk, dq_part, dq_scale, dq_slots, bases, dq, s),
             "dq reduce launch");
  }
  return ok();
}

hstu_status_t hstu_attn_bwd(const hstu_problem_t* p, const hstu_jagged_t* j, const void* q,
                            int64_t q_stride, const void* k, int64_t k_stride, const void* v,
                            int64_t v_stride, const void* d_out, void* dq, void* dk, void* dv,
                            float* d_rab_pos, float* d_rab_time, void* ws, size_t ws_bytes,
                            void* hip_stream) {
  try {
    Tensors t{q, q_stride, k, k_stride, v, v_stride};
    return attn_bwd_impl(p, j, t, d_out, nullptr, dq, dk, dv, d_rab_pos, d_rab_time, ws,
                         ws_bytes, (hipStream_t)hip_stream);
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_layer_bwd(const hstu_problem_t* p, const hstu_jagged_t* j, const void* q,
                             int64_t q_stride, const void* k, int64_t k_stride, const void* v,
                             int64_t v_stride, const void* u, int64_t u_stride,
                             const void* attn_out, const float* ln_weight, const float* ln_bias,
                             const float* ln_mean, const float* ln_rstd, const void* d_y,
                             void* dq, void* dk, void* dv, void* du, float* d_ln_weight,
                             float* d_ln_bias, float* d_rab_pos, float* d_rab_time, void* ws,
                             size_t ws_bytes, void* hip_stream) {
  try {
    hipStream_t s = (hipStream_t)hip_stream;
    Tensors t{q, q_stride, k, k_stride, v, v_stride};
    Layout l;
    HSTU_TRY(check_problem(p));
    HSTU_TRY(check_ws(p, ws, ws_bytes, &l));
    // dO of the attention, in the workspace: fp32, or for bf16 problems two
    // bf16 terms (high, then low) that the attention backward both uses.
    void* dout = (char*)ws + l.dout;
    const bool split = p->dtype == HSTU_BF16;
    void* dout_lo = split ? (char*)dout + 2 * (size_t)p->total_tokens * p->num_heads * p->d_v
                          : nullptr;
    HSTU_TRY(attn_bwd_check(p, j, t, dout, dq, dk, dv, d_rab_pos, d_rab_time, ws, ws_bytes, &l));
    const int64_t D = (int64_t)p->num_heads * p->d_v;
    if (D > 4096)
      return fail(HSTU_ERR_UNSUPPORTED, "h*d_v must be <= 4096 (got %lld)", (long long)D);
    HSTU_TRY(check_rows(p, "u", u, u_stride, D));
    HSTU_TRY(check_dense("attn_out", attn_out, 16));
    HSTU_TRY(check_dense("d_y", d_y, 16));
    HSTU_TRY(check_dense("du", du, 16));
    if (p->total_tokens > 0 && (!ln_mean || !ln_rstd))
      return fail(HSTU_ERR_INVALID_ARGUMENT,
                  "ln_mean and ln_rstd (saved by hstu_layer_fwd) are required");
    if (d_ln_weight) HSTU_HIP(launch_fill_f32(d_ln_weight, D, 0.0f, s), "fill launch");
    if (d_ln_bias) HSTU_HIP(launch_fill_f32(d_ln_bias, D, 0.0f, s), "fill launch");
    if (p->total_tokens > 0) {
      TimedScope ts("ln_gate_bwd", s);
      HSTU_HIP(launch_ln_gate_bwd(p->dtype == HSTU_BF16, p->total_tokens, (int32_t)D, attn_out, u,
                                  u_stride, d_y, ln_weight, ln_bias, ln_mean, ln_rstd, du, dout,
                                  dout_lo, d_ln_weight, d_ln_bias, s),
               "ln_gate_bwd launch");
    }
    return attn_bwd_impl(p, j, t, dout, dout_lo, dq, dk, dv, d_rab_pos, d_rab_time, ws, ws_bytes,
                         s);
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_layer_fwd(const hstu_problem_t* p, const hstu_jagged_t* j, const void* q,
                             int64_t q_stride, const void* k, int64_t k_stride, const void* v,
                             int64_t v_stride, const void* u, int64_t u_stride,
                             const float* ln_weight, const float* ln_bias, float ln_eps,
                             void* attn_out, void* y, float* ln_mean, float* ln_rstd, void* ws,
                             size_t ws_bytes, void* hip_stream) {
  try {
    hipStream_t s = (hipStream_t)hip_stream;
    HSTU_TRY(check_problem(p));
    const int64_t D = (int64_t)p->num_heads * p->d_v;
    if (D > 4096)
      return fail(HSTU_ERR_UNSUPPORTED, "h*d_v must be <= 4096 (got %lld)", (long long)D);
    HSTU_TRY(check_rows(p, "u", u, u_stride, D));
    HSTU_TRY(check_dense("y", y, 16));
    if (!(ln_eps >= 0.0f)) return fail(HSTU_ERR_INVALID_ARGUMENT, "ln_eps must be >= 0");
    Tensors t{q, q_stride, k, k_stride, v, v_stride};
    // The attention output stays fp32 for the layer norm (both dtypes).
    HSTU_TRY(attn_fwd_impl(p, j, t, attn_out, 1, ws, ws_bytes, s));
    if (p->total_tokens == 0) return ok();
    TimedScope ts("ln_gate", s);
    HSTU_HIP(launch_ln_gate(p->dtype == HSTU_BF16, p->total_tokens, (int32_t)D, attn_out, u,
                            u_stride, ln_weight, ln_bias, ln_eps, y, ln_mean, ln_rstd, s),
             "ln_gate launch");
    return ok();
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_time_bucketize(int32_t num_seqs, int64_t total_tokens, int32_t num_time_buckets,
                                  const int64_t* seq_offsets, const int64_t* timestamps,
                                  const int64_t* pair_offsets, int64_t total_pairs,
                                  uint8_t* buckets, void* hip_stream) {
  try {
    if (num_seqs < 1) return fail(HSTU_ERR_INVALID_ARGUMENT, "num_seqs must be >= 1");
    if (total_tokens < 0 || total_pairs < 0)
      return fail(HSTU_ERR_INVALID_ARGUMENT, "negative size");
    if (num_time_buckets < 1 || num_time_buckets > 256)
      return fail(HSTU_ERR_UNSUPPORTED, "num_time_buckets must be in [1, 256]");
    if (!seq_offsets || !pair_offsets) return fail(HSTU_ERR_INVALID_ARGUMENT, "offsets are NULL");
    if (total_pairs > 0) {
      if (!timestamps) return fail(HSTU_ERR_INVALID_ARGUMENT, "timestamps is NULL");
      HSTU_TRY(check_dense("buckets", buckets, 16));
    }
    TimedScope ts("bucketize", (hipStream_t)hip_stream);
    HSTU_HIP(launch_bucketize(num_seqs, total_tokens, num_time_buckets, seq_offsets, timestamps,
                              pair_offsets, total_pairs, buckets, (hipStream_t)hip_stream),
             "bucketize launch");
    return ok();
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_complete_cumsum(int32_t n, const int64_t* in, int64_t* out, void* hip_stream) {
  try {
    if (n < 0) return fail(HSTU_ERR_INVALID_ARGUMENT, "n must be >= 0");
    if (!out || (n > 0 && !in)) return fail(HSTU_ERR_INVALID_ARGUMENT, "NULL pointer");
    HSTU_HIP(launch_complete_cumsum(n, in, out, 0, (hipStream_t)hip_stream), "cumsum launch");
    return ok();
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_pair_offsets(int32_t num_seqs, const int64_t* seq_offsets, int64_t* pair_offsets,
                                void* hip_stream) {
  try {
    if (num_seqs < 1) return fail(HSTU_ERR_INVALID_ARGUMENT, "num_seqs must be >= 1");
    if (!seq_offsets || !pair_offsets) return fail(HSTU_ERR_INVALID_ARGUMENT, "NULL pointer");
    HSTU_HIP(launch_complete_cumsum(num_seqs, seq_offsets, pair_offsets, 1,
                                    (hipStream_t)hip_stream),
             "pair offsets launch");
    return ok();
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_validate(const hstu_problem_t* p, const hstu_jagged_t* j, void* hip_stream) {
  try {
    HSTU_TRY(check_problem(p));
    HSTU_TRY(check_jagged(j));
    hipStream_t s = (hipStream_t)hip_stream;
    const int B = p->num_seqs;
    const int64_t T = p->total_tokens;
    std::vector<int64_t> offs(B + 1), nt(B, 0), ts((size_t)T);
    HSTU_HIP(hipMemcpyAsync(offs.data(), j->seq_offsets, sizeof(int64_t) * (B + 1),
                            hipMemcpyDeviceToHost, s), "copy offsets");
    if (j->num_targets)
      HSTU_HIP(hipMemcpyAsync(nt.data(), j->num_targets, sizeof(int64_t) * B,
                              hipMemcpyDeviceToHost, s),
               "copy num_targets");
    if (T > 0)
      HSTU_HIP(hipMemcpyAsync(ts.data(), j->timestamps, sizeof(int64_t) * T,
                              hipMemcpyDeviceToHost, s),
               "copy timestamps");
    HSTU_HIP(hipStreamSynchronize(s), "synchronize");
    if (offs[0] != 0)
      return fail(HSTU_ERR_DATA, "seq_offsets[0] = %lld, expected 0", (long long)offs[0]);
    if (offs[B] != T)
      return fail(HSTU_ERR_DATA, "seq_offsets[B] = %lld, expected total_tokens %lld",
                  (long long)offs[B], (long long)T);
    for (int b = 0; b < B; b++) {
      const int64_t L = offs[b + 1] - offs[b];
      if (L < 0) return fail(HSTU_ERR_DATA, "seq_offsets decreases at b = %d", b);
      if (L > p->max_seq_len)
        return fail(HSTU_ERR_DATA, "sequence %d has length %lld > max_seq_len %d", b, (long long)L,
                    p->max_seq_len);
      if (nt[b] < 0 || nt[b] > L)
        return fail(HSTU_ERR_DATA, "num_targets[%d] = %lld outside [0, %lld]", b, (long long)nt[b],
                    (long long)L);
    }
    for (int64_t i = 0; i < T; i++)
      if (ts[i] < 0 || ts[i] >= ((int64_t)1 << 62))
        return fail(HSTU_ERR_DATA, "timestamps[%lld] = %lld outside [0, 2^62)", (long long)i,
                    (long long)ts[i]);
    return ok();
  } catch (...) {
    return fail(HSTU_ERR_INVALID_ARGUMENT, "internal error");
  }
}

hstu_status_t hstu_probe_mfma_bf16(int32_t iters, int32_t waves_per_simd, float* sink,
                                   double* flop, void* stream) {
  if (iters < 1 || iters > (1 << 24))
    return fail(HSTU_ERR_INVALID_ARGUMENT, "iters must be in [1, 2^24]");
  if (waves_per_simd < 1 || waves_per_simd > 2)
    return fail(HSTU_ERR_INVALID_ARGUMENT, "waves_per_simd must be 1 or 2");
  if (sink == nullptr || flop == nullptr)
    return fail(HSTU_ERR_INVALID_ARGUMENT, "sink and flop must not be null");
  hipStream_t s = (hipStream_t)stream;
  TimedScope ts("mfma_probe", s);
  HSTU_HIP(launch_mfma_probe(iters, waves_per_simd, sink, flop, s), "mfma probe launch");
  return ok();
}

hstu_status_t hstu_timing_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timing = on != 0;
  return ok();
}

hstu_status_t hstu_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_tmu);
  for (auto& p : g_pending) {
    (void)hipEventSynchronize(p.stop);
    (void)hipEventDestroy(p.start);
    (void)hipEventDestroy(p.stop);
  }
  g_pending.clear();
  g_acc.clear();
  return ok();
}

hstu_status_t hstu_timing_read(const char* name, double* total_ms, int64_t* launches) {
  if (!name || !total_ms || !launches) return fail(HSTU_ERR_INVALID_ARGUMENT, "NULL pointer");
  std::lock_guard<std::mutex> lk(g_tmu);
  for (auto& p : g_pending) {
    hipError_t e = hipEventSynchronize(p.stop);
    float ms = 0.0f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.start, p.stop);
    (void)hipEventDestroy(p.start);
    (void)hipEventDestroy(p.stop);
    if (e != hipSuccess) {
      g_pending.clear();
      return hip_fail(e, "timing events");
    }
    auto& a = g_acc[p.name];
    a.first += ms;
    a.second += 1;
  }
  g_pending.clear();
  auto it = g_acc.find(name);
  *total_ms = it == g_acc.end() ? 0.0 : it->second.first;
  *launches = it == g_acc.end() ? 0 : it->second.second;
  return ok();
}

}  // extern "C"
