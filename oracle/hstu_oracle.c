/*
 * HSTU jagged attention -- CPU ORACLE.  TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 statement of what the hot path computes, used to
 * check the GPU library.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may call it; the product never does.  It
 * shares no code, header or table with the GPU path.
 *
 * Definitions followed (Zhai et al., "Actions Speak Louder than Words",
 * ICML 2024):
 *   - Eq. 2 (spatial aggregation): A V = phi2(Q K^T + rab^{p,t}) V with
 *     phi2 = SiLU and no 1/sqrt(d) scaling;
 *   - Sec. 3.1 (pointwise aggregated attention): the aggregation is
 *     pointwise, normalised by a constant rather than a softmax; the
 *     normaliser is N = max sequence length, passed by the caller;
 *   - notation table, entry rab^{p,t}: one bias shared by all heads,
 *     built from positions and from a bucketisation of t_j - t_i; here
 *     rab = rab_pos[(N-1) + p(j) - p(i)] + rab_time[bucket(t_i - t_j)]
 *     with bucket(x) = min(B_t - 1, floor(log2(max(|x|, 1))));
 *   - Algorithm 1 (M-FALCON), mask construction: a lower-triangular mask
 *     (diagonal included) in which the last n_t tokens (candidates) may
 *     not see one another; every candidate sits at position n_h = L - n_t;
 *   - Eq. 3 (pointwise transformation): Norm(A V) (.) U, Norm = layer norm
 *     over the h*d_v features of a token, biased variance, optional affine,
 *     and its gradient by the chain rule;
 *   - Appendix on the fused kernels: the backward recomputes attention
 *     and the relative bias; gradients flow into both bias tables.
 *
 * Layouts: Q, K [T][h][d_qk]; V, U, O, dO [T][h][d_v]; all row-major fp64.
 * Sequence b occupies tokens [seq_offsets[b], seq_offsets[b+1]).
 *
 * Parallelism: one task per (sequence, head), each task strictly serial;
 * per-task bias-gradient partials are summed afterwards in task order, so
 * results do not depend on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---- scalar building blocks ------------------------------------------ */

/* floor(log2(x)) for x >= 1 by repeated halving (integer, exact). */
static int floor_log2_u64(uint64_t x) {
  int r = 0;
  while (x > 1) {
    x >>= 1;
    r++;
  }
  return r;
}

/* Time bucket of a timestamp difference: min(B_t-1, floor(log2(max(|dt|,1)))). */
int32_t oracle_time_bucket(int64_t dt, int32_t num_buckets) {
  uint64_t a = dt < 0 ? (uint64_t)0 - (uint64_t)dt : (uint64_t)dt;
  if (a < 1) a = 1;
  int b = floor_log2_u64(a);
  return b < num_buckets - 1 ? b : num_buckets - 1;
}

static double silu(double x) { return x / (1.0 + exp(-x)); }

/* d/dx SiLU(x) = sigma(x) * (1 + x * (1 - sigma(x))). */
static double silu_grad(double x) {
  double sg = 1.0 / (1.0 + exp(-x));
  return sg * (1.0 + x * (1.0 - sg));
}

/* Mask of Algorithm 1: causal with the diagonal, candidates (j >= n_h)
 * visible only to themselves. */
static int pair_valid(int64_t i, int64_t j, int64_t n_h) {
  return j <= i && (j < n_h || j == i);
}

/* Position used by the relative bias: candidates all sit at n_h. */
static int64_t bias_pos(int64_t x, int64_t n_h) { return x < n_h ? x : n_h; }

static double pair_bias(int64_t i, int64_t j, int64_t n_h, int32_t N,
                        const int64_t* ts, const double* rab_pos,
                        const double* rab_time, int32_t num_buckets) {
  int64_t pidx = (int64_t)(N - 1) + bias_pos(j, n_h) - bias_pos(i, n_h);
  int32_t tb = oracle_time_bucket(ts[i] - ts[j], num_buckets);
  return rab_pos[pidx] + rab_time[tb];
}

static int64_t seq_targets(const int64_t* num_targets, int32_t b) {
  return num_targets ? num_targets[b] : 0;
}

/* ---- prefix sums ---------------------------------------------------- */

/* out[0] = 0, out[i+1] = out[i] + in[i]   (n+1 outputs). */
void oracle_complete_cumsum(int32_t n, const int64_t* in, int64_t* out) {
  out[0] = 0;
  for (int32_t i = 0; i < n; i++) out[i + 1] = out[i] + in[i];
}

/* ---- standalone bucketisation --------------------------------------- */

/* For each sequence b, writes its L_b x L_b bucket matrix row-major at
 * pair_offsets[b]: entry (i, j) = bucket(t_i - t_j). */
void oracle_time_bucketize(int32_t num_seqs, const int64_t* seq_offsets,
                           const int64_t* timestamps, int32_t num_buckets,
                           const int64_t* pair_offsets, uint8_t* buckets) {
  for (int32_t b = 0; b < num_seqs; b++) {
    int64_t o = seq_offsets[b], L = seq_offsets[b + 1] - o;
    uint8_t* out = buckets + pair_offsets[b];
    for (int64_t i = 0; i < L; i++)
      for (int64_t j = 0; j < L; j++)
        out[i * L + j] = (uint8_t)oracle_time_bucket(
            timestamps[o + i] - timestamps[o + j], num_buckets);
  }
}

/* ---- attention forward (Eq. 2) -------------------------------------- */

void oracle_attn_fwd(int32_t num_seqs, const int64_t* seq_offsets,
                     int32_t N, int32_t H, int32_t dqk, int32_t dv,
                     const int64_t* timestamps, const int64_t* num_targets,
                     const double* rab_pos, const double* rab_time,
                     int32_t num_buckets, const double* q, const double* k,
                     const double* v, double* out) {
  int64_t ntask = (int64_t)num_seqs * H;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t task = 0; task < ntask; task++) {
    int32_t b = (int32_t)(task / H), a = (int32_t)(task % H);
    int64_t o = seq_offsets[b], L = seq_offsets[b + 1] - o;
    int64_t n_h = L - seq_targets(num_targets, b);
    const int64_t* ts = timestamps + o;
    for (int64_t i = 0; i < L; i++) {
      double* orow = out + ((o + i) * H + a) * dv;
      for (int32_t c = 0; c < dv; c++) orow[c] = 0.0;
      const double* qi = q + ((o + i) * H + a) * dqk;
      for (int64_t j = 0; j < L; j++) {
        if (!pair_valid(i, j, n_h)) continue;
        const double* kj = k + ((o + j) * H + a) * dqk;
        const double* vj = v + ((o + j) * H + a) * dv;
        double s = 0.0;
        for (int32_t c = 0; c < dqk; c++) s += qi[c] * kj[c];
        s += pair_bias(i, j, n_h, N, ts, rab_pos, rab_time, num_buckets);
        double att = silu(s) / (double)N;
        for (int32_t c = 0; c < dv; c++) orow[c] += att * vj[c];
      }
    }
  }
}

/* ---- attention backward --------------------------------------------- */

/* Given dO, the gradients of <O, dO> with respect to Q, K, V and both
 * bias tables.  All outputs are overwritten. */
void oracle_attn_bwd(int32_t num_seqs, const int64_t* seq_offsets,
                     int32_t N, int32_t H, int32_t dqk, int32_t dv,
                     const int64_t* timestamps, const int64_t* num_targets,
                     const double* rab_pos, const double* rab_time,
                     int32_t num_buckets, const double* q, const double* k,
                     const double* v, const double* d_out, double* dq,
                     double* dk, double* dv_out, double* d_rab_pos,
                     double* d_rab_time) {
  int64_t T = seq_offsets[num_seqs];
  int64_t npos = 2 * (int64_t)N - 1;
  int64_t ntask = (int64_t)num_seqs * H;
  memset(dq, 0, sizeof(double) * (size_t)(T * H * dqk));
  memset(dk, 0, sizeof(double) * (size_t)(T * H * dqk));
  memset(dv_out, 0, sizeof(double) * (size_t)(T * H * dv));
  double* part_pos = (double*)calloc((size_t)(ntask > 0 ? ntask : 1) * (size_t)npos, sizeof(double));
  double* part_time = (double*)calloc((size_t)(ntask > 0 ? ntask : 1) * (size_t)num_buckets, sizeof(double));

#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t task = 0; task < ntask; task++) {
    int32_t b = (int32_t)(task / H), a = (int32_t)(task % H);
    int64_t o = seq_offsets[b], L = seq_offsets[b + 1] - o;
    int64_t n_h = L - seq_targets(num_targets, b);
    const int64_t* ts = timestamps + o;
    double* ppos = part_pos + task * npos;
    double* ptime = part_time + task * num_buckets;
    for (int64_t i = 0; i < L; i++) {
      const double* qi = q + ((o + i) * H + a) * dqk;
      const double* doi = d_out + ((o + i) * H + a) * dv;
      double* dqi = dq + ((o + i) * H + a) * dqk;
      for (int64_t j = 0; j < L; j++) {
        if (!pair_valid(i, j, n_h)) continue;
        const double* kj = k + ((o + j) * H + a) * dqk;
        const double* vj = v + ((o + j) * H + a) * dv;
        double* dkj = dk + ((o + j) * H + a) * dqk;
        double* dvj = dv_out + ((o + j) * H + a) * dv;
        double s = 0.0, dp = 0.0;
        for (int32_t c = 0; c < dqk; c++) s += qi[c] * kj[c];
        s += pair_bias(i, j, n_h, N, ts, rab_pos, rab_time, num_buckets);
        for (int32_t c = 0; c < dv; c++) dp += doi[c] * vj[c];
        double att = silu(s) / (double)N;
        double ds = dp * silu_grad(s) / (double)N;
        for (int32_t c = 0; c < dv; c++) dvj[c] += att * doi[c];
        for (int32_t c = 0; c < dqk; c++) {
          dqi[c] += ds * kj[c];
          dkj[c] += ds * qi[c];
        }
        int64_t pidx = (int64_t)(N - 1) + bias_pos(j, n_h) - bias_pos(i, n_h);
        ppos[pidx] += ds;
        ptime[oracle_time_bucket(ts[i] - ts[j], num_buckets)] += ds;
      }
    }
  }
  for (int64_t e = 0; e < npos; e++) d_rab_pos[e] = 0.0;
  for (int32_t e = 0; e < num_buckets; e++) d_rab_time[e] = 0.0;
  for (int64_t task = 0; task < ntask; task++) {
    for (int64_t e = 0; e < npos; e++) d_rab_pos[e] += part_pos[task * npos + e];
    for (int32_t e = 0; e < num_buckets; e++)
      d_rab_time[e] += part_time[task * num_buckets + e];
  }
  free(part_pos);
  free(part_time);
}

/* ---- epilogue: LayerNorm(A V) (.) U  (Eq. 3) ------------------------ */

/* x, u, y: [T][D]; gamma, beta: [D] or NULL (identity affine);
 * mean, rstd: [T] or NULL. */
void oracle_ln_gate(int64_t T, int32_t D, const double* x, const double* u,
                    const double* gamma, const double* beta, double eps,
                    double* y, double* mean, double* rstd) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; t++) {
    const double* xr = x + t * D;
    double mu = 0.0, var = 0.0;
    for (int32_t c = 0; c < D; c++) mu += xr[c];
    mu /= (double)D;
    for (int32_t c = 0; c < D; c++) var += (xr[c] - mu) * (xr[c] - mu);
    var /= (double)D;
    double rs = 1.0 / sqrt(var + eps);
    for (int32_t c = 0; c < D; c++) {
      double g = gamma ? gamma[c] : 1.0, bb = beta ? beta[c] : 0.0;
      y[t * D + c] = ((xr[c] - mu) * rs * g + bb) * u[t * D + c];
    }
    if (mean) mean[t] = mu;
    if (rstd) rstd[t] = rs;
  }
}

/* Gradient of <Y, dY> for Y = (z * gamma + beta) (.) u, z = (x - mean) * rstd
 * (the epilogue above), by the chain rule written out per token:
 *   du = (z gamma + beta) dy,  dzn = dy u,  dgamma += dzn z,  dbeta += dzn,
 *   dz = dzn gamma,  dx = rstd (dz - mean(dz) - z mean(dz z)).
 * mean and rstd are recomputed from x.  dgamma, dbeta: [D] (overwritten)
 * or NULL; summed over tokens in token order. */
void oracle_ln_gate_bwd(int64_t T, int32_t D, const double* x, const double* u,
                        const double* dy, const double* gamma, const double* beta,
                        double eps, double* dx, double* du, double* dgamma,
                        double* dbeta) {
  if (dgamma)
    for (int32_t c = 0; c < D; c++) dgamma[c] = 0.0;
  if (dbeta)
    for (int32_t c = 0; c < D; c++) dbeta[c] = 0.0;
  double* z = (double*)malloc(sizeof(double) * (size_t)D);
  double* dz = (double*)malloc(sizeof(double) * (size_t)D);
  for (int64_t t = 0; t < T; t++) {
    const double* xr = x + t * D;
    double mu = 0.0, var = 0.0;
    for (int32_t c = 0; c < D; c++) mu += xr[c];
    mu /= (double)D;
    for (int32_t c = 0; c < D; c++) var += (xr[c] - mu) * (xr[c] - mu);
    var /= (double)D;
    const double rs = 1.0 / sqrt(var + eps);
    double m1 = 0.0, m2 = 0.0;
    for (int32_t c = 0; c < D; c++) {
      const double g = gamma ? gamma[c] : 1.0, bb = beta ? beta[c] : 0.0;
      z[c] = (xr[c] - mu) * rs;
      du[t * D + c] = (z[c] * g + bb) * dy[t * D + c];
      const double dzn = dy[t * D + c] * u[t * D + c];
      if (dgamma) dgamma[c] += dzn * z[c];
      if (dbeta) dbeta[c] += dzn;
      dz[c] = dzn * g;
      m1 += dz[c];
      m2 += dz[c] * z[c];
    }
    m1 /= (double)D;
    m2 /= (double)D;
    for (int32_t c = 0; c < D; c++) dx[t * D + c] = rs * (dz[c] - m1 - z[c] * m2);
  }
  free(z);
  free(dz);
}

int32_t oracle_num_threads(void) {
#ifdef _OPENMP
  return (int32_t)omp_get_max_threads();
#else
  return 1;
#endif
}
