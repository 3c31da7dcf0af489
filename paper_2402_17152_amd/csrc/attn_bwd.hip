// Fused jagged pointwise-attention backward, bf16 MFMA (gfx950).
//
// Gradients of <O, dO> for O = (1/N) SiLU(Q K^T + rab) V (Eq. 2).  As the
// paper's kernel appendix describes, attention and the relative bias are
// recomputed rather than stored, and the bias gradients are accumulated
// on chip before they reach HBM.  Pointwise aggregation means no row
// statistics are needed: with S = Q K^T + rab,
//   P  = SiLU(S) (masked),            dV = (1/N) P^T dO
//   dP = dO V^T,  dS = dP SiLU'(S) (masked)
//   dK = (1/N) dS^T Q,  dQ = (1/N) dS K
//   d rab_pos[(N-1)+p(j)-p(i)] += dS/N,  d rab_time[bkt] += dS/N.
//
// Workgroup = 4 waves = one (sequence, 128-key block, head) work item.
// Wave w owns keys j0 + 32w .. +31 and accumulates their dK, dV in
// registers for the whole item; K and V of the block stay in LDS.  The workgroup walks query steps of 32 rows; each step's Q and dO
// rows are staged row-major in LDS (prefetched into registers during the
// previous step).  Per step and wave, on v_mfma_f32_32x32x16_bf16:
//   S  = Q K^T (accumulator seeded with the bias), dP = dO V^T;
//   dV += P^T dO and dK += dS^T Q straight from the accumulator registers,
//         the Q / dO operand fetched with transposing LDS reads in the
//         accumulator's row order;
//   dS -> LDS tile; then the whole workgroup forms dQ(step) = dS K
//         (added to an fp32 workspace with float atomics).
// Bias gradients:
//   time table: per wave and step the slot range of the tile is bounded
//         from timestamp extremes; each slot's dS is summed in registers,
//         reduced across the wave and added to a per-wave LDS row (one
//         slot in far-from-diagonal tiles);
//   position table: after the step, threads own the 159 diagonals of the
//         32 x 128 dS tile and add their sums to an LDS array indexed by
//         p(i) - p(j) -- no atomics, one read-modify-write per diagonal.
// Both are flushed with one global atomic per touched entry at the end.
#include "bias.h"
#include "kernels.h"

namespace hstu {

namespace {

constexpr int64_t kI64Max = 0x7fffffffffffffffll;
constexpr int64_t kI64Min = -kI64Max - 1;

template <int DQK, int DV>
struct BwdShared {
  static constexpr int BN = kBwdBN, BM = kBwdBM;
  static constexpr int Q_LD = DQK + 8, DO_LD = DV + 8;  // row-major step tiles
  static constexpr int DS_LD = BN + 8;
  static constexpr int DS32_LD = BN + 1;
  static constexpr int K_LD = DQK + 8, V_LD = DV + 8;    // the block's keys, row-major
  static constexpr int NWIN = BM + BN;                   // reversed rab_pos window
  __align__(16) uint16_t sQ[BM * Q_LD];
  __align__(16) uint16_t sdO[BM * DO_LD];
  __align__(16) uint16_t sdS[BM * DS_LD];
  float sdS32[BM * DS32_LD];       // dS in fp32 for the bias-table gradients
  __align__(16) uint16_t sK[BN * K_LD];
  __align__(16) uint16_t sV[BN * V_LD];
  __align__(16) uint32_t sTr[BM];  // step row timestamps, rebased (fast path)
  int64_t sTr64[BM];               // step row timestamps (exact path)
  float sWin[NWIN];
  float sTab[64];                  // rab_time by slot
  float sTacc[4][64];              // per-wave time-gradient sums by slot
  int64_t sRange[2];               // extremes of the step's row timestamps
  int64_t sRed[2][4];
};

struct BwdArgs {
  JaggedArgs ja;
  Tensors t;
  const uint16_t* dO;
  float* dq_acc;
  uint16_t* dK;
  uint16_t* dV;
  float* d_rab_pos;
  float* d_rab_time;
  int pos_in_lds;
};

// Slot of t_i - t_j: 32-bit rebased form on the fast path, exact 64-bit otherwise.
template <bool FAST>
__device__ __forceinline__ int slot_of(uint32_t ri, uint32_t rj, int64_t ti, int64_t tj) {
  if constexpr (FAST)
    return slot32(ri, rj);
  else
    return slot64(ti - tj);
}

template <int DQK, int DV, bool FAST>
__device__ __forceinline__ void bwd_item(BwdShared<DQK, DV>& sm, float* __restrict__ sPosAcc,
                                         const BwdArgs& A, int64_t o, int L, int n_h, int j0,
                                         int head, int64_t tbase) {
  using S = BwdShared<DQK, DV>;
  constexpr int BN = S::BN, BM = S::BM, Q_LD = S::Q_LD, DO_LD = S::DO_LD, DS_LD = S::DS_LD,
                DS32_LD = S::DS32_LD, K_LD = S::K_LD, V_LD = S::V_LD, NWIN = S::NWIN;
  constexpr int QCH = BM * DQK / 8, OCH = BM * DV / 8;
  constexpr int QPT = (QCH + 255) / 256, OPT = (OCH + 255) / 256;
  const JaggedArgs& ja = A.ja;
  const int H = ja.num_heads, N = ja.max_seq_len, NB = ja.num_buckets;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  const int jw0 = j0 + 32 * wave;
  const int my_j = jw0 + col;
  const bool key_ok = my_j < L;
  const int pj = bias_pos(my_j, n_h);
  const float invN = 1.0f / (float)N;
  const int64_t* __restrict__ ts = ja.timestamps + o;
  const uint16_t* __restrict__ qg = (const uint16_t*)A.t.q;
  const int R = L - j0;  // p(i) - p(j) of kept pairs lies in [0, R)

  const int64_t tj64 = key_ok ? ts[my_j] : tbase;
  const uint32_t tjr = (uint32_t)(tj64 - tbase);
  const int64_t klo = wave_min_i64(key_ok ? tj64 : kI64Max);
  const int64_t khi = wave_max_i64(key_ok ? tj64 : kI64Min);

  f32x16 dkacc[DQK / 32], dvacc[DV / 32];
#pragma unroll
  for (int nb = 0; nb < DQK / 32; nb++)
#pragma unroll
    for (int q = 0; q < 16; q++) dkacc[nb][q] = 0.0f;
#pragma unroll
  for (int nb = 0; nb < DV / 32; nb++)
#pragma unroll
    for (int q = 0; q < 16; q++) dvacc[nb][q] = 0.0f;

  // Lane addressing of the transposing reads (see lds_read_tr16): lane
  // 16g + r reads row 4*(g/2) + r/4 (+ 8 for the second half of the
  // k-group) and columns 16*(g%2) + 4*(r%4) .. +3 of a 32-column block.
  const int tr_row = 4 * (lane >> 5) + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  // Staging registers for the next step.
  u32x4 pq[QPT], po[OPT];
  int64_t pt = 0;
  float pw = 0.0f;
  auto prefetch = [&](int i0) {
#pragma unroll
    for (int k = 0; k < QPT; k++) {
      const int c = tid + 256 * k;
      if (c < QCH) {
        const int r = c / (DQK / 8), cc = (c % (DQK / 8)) * 8, i = i0 + r;
        pq[k] = i < L ? *reinterpret_cast<const u32x4*>(qg + (o + i) * A.t.q_stride + head * DQK + cc)
                      : zero_u32x4();
      }
    }
#pragma unroll
    for (int k = 0; k < OPT; k++) {
      const int c = tid + 256 * k;
      if (c < OCH) {
        const int r = c / (DV / 8), cc = (c % (DV / 8)) * 8, i = i0 + r;
        po[k] = i < L ? *reinterpret_cast<const u32x4*>(A.dO + ((o + i) * H + head) * DV + cc)
                      : zero_u32x4();
      }
    }
    if (tid < BM) pt = (i0 + tid < L) ? ts[i0 + tid] : tbase;
    if (tid < NWIN) {
      // rab_pos entries reachable from (query step, key block), reversed.
      const int pos_base = (N - 1) + min(j0, n_h) - min(i0 + BM - 1, n_h);
      const int g = pos_base + (NWIN - 1 - tid);
      pw = (g >= 0 && g <= 2 * N - 2) ? ja.rab_pos[g] : 0.0f;
    }
  };

  // Candidate keys see only themselves; otherwise every later row sees them.
  const int i_end = j0 >= n_h ? min(j0 + BN, L) : L;
  prefetch(j0);

  for (int i0 = j0; i0 < i_end; i0 += BM) {
    __syncthreads();  // previous step's LDS tiles consumed
#pragma unroll
    for (int k = 0; k < QPT; k++) {
      const int c = tid + 256 * k;
      if (c < QCH) *reinterpret_cast<u32x4*>(sm.sQ + (c / (DQK / 8)) * Q_LD + (c % (DQK / 8)) * 8) = pq[k];
    }
#pragma unroll
    for (int k = 0; k < OPT; k++) {
      const int c = tid + 256 * k;
      if (c < OCH) *reinterpret_cast<u32x4*>(sm.sdO + (c / (DV / 8)) * DO_LD + (c % (DV / 8)) * 8) = po[k];
    }
    if (tid < BM) {
      if constexpr (FAST)
        sm.sTr[tid] = (uint32_t)(pt - tbase);
      else
        sm.sTr64[tid] = pt;
    }
    if (tid < NWIN) sm.sWin[tid] = pw;
    if (wave == 0) {
      const bool okr = lane < BM && i0 + lane < L;
      const int64_t rlo = wave_min_i64(okr ? pt : kI64Max);
      const int64_t rhi = wave_max_i64(okr ? pt : kI64Min);
      if (lane == 0) {
        sm.sRange[0] = rlo;
        sm.sRange[1] = rhi;
      }
    }
    __syncthreads();
    if (i0 + BM < i_end) prefetch(i0 + BM);

    // Does any kept pair fall in (rows i0..i0+31) x (this wave's keys)?
    const int imax = min(i0 + BM - 1, L - 1);
    bool active = jw0 < L && jw0 <= imax;
    if (jw0 >= n_h && jw0 != i0) active = false;  // candidate keys: diagonal block only

    // dS of this wave's block as bf16 pairs: da[st][e] holds accumulator
    // entries 8st+2e and 8st+2e+1.  The contractions run for every wave:
    // a wave without kept pairs in this step gets an all-zero mask from
    // the general path, so its P and dS are zero and the accumulators
    // stay in straight-line code (no merge of the dK/dV registers).
    u32x4 da[2];
    {
      // Accumulator lane holds (i = i0 + 8g + 4*half + m, j = my_j).
      const bool full = active && (jw0 + 31 <= i0) && (i0 + BM - 1 < L) && (i0 + BM - 1 < n_h);
      f32x16 sacc, pacc;
      uint32_t vmask = 0xffffu;
      if (full) {
        const int yb = (NWIN - 32 - 32 * wave - col) + 4 * half;
        int sl[16];
        float wv[16], tv[16];
#pragma unroll
        for (int q = 0; q < 16; q++) {
          const int il = 8 * (q >> 2) + 4 * half + (q & 3);
          sl[q] = slot_of<FAST>(sm.sTr[il], tjr, sm.sTr64[il], tj64);
        }
#pragma unroll
        for (int q = 0; q < 16; q++) {
          wv[q] = sm.sWin[yb + 8 * (q >> 2) + (q & 3)];
          tv[q] = sm.sTab[sl[q]];
        }
#pragma unroll
        for (int q = 0; q < 16; q++) sacc[q] = wv[q] + tv[q];
      } else {
        vmask = 0;
        const int pos_base = (N - 1) + min(j0, n_h) - min(i0 + BM - 1, n_h);
#pragma unroll
        for (int q = 0; q < 16; q++) {
          const int il = 8 * (q >> 2) + 4 * half + (q & 3);
          const int i = i0 + il;
          const bool ok = key_ok && i < L && pair_valid(i, my_j, n_h);
          const int x = ok ? (N - 1) + pj - bias_pos(i, n_h) - pos_base : 0;
          const int sl = slot_of<FAST>(sm.sTr[il], tjr, sm.sTr64[il], tj64);
          const float b = sm.sWin[NWIN - 1 - x] + sm.sTab[sl];
          sacc[q] = ok ? b : 0.0f;
          vmask |= (uint32_t)ok << q;
        }
      }
#pragma unroll
      for (int q = 0; q < 16; q++) pacc[q] = 0.0f;
      // The S and dP chains are independent: interleave them so each
      // MFMA's accumulator dependency is covered by the other chain.
      constexpr int SMAX = DQK > DV ? DQK / 16 : DV / 16;
#pragma unroll
      for (int s = 0; s < SMAX; s++) {
        if (s < DQK / 16) {
          u32x4 a = *reinterpret_cast<const u32x4*>(sm.sQ + col * Q_LD + 16 * s + 8 * half);
          u32x4 b = *reinterpret_cast<const u32x4*>(sm.sK + (32 * wave + col) * K_LD + 16 * s + 8 * half);
          sacc = mfma32x32x16(as_bf16x8(a), as_bf16x8(b), sacc);
        }
        if (s < DV / 16) {
          u32x4 a = *reinterpret_cast<const u32x4*>(sm.sdO + col * DO_LD + 16 * s + 8 * half);
          u32x4 b = *reinterpret_cast<const u32x4*>(sm.sV + (32 * wave + col) * V_LD + 16 * s + 8 * half);
          pacc = mfma32x32x16(as_bf16x8(a), as_bf16x8(b), pacc);
        }
      }
      float pv[16], dsv[16], sg[16];
#pragma unroll
      for (int q = 0; q < 16; q++) sg[q] = __builtin_amdgcn_exp2f(-sacc[q] * kLog2e);
#pragma unroll
      for (int q = 0; q < 16; q++) sg[q] = __builtin_amdgcn_rcpf(1.0f + sg[q]);
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const float sl = sacc[q] * sg[q];
        const bool ok = (vmask >> q) & 1u;
        pv[q] = ok ? sl : 0.0f;
        dsv[q] = ok ? pacc[q] * (sg[q] + sl * (1.0f - sg[q])) : 0.0f;
      }
      // Time-table gradient: sum dS per slot over the slots this tile spans
      // (a single slot away from the diagonal).
      if (active) {
        int s_lo, s_hi;
        slot_range(sm.sRange[0], sm.sRange[1], klo, khi, s_lo, s_hi);
        if (s_lo == s_hi) {
          float sum = 0.0f;
#pragma unroll
          for (int q = 0; q < 16; q++) sum += dsv[q];
          sum = wave_sum_f32(sum);
          if (lane == 0) sm.sTacc[wave][s_lo] += sum;
        } else {
          for (int s = s_lo; s <= s_hi; s++) {
            float sum = 0.0f;
#pragma unroll
            for (int q = 0; q < 16; q++) {
              const int il = 8 * (q >> 2) + 4 * half + (q & 3);
              const int sl = slot_of<FAST>(sm.sTr[il], tjr, sm.sTr64[il], tj64);
              sum += sl == s ? dsv[q] : 0.0f;
            }
            sum = wave_sum_f32(sum);
            if (lane == 0) sm.sTacc[wave][s] += sum;
          }
        }
      }
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int il = 8 * (q >> 2) + 4 * half + (q & 3);
        sm.sdS32[il * DS32_LD + 32 * wave + col] = dsv[q];
      }
      u32x4 pa[2];
#pragma unroll
      for (int q = 0; q < 16; q += 2) {
        pa[q >> 3][(q & 7) >> 1] = pack_bf16x2(pv[q], pv[q + 1]);
        da[q >> 3][(q & 7) >> 1] = pack_bf16x2(dsv[q], dsv[q + 1]);
      }
      // dV += P^T dO, dK += dS^T Q  (contraction over the step's 32 rows).
#pragma unroll
      for (int st = 0; st < 2; st++) {
        const int row = 16 * st + tr_row;
#pragma unroll
        for (int nb = 0; nb < DV / 32; nb++) {
          const uint16_t* base = sm.sdO + row * DO_LD + 32 * nb + tr_col;
          const uint2 lo = lds_read_tr16(base), hi = lds_read_tr16(base + 8 * DO_LD);
          u32x4 b = {lo.x, lo.y, hi.x, hi.y};
          dvacc[nb] = mfma32x32x16(as_bf16x8(pa[st]), as_bf16x8(b), dvacc[nb]);
        }
#pragma unroll
        for (int nb = 0; nb < DQK / 32; nb++) {
          const uint16_t* base = sm.sQ + row * Q_LD + 32 * nb + tr_col;
          const uint2 lo = lds_read_tr16(base), hi = lds_read_tr16(base + 8 * Q_LD);
          u32x4 b = {lo.x, lo.y, hi.x, hi.y};
          dkacc[nb] = mfma32x32x16(as_bf16x8(da[st]), as_bf16x8(b), dkacc[nb]);
        }
      }
    }
    // dS tile, row-major [32 rows][128 keys] (bf16).
#pragma unroll
    for (int q = 0; q < 16; q++) {
      const int il = 8 * (q >> 2) + 4 * half + (q & 3);
      const uint32_t w = da[q >> 3][(q & 7) >> 1];
      sm.sdS[il * DS_LD + 32 * wave + col] = (uint16_t)((q & 1) ? (w >> 16) : (w & 0xffffu));
    }
    __syncthreads();

    // dQ(step rows) += dS K: each wave one 32-wide d block over a share of keys.
    {
      constexpr int NBLK = DQK / 32;
      constexpr int KSPLIT = 4 / NBLK;
      constexpr int STEPS = (BN / 16) / KSPLIT;
      const int nbq = wave % NBLK, ks = wave / NBLK;
      f32x16 qacc;
#pragma unroll
      for (int q = 0; q < 16; q++) qacc[q] = 0.0f;
#pragma unroll
      for (int st = 0; st < STEPS; st++) {
        const int kk = (ks * STEPS + st) * 16;
        u32x4 a = *reinterpret_cast<const u32x4*>(sm.sdS + col * DS_LD + kk + 8 * half);
        // B = K[kk + 8*half + e][32*nbq + col]: down the rows of the K tile.
        const uint16_t* base = sm.sK + (kk + (tr_row & 3) + 4 * (tr_row >> 2) * 2) * K_LD + 32 * nbq + tr_col;
        const uint2 lo = lds_read_tr16(base), hi = lds_read_tr16(base + 4 * K_LD);
        u32x4 b = {lo.x, lo.y, hi.x, hi.y};
        qacc = mfma32x32x16(as_bf16x8(a), as_bf16x8(b), qacc);
      }
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int i = i0 + 8 * (q >> 2) + 4 * half + (q & 3);
        if (i < L) unsafeAtomicAdd(&A.dq_acc[((o + i) * H + head) * DQK + 32 * nbq + col], qacc[q]);
      }
    }

    // Position-table gradient, history rows: thread tid owns diagonal
    // i_local - j_local = tid - 127, i.e. p(i) - p(j) = i0 - j0 + tid - 127.
    const int rh = max(0, min(BM, n_h - i0));
    if (tid < NWIN - 1) {
      const int dd = tid - (BN - 1);
      const int k = i0 - j0 + dd;
      if (k >= 0) {
        const int ilo = max(0, dd), ihi = min(rh, BN + dd);
        // Rows outside [ilo, ihi) are skipped by predication; the eight
        // partial sums keep the LDS reads independent.
        float part[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int il = 0; il < BM; il++) {
          const int c = il - dd;
          const float v = sm.sdS32[il * DS32_LD + (c < 0 ? 0 : (c > BN - 1 ? BN - 1 : c))];
          part[il & 7] += (il >= ilo && il < ihi) ? v : 0.0f;
        }
        const float sum = ((part[0] + part[1]) + (part[2] + part[3])) +
                          ((part[4] + part[5]) + (part[6] + part[7]));
        if (sum != 0.0f) {
          if (A.pos_in_lds)
            sPosAcc[k] += sum;
          else
            unsafeAtomicAdd(&A.d_rab_pos[(N - 1) - k], sum * invN);
        }
      }
    }
    // Candidate rows (p(i) = n_h): key j < n_h lands on n_h - j, the
    // diagonal (j = i) on 0.
    if (rh < BM && i0 + rh < L) {
      __syncthreads();
      if (tid < BN) {
        const int j = j0 + tid;
        float sum = 0.0f;
        for (int il = rh; il < BM; il++) sum += sm.sdS32[il * DS32_LD + tid];
        if (sum != 0.0f) {
          const int k = j < n_h ? n_h - j : 0;
          if (A.pos_in_lds)
            atomicAdd(&sPosAcc[k], sum);
          else
            unsafeAtomicAdd(&A.d_rab_pos[(N - 1) - k], sum * invN);
        }
      }
    }
  }

  // dK, dV of the wave's keys: lane holds (j = jw0 + 8g + 4*half + m, d = 32nb + col).
#pragma unroll
  for (int q = 0; q < 16; q++) {
    const int j = jw0 + 8 * (q >> 2) + 4 * half + (q & 3);
    if (j < L) {
#pragma unroll
      for (int nb = 0; nb < DQK / 32; nb++)
        A.dK[((o + j) * H + head) * DQK + 32 * nb + col] = f32_to_bf16_bits(dkacc[nb][q] * invN);
#pragma unroll
      for (int nb = 0; nb < DV / 32; nb++)
        A.dV[((o + j) * H + head) * DV + 32 * nb + col] = f32_to_bf16_bits(dvacc[nb][q] * invN);
    }
  }

  __syncthreads();
  if (A.pos_in_lds)
    for (int x = tid; x < R; x += 256) {
      const float v = sPosAcc[x];
      if (v != 0.0f) unsafeAtomicAdd(&A.d_rab_pos[(N - 1) - x], v * invN);
    }
  if (tid < 64) {
    const float v = sm.sTacc[0][tid] + sm.sTacc[1][tid] + sm.sTacc[2][tid] + sm.sTacc[3][tid];
    if (v != 0.0f) unsafeAtomicAdd(&A.d_rab_time[min(63 - tid, NB - 1)], v * invN);
  }
}

template <int DQK, int DV>
__global__ __launch_bounds__(256, 1) void attn_bwd_bf16_kernel(BwdArgs A,
                                                               const WorkItem* __restrict__ items,
                                                               const int32_t* __restrict__ count) {
  using S = BwdShared<DQK, DV>;
  constexpr int BN = S::BN, K_LD = S::K_LD, V_LD = S::V_LD;
  __shared__ S sm;
  extern __shared__ float sPosAcc[];  // [N] when pos_in_lds

  if ((int)blockIdx.x >= *count) return;
  const WorkItem it = items[blockIdx.x];
  const int head = blockIdx.y;
  const JaggedArgs& ja = A.ja;
  const int NB = ja.num_buckets;
  const int64_t o = ja.seq_offsets[it.seq];
  const int L = (int)(ja.seq_offsets[it.seq + 1] - o);
  const int n_h = L - (ja.num_targets ? (int)ja.num_targets[it.seq] : 0);
  const int j0 = it.blk * BN;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t* __restrict__ ts = ja.timestamps + o;
  const uint16_t* __restrict__ kg = (const uint16_t*)A.t.k;
  const uint16_t* __restrict__ vg = (const uint16_t*)A.t.v;

  // Timestamp extremes over the tokens this item touches, [j0, L): the
  // 32-bit fast path applies when they span less than 2^31.
  int64_t tlo = kI64Max, thi = kI64Min;
  for (int x = j0 + tid; x < L; x += 256) {
    const int64_t v = ts[x];
    tlo = v < tlo ? v : tlo;
    thi = v > thi ? v : thi;
  }
  tlo = wave_min_i64(tlo);
  thi = wave_max_i64(thi);
  if (lane == 0) {
    sm.sRed[0][wave] = tlo;
    sm.sRed[1][wave] = thi;
  }
  for (int x = tid; x < 64; x += 256) sm.sTab[x] = ja.rab_time[min(63 - x, NB - 1)];
  for (int x = tid; x < 4 * 64; x += 256) (&sm.sTacc[0][0])[x] = 0.0f;
  if (A.pos_in_lds)
    for (int x = tid; x < L - j0; x += 256) sPosAcc[x] = 0.0f;
  // K and V of the 128-key block, row-major: operands of S = Q K^T and
  // dP = dO V^T (16-byte reads along a key row) and of dQ = dS K
  // (transposing reads down the key rows).
  constexpr int KCH = BN * DQK / 8, VCH = BN * DV / 8;
  for (int c = tid; c < KCH; c += 256) {
    const int r = c / (DQK / 8), cc = (c % (DQK / 8)) * 8;
    const int j = j0 + r;
    *reinterpret_cast<u32x4*>(sm.sK + r * K_LD + cc) =
        j < L ? *reinterpret_cast<const u32x4*>(kg + (o + j) * A.t.k_stride + head * DQK + cc)
              : zero_u32x4();
  }
  for (int c = tid; c < VCH; c += 256) {
    const int r = c / (DV / 8), cc = (c % (DV / 8)) * 8;
    const int j = j0 + r;
    *reinterpret_cast<u32x4*>(sm.sV + r * V_LD + cc) =
        j < L ? *reinterpret_cast<const u32x4*>(vg + (o + j) * A.t.v_stride + head * DV + cc)
              : zero_u32x4();
  }
  __syncthreads();
  tlo = sm.sRed[0][0];
  thi = sm.sRed[1][0];
#pragma unroll
  for (int w = 1; w < 4; w++) {
    tlo = sm.sRed[0][w] < tlo ? sm.sRed[0][w] : tlo;
    thi = sm.sRed[1][w] > thi ? sm.sRed[1][w] : thi;
  }
  if (thi - tlo < ((int64_t)1 << 31))
    bwd_item<DQK, DV, true>(sm, sPosAcc, A, o, L, n_h, j0, head, tlo);
  else
    bwd_item<DQK, DV, false>(sm, sPosAcc, A, o, L, n_h, j0, head, tlo);
}

template <int DQK, int DV>
hipError_t launch_bwd(const JaggedArgs& ja, const Tensors& t, const void* d_out, float* dq_acc,
                      void* dk, void* dv, float* d_rab_pos, float* d_rab_time,
                      const WorkItem* items, const int32_t* count, int64_t max_items,
                      hipStream_t s) {
  BwdArgs A;
  A.ja = ja;
  A.t = t;
  A.dO = (const uint16_t*)d_out;
  A.dq_acc = dq_acc;
  A.dK = (uint16_t*)dk;
  A.dV = (uint16_t*)dv;
  A.d_rab_pos = d_rab_pos;
  A.d_rab_time = d_rab_time;
  // The position-gradient accumulator (N floats) joins the static LDS when
  // both fit in the 160 KiB a gfx950 workgroup may use.
  A.pos_in_lds = sizeof(BwdShared<DQK, DV>) + sizeof(float) * (size_t)ja.max_seq_len <= kLdsBytes;
  const size_t lds = A.pos_in_lds ? sizeof(float) * (size_t)ja.max_seq_len : 0;
  dim3 grid((unsigned)max_items, (unsigned)ja.num_heads);
  hipLaunchKernelGGL((attn_bwd_bf16_kernel<DQK, DV>), grid, dim3(256), lds, s, A, items, count);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bwd_bf16(const JaggedArgs& ja, const Tensors& t, int dqk, int dv,
                                const void* d_out, float* dq_acc, void* dk, void* dv_out,
                                float* d_rab_pos, float* d_rab_time, const WorkItem* items,
                                const int32_t* count, int64_t max_items, hipStream_t s) {
#define HSTU_BWD_CASE(A, B)                                                                  \
  if (dqk == A && dv == B)                                                                   \
    return launch_bwd<A, B>(ja, t, d_out, dq_acc, dk, dv_out, d_rab_pos, d_rab_time, items, \
                            count, max_items, s);
  HSTU_BWD_CASE(32, 32)
  HSTU_BWD_CASE(32, 64)
  HSTU_BWD_CASE(32, 128)
  HSTU_BWD_CASE(64, 32)
  HSTU_BWD_CASE(64, 64)
  HSTU_BWD_CASE(64, 128)
  HSTU_BWD_CASE(128, 32)
  HSTU_BWD_CASE(128, 64)
  HSTU_BWD_CASE(128, 128)
#undef HSTU_BWD_CASE
  return hipErrorInvalidValue;
}

}  // namespace hstu
