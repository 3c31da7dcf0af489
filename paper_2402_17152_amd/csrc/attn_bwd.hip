// Fused jagged pointwise-attention backward, bf16 MFMA (gfx950).
//
// Gradients of <O, dO> for O = (1/N) SiLU(Q K^T + rab) V (Eq. 2).  As the
// paper's Appendix G describes, attention and the relative bias are
// recomputed rather than stored, and the bias gradients are accumulated
// on chip before they reach HBM.  Pointwise aggregation means no row
// statistics are needed: with S = Q K^T + rab,
//   P  = SiLU(S) (masked),            dV = (1/N) P^T dO
//   dP = dO V^T,  dS = dP SiLU'(S) (masked)
//   dK = (1/N) dS^T Q,  dQ = (1/N) dS K
//   d rab_pos[(N-1)+p(j)-p(i)] += dS/N,  d rab_time[bkt] += dS/N.
//
// Workgroup = 8 waves = one (sequence, 128-key block, head) work item;
// two waves share each SIMD so one wave's MFMA work overlaps the other's
// SiLU and bias arithmetic.  Wave w owns keys j0 + 16w .. +15: their K and
// V sit in registers as MFMA operands and their dK, dV accumulate in
// registers (64 per lane at d = 128) for the whole item.  The workgroup
// walks query steps of 32 rows; each step's Q and dO rows are staged
// row-major in LDS (prefetched into registers during the previous step).
// Per step and wave, on v_mfma_f32_16x16x32_bf16:
//   S  = Q K^T (accumulator seeded with the bias), dP = dO V^T: two 16-row
//        blocks each, lane = key, 4 rows per block in registers;
//   dV += P^T dO and dK += dS^T Q straight from those registers, the
//        contraction order permuted to the accumulator's rows and the
//        Q / dO operand fetched with transposing LDS reads in that order;
//   dS -> LDS (bf16 for dQ, fp32 for the bias gradients); then each wave
//        forms its 16x16 blocks of dQ(step) = dS K over the 128 keys and
//        adds them to an fp32 workspace with float atomics.
// Bias gradients (no per-element atomics):
//   time table: per wave and step the slot range of the tile is bounded
//        from timestamp extremes (usually one slot away from the
//        diagonal); dS is summed per slot, reduced across the wave and
//        added to the wave's LDS row;
//   position table: pairs of threads own the 159 diagonals of the 32x128
//        fp32 dS tile and add their sums to an LDS array indexed by
//        p(i) - p(j).
// Both are flushed with one global atomic per touched entry at the end.
#include "bias.h"
#include "kernels.h"

namespace hstu {

namespace {

constexpr int64_t kI64Max = 0x7fffffffffffffffll;
constexpr int64_t kI64Min = -kI64Max - 1;
constexpr int kBwdThreads = 512;
constexpr int kBwdWaves = kBwdThreads / 64;

template <int DQK, int DV>
struct BwdShared {
  static constexpr int BN = kBwdBN, BM = kBwdBM;
  static constexpr int Q_LD = DQK + 8, DO_LD = DV + 8;  // row-major step tiles
  static constexpr int DS_LD = BN + 8, DS32_LD = BN + 1;
  static constexpr int K_LD = DQK + 8;                   // the block's keys, row-major
  static constexpr int NWIN = BM + BN;                   // reversed rab_pos window
  __align__(16) uint16_t sQ[BM * Q_LD];
  __align__(16) uint16_t sdO[BM * DO_LD];
  __align__(16) uint16_t sdS[BM * DS_LD];
  __align__(16) uint16_t sK[BN * K_LD];
  float sdS32[BM * DS32_LD];         // dS in fp32 for the bias-table gradients
  __align__(16) uint32_t sTr[BM];    // step row timestamps, rebased (fast path)
  int64_t sTr64[BM];                 // step row timestamps (exact path)
  float sWin[NWIN];
  float sTab[64];                    // rab_time by slot
  float sTacc[kBwdWaves][64];        // per-wave time-gradient sums by slot
  int64_t sRange[2];                 // extremes of the step's row timestamps
  int64_t sRed[2][kBwdWaves];
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
                DS32_LD = S::DS32_LD, K_LD = S::K_LD, NWIN = S::NWIN;
  constexpr int QCH = BM * DQK / 8, OCH = BM * DV / 8;
  constexpr int QPT = (QCH + kBwdThreads - 1) / kBwdThreads;
  constexpr int OPT = (OCH + kBwdThreads - 1) / kBwdThreads;
  const JaggedArgs& ja = A.ja;
  const int H = ja.num_heads, N = ja.max_seq_len, NB = ja.num_buckets;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c16 = lane & 15, kg = lane >> 4;
  const int jw0 = j0 + 16 * wave;
  const int my_j = jw0 + c16;
  const bool key_ok = my_j < L;
  const int pj = bias_pos(my_j, n_h);
  const float invN = 1.0f / (float)N;
  const int64_t* __restrict__ ts = ja.timestamps + o;
  const uint16_t* __restrict__ qg = (const uint16_t*)A.t.q + (o * A.t.q_stride + head * DQK);
  const uint16_t* __restrict__ dog = A.dO + (o * H + head) * DV;
  const uint16_t* __restrict__ kg_ = (const uint16_t*)A.t.k;
  const uint16_t* __restrict__ vg_ = (const uint16_t*)A.t.v;
  const int R = L - j0;  // p(i) - p(j) of kept pairs lies in [0, R)

  const int64_t tj64 = key_ok ? ts[my_j] : tbase;
  const uint32_t tjr = (uint32_t)(tj64 - tbase);
  const int64_t klo = wave_min_i64(key_ok ? tj64 : kI64Max);
  const int64_t khi = wave_max_i64(key_ok ? tj64 : kI64Min);

  // K, V of the wave's keys as B operands (lane = key, 8 features per step).
  u32x4 kf[DQK / 32], vf[DV / 32];
#pragma unroll
  for (int s = 0; s < DQK / 32; s++)
    kf[s] = key_ok ? *reinterpret_cast<const u32x4*>(kg_ + (o + my_j) * A.t.k_stride + head * DQK +
                                                     32 * s + 8 * kg)
                   : zero_u32x4();
#pragma unroll
  for (int s = 0; s < DV / 32; s++)
    vf[s] = key_ok ? *reinterpret_cast<const u32x4*>(vg_ + (o + my_j) * A.t.v_stride + head * DV +
                                                     32 * s + 8 * kg)
                   : zero_u32x4();

  // dV, dK accumulators: lane holds keys jw0 + 4kg + m (m = 0..3), feature 16cb + c16.
  f32x4 dvacc[DV / 16], dkacc[DQK / 16];
#pragma unroll
  for (int cb = 0; cb < DV / 16; cb++) dvacc[cb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int cb = 0; cb < DQK / 16; cb++) dkacc[cb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  // Transposing reads (lds_read_tr16): lane 16g + r reads row (r >> 2) of
  // the group's 4-row strip and 4 columns starting at 4*(r & 3).
  const int tr_r = c16 >> 2, tr_c = 4 * (c16 & 3);

  // Staging registers for the next step.
  u32x4 pq[QPT], po[OPT];
  int64_t pt = 0;
  float pw = 0.0f;

  // Candidate keys see only themselves; otherwise every later row sees them.
  const int i_end = j0 >= n_h ? min(j0 + BN, L) : L;

  auto prefetch = [&](int i0) {
#pragma unroll
    for (int k = 0; k < QPT; k++) {
      const int c = tid + kBwdThreads * k;
      if (c < QCH) {
        const int r = c / (DQK / 8), cc = (c % (DQK / 8)) * 8, i = i0 + r;
        pq[k] = i < L ? *reinterpret_cast<const u32x4*>(qg + (int64_t)i * A.t.q_stride + cc)
                      : zero_u32x4();
      }
    }
#pragma unroll
    for (int k = 0; k < OPT; k++) {
      const int c = tid + kBwdThreads * k;
      if (c < OCH) {
        const int r = c / (DV / 8), cc = (c % (DV / 8)) * 8, i = i0 + r;
        po[k] = i < L ? *reinterpret_cast<const u32x4*>(dog + (int64_t)i * H * DV + cc)
                      : zero_u32x4();
      }
    }
    if (tid < BM) pt = (i0 + tid < L) ? ts[i0 + tid] : tbase;
    if (tid >= 64 && tid < 64 + NWIN) {
      // rab_pos entries reachable from (query step, key block), reversed.
      const int x = tid - 64;
      const int pos_base = (N - 1) + min(j0, n_h) - min(i0 + BM - 1, n_h);
      const int g = pos_base + (NWIN - 1 - x);
      pw = (g >= 0 && g <= 2 * N - 2) ? ja.rab_pos[g] : 0.0f;
    }
  };

  prefetch(j0);

  for (int i0 = j0; i0 < i_end; i0 += BM) {
    __syncthreads();  // previous step's LDS tiles consumed
#pragma unroll
    for (int k = 0; k < QPT; k++) {
      const int c = tid + kBwdThreads * k;
      if (c < QCH) *reinterpret_cast<u32x4*>(sm.sQ + (c / (DQK / 8)) * Q_LD + (c % (DQK / 8)) * 8) = pq[k];
    }
#pragma unroll
    for (int k = 0; k < OPT; k++) {
      const int c = tid + kBwdThreads * k;
      if (c < OCH) *reinterpret_cast<u32x4*>(sm.sdO + (c / (DV / 8)) * DO_LD + (c % (DV / 8)) * 8) = po[k];
    }
    if (tid < BM) {
      if constexpr (FAST)
        sm.sTr[tid] = (uint32_t)(pt - tbase);
      else
        sm.sTr64[tid] = pt;
    }
    if (tid >= 64 && tid < 64 + NWIN) sm.sWin[tid - 64] = pw;
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
    if (jw0 >= n_h && (jw0 + 15 < i0 || jw0 > imax)) active = false;  // candidates: diagonal only
    // Every key of the wave precedes every row, all rows are history rows.
    const bool full = (jw0 + 15 <= i0) && (i0 + BM - 1 < L) && (i0 + BM - 1 < n_h);

    // Scores and dP, accumulator seeded with the bias.  sacc[rb][m] holds
    // (row i0 + 16rb + 4kg + m, key my_j).  A wave without kept pairs gets
    // an all-zero mask from the general branch, so its P and dS vanish and
    // the contractions below stay unconditional.
    f32x4 sacc[2], pacc[2];
    uint32_t vmask = 0xffu;
    if (full) {
      const int yb = (NWIN - 32 - 16 * wave - c16) + 4 * kg;
      int sl[8];
      float wv[8], tv[8];
#pragma unroll
      for (int q = 0; q < 8; q++) {
        const int il = 16 * (q >> 2) + 4 * kg + (q & 3);
        sl[q] = slot_of<FAST>(sm.sTr[il], tjr, sm.sTr64[il], tj64);
      }
#pragma unroll
      for (int q = 0; q < 8; q++) {
        wv[q] = sm.sWin[yb + 16 * (q >> 2) + (q & 3)];
        tv[q] = sm.sTab[sl[q]];
      }
#pragma unroll
      for (int q = 0; q < 8; q++) sacc[q >> 2][q & 3] = wv[q] + tv[q];
    } else {
      vmask = 0;
      const int pos_base = (N - 1) + min(j0, n_h) - min(i0 + BM - 1, n_h);
#pragma unroll
      for (int q = 0; q < 8; q++) {
        const int il = 16 * (q >> 2) + 4 * kg + (q & 3);
        const int i = i0 + il;
        const bool ok = key_ok && i < L && pair_valid(i, my_j, n_h);
        const int x = ok ? (N - 1) + pj - bias_pos(i, n_h) - pos_base : 0;
        const int sl = slot_of<FAST>(sm.sTr[il], tjr, sm.sTr64[il], tj64);
        const float b = sm.sWin[NWIN - 1 - x] + sm.sTab[sl];
        sacc[q >> 2][q & 3] = ok ? b : 0.0f;
        vmask |= (uint32_t)ok << q;
      }
    }
    pacc[0] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    pacc[1] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    {
      constexpr int SMAX = DQK > DV ? DQK / 32 : DV / 32;
#pragma unroll
      for (int s = 0; s < SMAX; s++) {
#pragma unroll
        for (int rb = 0; rb < 2; rb++) {
          if (s < DQK / 32) {
            u32x4 a = *reinterpret_cast<const u32x4*>(sm.sQ + (16 * rb + c16) * Q_LD + 32 * s + 8 * kg);
            sacc[rb] = mfma16x16x32(as_bf16x8(a), as_bf16x8(kf[s]), sacc[rb]);
          }
          if (s < DV / 32) {
            u32x4 a = *reinterpret_cast<const u32x4*>(sm.sdO + (16 * rb + c16) * DO_LD + 32 * s + 8 * kg);
            pacc[rb] = mfma16x16x32(as_bf16x8(a), as_bf16x8(vf[s]), pacc[rb]);
          }
        }
      }
    }
    // SiLU, SiLU' and dS in fp32.
    float pv[8], dsv[8], sg[8];
#pragma unroll
    for (int q = 0; q < 8; q++) sg[q] = __builtin_amdgcn_exp2f(-sacc[q >> 2][q & 3] * kLog2e);
#pragma unroll
    for (int q = 0; q < 8; q++) sg[q] = __builtin_amdgcn_rcpf(1.0f + sg[q]);
#pragma unroll
    for (int q = 0; q < 8; q++) {
      const float x = sacc[q >> 2][q & 3];
      const float sl = x * sg[q];
      const bool ok = (vmask >> q) & 1u;
      pv[q] = ok ? sl : 0.0f;
      dsv[q] = ok ? pacc[q >> 2][q & 3] * (sg[q] + sl * (1.0f - sg[q])) : 0.0f;
    }
    // Time-table gradient: sum dS per slot over the slots this tile spans.
    if (active) {
      int s_lo, s_hi;
      slot_range(sm.sRange[0], sm.sRange[1], klo, khi, s_lo, s_hi);
      if (s_lo == s_hi) {
        float sum = 0.0f;
#pragma unroll
        for (int q = 0; q < 8; q++) sum += dsv[q];
        sum = wave_sum_f32(sum);
        if (lane == 0) sm.sTacc[wave][s_lo] += sum;
      } else {
        for (int s = s_lo; s <= s_hi; s++) {
          float sum = 0.0f;
#pragma unroll
          for (int q = 0; q < 8; q++) {
            const int il = 16 * (q >> 2) + 4 * kg + (q & 3);
            const int sl = slot_of<FAST>(sm.sTr[il], tjr, sm.sTr64[il], tj64);
            sum += sl == s ? dsv[q] : 0.0f;
          }
          sum = wave_sum_f32(sum);
          if (lane == 0) sm.sTacc[wave][s] += sum;
        }
      }
    }
    // P^T and dS^T as A operands: k-slots 0..3 = rows 4kg + 0..3,
    // k-slots 4..7 = rows 16 + 4kg + 0..3 (the accumulator's own rows).
    u32x4 pa, da;
    pa[0] = pack_bf16x2(pv[0], pv[1]);
    pa[1] = pack_bf16x2(pv[2], pv[3]);
    pa[2] = pack_bf16x2(pv[4], pv[5]);
    pa[3] = pack_bf16x2(pv[6], pv[7]);
    da[0] = pack_bf16x2(dsv[0], dsv[1]);
    da[1] = pack_bf16x2(dsv[2], dsv[3]);
    da[2] = pack_bf16x2(dsv[4], dsv[5]);
    da[3] = pack_bf16x2(dsv[6], dsv[7]);
    // dS tiles: bf16 for dQ, fp32 for the bias gradients.
#pragma unroll
    for (int q = 0; q < 8; q++) {
      const int il = 16 * (q >> 2) + 4 * kg + (q & 3);
      sm.sdS32[il * DS32_LD + 16 * wave + c16] = dsv[q];
      const uint32_t w = da[q >> 1];
      sm.sdS[il * DS_LD + 16 * wave + c16] = (uint16_t)((q & 1) ? (w >> 16) : (w & 0xffffu));
    }
    // dV += P^T dO, dK += dS^T Q (contraction over the step's 32 rows).
    {
      const int row0 = 4 * kg + tr_r;
#pragma unroll
      for (int cb = 0; cb < DV / 16; cb++) {
        const uint16_t* base = sm.sdO + row0 * DO_LD + 16 * cb + tr_c;
        const uint2 lo = lds_read_tr16(base), hi = lds_read_tr16(base + 16 * DO_LD);
        u32x4 b = {lo.x, lo.y, hi.x, hi.y};
        dvacc[cb] = mfma16x16x32(as_bf16x8(pa), as_bf16x8(b), dvacc[cb]);
      }
#pragma unroll
      for (int cb = 0; cb < DQK / 16; cb++) {
        const uint16_t* base = sm.sQ + row0 * Q_LD + 16 * cb + tr_c;
        const uint2 lo = lds_read_tr16(base), hi = lds_read_tr16(base + 16 * Q_LD);
        u32x4 b = {lo.x, lo.y, hi.x, hi.y};
        dkacc[cb] = mfma16x16x32(as_bf16x8(da), as_bf16x8(b), dkacc[cb]);
      }
    }
    __syncthreads();

    // dQ(step rows) += dS K: 2 row blocks x DQK/16 column blocks shared by
    // the 8 waves; each wave takes row block w & 1 and its share of the
    // column blocks, contracting over all 128 keys (or half of them when
    // there are fewer column blocks than wave pairs).
    {
      constexpr int NCB = DQK / 16;
      constexpr int CB_PER = NCB >= 4 ? NCB / 4 : 1;       // column blocks per wave
      constexpr int KSPLIT = NCB >= 4 ? 1 : 4 / NCB;       // key splits per block
      constexpr int KSTEPS = (BN / 32) / KSPLIT;
      const int rb = wave & 1;
      const int grp = wave >> 1;                           // 0..3
      const int cb0 = (grp / KSPLIT) * CB_PER;
      const int ks0 = (grp % KSPLIT) * KSTEPS;
#pragma unroll
      for (int u = 0; u < CB_PER; u++) {
        const int cb = cb0 + u;
        f32x4 qacc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ks++) {
          const int kk = 32 * (ks0 + ks);
          u32x4 a = *reinterpret_cast<const u32x4*>(sm.sdS + (16 * rb + c16) * DS_LD + kk + 8 * kg);
          // B = K[kk + 8kg + e][16cb + c16]: down the rows of the key tile.
          const uint16_t* base = sm.sK + (kk + 8 * kg + tr_r) * K_LD + 16 * cb + tr_c;
          const uint2 lo = lds_read_tr16(base), hi = lds_read_tr16(base + 4 * K_LD);
          u32x4 b = {lo.x, lo.y, hi.x, hi.y};
          qacc = mfma16x16x32(as_bf16x8(a), as_bf16x8(b), qacc);
        }
#pragma unroll
        for (int m = 0; m < 4; m++) {
          const int i = i0 + 16 * rb + 4 * kg + m;
          if (i < L) unsafeAtomicAdd(&A.dq_acc[((o + i) * H + head) * DQK + 16 * cb + c16], qacc[m]);
        }
      }
    }

    // Position-table gradient, history rows: threads 2t, 2t+1 own diagonal
    // i_local - j_local = t - 127 (rows 0..15 and 16..31 respectively),
    // i.e. p(i) - p(j) = i0 - j0 + t - 127.
    const int rh = max(0, min(BM, n_h - i0));
    if (tid < 2 * (NWIN - 1)) {
      const int dd = (tid >> 1) - (BN - 1);
      const int k = i0 - j0 + dd;
      const int lo = max(max(0, dd), 16 * (tid & 1)), hi = min(min(rh, BN + dd), 16 * (tid & 1) + 16);
      float part[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int u = 0; u < 16; u++) {
        const int il = 16 * (tid & 1) + u;
        const int c = il - dd;
        const float v = sm.sdS32[il * DS32_LD + (c < 0 ? 0 : (c > BN - 1 ? BN - 1 : c))];
        part[u & 3] += (il >= lo && il < hi) ? v : 0.0f;
      }
      float sum = (part[0] + part[1]) + (part[2] + part[3]);
      sum += __shfl_xor(sum, 1, 64);
      if ((tid & 1) == 0 && k >= 0 && sum != 0.0f) {
        if (A.pos_in_lds)
          sPosAcc[k] += sum;
        else
          unsafeAtomicAdd(&A.d_rab_pos[(N - 1) - k], sum * invN);
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

  // dK, dV of the wave's keys: lane holds (j = jw0 + 4kg + m, d = 16cb + c16).
#pragma unroll
  for (int m = 0; m < 4; m++) {
    const int j = jw0 + 4 * kg + m;
    if (j < L) {
#pragma unroll
      for (int cb = 0; cb < DQK / 16; cb++)
        A.dK[((o + j) * H + head) * DQK + 16 * cb + c16] = f32_to_bf16_bits(dkacc[cb][m] * invN);
#pragma unroll
      for (int cb = 0; cb < DV / 16; cb++)
        A.dV[((o + j) * H + head) * DV + 16 * cb + c16] = f32_to_bf16_bits(dvacc[cb][m] * invN);
    }
  }

  __syncthreads();
  if (A.pos_in_lds)
    for (int x = tid; x < R; x += kBwdThreads) {
      const float v = sPosAcc[x];
      if (v != 0.0f) unsafeAtomicAdd(&A.d_rab_pos[(N - 1) - x], v * invN);
    }
  if (tid < 64) {
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < kBwdWaves; w++) v += sm.sTacc[w][tid];
    if (v != 0.0f) unsafeAtomicAdd(&A.d_rab_time[min(63 - tid, NB - 1)], v * invN);
  }
}

template <int DQK, int DV>
__global__ __launch_bounds__(kBwdThreads, 1) void attn_bwd_bf16_kernel(
    BwdArgs A, const WorkItem* __restrict__ items, const int32_t* __restrict__ count) {
  using S = BwdShared<DQK, DV>;
  constexpr int BN = S::BN, K_LD = S::K_LD;
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

  // Timestamp extremes over the tokens this item touches, [j0, L): the
  // 32-bit fast path applies when they span less than 2^31.
  int64_t tlo = kI64Max, thi = kI64Min;
  for (int x = j0 + tid; x < L; x += kBwdThreads) {
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
  for (int x = tid; x < 64; x += kBwdThreads) sm.sTab[x] = ja.rab_time[min(63 - x, NB - 1)];
  for (int x = tid; x < kBwdWaves * 64; x += kBwdThreads) (&sm.sTacc[0][0])[x] = 0.0f;
  if (A.pos_in_lds)
    for (int x = tid; x < L - j0; x += kBwdThreads) sPosAcc[x] = 0.0f;
  // K of the 128-key block, row-major: operand of dQ = dS K (read down
  // the key rows with transposing reads).
  constexpr int KCH = BN * DQK / 8;
  for (int c = tid; c < KCH; c += kBwdThreads) {
    const int r = c / (DQK / 8), cc = (c % (DQK / 8)) * 8;
    const int j = j0 + r;
    *reinterpret_cast<u32x4*>(sm.sK + r * K_LD + cc) =
        j < L ? *reinterpret_cast<const u32x4*>(kg + (o + j) * A.t.k_stride + head * DQK + cc)
              : zero_u32x4();
  }
  __syncthreads();
  tlo = sm.sRed[0][0];
  thi = sm.sRed[1][0];
#pragma unroll
  for (int w = 1; w < kBwdWaves; w++) {
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
  hipLaunchKernelGGL((attn_bwd_bf16_kernel<DQK, DV>), grid, dim3(kBwdThreads), lds, s, A, items,
                     count);
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
