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
// Wave w owns keys j0 + 32w .. +31: their K and V sit in registers as
// MFMA operands and their dK, dV accumulate in registers for the whole
// item.  The workgroup walks query steps of 32 rows; each step's Q and dO
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
__global__ __launch_bounds__(256, 1) void attn_bwd_bf16_kernel(
    JaggedArgs ja, Tensors t, const uint16_t* __restrict__ dO, float* __restrict__ dq_acc,
    uint16_t* __restrict__ dK, uint16_t* __restrict__ dV, float* __restrict__ d_rab_pos,
    float* __restrict__ d_rab_time, const WorkItem* __restrict__ items,
    const int32_t* __restrict__ count, int pos_in_lds) {
  constexpr int BN = kBwdBN, BM = kBwdBM;
  constexpr int Q_LD = DQK + 8, DO_LD = DV + 8;  // row-major step tiles
  constexpr int DS_LD = BN + 8, KT_LD = BN + 8;
  constexpr int NWIN = BM + BN;                   // reversed rab_pos window
  constexpr int QCH = BM * DQK / 8, OCH = BM * DV / 8;
  constexpr int QPT = (QCH + 255) / 256, OPT = (OCH + 255) / 256;
  static_assert(BN == 128 && BM == 32, "4 waves x 32 keys, 32-row query steps");

  __shared__ __align__(16) uint16_t sQ[BM * Q_LD];
  __shared__ __align__(16) uint16_t sdO[BM * DO_LD];
  __shared__ __align__(16) uint16_t sdS[BM * DS_LD];
  __shared__ __align__(16) uint16_t sKT[DQK * KT_LD];
  __shared__ __align__(16) uint32_t sTr[BM];   // step row timestamps, rebased
  __shared__ int64_t sTr64[BM];                // step row timestamps
  __shared__ float sWin[NWIN];
  __shared__ float sTab[64];                   // rab_time by slot
  __shared__ float sTacc[4][64];               // per-wave time-gradient sums by slot
  __shared__ int64_t sRange[2];                // extremes of the step's row timestamps
  __shared__ int64_t sRed[2][4];
  extern __shared__ float sPosAcc[];           // [N] when pos_in_lds

  if ((int)blockIdx.x >= *count) return;
  const WorkItem it = items[blockIdx.x];
  const int head = blockIdx.y;
  const int H = ja.num_heads, N = ja.max_seq_len, NB = ja.num_buckets;
  const int64_t o = ja.seq_offsets[it.seq];
  const int L = (int)(ja.seq_offsets[it.seq + 1] - o);
  const int n_h = L - (ja.num_targets ? (int)ja.num_targets[it.seq] : 0);
  const int j0 = it.blk * BN;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  const int jw0 = j0 + 32 * wave;
  const int my_j = jw0 + col;
  const bool key_ok = my_j < L;
  const int pj = bias_pos(my_j, n_h);
  const float invN = 1.0f / (float)N;
  const int64_t* __restrict__ ts = ja.timestamps + o;

  const uint16_t* __restrict__ qg = (const uint16_t*)t.q;
  const uint16_t* __restrict__ kg = (const uint16_t*)t.k;
  const uint16_t* __restrict__ vg = (const uint16_t*)t.v;

  // Timestamp extremes over the tokens this item touches, [j0, L).
  int64_t tlo = kI64Max, thi = kI64Min;
  for (int x = j0 + tid; x < L; x += 256) {
    const int64_t v = ts[x];
    tlo = v < tlo ? v : tlo;
    thi = v > thi ? v : thi;
  }
  tlo = wave_min_i64(tlo);
  thi = wave_max_i64(thi);
  if (lane == 0) {
    sRed[0][wave] = tlo;
    sRed[1][wave] = thi;
  }
  for (int x = tid; x < 64; x += 256) sTab[x] = ja.rab_time[min(63 - x, NB - 1)];
  for (int x = tid; x < 4 * 64; x += 256) (&sTacc[0][0])[x] = 0.0f;
  const int R = L - j0;  // p(i) - p(j) of kept pairs lies in [0, R)
  if (pos_in_lds)
    for (int x = tid; x < R; x += 256) sPosAcc[x] = 0.0f;
  // K^T of the 128-key block (operand of dQ = dS K).
  constexpr int KCH = BN * DQK / 8;
  for (int c = tid; c < KCH; c += 256) {
    const int r = c / (DQK / 8), cc = (c % (DQK / 8)) * 8;
    const int j = j0 + r;
    u32x4 v = j < L ? *reinterpret_cast<const u32x4*>(kg + (o + j) * t.k_stride + head * DQK + cc)
                    : zero_u32x4();
#pragma unroll
    for (int e = 0; e < 8; e++) sKT[(cc + e) * KT_LD + r] = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
  }
  __syncthreads();
  tlo = sRed[0][0];
  thi = sRed[1][0];
#pragma unroll
  for (int w = 1; w < 4; w++) {
    tlo = sRed[0][w] < tlo ? sRed[0][w] : tlo;
    thi = sRed[1][w] > thi ? sRed[1][w] : thi;
  }
  const bool fast = (thi - tlo) < ((int64_t)1 << 31);
  const int64_t tbase = tlo;
  const int64_t tj64 = key_ok ? ts[my_j] : tbase;
  const uint32_t tjr = (uint32_t)(tj64 - tbase);
  const int64_t klo = wave_min_i64(key_ok ? tj64 : kI64Max);
  const int64_t khi = wave_max_i64(key_ok ? tj64 : kI64Min);

  // K, V of the wave's keys as B operands (lane = key, 8 features per step).
  u32x4 kf[DQK / 16], vf[DV / 16];
#pragma unroll
  for (int s = 0; s < DQK / 16; s++)
    kf[s] = key_ok ? *reinterpret_cast<const u32x4*>(kg + (o + my_j) * t.k_stride + head * DQK +
                                                     16 * s + 8 * half)
                   : zero_u32x4();
#pragma unroll
  for (int s = 0; s < DV / 16; s++)
    vf[s] = key_ok ? *reinterpret_cast<const u32x4*>(vg + (o + my_j) * t.v_stride + head * DV +
                                                     16 * s + 8 * half)
                   : zero_u32x4();

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
        pq[k] = i < L ? *reinterpret_cast<const u32x4*>(qg + (o + i) * t.q_stride + head * DQK + cc)
                      : zero_u32x4();
      }
    }
#pragma unroll
    for (int k = 0; k < OPT; k++) {
      const int c = tid + 256 * k;
      if (c < OCH) {
        const int r = c / (DV / 8), cc = (c % (DV / 8)) * 8, i = i0 + r;
        po[k] = i < L ? *reinterpret_cast<const u32x4*>(dO + ((o + i) * H + head) * DV + cc)
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
      if (c < QCH) *reinterpret_cast<u32x4*>(sQ + (c / (DQK / 8)) * Q_LD + (c % (DQK / 8)) * 8) = pq[k];
    }
#pragma unroll
    for (int k = 0; k < OPT; k++) {
      const int c = tid + 256 * k;
      if (c < OCH) *reinterpret_cast<u32x4*>(sdO + (c / (DV / 8)) * DO_LD + (c % (DV / 8)) * 8) = po[k];
    }
    if (tid < BM) {
      sTr64[tid] = pt;
      sTr[tid] = (uint32_t)(pt - tbase);
    }
    if (tid < NWIN) sWin[tid] = pw;
    if (wave == 0) {
      const bool okr = lane < BM && i0 + lane < L;
      const int64_t rlo = wave_min_i64(okr ? pt : kI64Max);
      const int64_t rhi = wave_max_i64(okr ? pt : kI64Min);
      if (lane == 0) {
        sRange[0] = rlo;
        sRange[1] = rhi;
      }
    }
    __syncthreads();
    if (i0 + BM < i_end) prefetch(i0 + BM);

    // Does any kept pair fall in (rows i0..i0+31) x (this wave's keys)?
    const int imax = min(i0 + BM - 1, L - 1);
    bool active = jw0 < L && jw0 <= imax;
    if (jw0 >= n_h && jw0 != i0) active = false;  // candidate keys: diagonal block only

    float ds[16];
    if (active) {
      // Accumulator lane holds (i = i0 + 8g + 4*half + m, j = my_j).
      const bool full = (jw0 + 31 <= i0) && (i0 + BM - 1 < L) && (i0 + BM - 1 < n_h);
      f32x16 sacc, pacc;
      int slot[16];
      uint32_t vmask = 0xffffu;
      if (full) {
        const int yb = (NWIN - 32 - 32 * wave - col) + 4 * half;
#pragma unroll
        for (int q = 0; q < 16; q++) {
          const int il = 8 * (q >> 2) + 4 * half + (q & 3);
          slot[q] = fast ? slot32(sTr[il], tjr) : slot64(sTr64[il] - tj64);
          sacc[q] = sWin[yb + 8 * (q >> 2) + (q & 3)] + sTab[slot[q]];
        }
      } else {
        vmask = 0;
        const int pos_base = (N - 1) + min(j0, n_h) - min(i0 + BM - 1, n_h);
#pragma unroll
        for (int q = 0; q < 16; q++) {
          const int il = 8 * (q >> 2) + 4 * half + (q & 3);
          const int i = i0 + il;
          float b = 0.0f;
          int s = 0;
          if (key_ok && i < L && pair_valid(i, my_j, n_h)) {
            const int x = (N - 1) + pj - bias_pos(i, n_h) - pos_base;
            s = fast ? slot32(sTr[il], tjr) : slot64(sTr64[il] - tj64);
            b = sWin[NWIN - 1 - x] + sTab[s];
            vmask |= 1u << q;
          }
          slot[q] = s;
          sacc[q] = b;
        }
      }
#pragma unroll
      for (int q = 0; q < 16; q++) pacc[q] = 0.0f;
#pragma unroll
      for (int s = 0; s < DQK / 16; s++) {
        u32x4 a = *reinterpret_cast<const u32x4*>(sQ + col * Q_LD + 16 * s + 8 * half);
        sacc = mfma32x32x16(as_bf16x8(a), as_bf16x8(kf[s]), sacc);
      }
#pragma unroll
      for (int s = 0; s < DV / 16; s++) {
        u32x4 a = *reinterpret_cast<const u32x4*>(sdO + col * DO_LD + 16 * s + 8 * half);
        pacc = mfma32x32x16(as_bf16x8(a), as_bf16x8(vf[s]), pacc);
      }
      float p[16];
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const float x = sacc[q];
        const float sg = sigmoid_fast(x);
        const float sl = x * sg;
        const bool ok = (vmask >> q) & 1u;
        p[q] = ok ? sl : 0.0f;
        ds[q] = ok ? pacc[q] * (sg + sl * (1.0f - sg)) : 0.0f;
      }
      // dV += P^T dO, dK += dS^T Q  (contraction over the step's 32 rows).
#pragma unroll
      for (int st = 0; st < 2; st++) {
        u32x4 pa, da;
#pragma unroll
        for (int e = 0; e < 4; e++) {
          pa[e] = pack_bf16x2(p[8 * st + 2 * e], p[8 * st + 2 * e + 1]);
          da[e] = pack_bf16x2(ds[8 * st + 2 * e], ds[8 * st + 2 * e + 1]);
        }
        const int row = 16 * st + tr_row;
#pragma unroll
        for (int nb = 0; nb < DV / 32; nb++) {
          const uint16_t* base = sdO + row * DO_LD + 32 * nb + tr_col;
          const uint2 lo = lds_read_tr16(base), hi = lds_read_tr16(base + 8 * DO_LD);
          u32x4 b = {lo.x, lo.y, hi.x, hi.y};
          dvacc[nb] = mfma32x32x16(as_bf16x8(pa), as_bf16x8(b), dvacc[nb]);
        }
#pragma unroll
        for (int nb = 0; nb < DQK / 32; nb++) {
          const uint16_t* base = sQ + row * Q_LD + 32 * nb + tr_col;
          const uint2 lo = lds_read_tr16(base), hi = lds_read_tr16(base + 8 * Q_LD);
          u32x4 b = {lo.x, lo.y, hi.x, hi.y};
          dkacc[nb] = mfma32x32x16(as_bf16x8(da), as_bf16x8(b), dkacc[nb]);
        }
      }
      // Time-table gradient: sum dS per slot over the slots this tile spans.
      int s_lo, s_hi;
      slot_range(sRange[0], sRange[1], klo, khi, s_lo, s_hi);
      if (s_lo == s_hi) {
        float sum = 0.0f;
#pragma unroll
        for (int q = 0; q < 16; q++) sum += ds[q];
        sum = wave_sum_f32(sum);
        if (lane == 0) sTacc[wave][s_lo] += sum;
      } else {
        for (int s = s_lo; s <= s_hi; s++) {
          float sum = 0.0f;
#pragma unroll
          for (int q = 0; q < 16; q++) sum += slot[q] == s ? ds[q] : 0.0f;
          sum = wave_sum_f32(sum);
          if (lane == 0) sTacc[wave][s] += sum;
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < 16; q++) ds[q] = 0.0f;
    }
    // dS tile, row-major [32 rows][128 keys] (bf16).
#pragma unroll
    for (int q = 0; q < 16; q++) {
      const int il = 8 * (q >> 2) + 4 * half + (q & 3);
      sdS[il * DS_LD + 32 * wave + col] = f32_to_bf16_bits(ds[q]);
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
        const int kk = (ks * STEPS + st) * 16 + 8 * half;
        u32x4 a = *reinterpret_cast<const u32x4*>(sdS + col * DS_LD + kk);
        u32x4 b = *reinterpret_cast<const u32x4*>(sKT + (32 * nbq + col) * KT_LD + kk);
        qacc = mfma32x32x16(as_bf16x8(a), as_bf16x8(b), qacc);
      }
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int i = i0 + 8 * (q >> 2) + 4 * half + (q & 3);
        if (i < L) unsafeAtomicAdd(&dq_acc[((o + i) * H + head) * DQK + 32 * nbq + col], qacc[q]);
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
        float sum = 0.0f;
        for (int il = ilo; il < ihi; il++)
          sum += bf16_bits_to_f32(sdS[il * DS_LD + il - dd]);
        if (sum != 0.0f) {
          if (pos_in_lds)
            sPosAcc[k] += sum;
          else
            unsafeAtomicAdd(&d_rab_pos[(N - 1) - k], sum * invN);
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
        for (int il = rh; il < BM; il++) sum += bf16_bits_to_f32(sdS[il * DS_LD + tid]);
        if (sum != 0.0f) {
          const int k = j < n_h ? n_h - j : 0;
          if (pos_in_lds)
            atomicAdd(&sPosAcc[k], sum);
          else
            unsafeAtomicAdd(&d_rab_pos[(N - 1) - k], sum * invN);
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
        dK[((o + j) * H + head) * DQK + 32 * nb + col] = f32_to_bf16_bits(dkacc[nb][q] * invN);
#pragma unroll
      for (int nb = 0; nb < DV / 32; nb++)
        dV[((o + j) * H + head) * DV + 32 * nb + col] = f32_to_bf16_bits(dvacc[nb][q] * invN);
    }
  }

  __syncthreads();
  if (pos_in_lds)
    for (int x = tid; x < R; x += 256) {
      const float v = sPosAcc[x];
      if (v != 0.0f) unsafeAtomicAdd(&d_rab_pos[(N - 1) - x], v * invN);
    }
  if (tid < 64) {
    const float v = sTacc[0][tid] + sTacc[1][tid] + sTacc[2][tid] + sTacc[3][tid];
    if (v != 0.0f) unsafeAtomicAdd(&d_rab_time[min(63 - tid, NB - 1)], v * invN);
  }
}

template <int DQK, int DV>
hipError_t launch_bwd(const JaggedArgs& ja, const Tensors& t, const void* d_out, float* dq_acc,
                      void* dk, void* dv, float* d_rab_pos, float* d_rab_time,
                      const WorkItem* items, const int32_t* count, int64_t max_items,
                      hipStream_t s) {
  const int pos_in_lds = ja.max_seq_len <= kBwdMaxLdsPos ? 1 : 0;
  const size_t lds = pos_in_lds ? sizeof(float) * (size_t)ja.max_seq_len : 0;
  dim3 grid((unsigned)max_items, (unsigned)ja.num_heads);
  hipLaunchKernelGGL((attn_bwd_bf16_kernel<DQK, DV>), grid, dim3(256), lds, s, ja, t,
                     (const uint16_t*)d_out, dq_acc, (uint16_t*)dk, (uint16_t*)dv, d_rab_pos,
                     d_rab_time, items, count, pos_in_lds);
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
