// Fused jagged pointwise-attention backward, bf16 MFMA (gfx950).
//
// Gradients of <O, dO> for O = (1/N) SiLU(Q K^T + rab) V (Eq. 2).  As the
// paper's kernel appendix describes, attention and the relative bias are
// recomputed rather than stored, and the bias gradients are accumulated
// in on-chip shared memory before they reach HBM.  Pointwise aggregation
// means no row statistics are needed: with S = Q K^T + rab,
//   P  = SiLU(S) (masked),            dV = (1/N) P^T dO
//   dP = dO V^T,  dS = dP SiLU'(S) (masked)
//   dK = (1/N) dS^T Q,  dQ = (1/N) dS K
//   d rab_pos[(N-1)+p(j)-p(i)] += dS/N,  d rab_time[bkt] += dS/N.
//
// Workgroup = 4 waves = one (sequence, 128-key block, head) work item.
// Wave w owns keys j0 + 32w .. +31 and keeps their K, V (as MFMA
// operands) and dK, dV accumulators in registers for the whole item.  It
// walks query steps of 32 rows: Q and dO of the step are staged in LDS
// both row-major (operand of S and dP) and transposed in the
// accumulator-matched order (operand of dK and dV).  dS is written to LDS
// so all four waves can form the step's dQ = dS K block, which is added
// to an fp32 workspace with hardware float atomics (converted to bf16 by
// a separate pass).  Bias-position gradients are summed in an LDS array
// indexed by p(i) - p(j) and time-bucket gradients in an LDS histogram;
// each workgroup flushes them with one atomic per touched entry.
#include "kernels.h"

namespace hstu {

namespace {

template <int DQK, int DV>
__global__ __launch_bounds__(256, 1) void attn_bwd_bf16_kernel(
    JaggedArgs ja, Tensors t, const uint16_t* __restrict__ dO, float* __restrict__ dq_acc,
    uint16_t* __restrict__ dK, uint16_t* __restrict__ dV, float* __restrict__ d_rab_pos,
    float* __restrict__ d_rab_time, const WorkItem* __restrict__ items,
    const int32_t* __restrict__ count, int pos_in_lds) {
  constexpr int BN = kBwdBN, BM = kBwdBM;
  constexpr int Q_LD = DQK + 8, DO_LD = DV + 8;  // row-major tiles
  constexpr int QT_LD = BM + 8, DOT_LD = BM + 8;  // transposed tiles
  constexpr int DS_LD = BN + 8, KT_LD = BN + 8;
  constexpr int NWIN = BM + BN;
  static_assert(BN == 128 && BM == 32, "4 waves x 32 keys, 32-row query steps");

  __shared__ __align__(16) uint16_t sQ[BM * Q_LD];
  __shared__ __align__(16) uint16_t sQT[DQK * QT_LD];
  __shared__ __align__(16) uint16_t sdO[BM * DO_LD];
  __shared__ __align__(16) uint16_t sdOT[DV * DOT_LD];
  __shared__ __align__(16) uint16_t sdS[BM * DS_LD];
  __shared__ __align__(16) uint16_t sKT[DQK * KT_LD];
  __shared__ int64_t sTi[BM];
  __shared__ float sPos[NWIN];
  __shared__ float sTime[256];
  __shared__ float sHist[256];
  extern __shared__ float sPosAcc[];  // [N] when pos_in_lds

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
  const int64_t tj = key_ok ? ja.timestamps[o + my_j] : 0;
  const float invN = 1.0f / (float)N;

  const uint16_t* __restrict__ qg = (const uint16_t*)t.q;
  const uint16_t* __restrict__ kg = (const uint16_t*)t.k;
  const uint16_t* __restrict__ vg = (const uint16_t*)t.v;

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

  // K^T of the whole 128-key block (operand of dQ = dS K).
  constexpr int KCH = BN * DQK / 8;
  for (int c = tid; c < KCH; c += 256) {
    const int r = c / (DQK / 8), cc = (c % (DQK / 8)) * 8;
    const int j = j0 + r;
    u32x4 v = j < L ? *reinterpret_cast<const u32x4*>(kg + (o + j) * t.k_stride + head * DQK + cc)
                    : zero_u32x4();
#pragma unroll
    for (int e = 0; e < 8; e++) sKT[(cc + e) * KT_LD + r] = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
  }
  for (int x = tid; x < NB; x += 256) {
    sTime[x] = ja.rab_time[x];
    sHist[x] = 0.0f;
  }
  const int R = L - j0;  // p(i) - p(j) of kept pairs lies in [0, R)
  if (pos_in_lds)
    for (int x = tid; x < R; x += 256) sPosAcc[x] = 0.0f;

  f32x16 dkacc[DQK / 32], dvacc[DV / 32];
#pragma unroll
  for (int nb = 0; nb < DQK / 32; nb++)
#pragma unroll
    for (int q = 0; q < 16; q++) dkacc[nb][q] = 0.0f;
#pragma unroll
  for (int nb = 0; nb < DV / 32; nb++)
#pragma unroll
    for (int q = 0; q < 16; q++) dvacc[nb][q] = 0.0f;

  // Candidate keys see only themselves; otherwise every later row sees them.
  const int i_end = j0 >= n_h ? min(j0 + BN, L) : L;

  for (int i0 = j0; i0 < i_end; i0 += BM) {
    __syncthreads();  // previous step's tiles consumed
    constexpr int QCH = BM * DQK / 8;
    for (int c = tid; c < QCH; c += 256) {
      const int r = c / (DQK / 8), cc = (c % (DQK / 8)) * 8;
      const int i = i0 + r;
      u32x4 v = i < L ? *reinterpret_cast<const u32x4*>(qg + (o + i) * t.q_stride + head * DQK + cc)
                      : zero_u32x4();
      *reinterpret_cast<u32x4*>(sQ + r * Q_LD + cc) = v;
      const int pos = swap_bits23(r);
#pragma unroll
      for (int e = 0; e < 8; e++)
        sQT[(cc + e) * QT_LD + pos] = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
    }
    constexpr int OCH = BM * DV / 8;
    for (int c = tid; c < OCH; c += 256) {
      const int r = c / (DV / 8), cc = (c % (DV / 8)) * 8;
      const int i = i0 + r;
      u32x4 v = i < L ? *reinterpret_cast<const u32x4*>(dO + ((o + i) * H + head) * DV + cc)
                      : zero_u32x4();
      *reinterpret_cast<u32x4*>(sdO + r * DO_LD + cc) = v;
      const int pos = swap_bits23(r);
#pragma unroll
      for (int e = 0; e < 8; e++)
        sdOT[(cc + e) * DOT_LD + pos] = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
    }
    if (tid < BM) sTi[tid] = (i0 + tid < L) ? ja.timestamps[o + i0 + tid] : 0;
    // rab_pos entries reachable from (query step, key block).
    const int pos_base = (N - 1) + min(j0, n_h) - min(i0 + BM - 1, n_h);
    for (int x = tid; x < NWIN; x += 256) {
      const int g = pos_base + x;
      sPos[x] = (g >= 0 && g <= 2 * N - 2) ? ja.rab_pos[g] : 0.0f;
    }
    __syncthreads();

    // Does any kept pair fall in (rows i0..i0+31) x (this wave's keys)?
    bool active = jw0 < L && jw0 <= i0 + BM - 1;
    if (jw0 >= n_h && jw0 != i0) active = false;  // candidate keys: diagonal block only

    float ds[16];
    if (active) {
      // Accumulator lane holds (i = i0 + 8g + 4*half + m, j = my_j).
      f32x16 sacc, pacc;
      uint32_t vmask = 0;
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int il = 8 * (q >> 2) + 4 * half + (q & 3);
        const int i = i0 + il;
        float bias = 0.0f;
        if (key_ok && i < L && pair_valid(i, my_j, n_h)) {
          const int widx = (N - 1) + pj - bias_pos(i, n_h) - pos_base;
          bias = sPos[widx] + sTime[time_bucket64(sTi[il] - tj, NB)];
          vmask |= 1u << q;
        }
        sacc[q] = bias;
        pacc[q] = 0.0f;
      }
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
#pragma unroll
        for (int nb = 0; nb < DV / 32; nb++) {
          u32x4 b = *reinterpret_cast<const u32x4*>(sdOT + (32 * nb + col) * DOT_LD + 16 * st + 8 * half);
          dvacc[nb] = mfma32x32x16(as_bf16x8(pa), as_bf16x8(b), dvacc[nb]);
        }
#pragma unroll
        for (int nb = 0; nb < DQK / 32; nb++) {
          u32x4 b = *reinterpret_cast<const u32x4*>(sQT + (32 * nb + col) * QT_LD + 16 * st + 8 * half);
          dkacc[nb] = mfma32x32x16(as_bf16x8(da), as_bf16x8(b), dkacc[nb]);
        }
      }
      // Bias gradients: position by p(i) - p(j), time by bucket.
#pragma unroll
      for (int q = 0; q < 16; q++) {
        if ((vmask >> q) & 1u) {
          const int il = 8 * (q >> 2) + 4 * half + (q & 3);
          const int i = i0 + il;
          const int kpos = bias_pos(i, n_h) - pj;
          if (pos_in_lds)
            atomicAdd(&sPosAcc[kpos], ds[q]);
          else
            unsafeAtomicAdd(&d_rab_pos[(N - 1) - kpos], ds[q] * invN);
          atomicAdd(&sHist[time_bucket64(sTi[il] - tj, NB)], ds[q]);
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
  for (int x = tid; x < NB; x += 256) {
    const float v = sHist[x];
    if (v != 0.0f) unsafeAtomicAdd(&d_rab_time[x], v * invN);
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
