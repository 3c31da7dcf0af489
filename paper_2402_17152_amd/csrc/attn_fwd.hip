// Fused jagged pointwise-attention forward, bf16 MFMA (gfx950).
//
// Computes Eq. 2 of the paper, O = (1/N) SiLU(Q K^T + rab^{p,t}) V, over a
// jagged batch without padding (Sec. 3.2, "fully raggified" attention),
// with the relative bias built in registers from the position table and
// the time-bucket table (notation table, rab^{p,t}; kernel appendix: bias
// construction fused into the attention kernel).  Pointwise aggregation
// needs no running max, rescale or row sum, so each key tile is consumed
// once and forgotten.
//
// Workgroup = 4 waves = one (sequence, 128-row query block, head) work
// item from the scheduler.  Wave w owns query rows i0 + 32w .. +31.
// Per 32-key tile:
//   S^T = K_tile Q^T via v_mfma_f32_32x32x16_bf16 (accumulator seeded with
//         the bias), so each lane holds one query row and 16 keys;
//   P   = SiLU(S) in fp32 registers (masked only on diagonal, ragged and
//         candidate tiles), rounded to bf16;
//   O  += P V_tile, P taken straight from the accumulator registers: the
//         contraction index is permuted to match the accumulator layout
//         and V is fetched from its row-major LDS tile with transposing
//         reads in that same order.
// The next tile's K, V, timestamps and rab_pos slice are loaded into
// registers while the current tile is computed.  Timestamps are rebased
// to 32 bits when the item's span allows (see bias.h).
#include "bias.h"
#include "kernels.h"

namespace hstu {

namespace {

constexpr int64_t kI64Max = 0x7fffffffffffffffll;
constexpr int64_t kI64Min = -kI64Max - 1;

template <int DQK, int DV>
struct FwdShared {
  static constexpr int BM = kFwdBM, BN = kFwdBN;
  static constexpr int K_LD = DQK + 8;   // LDS row pitch of the K tile (bf16 elements)
  static constexpr int V_LD = DV + 8;    // LDS row pitch of the V tile
  static constexpr int NWIN = BM + BN;   // rab_pos slice per tile (BM + BN - 1 used)
  __align__(16) uint16_t sK[BN * K_LD];
  __align__(16) uint16_t sV[BN * V_LD];
  __align__(16) uint32_t sTj[BN];  // key timestamps, rebased (fast path)
  int64_t sTj64[BN];               // key timestamps (exact path)
  float sWin[NWIN];
  float sTab[64];
  int64_t sRed[2][4];
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
__device__ __forceinline__ void fwd_item(FwdShared<DQK, DV>& sm, const JaggedArgs& ja,
                                         const Tensors& t, uint16_t* __restrict__ out, int64_t o,
                                         int L, int n_h, int i0, int head, int64_t tbase) {
  using Sh = FwdShared<DQK, DV>;
  constexpr int BM = Sh::BM, BN = Sh::BN, K_LD = Sh::K_LD, V_LD = Sh::V_LD, NWIN = Sh::NWIN;
  constexpr int KCH = BN * DQK / 8, VCH = BN * DV / 8;
  constexpr int KPT = (KCH + 255) / 256, VPT = (VCH + 255) / 256;
  static_assert(BN == 32, "one 32x32 score block per wave and tile");
  const int H = ja.num_heads, N = ja.max_seq_len;
  const int rows_end = min(i0 + BM, L);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  const int iw0 = i0 + wave * 32;
  const int my_i = iw0 + col;
  const bool row_ok = my_i < L;
  const int wave_last = min(iw0 + 31, L - 1);
  const int64_t* __restrict__ ts = ja.timestamps + o;
  const uint16_t* __restrict__ qg = (const uint16_t*)t.q;
  const uint16_t* __restrict__ kg = (const uint16_t*)t.k;
  const uint16_t* __restrict__ vg = (const uint16_t*)t.v;

  // Q fragment: B operand of S^T = K Q^T (lane = query row, 8 d's per step).
  u32x4 qf[DQK / 16];
#pragma unroll
  for (int s = 0; s < DQK / 16; s++)
    qf[s] = row_ok ? *reinterpret_cast<const u32x4*>(qg + (o + my_i) * t.q_stride + head * DQK +
                                                     16 * s + 8 * half)
                   : zero_u32x4();
  const int64_t ti64 = row_ok ? ts[my_i] : tbase;
  const uint32_t tir = (uint32_t)(ti64 - tbase);
  const int pi = bias_pos(my_i, n_h);

  f32x16 oacc[DV / 32];
#pragma unroll
  for (int nb = 0; nb < DV / 32; nb++)
#pragma unroll
    for (int q = 0; q < 16; q++) oacc[nb][q] = 0.0f;

  const int kend = (rows_end + BN - 1) / BN;
  const int nh_blk = (n_h + BN - 1) / BN;
  // Key tiles made only of candidates that precede every row of the
  // block are fully masked and skipped.
  auto skipped = [&](int kb) { return kb >= nh_blk && (kb + 1) * BN <= i0; };

  const int tr_row = 4 * (lane >> 5) + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  u32x4 pk[KPT], pv[VPT];
  int64_t pt = 0;
  float pw = 0.0f;
  auto prefetch = [&](int kb) {
    const int j0 = kb * BN;
#pragma unroll
    for (int k = 0; k < KPT; k++) {
      const int c = tid + 256 * k;
      if (c < KCH) {
        const int r = c / (DQK / 8), cc = (c % (DQK / 8)) * 8, j = j0 + r;
        pk[k] = j < L ? *reinterpret_cast<const u32x4*>(kg + (o + j) * t.k_stride + head * DQK + cc)
                      : zero_u32x4();
      }
    }
#pragma unroll
    for (int k = 0; k < VPT; k++) {
      const int c = tid + 256 * k;
      if (c < VCH) {
        const int r = c / (DV / 8), cc = (c % (DV / 8)) * 8, j = j0 + r;
        pv[k] = j < L ? *reinterpret_cast<const u32x4*>(vg + (o + j) * t.v_stride + head * DV + cc)
                      : zero_u32x4();
      }
    }
    if (tid < BN) pt = (j0 + tid < L) ? ts[j0 + tid] : tbase;
    if (tid < NWIN) {
      // rab_pos entries reachable from (query block, key tile):
      // (N-1) + p(j) - p(i), p(i) in [min(i0,n_h), min(i0+BM-1,n_h)],
      // p(j) in [min(j0,n_h), min(j0+BN-1,n_h)].
      const int pos_base = (N - 1) + min(j0, n_h) - min(i0 + BM - 1, n_h);
      const int g = pos_base + tid;
      pw = (g >= 0 && g <= 2 * N - 2) ? ja.rab_pos[g] : 0.0f;
    }
  };

  int kb = 0;
  while (kb < kend && skipped(kb)) kb++;
  if (kb < kend) prefetch(kb);

  while (kb < kend) {
    const int j0 = kb * BN;
    int kn = kb + 1;
    while (kn < kend && skipped(kn)) kn++;
    __syncthreads();  // previous tile fully consumed
#pragma unroll
    for (int k = 0; k < KPT; k++) {
      const int c = tid + 256 * k;
      if (c < KCH) *reinterpret_cast<u32x4*>(sm.sK + (c / (DQK / 8)) * K_LD + (c % (DQK / 8)) * 8) = pk[k];
    }
#pragma unroll
    for (int k = 0; k < VPT; k++) {
      const int c = tid + 256 * k;
      if (c < VCH) *reinterpret_cast<u32x4*>(sm.sV + (c / (DV / 8)) * V_LD + (c % (DV / 8)) * 8) = pv[k];
    }
    if (tid < BN) {
      if constexpr (FAST)
        sm.sTj[tid] = (uint32_t)(pt - tbase);
      else
        sm.sTj64[tid] = pt;
    }
    if (tid < NWIN) sm.sWin[tid] = pw;
    __syncthreads();
    if (kn < kend) prefetch(kn);

    const bool active = iw0 < L && j0 <= wave_last && !(kb >= nh_blk && j0 + BN <= iw0);
    if (active) {
      // Lane holds (j = j0 + 8g + 4*half + m, i = my_i).
      const bool full = (j0 + BN - 1 <= iw0) && (iw0 + 31 < L) && (iw0 + 31 < n_h);
      const int pos_base = (N - 1) + min(j0, n_h) - min(i0 + BM - 1, n_h);
      f32x16 sacc;
      uint32_t vmask = 0xffffu;
      if (full) {
        // window index = j_local + (min(i0+BM-1, n_h) - i) for history rows
        const int xb = min(i0 + BM - 1, n_h) - my_i + 4 * half;
#pragma unroll
        for (int q = 0; q < 16; q++) {
          const int jl = 8 * (q >> 2) + 4 * half + (q & 3);
          const int s = slot_of<FAST>(tir, sm.sTj[jl], ti64, sm.sTj64[jl]);
          sacc[q] = sm.sWin[xb + 8 * (q >> 2) + (q & 3)] + sm.sTab[s];
        }
      } else {
        vmask = 0;
#pragma unroll
        for (int q = 0; q < 16; q++) {
          const int jl = 8 * (q >> 2) + 4 * half + (q & 3);
          const int j = j0 + jl;
          float b = 0.0f;
          if (row_ok && j < L && pair_valid(my_i, j, n_h)) {
            const int x = (N - 1) + bias_pos(j, n_h) - pi - pos_base;
            const int s = slot_of<FAST>(tir, sm.sTj[jl], ti64, sm.sTj64[jl]);
            b = sm.sWin[x] + sm.sTab[s];
            vmask |= 1u << q;
          }
          sacc[q] = b;
        }
      }
#pragma unroll
      for (int s = 0; s < DQK / 16; s++) {
        u32x4 kf = *reinterpret_cast<const u32x4*>(sm.sK + col * K_LD + 16 * s + 8 * half);
        sacc = mfma32x32x16(as_bf16x8(kf), as_bf16x8(qf[s]), sacc);
      }
      float p[16];
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const float x = sacc[q];
        p[q] = ((vmask >> q) & 1u) ? x * sigmoid_fast(x) : 0.0f;
      }
#pragma unroll
      for (int st = 0; st < 2; st++) {
        u32x4 pa;
        pa[0] = pack_bf16x2(p[8 * st + 0], p[8 * st + 1]);
        pa[1] = pack_bf16x2(p[8 * st + 2], p[8 * st + 3]);
        pa[2] = pack_bf16x2(p[8 * st + 4], p[8 * st + 5]);
        pa[3] = pack_bf16x2(p[8 * st + 6], p[8 * st + 7]);
        const int row = 16 * st + tr_row;
#pragma unroll
        for (int nb = 0; nb < DV / 32; nb++) {
          const uint16_t* base = sm.sV + row * V_LD + 32 * nb + tr_col;
          const uint2 lo = lds_read_tr16(base), hi = lds_read_tr16(base + 8 * V_LD);
          u32x4 vb = {lo.x, lo.y, hi.x, hi.y};
          oacc[nb] = mfma32x32x16(as_bf16x8(pa), as_bf16x8(vb), oacc[nb]);
        }
      }
    }
    kb = kn;
  }

  // O accumulator: lane holds (i = iw0 + 8g + 4*half + m, c = 32nb + col).
  const float invN = 1.0f / (float)N;
  uint16_t* __restrict__ og = out + (o * H + head) * DV;
#pragma unroll
  for (int nb = 0; nb < DV / 32; nb++)
#pragma unroll
    for (int q = 0; q < 16; q++) {
      const int i = iw0 + 8 * (q >> 2) + 4 * half + (q & 3);
      if (i < L) og[(int64_t)i * H * DV + 32 * nb + col] = f32_to_bf16_bits(oacc[nb][q] * invN);
    }
}

template <int DQK, int DV>
__global__ __launch_bounds__(256, 2) void attn_fwd_bf16_kernel(JaggedArgs ja, Tensors t,
                                                               uint16_t* __restrict__ out,
                                                               const WorkItem* __restrict__ items,
                                                               const int32_t* __restrict__ count) {
  using Sh = FwdShared<DQK, DV>;
  __shared__ Sh sm;
  if ((int)blockIdx.x >= *count) return;
  const WorkItem it = items[blockIdx.x];
  const int head = blockIdx.y;
  const int NB = ja.num_buckets;
  const int64_t o = ja.seq_offsets[it.seq];
  const int L = (int)(ja.seq_offsets[it.seq + 1] - o);
  const int n_h = L - (ja.num_targets ? (int)ja.num_targets[it.seq] : 0);
  const int i0 = it.blk * Sh::BM;
  const int rows_end = min(i0 + Sh::BM, L);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t* __restrict__ ts = ja.timestamps + o;

  // Timestamp extremes over the tokens this item touches, [0, rows_end):
  // the 32-bit fast path applies when they span less than 2^31.
  int64_t tlo = kI64Max, thi = kI64Min;
  for (int x = tid; x < rows_end; x += 256) {
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
  __syncthreads();
  tlo = sm.sRed[0][0];
  thi = sm.sRed[1][0];
#pragma unroll
  for (int w = 1; w < 4; w++) {
    tlo = sm.sRed[0][w] < tlo ? sm.sRed[0][w] : tlo;
    thi = sm.sRed[1][w] > thi ? sm.sRed[1][w] : thi;
  }
  if (thi - tlo < ((int64_t)1 << 31))
    fwd_item<DQK, DV, true>(sm, ja, t, out, o, L, n_h, i0, head, tlo);
  else
    fwd_item<DQK, DV, false>(sm, ja, t, out, o, L, n_h, i0, head, tlo);
}

template <int DQK, int DV>
hipError_t launch_fwd(const JaggedArgs& ja, const Tensors& t, void* out, const WorkItem* items,
                      const int32_t* count, int64_t max_items, hipStream_t s) {
  dim3 grid((unsigned)max_items, (unsigned)ja.num_heads);
  hipLaunchKernelGGL((attn_fwd_bf16_kernel<DQK, DV>), grid, dim3(256), 0, s, ja, t,
                     (uint16_t*)out, items, count);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_fwd_bf16(const JaggedArgs& ja, const Tensors& t, int dqk, int dv, void* out,
                                const WorkItem* items, const int32_t* count, int64_t max_items,
                                hipStream_t s) {
#define HSTU_FWD_CASE(A, B) \
  if (dqk == A && dv == B) return launch_fwd<A, B>(ja, t, out, items, count, max_items, s);
  HSTU_FWD_CASE(32, 32)
  HSTU_FWD_CASE(32, 64)
  HSTU_FWD_CASE(32, 128)
  HSTU_FWD_CASE(64, 32)
  HSTU_FWD_CASE(64, 64)
  HSTU_FWD_CASE(64, 128)
  HSTU_FWD_CASE(128, 32)
  HSTU_FWD_CASE(128, 64)
  HSTU_FWD_CASE(128, 128)
#undef HSTU_FWD_CASE
  return hipErrorInvalidValue;
}

}  // namespace hstu
