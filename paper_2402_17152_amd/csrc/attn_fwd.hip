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
//   P   = mask ? SiLU(S) : 0 in fp32 registers, rounded to bf16;
//   O  += P V_tile, P taken straight from the accumulator registers: the
//         contraction index is permuted to match the accumulator layout
//         and V is stored transposed in LDS in that same order.
// K and V^T tiles, the tile's timestamps and the slice of rab_pos it can
// touch are staged in LDS; rab_time lives in LDS for the whole item.
#include "kernels.h"

namespace hstu {

namespace {

template <int DQK, int DV>
__global__ __launch_bounds__(256, 2) void attn_fwd_bf16_kernel(JaggedArgs ja, Tensors t,
                                                               uint16_t* __restrict__ out,
                                                               const WorkItem* __restrict__ items,
                                                               const int32_t* __restrict__ count) {
  constexpr int BM = kFwdBM, BN = kFwdBN;
  constexpr int K_LD = DQK + 8;   // LDS row pitch of the K tile (bf16 elements)
  constexpr int VT_LD = BN + 8;   // LDS row pitch of the V^T tile
  constexpr int NWIN = BM + BN;   // rab_pos slice per tile (BM + BN - 1 used)
  static_assert(BN == 32, "one 32x32 score block per wave and tile");

  __shared__ __align__(16) uint16_t sK[BN * K_LD];
  __shared__ __align__(16) uint16_t sVT[DV * VT_LD];
  __shared__ int64_t sTj[BN];
  __shared__ float sPos[NWIN];
  __shared__ float sTime[256];

  if ((int)blockIdx.x >= *count) return;
  const WorkItem it = items[blockIdx.x];
  const int head = blockIdx.y;
  const int H = ja.num_heads, N = ja.max_seq_len, NB = ja.num_buckets;
  const int64_t o = ja.seq_offsets[it.seq];
  const int L = (int)(ja.seq_offsets[it.seq + 1] - o);
  const int n_h = L - (ja.num_targets ? (int)ja.num_targets[it.seq] : 0);
  const int i0 = it.blk * BM;
  const int rows_end = min(i0 + BM, L);

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  const int iw0 = i0 + wave * 32;
  const int my_i = iw0 + col;
  const bool row_ok = my_i < L;
  const int wave_last = min(iw0 + 31, L - 1);

  for (int x = tid; x < NB; x += 256) sTime[x] = ja.rab_time[x];

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
  const int64_t ti = row_ok ? ja.timestamps[o + my_i] : 0;
  const int pi = bias_pos(my_i, n_h);

  f32x16 oacc[DV / 32];
#pragma unroll
  for (int nb = 0; nb < DV / 32; nb++)
#pragma unroll
    for (int q = 0; q < 16; q++) oacc[nb][q] = 0.0f;

  const int kend = (rows_end + BN - 1) / BN;
  const int nh_blk = (n_h + BN - 1) / BN;

  for (int kb = 0; kb < kend; kb++) {
    const int j0 = kb * BN;
    // Key tile of candidates entirely before this block's rows: all masked.
    if (kb >= nh_blk && j0 + BN <= i0) continue;
    __syncthreads();  // previous tile fully consumed

    constexpr int KCH = BN * DQK / 8;
    for (int c = tid; c < KCH; c += 256) {
      const int r = c / (DQK / 8), cc = (c % (DQK / 8)) * 8;
      const int j = j0 + r;
      u32x4 v = j < L ? *reinterpret_cast<const u32x4*>(kg + (o + j) * t.k_stride + head * DQK + cc)
                      : zero_u32x4();
      *reinterpret_cast<u32x4*>(sK + r * K_LD + cc) = v;
    }
    constexpr int VCH = BN * DV / 8;
    for (int c = tid; c < VCH; c += 256) {
      const int r = c / (DV / 8), cc = (c % (DV / 8)) * 8;
      const int j = j0 + r;
      u32x4 v = j < L ? *reinterpret_cast<const u32x4*>(vg + (o + j) * t.v_stride + head * DV + cc)
                      : zero_u32x4();
      const int pos = swap_bits23(r);
#pragma unroll
      for (int e = 0; e < 8; e++)
        sVT[(cc + e) * VT_LD + pos] = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
    }
    if (tid < BN) sTj[tid] = (j0 + tid < L) ? ja.timestamps[o + j0 + tid] : 0;
    // rab_pos entries reachable from this (query block, key tile):
    // (N-1) + p(j) - p(i) with p(i) in [min(i0,n_h), min(i0+BM-1,n_h)] and
    // p(j) in [min(j0,n_h), min(j0+BN-1,n_h)].
    const int pos_base = (N - 1) + min(j0, n_h) - min(i0 + BM - 1, n_h);
    for (int x = tid; x < NWIN; x += 256) {
      const int g = pos_base + x;
      sPos[x] = (g >= 0 && g <= 2 * N - 2) ? ja.rab_pos[g] : 0.0f;
    }
    __syncthreads();

    if (iw0 >= L || j0 > wave_last) continue;           // no row of this wave sees the tile
    if (kb >= nh_blk && j0 + BN <= iw0) continue;         // candidate keys before the wave

    // Bias into the accumulator; lane holds (j = j0 + 8g + 4*half + m, i = my_i).
    f32x16 sacc;
    uint32_t vmask = 0;
#pragma unroll
    for (int q = 0; q < 16; q++) {
      const int jl = 8 * (q >> 2) + 4 * half + (q & 3);
      const int j = j0 + jl;
      float bias = 0.0f;
      if (row_ok && j < L && pair_valid(my_i, j, n_h)) {
        const int widx = (N - 1) + bias_pos(j, n_h) - pi - pos_base;
        bias = sPos[widx] + sTime[time_bucket64(ti - sTj[jl], NB)];
        vmask |= 1u << q;
      }
      sacc[q] = bias;
    }
#pragma unroll
    for (int s = 0; s < DQK / 16; s++) {
      u32x4 kf = *reinterpret_cast<const u32x4*>(sK + col * K_LD + 16 * s + 8 * half);
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
#pragma unroll
      for (int nb = 0; nb < DV / 32; nb++) {
        u32x4 vb = *reinterpret_cast<const u32x4*>(sVT + (32 * nb + col) * VT_LD + 16 * st + 8 * half);
        oacc[nb] = mfma32x32x16(as_bf16x8(pa), as_bf16x8(vb), oacc[nb]);
      }
    }
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
