// Fused jagged pointwise-attention forward, bf16 MFMA (gfx950).
//
// Computes Eq. 2 of the paper, O = (1/N) SiLU(Q K^T + rab^{p,t}) V, over a
// jagged batch without padding (Sec. 3.2),
// with the relative bias built on chip from the position table and the
// time-bucket table (notation table, rab^{p,t}; kernel appendix: bias
// construction fused into the attention kernel).  Pointwise aggregation
// needs no running max, rescale or row sum, so each key tile is consumed
// once and forgotten.
//
// Workgroup = 4 waves = one (sequence, 128-row query block, head) work
// item from the scheduler.  Wave w owns query rows i0 + 32w .. +31 and
// walks the block's 32-key tiles t = 0, 1, ...:
//   S^T(t) = K_t Q^T  (v_mfma_f32_32x32x16_bf16, accumulator seeded with
//            the bias; lane = one query row x 16 keys),
//   P(t)   = SiLU(S(t)) in fp32, rounded to bf16,
//   O     += P(t) V_t, P taken straight from the accumulator registers
//            (contraction index permuted to the accumulator layout, V read
//            with transposing LDS loads in that order).
// Pointwise SiLU costs about as much VALU issue time per score as the
// d = 128 contractions cost MFMA time, so the loop is software-pipelined:
// one straight-line block issues the MFMAs of S(t+1) and of P(t-1) V_{t-1}
// next to the SiLU of tile t.  Masked scores are seeded with a large
// negative bias, for which SiLU yields exactly -0, so the SiLU block has
// no selects.
//
// Bias on full tiles (every pair valid, all positions history): the
// position term rab_pos[(N-1) + j - i] is read as aligned 16-byte LDS
// loads from four shifted copies of the tile's table window, and when
// every |t_i - t_j| of the (wave, tile) falls in one log2 bucket (decided
// from the timestamp ranges) the time term is one constant.  Other tiles
// evaluate the mask and both terms per element.
//
// LDS staging by LDS DMA (buffer loads that write LDS directly): K tiles
// and rab_pos windows in rings of 3, issued three tiles ahead; V tiles in
// a ring of 4, issued two ahead (V of tile t is consumed one step after
// K); key timestamps five ahead.  One explicit vmcnt wait and one barrier
// per tile.
#include <type_traits>

#include "bias.h"
#include "kernels.h"

namespace hstu {

namespace {

constexpr int64_t kI64Max = 0x7fffffffffffffffll;
constexpr int64_t kI64Min = -kI64Max - 1;
// Bias of a masked pair: SiLU(x) with x ~ -1e30 evaluates to exactly -0
// (exp2 overflows to +inf, its reciprocal is 0).
constexpr float kMaskedBias = -1.0e30f;

// Padded row pitches, in 16-byte chunks.  K is read one 16-byte chunk
// per lane (8 lanes per LDS cycle, rows 0..7): an odd pitch spreads them
// over all banks.  V is read with 8-byte transposing loads (16 lanes per
// cycle: 4 rows x 2 chunks x 2 halves): a pitch of 8 dwords mod 32 (24 for
// d_v = 32) does the same.
constexpr int k_pitch_chunks(int d) { return d / 8 + 1; }
constexpr int v_pitch_chunks(int d) { return d == 128 ? 18 : d == 64 ? 10 : 6; }

template <int DQK, int DV>
struct FwdShared {
  static constexpr int BM = kFwdBM, BN = kFwdBN;
  static constexpr int KP = k_pitch_chunks(DQK), VP = v_pitch_chunks(DV);
  static constexpr int K_LD = KP * 8, V_LD = VP * 8;  // row pitches in bf16 elements
  // A tile is staged by 1 KB LDS-DMA operations (64 lanes x 16 bytes);
  // the pad chunks of each row are filled with a repeat of a data chunk.
  static constexpr int KOPS = (BN * KP + 63) / 64, VOPS = (BN * VP + 63) / 64;
  static constexpr int NWIN = BM + BN;  // rab_pos window per tile (BM + BN - 1 used)
  // Window copy c holds window[k + c] at index kWinPad + k, k in [0, 192).
  // Copy pitch 264 dwords = 8 mod 32 banks: the 16-byte reads of 8
  // neighbouring lanes (4 copies x 2 offsets) hit distinct banks.
  static constexpr int kWinPad = 4, WIN_LD = 264;
  // Rings: K and window tiles are staged three steps ahead (3 slots), V
  // two steps ahead and consumed one step after K (4 slots), timestamps
  // five steps ahead (8 slots).
  __align__(16) uint16_t sK[3][KOPS * 512];
  __align__(16) uint16_t sV[4][VOPS * 512];
  __align__(16) float sWin[3][4][WIN_LD];
  __align__(16) uint32_t sT[8][64];  // the tile's 32 int64 key timestamps
  __align__(16) uint32_t sTr[8][32];  // the same rebased to 32 bits (fast path)
  uint32_t sKr32[4][2];              // rebased key timestamp min / max per tile
  float sTab[64];                    // time bias by slot (bias.h)
};

__device__ __forceinline__ float silu(float x) {
  const float e = __builtin_amdgcn_exp2f(x * -kLog2e);
  return x * __builtin_amdgcn_rcpf(1.0f + e);
}

// SPLIT: P enters the second contraction as two bf16 terms, hi = bf16(P)
// and lo = bf16(P - hi) (two MFMAs per V operand), which leaves O with
// about 2^-17 relative error instead of bf16's 2^-9; used where O is
// normalised afterwards (the layer's LayerNorm rescales every row to unit
// spread and would magnify a bf16 P).
// Row i of the item is global row orow + i, key j global key okey + j;
// keys at or past key_lim do not exist (cross mode: the cached prefix has
// n_h keys).  TGT: self mode with candidate rows, whose blocks may visit
// candidate key tiles after the history tiles; otherwise step u's tile is
// kt0 + u.
template <int DQK, int DV, bool FAST, bool SPLIT, bool TGT>
__device__ __forceinline__ void fwd_item(FwdShared<DQK, DV>& sm, const JaggedArgs& ja,
                                         const Tensors& t, void* __restrict__ out, int out_f32,
                                         int64_t orow, int64_t okey, int L, int n_h, int key_lim,
                                         int kt0, int kt1, int i0, int head, int64_t tbase) {
  using Sh = FwdShared<DQK, DV>;
  constexpr int BM = Sh::BM, BN = Sh::BN, K_LD = Sh::K_LD, V_LD = Sh::V_LD;
  // Masked tiles with history keys read the window as full tiles do; the
  // instances that run three workgroups per CU (d_qk, d_v <= 64) keep
  // reading it entry by entry, as the other form costs them registers past
  // that occupancy.
  constexpr bool kMaskedWindowReads = DQK > 64 || DV > 64;
  constexpr int KCH = BN * DQK / 8, VCH = BN * DV / 8;
  constexpr int KPT = (KCH + 255) / 256, VPT = (VCH + 255) / 256;
  static_assert(BN == 32 && BM == 128, "4 waves x 32 rows, 32-key tiles");
  const int H = ja.num_heads, N = ja.max_seq_len;
  const int rows_end = min(i0 + BM, L);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, half = lane >> 5;
  const int iw0 = i0 + wave * 32;
  const int my_i = iw0 + col;
  const bool row_ok = my_i < L;
  const int wave_last = min(iw0 + 31, L - 1);
  const int R = min(i0 + BM - 1, n_h);  // largest row position of the block
  const int64_t* __restrict__ ts = ja.timestamps + orow;  // row timestamps
  const int64_t* __restrict__ tsk = (ja.key_timestamps ? ja.key_timestamps : ja.timestamps) + okey;
  const uint16_t* __restrict__ qg = (const uint16_t*)t.q;
  const uint16_t* __restrict__ kg = (const uint16_t*)t.k;
  const uint16_t* __restrict__ vg = (const uint16_t*)t.v;
  const float* tab32 = sm.sTab + 32;

  // Q fragment: B operand of S^T = K Q^T (lane = query row, 8 d's per step).
  u32x4 qf[DQK / 16];
#pragma unroll
  for (int s = 0; s < DQK / 16; s++)
    qf[s] = row_ok ? *reinterpret_cast<const u32x4*>(qg + (orow + my_i) * t.q_stride + head * DQK +
                                                     16 * s + 8 * half)
                   : zero_u32x4();
  const int64_t ti64 = row_ok ? ts[my_i] : tbase;
  const uint32_t tir = (uint32_t)(ti64 - tbase);
  const int pi = bias_pos(my_i, n_h);
  // Timestamp range of the wave's rows (used by full tiles, whose rows are all valid).
  const int64_t rlo = wave_min_i64(ti64), rhi = wave_max_i64(ti64);
  const uint32_t rlo32 = __builtin_amdgcn_readfirstlane((uint32_t)(rlo - tbase));
  const uint32_t rhi32 = __builtin_amdgcn_readfirstlane((uint32_t)(rhi - tbase));

  f32x16 oacc[DV / 32];
#pragma unroll
  for (int nb = 0; nb < DV / 32; nb++)
#pragma unroll
    for (int q = 0; q < 16; q++) oacc[nb][q] = 0.0f;

  // Key tiles visited: history tiles [kt0, min(kt1, kend)), then
  // candidate tiles [bstart, kend).  Tiles made only of candidates that
  // precede every row of the block are fully masked and skipped.  Self
  // mode passes [0, all history tiles); cross mode one chunk of the prefix.
  const int kend = (min(rows_end, key_lim) + BN - 1) / BN;
  const int nh_blk = (n_h + BN - 1) / BN;
  const int nA = max(0, min(kt1, kend) - kt0);
  const int bstart = max(nh_blk, i0 / BN);
  const int n = nA + max(0, kend - bstart);
  auto kb_of = [&](int u) {
    if constexpr (TGT)
      return u < nA ? kt0 + u : bstart + (u - nA);
    else
      return kt0 + u;
  };
  auto pos_base_of = [&](int j0) { return (N - 1) + min(j0, n_h) - R; };

  const int tr_row = 4 * (lane >> 5) + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  // ---- staging: LDS DMA straight from global memory ----
  // Buffer loads relative to the sequence start: rows past its end lie
  // past the descriptor's range and read as zeros.  Byte offsets fit in
  // 32 bits (the library rejects sequences spanning more than 2 GiB).
  // Every wave issues the same number of DMA operations per step, so one
  // vmcnt value before each barrier retires exactly the previous step's.
  constexpr int KP = Sh::KP, VP = Sh::VP, KOPS = Sh::KOPS, VOPS = Sh::VOPS;
  constexpr int KOPW = (KOPS + 3) / 4, VOPW = (VOPS + 3) / 4;
  constexpr int OPS_PER_STEP = KOPW + VOPW + 3 + 1;
  const __amdgpu_buffer_rsrc_t krs =
      make_rsrc(kg + okey * t.k_stride + head * DQK, (uint32_t)(key_lim * t.k_stride * 2));
  const __amdgpu_buffer_rsrc_t vrs =
      make_rsrc(vg + okey * t.v_stride + head * DV, (uint32_t)(key_lim * t.v_stride * 2));
  const __amdgpu_buffer_rsrc_t trs = make_rsrc(tsk, (uint32_t)key_lim * 8u);
  const __amdgpu_buffer_rsrc_t prs = make_rsrc(ja.rab_pos, (uint32_t)(2 * N - 1) * 4u);
  const uint32_t kstride_b = (uint32_t)t.k_stride * 2u, vstride_b = (uint32_t)t.v_stride * 2u;
  // Lane offsets of this wave's K / V operations: chunk g = 64 op + lane
  // of the padded tile is row g / P, chunk g % P (pad chunks repeat chunk
  // 0); operations past the tile's count repeat its last one.
  uint32_t koff[KOPW], voff[VOPW];
#pragma unroll
  for (int k = 0; k < KOPW; k++) {
    const int op = min(wave * KOPW + k, KOPS - 1), g = 64 * op + lane;
    const int ch = g % KP < DQK / 8 ? g % KP : 0;
    koff[k] = (uint32_t)(g / KP) * kstride_b + (uint32_t)ch * 16u;
  }
#pragma unroll
  for (int k = 0; k < VOPW; k++) {
    const int op = min(wave * VOPW + k, VOPS - 1), g = 64 * op + lane;
    const int ch = g % VP < DV / 8 ? g % VP : 0;
    voff[k] = (uint32_t)(g / VP) * vstride_b + (uint32_t)ch * 16u;
  }
  auto issue_k = [&](int u) {
    const uint32_t base = (uint32_t)(kb_of(u) * BN) * kstride_b;
#pragma unroll
    for (int k = 0; k < KOPW; k++)
      dma_to_lds16(krs, sm.sK[u % 3] + 512 * min(wave * KOPW + k, KOPS - 1), koff[k] + base);
  };
  auto issue_v = [&](int u) {
    const uint32_t base = (uint32_t)(kb_of(u) * BN) * vstride_b;
#pragma unroll
    for (int k = 0; k < VOPW; k++)
      dma_to_lds16(vrs, sm.sV[u & 3] + 512 * min(wave * VOPW + k, VOPS - 1), voff[k] + base);
  };
  // rab_pos window: 12 operations of 64 entries (4 shifted copies x 192
  // entries), three per wave.  Entries reachable from (query block, key
  // tile) are (N-1) + p(j) - p(i), p(i) in [min(i0, n_h), R],
  // p(j) in [min(j0, n_h), min(j0+BN-1, n_h)]; entries outside the table
  // (negative offsets wrap past its end) read as 0 and are never used by a
  // valid pair.
  auto issue_win = [&](int u) {
    const int pb = pos_base_of(kb_of(u) * BN);
#pragma unroll
    for (int k = 0; k < 3; k++) {
      const int op = 3 * wave + k, c = op / 3, ch = op % 3;
      dma_to_lds4(prs, &sm.sWin[u % 3][c][Sh::kWinPad + 64 * ch],
                  (uint32_t)(pb + 64 * ch + lane + c) * 4u);
    }
  };
  // Key timestamps as 64 dwords (all waves load the same data).
  auto issue_ts = [&](int u) {
    dma_to_lds4(trs, sm.sT[u & 7], (uint32_t)(kb_of(u) * BN) * 8u + 4u * (uint32_t)lane);
  };
  // Wave 0: rebased min / max of a staged tile's key timestamps (zeros past
  // the sequence end only enter ranges of tiles that are never full).
  auto reduce_ts = [&](int u) {
    if constexpr (FAST) {
      if (wave == 0) {
        const uint32_t v = sm.sT[u & 7][2 * (lane & 31)] - (uint32_t)tbase;
        uint32_t lo = v, hi = v;
#pragma unroll
        for (int off = 16; off > 0; off >>= 1) {
          lo = min(lo, (uint32_t)__shfl_xor((int)lo, off, 64));
          hi = max(hi, (uint32_t)__shfl_xor((int)hi, off, 64));
        }
        sm.sTr[u & 7][lane & 31] = v;
        if (lane < 2) sm.sKr32[u & 3][lane] = lane ? hi : lo;
      }
    }
  };

  // ---- bias path of tile u for this wave, decided two steps ahead ----
  // Full tiles (every pair valid, history positions) whose |t_i - t_j| all
  // lie in one log2 bucket take the rab_pos window plus one rab_time
  // constant ("uniform").  When every t_i >= every t_j (ordered
  // timestamps) and the pairs span two adjacent buckets b and b+1, the
  // time term is a select on t_j <= t_i - 2^(b+1) ("two").  Everything
  // else evaluates each pair ("general").
  enum { kUniform = 0, kTwo = 1, kGeneral = 2 };
  // Full tile: every pair valid, either history rows after every key
  // (j0 + BN - 1 <= iw0), or candidate rows (all at position n_h) against
  // history keys (j0 + BN - 1 < n_h); a wave mixing both has none.  Either
  // way the tiles with j0 <= full_lim (wave-uniform).
  const int full_lim = __builtin_amdgcn_readfirstlane(
      iw0 + 31 >= L ? -1 : iw0 + 31 < n_h ? iw0 - (BN - 1) : iw0 >= n_h ? n_h - BN : -1);
  auto full_tile = [&](int j0) { return j0 <= full_lim; };
  struct Path {
    int kind;
    float cb, cb_far;  // time term (nearer bucket) and, for "two", the farther one
    int thr;           // 2^(b+1) for "two"
  };
  auto classify = [&](int u) -> Path {
    Path r{kGeneral, 0.0f, 0.0f, 0};
    if (u >= n) {
      r.kind = kUniform;  // past the end: the seed is computed but never used
      return r;
    }
    const int j0 = kb_of(u) * BN;
    const bool full = full_tile(j0);
    if constexpr (FAST) {
      if (full) {
        const uint32_t klo = __builtin_amdgcn_readfirstlane(sm.sKr32[u & 3][0]);
        const uint32_t khi = __builtin_amdgcn_readfirstlane(sm.sKr32[u & 3][1]);
        const bool ordered = rlo32 >= khi;
        uint32_t dmin, dmax;
        if (ordered) {
          dmin = rlo32 - khi;
          dmax = rhi32 - klo;
        } else if (klo >= rhi32) {
          dmin = klo - rhi32;
          dmax = khi - rlo32;
        } else {
          dmin = 0;
          dmax = max(rhi32 - klo, khi - rlo32);
        }
        // floor(log2 |dt|) over [dmin, dmax] (|dt| <= 1 -> 0); all < 31.
        const int bnear = 31 - __clz((int)(dmin | 1u)), bfar = 31 - __clz((int)(dmax | 1u));
        if (bnear == bfar) {
          r.kind = kUniform;
          r.cb = sm.sTab[63 - bnear];
        } else if (ordered && bfar == bnear + 1) {
          r.kind = kTwo;
          r.cb = sm.sTab[63 - bnear];
          r.cb_far = sm.sTab[63 - bfar];
          r.thr = 1 << bfar;
        }
      }
    }
    return r;
  };

  // ---- bias seed of tile u for this wave ----
  const int a_win = R - pi + 4 * half;  // window index of (i, j0 + 4*half) in a full tile
  auto seed_uniform = [&](int u, float cb, f32x16& acc) {
    // window index of (i, j) = (j - j0) + (R - i); the lane reads
    // a + 8g + m, a = R - i + 4*half, from the copy that makes it aligned.
    const int c = a_win & 3;
    const float* wp = &sm.sWin[u % 3][c][Sh::kWinPad + a_win - c];
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const f32x4 w = *reinterpret_cast<const f32x4*>(wp + 8 * g);
#pragma unroll
      for (int m = 0; m < 4; m++) acc[4 * g + m] = w[m] + cb;
    }
  };
  auto seed_two = [&](int u, const Path& pth, f32x16& acc) {
    const int c = a_win & 3;
    const float* wp = &sm.sWin[u % 3][c][Sh::kWinPad + a_win - c];
    const uint32_t* tp = sm.sTr[u & 7] + 4 * half;
    const int lim = (int)tir - pth.thr;  // t_j <= lim: the farther bucket
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const f32x4 w = *reinterpret_cast<const f32x4*>(wp + 8 * g);
      const u32x4 tj = *reinterpret_cast<const u32x4*>(tp + 8 * g);
#pragma unroll
      for (int m = 0; m < 4; m++) acc[4 * g + m] = w[m] + ((int)tj[m] <= lim ? pth.cb_far : pth.cb);
    }
  };
  // Per-pair bias.  Branch-free, with every LDS lookup issued before any
  // is consumed, so the lookups of the 16 pairs overlap.  Time term on the
  // fast path: |t_i - t_j| < 2^31 by one v_sad_u32, its leading-zero count
  // z by v_ffbh_u32 (-1 for 0), then tab32[z] = tab[32 + z]; entry -1
  // (= tab[31], unused by the fast path) holds bucket 0, the bucket of
  // |dt| <= 1.
  auto time_terms = [&](int u, float (&tv)[16]) {
    // The lane's 16 keys are 4 runs of 4: jl = 8g + 4*half + m.
    if constexpr (FAST) {
      const uint32_t* tp = sm.sTr[u & 7] + 4 * half;
      uint32_t tj[16];
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(tp + 8 * g);
#pragma unroll
        for (int m = 0; m < 4; m++) tj[4 * g + m] = v[m];
      }
      int z[16];
#pragma unroll
      for (int q = 0; q < 16; q++) {
        uint32_t d, zz;
        asm("v_sad_u32 %0, %1, %2, 0" : "=v"(d) : "v"(tir), "v"(tj[q]));
        asm("v_ffbh_u32 %0, %1" : "=v"(zz) : "v"(d));
        z[q] = (int)zz;
      }
#pragma unroll
      for (int q = 0; q < 16; q++) tv[q] = tab32[z[q]];
    } else {
      // Staged as int64: each run of 4 keys is 8 dwords.
      const uint32_t* tp = sm.sT[u & 7] + 2 * (4 * half);
      uint32_t w[32];
#pragma unroll
      for (int g = 0; g < 4; g++)
#pragma unroll
        for (int h = 0; h < 2; h++) {
          const u32x4 v = *reinterpret_cast<const u32x4*>(tp + 16 * g + 4 * h);
#pragma unroll
          for (int e = 0; e < 4; e++) w[8 * g + 4 * h + e] = v[e];
        }
      int sl[16];
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int64_t tj = (int64_t)(((uint64_t)w[2 * q + 1] << 32) | w[2 * q]);
        sl[q] = slot64(ti64 - tj);
      }
#pragma unroll
      for (int q = 0; q < 16; q++) tv[q] = sm.sTab[sl[q]];
    }
  };
  auto seed_general = [&](int u, f32x16& acc) {
    const int ks = u % 3;
    const int j0 = kb_of(u) * BN;
    const bool full = full_tile(j0);
    if (!full && (iw0 >= L || j0 > wave_last || (j0 >= n_h && j0 + BN - 1 < iw0))) {
#pragma unroll
      for (int q = 0; q < 16; q++) acc[q] = kMaskedBias;
      return;
    }
    float tv[16], wv[16];
    if (full) {
      // Several buckets: position term as on uniform tiles, time term per pair.
      const int c = a_win & 3;
      const float* wp = &sm.sWin[ks][c][Sh::kWinPad + a_win - c];
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const f32x4 w = *reinterpret_cast<const f32x4*>(wp + 8 * g);
#pragma unroll
        for (int m = 0; m < 4; m++) wv[4 * g + m] = w[m];
      }
      time_terms(u, tv);
#pragma unroll
      for (int q = 0; q < 16; q++) acc[q] = wv[q] + tv[q];
    } else if constexpr (!kMaskedWindowReads) {
      // Masked, ragged or candidate pairs: invalid pairs read window entry 0.
      const int pb = min(j0, n_h);
      bool ok[16];
      int x[16];
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int j = j0 + 8 * (q >> 2) + 4 * half + (q & 3);
        ok[q] = row_ok && j < key_lim && pair_valid(my_i, j, n_h);
        x[q] = ok[q] ? bias_pos(j, n_h) - pb + R - pi : 0;
      }
#pragma unroll
      for (int q = 0; q < 16; q++) wv[q] = sm.sWin[ks][0][Sh::kWinPad + x[q]];
      time_terms(u, tv);
#pragma unroll
      for (int q = 0; q < 16; q++) acc[q] = ok[q] ? wv[q] + tv[q] : kMaskedBias;
    } else {
      // The same with history keys (position = index) by the window reads
      // of full tiles (they stay inside the window for every lane, valid
      // or not); candidate keys (all at position n_h) entry by entry.
      bool ok[16];
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int j = j0 + 8 * (q >> 2) + 4 * half + (q & 3);
        ok[q] = row_ok && j < key_lim && pair_valid(my_i, j, n_h);
      }
      if (!TGT || j0 + BN - 1 < n_h) {
        const int c = a_win & 3;
        const float* wp = &sm.sWin[ks][c][Sh::kWinPad + a_win - c];
#pragma unroll
        for (int g = 0; g < 4; g++) {
          const f32x4 w = *reinterpret_cast<const f32x4*>(wp + 8 * g);
#pragma unroll
          for (int m = 0; m < 4; m++) wv[4 * g + m] = w[m];
        }
      } else {
        const int pb = min(j0, n_h);
#pragma unroll
        for (int q = 0; q < 16; q++) {
          const int j = j0 + 8 * (q >> 2) + 4 * half + (q & 3);
          wv[q] = sm.sWin[ks][0][Sh::kWinPad + (ok[q] ? bias_pos(j, n_h) - pb + R - pi : 0)];
        }
      }
      time_terms(u, tv);
#pragma unroll
      for (int q = 0; q < 16; q++) acc[q] = ok[q] ? wv[q] + tv[q] : kMaskedBias;
    }
  };

  auto score = [&](int u, f32x16& acc) {
    const uint16_t* kp = sm.sK[u % 3] + col * K_LD + 8 * half;
#pragma unroll
    for (int s = 0; s < DQK / 16; s++) {
      const u32x4 kf = *reinterpret_cast<const u32x4*>(kp + 16 * s);
      acc = mfma32x32x16(as_bf16x8(kf), as_bf16x8(qf[s]), acc);
    }
  };
  // P operands of a tile: pa[st] the bf16 terms (pa[2 + st] the low
  // terms when SPLIT).
  constexpr int NPA = SPLIT ? 4 : 2;
  auto aggregate = [&](int u, const u32x4 (&pa)[NPA]) {
    const uint16_t* vp = sm.sV[u & 3] + tr_row * V_LD + tr_col;
#pragma unroll
    for (int st = 0; st < 2; st++)
#pragma unroll
      for (int nb = 0; nb < DV / 32; nb++) {
        const uint16_t* base = vp + 16 * st * V_LD + 32 * nb;
        const uint2 lo = lds_read_tr16(base), hi = lds_read_tr16(base + 8 * V_LD);
        const u32x4 vb = {lo.x, lo.y, hi.x, hi.y};
        oacc[nb] = mfma32x32x16(as_bf16x8(pa[st]), as_bf16x8(vb), oacc[nb]);
        if constexpr (SPLIT)
          oacc[nb] = mfma32x32x16(as_bf16x8(pa[2 + st]), as_bf16x8(vb), oacc[nb]);
      }
  };
  auto activate = [&](const f32x16& acc, u32x4 (&pa)[NPA]) {
    float p[16];
#pragma unroll
    for (int q = 0; q < 16; q++) p[q] = silu(acc[q]);
#pragma unroll
    for (int st = 0; st < 2; st++)
#pragma unroll
      for (int e = 0; e < 4; e++) {
        const uint32_t h = pack_bf16x2(p[8 * st + 2 * e], p[8 * st + 2 * e + 1]);
        pa[st][e] = h;
        if constexpr (SPLIT)
          pa[2 + st][e] = pack_bf16x2(p[8 * st + 2 * e] - __uint_as_float(h << 16),
                                      p[8 * st + 2 * e + 1] - __uint_as_float(h & 0xffff0000u));
      }
  };

  // One pipeline step for tile u: S(u+1) and P(u-1) V_{u-1} on the matrix
  // cores while tile u goes through SiLU.  Staging runs ahead: K and the
  // window of tile u+3, V of tile u+2, timestamps of tile u+5 (DMA issued
  // at step s is complete at the barrier of step s+2); tiles past the last
  // are staged too (zeros or unused data) so that every step issues the
  // same operations.
  Path path_next = {kUniform, 0.0f, 0.0f, 0};
  auto step = [&](auto has_prev, int u, f32x16& s_cur, f32x16& s_next, u32x4 (&p_prev)[NPA],
                  u32x4 (&p_cur)[NPA]) {
    wait_vmcnt_lgkmcnt0<OPS_PER_STEP>();
    barrier_no_fence();
    issue_k(u + 3);
    issue_win(u + 3);
    issue_v(u + 2);
    issue_ts(u + 5);
    if (path_next.kind == kUniform)
      seed_uniform(u + 1, path_next.cb, s_next);
    else if (path_next.kind == kTwo)
      seed_two(u + 1, path_next, s_next);
    else
      seed_general(u + 1, s_next);
    score(u + 1, s_next);
    activate(s_cur, p_cur);
    if constexpr (decltype(has_prev)::value) aggregate(u - 1, p_prev);
    // Keeps the SiLU of tile u in this block (it would otherwise be sunk
    // towards its use in the next step, away from the MFMAs).
    asm volatile("" ::"v"(p_cur[0]), "v"(p_cur[1]));
    if constexpr (SPLIT) asm volatile("" ::"v"(p_cur[2]), "v"(p_cur[3]));
    path_next = classify(u + 2);
    reduce_ts(u + 3);
  };

  // Prologue: stage timestamps 0..4, K / window 0..2, V 0..1; key ranges
  // of tiles 0..2; then tile 0 is scored.
  for (int v = 0; v < 5; v++) issue_ts(v);
  for (int v = 0; v < 3; v++) {
    issue_k(v);
    issue_win(v);
  }
  issue_v(0);
  issue_v(1);
  wait_vmcnt_lgkmcnt0<0>();
  barrier_no_fence();
  for (int v = 0; v < 3; v++) reduce_ts(v);
  wait_vmcnt_lgkmcnt0<0>();
  barrier_no_fence();
  f32x16 sA, sB;
  u32x4 pA[NPA], pB[NPA];
  {
    const Path p0 = classify(0);
    if (p0.kind == kUniform)
      seed_uniform(0, p0.cb, sA);
    else if (p0.kind == kTwo)
      seed_two(0, p0, sA);
    else
      seed_general(0, sA);
    score(0, sA);
  }
  path_next = classify(1);
  step(std::false_type{}, 0, sA, sB, pB, pA);
  int u = 1;
  for (; u + 1 < n; u += 2) {
    step(std::true_type{}, u, sB, sA, pA, pB);
    step(std::true_type{}, u + 1, sA, sB, pB, pA);
  }
  if (u < n) {
    step(std::true_type{}, u, sB, sA, pA, pB);
    aggregate(u, pB);
  } else {
    aggregate(u - 1, pA);
  }
  // No LDS-DMA may land after the workgroup ends.
  wait_vmcnt_lgkmcnt0<0>();

  // O accumulator: lane holds (i = iw0 + 8g + 4*half + m, c = 32nb + col);
  // stored as bf16, or as fp32 for a consumer that normalises it.
  const float invN = 1.0f / (float)N;
  if (out_f32) {
    float* __restrict__ og = (float*)out + (orow * H + head) * DV;
#pragma unroll
    for (int nb = 0; nb < DV / 32; nb++)
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int i = iw0 + 8 * (q >> 2) + 4 * half + (q & 3);
        if (i < L) og[(int64_t)i * H * DV + 32 * nb + col] = oacc[nb][q] * invN;
      }
  } else {
    uint16_t* __restrict__ og = (uint16_t*)out + (orow * H + head) * DV;
#pragma unroll
    for (int nb = 0; nb < DV / 32; nb++)
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int i = iw0 + 8 * (q >> 2) + 4 * half + (q & 3);
        if (i < L) og[(int64_t)i * H * DV + 32 * nb + col] = f32_to_bf16_bits(oacc[nb][q] * invN);
      }
  }
}

template <int DQK, int DV, bool SPLIT, bool TGT>
__global__ __launch_bounds__(256, 2) void attn_fwd_bf16_kernel(JaggedArgs ja, Tensors t,
                                                               void* __restrict__ out, int out_f32,
                                                               const WorkItem* __restrict__ items,
                                                               const int32_t* __restrict__ count) {
  using Sh = FwdShared<DQK, DV>;
  __shared__ Sh sm;
  // Workgroup id = item * H + head: the dispatcher walks the (longest
  // first) work list with all heads of an item together, so the long items
  // of every head start early.
  const int item = (int)(blockIdx.x / (unsigned)ja.num_heads);
  const int head = (int)blockIdx.x - item * ja.num_heads;
  if (item >= *count) return;
  const WorkItem it = items[item];
  const int NB = ja.num_buckets;
  const int64_t o = ja.seq_offsets[it.seq];
  const int Lr = (int)(ja.seq_offsets[it.seq + 1] - o);
  // Self-attention: rows and keys are the sequence's L tokens.  Cross mode:
  // the rows are its candidates, virtual positions n_h .. n_h + Lr - 1
  // after the n_h keys of its cached prefix.
  // Cross mode splits the prefix keys into chunks of kCrossChunk, one item
  // each, whose fp32 partial outputs go to separate slots.
  int64_t orow = o, okey = o;
  int L = Lr, n_h = Lr - (ja.num_targets ? (int)ja.num_targets[it.seq] : 0), key_lim = Lr, i0;
  int kt0 = 0, kt1 = (n_h + Sh::BN - 1) / Sh::BN;
  void* outp = out;
  if (ja.key_offsets) {
    okey = ja.key_offsets[it.seq];
    n_h = (int)(ja.key_offsets[it.seq + 1] - okey);
    L = n_h + Lr;
    orow = o - n_h;
    key_lim = n_h;
    const int qb = it.blk / ja.key_chunks, ch = it.blk - qb * ja.key_chunks;
    i0 = n_h + qb * Sh::BM;
    kt0 = ch * (kCrossChunk / Sh::BN);
    kt1 = min((n_h + Sh::BN - 1) / Sh::BN, kt0 + kCrossChunk / Sh::BN);
    outp = (float*)out + (int64_t)ch * ja.chunk_stride;
  } else {
    i0 = it.blk * Sh::BM;
  }
  const int tid = threadIdx.x;

  // The 32-bit fast path applies when the sequence's timestamps span less
  // than 2^31; they are then rebased to its smallest one.
  const int64_t tlo = ja.seq_trange[2 * it.seq], thi = ja.seq_trange[2 * it.seq + 1];
  // Time bias by slot; when every |dt| < 2^31, slots 0..32 are unreachable
  // and entry 31 becomes the fast path's entry for dt = 0 (bucket 0).
  const bool fast = thi - tlo < ((int64_t)1 << 31);
  for (int x = tid; x < 64; x += 256)
    sm.sTab[x] = (fast && x == 31) ? ja.rab_time[0] : ja.rab_time[min(63 - x, NB - 1)];
  __syncthreads();
  if (fast) {
    fwd_item<DQK, DV, true, SPLIT, TGT>(sm, ja, t, outp, out_f32, orow, okey, L, n_h, key_lim, kt0,
                                        kt1, i0, head, tlo);
  } else {
    fwd_item<DQK, DV, false, SPLIT, TGT>(sm, ja, t, outp, out_f32, orow, okey, L, n_h, key_lim, kt0,
                                         kt1, i0, head, tlo);
  }
}

template <int DQK, int DV>
hipError_t launch_fwd(const JaggedArgs& ja, const Tensors& t, void* out, int out_f32, int split,
                      const WorkItem* items, const int32_t* count, int64_t max_items,
                      hipStream_t s) {
  dim3 grid((unsigned)(max_items * ja.num_heads));
  // Candidate key tiles exist only for self attention with targets (cross
  // mode's keys are the cached prefix alone).
  const bool tgt = ja.num_targets && !ja.key_offsets;
#define HSTU_LAUNCH_FWD(SP, TG)                                                                  \
  hipLaunchKernelGGL((attn_fwd_bf16_kernel<DQK, DV, SP, TG>), grid, dim3(256), 0, s, ja, t, out, \
                     out_f32, items, count)
  if (split) {
    if (tgt)
      HSTU_LAUNCH_FWD(true, true);
    else
      HSTU_LAUNCH_FWD(true, false);
  } else {
    if (tgt)
      HSTU_LAUNCH_FWD(false, true);
    else
      HSTU_LAUNCH_FWD(false, false);
  }
#undef HSTU_LAUNCH_FWD
  return hipGetLastError();
}

// Self term of the cached candidate pass: the cross-mode items leave out
// each candidate's own key (position n_h, dt = 0, so rab = rab_pos[N-1] +
// rab_time[0]).  One wave per candidate row and all its heads adds the
// fp32 partials of the row's key chunks in chunk order, then SiLU(q.k +
// rab) v / N, and stores the result once (bf16).  Each lane takes 8
// consecutive features (16-byte loads of q, k, v, the partials and the
// output; rows are 16-byte aligned), the QL = DQK / 8 lanes of a head
// reduce q.k among themselves, and each head's SiLU(q.k + rab) / N passes
// through LDS to the lanes of its output.  The row's sequence comes from
// one load per lane and a ballot when there are fewer than 64 sequences,
// else from a binary search.  Per (row, head) the arithmetic is the same
// for every partition of the candidates into passes.
constexpr int kSelfMaxHeads = 64;
template <int DQK, int DV>
__global__ __launch_bounds__(256) void cached_self_rows_kernel(JaggedArgs ja, Tensors t,
                                                               const float* __restrict__ o32,
                                                               uint16_t* __restrict__ out) {
  __shared__ float spn[4][kSelfMaxHeads];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int H = ja.num_heads, N = ja.max_seq_len, B = ja.num_seqs;
  const int64_t row = (int64_t)blockIdx.x * 4 + wave;
  if (row >= ja.total_tokens) return;
  int b;
  if (B < 64) {
    const int64_t ov = lane <= B ? ja.seq_offsets[lane] : INT64_MAX;
    b = __popcll(__ballot(ov <= row)) - 1;  // offsets non-decreasing, offsets[B] > row
  } else {
    int lo = 0, hi = B - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (ja.seq_offsets[mid] <= row) lo = mid; else hi = mid - 1;
    }
    b = lo;
  }
  const int n_h = (int)(ja.key_offsets[b + 1] - ja.key_offsets[b]);
  const int nch = min((n_h + kCrossChunk - 1) / kCrossChunk, ja.key_chunks);
  const float bias = ja.rab_pos[N - 1] + ja.rab_time[0];
  const float invN = 1.0f / (float)N;
  constexpr int QL = DQK / 8, VL = DV / 8;
  const uint16_t* qr = (const uint16_t*)t.q + row * t.q_stride;
  const uint16_t* kr = (const uint16_t*)t.k + row * t.k_stride;
  const uint16_t* vr = (const uint16_t*)t.v + row * t.v_stride;
  for (int g0 = 0; g0 < H * QL; g0 += 64) {
    const int g = g0 + lane;
    float part = 0.0f;
    if (g < H * QL) {
      const u32x4 qa = *reinterpret_cast<const u32x4*>(qr + 8 * g);
      const u32x4 ka = *reinterpret_cast<const u32x4*>(kr + 8 * g);
#pragma unroll
      for (int e = 0; e < 4; e++) {
        part = __builtin_fmaf(__uint_as_float(qa[e] << 16), __uint_as_float(ka[e] << 16), part);
        part = __builtin_fmaf(__uint_as_float(qa[e] & 0xffff0000u),
                              __uint_as_float(ka[e] & 0xffff0000u), part);
      }
    }
#pragma unroll
    for (int off = QL / 2; off > 0; off >>= 1) part += __shfl_xor(part, off, 64);
    if (g < H * QL && g % QL == 0) spn[wave][g / QL] = silu(part + bias) * invN;
  }
  // LDS accesses of one wave complete in order; this keeps the compiler's too.
  asm volatile("" ::: "memory");
  for (int g0 = 0; g0 < H * VL; g0 += 64) {
    const int g = g0 + lane;
    if (g >= H * VL) break;
    const float pN = spn[wave][g / VL];
    const int64_t oi = row * H * DV + 8 * (int64_t)g;
    float y[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int ch = 0; ch < nch; ch++) {
      const f32x4 a = *reinterpret_cast<const f32x4*>(o32 + (int64_t)ch * ja.chunk_stride + oi);
      const f32x4 c = *reinterpret_cast<const f32x4*>(o32 + (int64_t)ch * ja.chunk_stride + oi + 4);
#pragma unroll
      for (int e = 0; e < 4; e++) {
        y[e] += a[e];
        y[4 + e] += c[e];
      }
    }
    const u32x4 va = *reinterpret_cast<const u32x4*>(vr + 8 * g);
    u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; e++) {
      const float lo = y[2 * e] + pN * __uint_as_float(va[e] << 16);
      const float hi = y[2 * e + 1] + pN * __uint_as_float(va[e] & 0xffff0000u);
      o[e] = (uint32_t)f32_to_bf16_bits(lo) | ((uint32_t)f32_to_bf16_bits(hi) << 16);
    }
    *reinterpret_cast<u32x4*>(out + oi) = o;
  }
}

}  // namespace

hipError_t launch_cached_self(const JaggedArgs& ja, int32_t dqk, int32_t dv, const Tensors& t,
                              const float* o32, void* out, hipStream_t s) {
  if (ja.total_tokens <= 0) return hipSuccess;
  if (ja.num_heads > kSelfMaxHeads) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((ja.total_tokens + 3) / 4));
#define HSTU_SELF_CASE(A, B_)                                                              \
  if (dqk == A && dv == B_) {                                                              \
    hipLaunchKernelGGL((cached_self_rows_kernel<A, B_>), grid, dim3(256), 0, s, ja, t, o32, \
                       (uint16_t*)out);                                                    \
    return hipGetLastError();                                                              \
  }
  HSTU_SELF_CASE(32, 32)
  HSTU_SELF_CASE(32, 64)
  HSTU_SELF_CASE(32, 128)
  HSTU_SELF_CASE(64, 32)
  HSTU_SELF_CASE(64, 64)
  HSTU_SELF_CASE(64, 128)
  HSTU_SELF_CASE(128, 32)
  HSTU_SELF_CASE(128, 64)
  HSTU_SELF_CASE(128, 128)
#undef HSTU_SELF_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_attn_fwd_bf16(const JaggedArgs& ja, const Tensors& t, int dqk, int dv, void* out,
                                int out_f32, int split, const WorkItem* items,
                                const int32_t* count, int64_t max_items, hipStream_t s) {
#define HSTU_FWD_CASE(A, B) \
  if (dqk == A && dv == B)  \
    return launch_fwd<A, B>(ja, t, out, out_f32, split, items, count, max_items, s);
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
