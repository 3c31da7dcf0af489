// Fused jagged pointwise-attention backward, bf16 MFMA (gfx950).
//
// Gradients of <O, dO> for O = (1/N) SiLU(Q K^T + rab) V (Eq. 2).  As the
// paper's appendix on the fused kernels describes, attention and the
// relative bias are recomputed rather than stored, and the bias gradients
// are accumulated on chip before they reach HBM.  Pointwise aggregation
// means no row statistics are needed: with S = Q K^T + rab,
//   P  = SiLU(S) (masked),            dV = (1/N) P^T dO
//   dP = dO V^T,  dS = dP SiLU'(S) (masked)
//   dK = (1/N) dS^T Q,  dQ = (1/N) dS K
//   d rab_pos[(N-1)+p(j)-p(i)] += dS/N,  d rab_time[bkt] += dS/N.
//
// Workgroup = 4 waves, one per SIMD, = one (sequence, 128-key block,
// head) work item.  Wave w owns keys j0 + 32w .. +31: their K and V sit in
// registers as MFMA operands and their dK, dV accumulate in registers for
// the whole item (one wave per SIMD leaves room for all of it).  Owning 32
// keys per wave halves the LDS traffic of the step tiles per MFMA compared
// with 16.  The workgroup walks query steps of 32 rows; per step and wave,
// on v_mfma_f32_32x32x16_bf16:
//   S  = Q K^T (accumulator seeded with the bias), dP = dO V^T: lane = key,
//        16 rows in registers;
//   dV += P^T dO and dK += dS^T Q straight from those registers (the
//        contraction order permuted to the accumulator rows, dO / Q read
//        with transposing LDS loads in that order);
//   dS^T -> LDS; one step later each wave forms its 32-column block of
//        dQ = dS K over the block's keys and adds it to an fp32 workspace
//        with float atomics.
// The step is software-pipelined: S and dP of step u+1 are issued while
// step u goes through SiLU'.  Step tiles (Q, dO, timestamps, rab_pos
// window) arrive by LDS DMA several steps ahead.
// Bias gradients, without per-element atomics on full tiles:
//   time table: a (wave, step) tile whose |t_i - t_j| fall in one or two
//        log2 buckets adds its dS sum to a running per-lane sum (flushed
//        when the bucket changes);
//   position table: history pairs have p(i) - p(j) = i - j.  Rotating
//        register q of every lane by its row offset (ds_bpermute) puts a
//        lane's values on one diagonal, except those that crossed into
//        the other half of the wave, which lie on the diagonal that the
//        partner lane (other half) owns one step later and are handed to
//        it.  Each lane then stores one sum per step, with a plain LDS
//        store, into a ring of diagonals of its own (wave, half); a chunk
//        of 32 diagonals is complete once the rows have moved past it and
//        is then summed over the rings, added to the table in HBM and
//        cleared.  Masked pairs carry dS = 0, so every tile takes this
//        path; candidate rows (all at position n_h) put every pair of a
//        key on one entry, which each lane sums in an LDS word of its own
//        and adds to HBM once per item.
// Tiles whose bucket is not fixed by the timestamp extremes (near the
// diagonal, ragged, 64-bit timestamps): each lane walks its 16 pairs in
// row order and adds every run of equal bucket to the LDS table with one
// float atomic (sweeping the tile's bucket range with a wave reduction per
// bucket cost several times a one-bucket step).
// SPLIT (the layer's backward): dO arrives as two bf16 terms, hi + lo
// (its own LayerNorm backward produces it in fp32, with a dynamic range
// across rows that a single bf16 would turn into several percent of error
// after the cancellations of the contractions); both are staged and each
// dO contraction runs on both.  For the same reason P and dS enter dV, dK
// and dQ as two bf16 terms as well (hi P with both dO terms, lo P with hi
// dO; hi and lo dS with Q and with K).
#include <algorithm>
#include <type_traits>

#include "bias.h"
#include "kernels.h"

namespace hstu {

namespace {

constexpr int64_t kI64Max = 0x7fffffffffffffffll;
constexpr int64_t kI64Min = -kI64Max - 1;
constexpr int kBwdThreads = 256;
constexpr int kBwdWaves = kBwdThreads / 64;
// Bias of a masked pair: SiLU and SiLU' of x ~ -1e30 are exactly -0.
constexpr float kMaskedBias = -1.0e30f;

// Step tile of 32 rows x D features (Q or dO), read two ways: 16-byte row
// chunks (MFMA A operand, one row per lane) and 8-byte transposing loads
// (B operand, 16 lanes = 4 rows x 2 chunks x 2 halves).  For D >= 64 the
// row is unpadded and chunk c of row r sits at chunk c ^ swz(r); swz takes
// 8 values, so 16 consecutive rows would meet each bank group twice: each
// group of 8 rows therefore starts GSH bytes (half of 64 four-byte banks)
// further on than the one before, and the 16 rows of an A-operand read
// cover every bank once (GS = false leaves the groups unshifted, for a
// kernel short of LDS).  For D = 32 rows carry one pad chunk.
template <int D, bool GS = true>
struct StepTile {
  static constexpr int CPR = D / 8;                  // data chunks per row
  static constexpr bool SWZ = D >= 64;
  static constexpr int PC = SWZ ? CPR : CPR + 1;     // chunks per row
  static constexpr int RB = PC * 16;                 // row bytes
  static constexpr int GSH = SWZ && GS ? 128 : 0;    // shift per group of 8 rows
  static constexpr int OPS = (32 * PC + 63) / 64;    // 1 KB DMA operations per tile
  static constexpr int OPW = (OPS + 3) / 4;          // per wave
  static constexpr int BYTES = OPS * 1024 + 3 * GSH;
  __device__ static int swz(int r) { return SWZ ? 2 * (r & 3) + ((r >> 2) & 1) : 0; }
  // Byte offset of row r, and of DMA operation o (1 KB: whole rows when
  // SWZ, so that one operation never straddles a row group).
  __device__ static constexpr int row_base(int r) { return r * RB + GSH * (r >> 3); }
  __device__ static constexpr int op_base(int o) {
    return 1024 * o + GSH * ((o * (1024 / RB)) >> 3);
  }
  static_assert(!SWZ || 1024 % RB == 0, "a DMA operation covers whole rows");
};

// The single-role kernel runs the two-term (SPLIT) backward of heads
// larger than 64, whose staging rings nearly fill LDS: its step tiles go
// without the row-group shift, its dS^T tiles use the 72-byte pitch and
// its window copies a 200-float pitch (8 banks apart, as 264).
template <int DQK, int DV, bool SPLIT>
struct BwdShared {
  using QT = StepTile<DQK, false>;
  using OT = StepTile<DV, false>;
  static constexpr int BN = kBwdBN, BM = kBwdBM;
  // dS^T tile [128 keys][32 rows] bf16, pitch 72 bytes.
  static constexpr int DST_LD = 36;
  // The block's K, row-major, staged once per item to build the dQ
  // operand (pitch 8 dwords mod 32 banks for transposing reads).
  static constexpr int KB_LD = DQK + 16;
  static constexpr int NWIN = BM + BN;  // reversed rab_pos window (BM + BN - 1 used)
  // Each copy is filled at kWinPad .. kWinPad + 191 (three 64-float DMAs).
  static constexpr int kWinPad = 4, WIN_LD = 200;
  static constexpr int NLO = SPLIT ? 4 : 1, LOB = SPLIT ? OT::BYTES : 16;
  union Ring {
    struct {
      __align__(16) uint8_t q[4][QT::BYTES];
      __align__(16) uint8_t dO[4][OT::BYTES];
      __align__(16) uint8_t dOl[NLO][LOB];  // low terms of dO (SPLIT)
    } t;
    __align__(16) uint16_t kblk[BN * KB_LD];  // prologue only
  };
  Ring ring;
  __align__(16) uint16_t sdST[2][BN * DST_LD];
  // SPLIT: the low bf16 terms of dS^T, laid out as sdST.
  __align__(16) uint16_t sdSTl[SPLIT ? 2 : 1][SPLIT ? BN * DST_LD : 8];
  __align__(16) float sWin[4][4][WIN_LD];  // copy c holds window[k + c] at kWinPad + k
  __align__(16) uint32_t sT[8][64];        // step row timestamps (32 int64)
  __align__(16) uint32_t sTr[8][32];       // the same rebased (fast path)
  uint32_t sRr[4][2];                      // rebased row timestamp min / max per step
  float sTab[64];                          // rab_time by slot (bias.h)
  float sTacc[64];                         // time-table gradient by slot
  // Position-gradient rings, one per (wave, half): diagonal k at k % 256.
  static constexpr int kRing = 256;
  float sRing[kBwdWaves][2][kRing];
  float sCand[kBwdWaves][64];  // per lane: dS of candidate rows at its key
};

struct BwdArgs {
  JaggedArgs ja;
  Tensors t;
  const uint16_t* dO;
  const uint16_t* dO_lo;  // SPLIT only
  float* dq_acc;         // single-role kernel: fp32 [h][T][d_qk], atomics
  uint16_t* dq_part;     // two-role kernel: f16 partial dQ blocks (see dq_step)
  float* dq_scale;       // two-role kernel: one power-of-two scale per partial block
  const int64_t* pbase;  // two-role kernel: [B+1] first partial slot of each sequence
  int64_t dq_slots;      // two-role kernel: slots the partial buffer holds (sized for L <= N;
                         // slots past it, only reachable with longer sequences, are skipped)
  uint16_t* dK;
  uint16_t* dV;
  float* d_rab_pos;
  float* d_rab_time;
};

__device__ __forceinline__ float silu_sigma(float x) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x * -kLog2e));
}

template <int DQK, int DV, bool FAST, bool SPLIT>
__device__ __forceinline__ void bwd_item(BwdShared<DQK, DV, SPLIT>& sm, const BwdArgs& A,
                                         int64_t o, int L, int n_h, int j0, int head,
                                         int64_t tbase) {
  using Sh = BwdShared<DQK, DV, SPLIT>;
  using QT = typename Sh::QT;
  using OT = typename Sh::OT;
  constexpr int BN = Sh::BN, BM = Sh::BM, DST_LD = Sh::DST_LD, KB_LD = Sh::KB_LD;
  static_assert(BN == 128 && BM == 32, "4 waves x 32 keys, 32-row steps");
  const JaggedArgs& ja = A.ja;
  const int H = ja.num_heads, N = ja.max_seq_len;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, half = lane >> 5;
  const int jw0 = j0 + 32 * wave;  // the wave's first key
  const int my_j = jw0 + col;       // the lane's key (column of S and dP)
  const bool key_ok = my_j < L;
  const int pj = bias_pos(my_j, n_h);
  const int64_t* __restrict__ ts = ja.timestamps + o;
  const uint16_t* __restrict__ kg = (const uint16_t*)A.t.k + o * A.t.k_stride + head * DQK;
  const uint16_t* __restrict__ vg = (const uint16_t*)A.t.v + o * A.t.v_stride + head * DV;
  const uint16_t* __restrict__ qg = (const uint16_t*)A.t.q + o * A.t.q_stride + head * DQK;
  const uint16_t* __restrict__ dog = A.dO + (o * H + head) * DV;
  const uint16_t* __restrict__ dogl = SPLIT ? A.dO_lo + (o * H + head) * DV : dog;
  const uint32_t kstride_b = (uint32_t)A.t.k_stride * 2u, vstride_b = (uint32_t)A.t.v_stride * 2u;
  const uint32_t qstride_b = (uint32_t)A.t.q_stride * 2u, dostride_b = (uint32_t)(H * DV) * 2u;
  const float invN = 1.0f / (float)N;

  // Candidate keys see only themselves; otherwise every later row sees them.
  const int i_end = j0 >= n_h ? min(j0 + BN, L) : L;
  const int nsteps = (i_end - j0 + BM - 1) / BM;
  auto row0 = [&](int u) { return j0 + BM * u; };

  // ---- per-item operands held in registers ----
  // K, V of the wave's keys: B operands of S = Q K^T and dP = dO V^T
  // (lane = key, 8 features per 16-feature step).  Keys past the sequence
  // end read as zeros.
  const __amdgpu_buffer_rsrc_t krs = make_rsrc(kg, (uint32_t)(L * A.t.k_stride * 2));
  const __amdgpu_buffer_rsrc_t vrs = make_rsrc(vg, (uint32_t)(L * A.t.v_stride * 2));
  u32x4 kf[DQK / 16], vf[DV / 16];
#pragma unroll
  for (int s = 0; s < DQK / 16; s++)
    kf[s] = buffer_load16(krs, (uint32_t)my_j * kstride_b + (uint32_t)(16 * s + 8 * half) * 2u);
#pragma unroll
  for (int s = 0; s < DV / 16; s++)
    vf[s] = buffer_load16(vrs, (uint32_t)my_j * vstride_b + (uint32_t)(16 * s + 8 * half) * 2u);

  // dQ = dS K: the DQK/32 column blocks are shared by the 4 waves; with
  // fewer blocks than waves, each wave of a block takes a share of keys.
  constexpr int NCB = DQK / 32, WPB = kBwdWaves / NCB, KPW = BN / WPB, KSTEPS = KPW / 16;
  const int cbw = wave / WPB, kbase = (wave % WPB) * KPW;
  const int tr_row = 4 * half + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  u32x4 kq[KSTEPS];
  {
    // Stage the block's K row-major, then read the operand down its rows.
    constexpr int KCH = BN * DQK / 8;
    for (int c = tid; c < KCH; c += kBwdThreads) {
      const int r = c / (DQK / 8), cc = c % (DQK / 8);
      *reinterpret_cast<u32x4*>(sm.ring.kblk + r * KB_LD + 8 * cc) =
          buffer_load16(krs, (uint32_t)(j0 + r) * kstride_b + (uint32_t)cc * 16u);
    }
    __syncthreads();
    const uint16_t* kp = sm.ring.kblk + (kbase + tr_row) * KB_LD + 32 * cbw + tr_col;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ks++) {
      const uint2 lo = lds_read_tr16(kp + 16 * ks * KB_LD);
      const uint2 hi = lds_read_tr16(kp + (16 * ks + 8) * KB_LD);
      kq[ks] = u32x4{lo.x, lo.y, hi.x, hi.y};
    }
    __syncthreads();  // the ring may be overwritten from here on
  }

  // Key timestamps (fixed for the item) and the wave's key range.
  const int64_t tj64 = key_ok ? ts[my_j] : tbase;
  const uint32_t tjr = (uint32_t)(tj64 - tbase);
  const uint32_t klo32 =
      __builtin_amdgcn_readfirstlane((uint32_t)(wave_min_i64(key_ok ? tj64 : kI64Max) - tbase));
  const uint32_t khi32 =
      __builtin_amdgcn_readfirstlane((uint32_t)(wave_max_i64(key_ok ? tj64 : kI64Min) - tbase));

  // dK, dV accumulators: lane holds (key jw0 + 8g + 4*half + m, feature 32nb + col).
  f32x16 dkacc[DQK / 32], dvacc[DV / 32];
#pragma unroll
  for (int nb = 0; nb < DQK / 32; nb++)
#pragma unroll
    for (int q = 0; q < 16; q++) dkacc[nb][q] = 0.0f;
#pragma unroll
  for (int nb = 0; nb < DV / 32; nb++)
#pragma unroll
    for (int q = 0; q < 16; q++) dvacc[nb][q] = 0.0f;

  // ---- step-tile addressing ----
  // A-operand reads of row `col`, 16-byte chunk (2s + half).
  auto a_base = [&](auto tile_tag, uint32_t (&ab)[4]) {
    using T = decltype(tile_tag);
    const int sw = T::swz(col);
#pragma unroll
    for (int k = 0; k < 4; k++)
      ab[k] = (uint32_t)(T::row_base(col) + 16 * (half ^ (sw & 1)) + 32 * (k ^ (sw >> 1)));
  };
  auto a_off = [&](auto tile_tag, const uint32_t (&ab)[4], int s) -> uint32_t {
    using T = decltype(tile_tag);
    if constexpr (T::SWZ)
      return ab[s & 3] + 128u * (uint32_t)(s >> 2);
    else
      return (uint32_t)(col * T::RB + 16 * (2 * s + half));
  };
  // Transposing reads: rows (16 st + tr_row [+8]), 4 columns at 32 nb + tr_col.
  // The swizzle of those rows depends on tr_row only.
  auto tr_base = [&](auto tile_tag, uint32_t (&tb)[2]) {
    using T = decltype(tile_tag);
    const int sw = T::swz(tr_row);
    const int c1 = tr_col >> 3, off = (tr_col & 7) * 2;
    const int b = tr_row * T::RB + 16 * (c1 ^ (sw & 3)) + off;
    tb[0] = (uint32_t)(b + 64 * (sw >> 2));  // even 32-column blocks
    tb[1] = (uint32_t)(b - 64 * (sw >> 2));  // odd
  };
  auto tr_off = [&](auto tile_tag, const uint32_t (&tb)[2], int st, int hi, int nb) -> uint32_t {
    using T = decltype(tile_tag);
    const int rows = T::row_base(16 * st + 8 * hi);  // tr_row < 8: same row group
    if constexpr (T::SWZ)
      return tb[nb & 1] + (uint32_t)(rows + 64 * nb);
    else
      return (uint32_t)(tr_row * T::RB + rows + 64 * nb + tr_col * 2);
  };
  uint32_t qa[4], oa[4], qt[2], ot[2];
  a_base(QT{}, qa);
  a_base(OT{}, oa);
  tr_base(QT{}, qt);
  tr_base(OT{}, ot);

  // ---- staging: LDS DMA straight from global memory ----
  // Q, dO and the rab_pos window of step u travel three steps ahead (ring
  // of 4), row timestamps five (ring of 8).  vmcnt counts the DMA
  // operations and the dQ atomics in issue order.  Every wave issues, per
  // step, its DMA operations first and then (from step 1 on) 16 dQ
  // atomics, and possibly a few more atomics (flushes, candidate rows);
  // extra operations only make a vmcnt wait stricter.  Step u needs the
  // DMA of step u - 2, which is followed by that step's atomics and all of
  // step u - 1's operations: the wait lets those stay in flight, so the
  // atomics get about two steps to complete.
  constexpr int OPS_PER_STEP = QT::OPW + (SPLIT ? 2 : 1) * OT::OPW + 3 + 1 + 16;
  const u32x4 qrs = rsrc_words(qg, (uint32_t)(L * A.t.q_stride * 2));
  const u32x4 ors = rsrc_words(dog, (uint32_t)L * dostride_b);
  const u32x4 orsl = rsrc_words(dogl, (uint32_t)L * dostride_b);
  const u32x4 trs = rsrc_words(ts, (uint32_t)L * 8u);
  const u32x4 prs = rsrc_words(ja.rab_pos, (uint32_t)(2 * N - 1) * 4u);
  // Lane offsets of this wave's tile operations: linear chunk g = 64 op +
  // lane is row g / PC, stored chunk g % PC, holding logical chunk
  // (g % PC) ^ swz(row) (pad chunks repeat chunk 0); operations past the
  // tile's count repeat its last one.
  uint32_t qoffs[QT::OPW], ooffs[OT::OPW];
  auto tile_offs = [&](auto tile_tag, uint32_t* offs, uint32_t stride_b) {
    using T = decltype(tile_tag);
#pragma unroll
    for (int k = 0; k < T::OPW; k++) {
      const int op = min(wave * T::OPW + k, T::OPS - 1), g = 64 * op + lane;
      const int r = g / T::PC, p = g % T::PC;
      const int c = p < T::CPR ? (p ^ T::swz(r)) : 0;
      offs[k] = (uint32_t)r * stride_b + (uint32_t)c * 16u;
    }
  };
  tile_offs(QT{}, qoffs, qstride_b);
  tile_offs(OT{}, ooffs, dostride_b);
  auto issue_tiles = [&](int u) {
    const int i0 = row0(u), slot = u & 3;
#pragma unroll
    for (int k = 0; k < QT::OPW; k++)
      dma_to_lds16_asm(qrs, sm.ring.t.q[slot] + QT::op_base(min(wave * QT::OPW + k, QT::OPS - 1)),
                   qoffs[k] + (uint32_t)i0 * qstride_b);
#pragma unroll
    for (int k = 0; k < OT::OPW; k++)
      dma_to_lds16_asm(ors, sm.ring.t.dO[slot] + OT::op_base(min(wave * OT::OPW + k, OT::OPS - 1)),
                   ooffs[k] + (uint32_t)i0 * dostride_b);
    if constexpr (SPLIT) {
#pragma unroll
      for (int k = 0; k < OT::OPW; k++)
        dma_to_lds16_asm(orsl,
                         sm.ring.t.dOl[slot] + OT::op_base(min(wave * OT::OPW + k, OT::OPS - 1)),
                         ooffs[k] + (uint32_t)i0 * dostride_b);
    }
  };
  // Reversed rab_pos window of step u: W[y] = rab_pos[pb - y] with
  // pb = (N-1) + min(j0 + 127, n_h) - min(i0, n_h), so that a pair's entry
  // is y = (min(j0 + 127, n_h) - p(j)) + (p(i) - min(i0, n_h)) in [0, 158].
  // Entries outside the table read as 0 and are never used by a valid pair.
  const int Pk = min(j0 + BN - 1, n_h);
  auto issue_win = [&](int u) {
    const int pb = (N - 1) + Pk - min(row0(u), n_h);
#pragma unroll
    for (int k = 0; k < 3; k++) {
      const int op = 3 * wave + k, c = op / 3, ch = op % 3;
      dma_to_lds4_asm(prs, &sm.sWin[u & 3][c][Sh::kWinPad + 64 * ch],
                  (uint32_t)(pb - 64 * ch - lane - c) * 4u);
    }
  };
  auto issue_ts = [&](int u) {
    dma_to_lds4_asm(trs, sm.sT[u & 7], (uint32_t)row0(u) * 8u + 4u * (uint32_t)lane);
  };
  // Wave 0: rebased row timestamps of a staged step and their range (zeros
  // past the sequence end only enter steps that are never full).
  auto reduce_ts = [&](int u) {
    if constexpr (FAST) {
      if (wave == 0) {
        // Both halves hold the 32 values, so whole-wave extremes are theirs.
        const uint32_t v = sm.sT[u & 7][2 * (lane & 31)] - (uint32_t)tbase;
        const uint32_t lo = wave_min_dpp(v), hi = wave_max_dpp(v);
        sm.sTr[u & 7][lane & 31] = v;
        if (lane < 2) sm.sRr[u & 3][lane] = lane ? hi : lo;
      }
    }
  };

  // ---- bias path of a (wave, step) tile ----
  // Full: every key of the wave precedes every row and all rows are
  // history rows, so every pair is valid with p(i) - p(j) = i - j.  A full
  // tile whose |t_i - t_j| lie in one log2 bucket is "uniform"; one whose
  // t_i all follow the t_j and span two adjacent buckets b, b+1 is "two"
  // (t_i >= t_j + 2^(b+1) selects b+1); everything else is "general".
  enum { kUniform = 0, kTwo = 1, kGeneral = 2 };
  struct Path {
    int code;          // kind | near slot << 2 | far slot << 8 | far bucket << 14
    float cb, cb_far;  // rab_time of the near / far bucket
    __device__ int kind() const { return code & 3; }
    __device__ int slot() const { return (code >> 2) & 63; }
    __device__ int slot_far() const { return (code >> 8) & 63; }
    __device__ uint32_t thr() const { return 1u << ((code >> 14) & 31); }  // 2^(b+1) for "two"
  };
  auto full_tile = [&](int i0) {
    return (jw0 + 31 <= i0) && (i0 + BM - 1 < L) && (i0 + BM - 1 < n_h);
  };
  auto classify = [&](int u) -> Path {
    Path r{kGeneral, 0.0f, 0.0f};
    if (u >= nsteps) {
      r.code = kUniform;  // past the end: computed but never used
      return r;
    }
    if constexpr (FAST) {
      if (full_tile(row0(u))) {
        const uint32_t rlo = __builtin_amdgcn_readfirstlane(sm.sRr[u & 3][0]);
        const uint32_t rhi = __builtin_amdgcn_readfirstlane(sm.sRr[u & 3][1]);
        const bool ordered = rlo >= khi32;
        uint32_t dmin, dmax;
        if (ordered) {
          dmin = rlo - khi32;
          dmax = rhi - klo32;
        } else if (klo32 >= rhi) {
          dmin = klo32 - rhi;
          dmax = khi32 - rlo;
        } else {
          dmin = 0;
          dmax = max(rhi - klo32, khi32 - rlo);
        }
        // floor(log2 |dt|) over [dmin, dmax] (|dt| <= 1 -> 0); all < 31.
        const int bnear = 31 - __clz((int)(dmin | 1u)), bfar = 31 - __clz((int)(dmax | 1u));
        if (bnear == bfar) {
          r.code = kUniform | (63 - bnear) << 2;
          r.cb = sm.sTab[63 - bnear];
        } else if (ordered && bfar == bnear + 1) {
          r.code = kTwo | (63 - bnear) << 2 | (63 - bfar) << 8 | bfar << 14;
          r.cb = sm.sTab[63 - bnear];
          r.cb_far = sm.sTab[63 - bfar];
        }
      }
    }
    return r;
  };

  // ---- bias seed of step u (lane = key, rows 8g + 4*half + m) ----
  const int a_y = Pk - my_j + 4 * half;  // window entry of (row i0 + 4*half, key) on a full tile
  auto win_reads = [&](int u, float (&w)[16]) {
    const int c = a_y & 3;
    const float* wp = &sm.sWin[u & 3][c][Sh::kWinPad + a_y - c];
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(wp + 8 * g);
#pragma unroll
      for (int m = 0; m < 4; m++) w[4 * g + m] = v[m];
    }
  };
  auto row_ts = [&](int u, uint32_t (&ti)[16]) {
    const uint32_t* tp = sm.sTr[u & 7] + 4 * half;
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(tp + 8 * g);
#pragma unroll
      for (int m = 0; m < 4; m++) ti[4 * g + m] = v[m];
    }
  };
  // Time-table slot of every pair (fast path: |dt| < 2^31 by v_sad_u32,
  // z = v_ffbh_u32 (-1 for 0), slot 32 + z; slot 31 stands for dt = 0,
  // bucket 0, and its rab_time entry is set accordingly).
  auto pair_slots = [&](int u, int (&sl)[16]) {
    if constexpr (FAST) {
      uint32_t ti[16];
      row_ts(u, ti);
#pragma unroll
      for (int q = 0; q < 16; q++) {
        uint32_t d, z;
        asm("v_sad_u32 %0, %1, %2, 0" : "=v"(d) : "v"(ti[q]), "v"(tjr));
        asm("v_ffbh_u32 %0, %1" : "=v"(z) : "v"(d));
        sl[q] = 32 + (int)z;
      }
    } else {
      const uint32_t* tp = sm.sT[u & 7] + 2 * (4 * half);
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int r = 8 * (q >> 2) + (q & 3);
        const int64_t ti = (int64_t)(((uint64_t)tp[2 * r + 1] << 32) | tp[2 * r]);
        sl[q] = slot64(ti - tj64);
      }
    }
  };
  auto seed = [&](int u, const Path& pth, f32x16& acc) {
    if (pth.kind() == kUniform) {
      float w[16];
      win_reads(u, w);
#pragma unroll
      for (int q = 0; q < 16; q++) acc[q] = w[q] + pth.cb;
    } else if (pth.kind() == kTwo) {
      float w[16];
      uint32_t ti[16];
      win_reads(u, w);
      row_ts(u, ti);
      const uint32_t lim = tjr + pth.thr();
#pragma unroll
      for (int q = 0; q < 16; q++) acc[q] = w[q] + (ti[q] >= lim ? pth.cb_far : pth.cb);
    } else {
      const int i0 = row0(u), pi0 = min(i0, n_h);
      int sl[16];
      pair_slots(u, sl);
      bool ok[16];
      int y[16];
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int i = i0 + 8 * (q >> 2) + 4 * half + (q & 3);
        ok[q] = key_ok && i < L && pair_valid(i, my_j, n_h);
        y[q] = ok[q] ? (Pk - pj) + (bias_pos(i, n_h) - pi0) : 0;
      }
      float w[16], tv[16];
#pragma unroll
      for (int q = 0; q < 16; q++) {
        w[q] = sm.sWin[u & 3][0][Sh::kWinPad + y[q]];
        tv[q] = sm.sTab[sl[q]];
      }
#pragma unroll
      for (int q = 0; q < 16; q++) acc[q] = ok[q] ? w[q] + tv[q] : kMaskedBias;
    }
  };

  // ---- contractions ----
  auto scores = [&](int u, f32x16& sacc, f32x16& pacc) {
    const uint8_t* qb = sm.ring.t.q[u & 3];
    const uint8_t* ob = sm.ring.t.dO[u & 3];
    pacc = f32x16{};
    constexpr int SMAX = DQK > DV ? DQK / 16 : DV / 16;
#pragma unroll
    for (int s = 0; s < SMAX; s++) {
      if (s < DQK / 16) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(qb + a_off(QT{}, qa, s));
        sacc = mfma32x32x16(as_bf16x8(a), as_bf16x8(kf[s]), sacc);
      }
      if (s < DV / 16) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(ob + a_off(OT{}, oa, s));
        pacc = mfma32x32x16(as_bf16x8(a), as_bf16x8(vf[s]), pacc);
        if constexpr (SPLIT) {
          const u32x4 al =
              *reinterpret_cast<const u32x4*>(sm.ring.t.dOl[u & 3] + a_off(OT{}, oa, s));
          pacc = mfma32x32x16(as_bf16x8(al), as_bf16x8(vf[s]), pacc);
        }
      }
    }
  };
  // dV += P^T dO, dK += dS^T Q: k-slots (st, e) of the A operands are the
  // accumulator rows 16 st + 8 (e / 4) + 4*half + e % 4.
  // pl, dl: the low bf16 terms of P and dS (SPLIT only).
  auto key_grads = [&](int u, const u32x4 (&pa)[2], const u32x4 (&da)[2], const u32x4 (&pl)[2],
                       const u32x4 (&dl)[2]) {
    const uint8_t* qb = sm.ring.t.q[u & 3];
    const uint8_t* ob = sm.ring.t.dO[u & 3];
#pragma unroll
    for (int st = 0; st < 2; st++) {
#pragma unroll
      for (int nb = 0; nb < DV / 32; nb++) {
        const uint2 lo = lds_read_tr16((const uint16_t*)(ob + tr_off(OT{}, ot, st, 0, nb)));
        const uint2 hi = lds_read_tr16((const uint16_t*)(ob + tr_off(OT{}, ot, st, 1, nb)));
        dvacc[nb] = mfma32x32x16(as_bf16x8(pa[st]),
                                 as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y}), dvacc[nb]);
        if constexpr (SPLIT) {
          dvacc[nb] = mfma32x32x16(as_bf16x8(pl[st]),
                                 as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y}), dvacc[nb]);
          const uint8_t* obl = sm.ring.t.dOl[u & 3];
          const uint2 l2 = lds_read_tr16((const uint16_t*)(obl + tr_off(OT{}, ot, st, 0, nb)));
          const uint2 h2 = lds_read_tr16((const uint16_t*)(obl + tr_off(OT{}, ot, st, 1, nb)));
          dvacc[nb] = mfma32x32x16(as_bf16x8(pa[st]),
                                 as_bf16x8(u32x4{l2.x, l2.y, h2.x, h2.y}), dvacc[nb]);
        }
      }
#pragma unroll
      for (int nb = 0; nb < DQK / 32; nb++) {
        const uint2 lo = lds_read_tr16((const uint16_t*)(qb + tr_off(QT{}, qt, st, 0, nb)));
        const uint2 hi = lds_read_tr16((const uint16_t*)(qb + tr_off(QT{}, qt, st, 1, nb)));
        dkacc[nb] = mfma32x32x16(as_bf16x8(da[st]),
                                 as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y}), dkacc[nb]);
        if constexpr (SPLIT)
          dkacc[nb] = mfma32x32x16(as_bf16x8(dl[st]),
                                 as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y}), dkacc[nb]);
      }
    }
  };
  // dS^T of step u into its LDS slot: the lane (key) writes 4 runs of 4
  // rows (SPLIT: the low terms likewise).
  auto store_dst = [&](int u, const u32x4 (&da)[2], const u32x4 (&dl)[2]) {
    uint16_t* dp = sm.sdST[u & 1] + (32 * wave + col) * DST_LD + 4 * half;
#pragma unroll
    for (int st = 0; st < 2; st++) {
      *reinterpret_cast<uint2*>(dp + 16 * st) = uint2{da[st][0], da[st][1]};
      *reinterpret_cast<uint2*>(dp + 16 * st + 8) = uint2{da[st][2], da[st][3]};
    }
    if constexpr (SPLIT) {
      uint16_t* dpl = sm.sdSTl[u & 1] + (32 * wave + col) * DST_LD + 4 * half;
#pragma unroll
      for (int st = 0; st < 2; st++) {
        *reinterpret_cast<uint2*>(dpl + 16 * st) = uint2{dl[st][0], dl[st][1]};
        *reinterpret_cast<uint2*>(dpl + 16 * st + 8) = uint2{dl[st][2], dl[st][3]};
      }
    }
  };
  // dQ(rows of step u, the wave's 32 columns) over its keys, added to the
  // fp32 workspace [h][T][d_qk] of the head with buffer atomics: lane holds
  // (row i0 + 8g + 4*half + m, column 32 cbw + col); the row group goes
  // into the lane offset and m into the immediate offset.  Rows past the
  // sequence end fall outside the buffer and are dropped by the hardware.
  // The atomics go out after the next seed, among the step's contractions.
  const __amdgpu_buffer_rsrc_t dqrs =
      make_rsrc(A.dq_acc + ((size_t)head * (size_t)ja.total_tokens + (size_t)o) * DQK,
                (uint32_t)L * (uint32_t)DQK * 4u);
  const uint32_t dq_lane = (uint32_t)((4 * half * DQK + 32 * cbw + col) * 4);
  auto dq_mfma = [&](int u, f32x16& qacc) {
    const uint16_t* dp = sm.sdST[u & 1] + (kbase + tr_row) * DST_LD + tr_col;
    qacc = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ks++) {
      const uint2 lo = lds_read_tr16(dp + 16 * ks * DST_LD);
      const uint2 hi = lds_read_tr16(dp + (16 * ks + 8) * DST_LD);
      qacc = mfma32x32x16(as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y}), as_bf16x8(kq[ks]), qacc);
    }
    if constexpr (SPLIT) {
      const uint16_t* dpl = sm.sdSTl[u & 1] + (kbase + tr_row) * DST_LD + tr_col;
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ks++) {
        const uint2 lo = lds_read_tr16(dpl + 16 * ks * DST_LD);
        const uint2 hi = lds_read_tr16(dpl + (16 * ks + 8) * DST_LD);
        qacc = mfma32x32x16(as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y}), as_bf16x8(kq[ks]), qacc);
      }
    }
  };
  auto dq_atomics = [&](int u, const f32x16& qacc) {
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const uint32_t vo = dq_lane + (uint32_t)((row0(u) + 8 * g) * DQK * 4);
#pragma unroll
      for (int m = 0; m < 4; m++)
        __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(qacc[4 * g + m], dqrs, vo + m * DQK * 4, 0,
                                                        0);
    }
  };

  // ---- bias gradients ----
  // Time table: running per-lane sums for up to two slots (the near and
  // the far bucket of a tile), each flushed when its slot changes.
  int run_slot[2] = {-1, -1};
  float run_acc[2] = {0.0f, 0.0f};
  auto time_flush = [&](int r) {
    if (run_slot[r] >= 0) {
      const float v = wave_sum_dpp(run_acc[r]);
      if (lane == 0) atomicAdd(&sm.sTacc[run_slot[r]], v);
    }
    run_acc[r] = 0.0f;
  };
  auto time_add = [&](int r, int slot, float v) {
    if (slot != run_slot[r]) {
      time_flush(r);
      run_slot[r] = slot;
    }
    run_acc[r] += v;
  };

  // Position table.  Lane (col, half) reads register q = 4g + m from lane
  // + r0, r0 = 8g + m (mod 64): the pair (row 8g + 4*half' + m, key col')
  // then lies on diagonal D1 = (i0 - jw0) - col + 4*half if col + r0 < 32,
  // else on D1 of the partner lane (col, 1 - half) one step later.
  constexpr int kRing = Sh::kRing;
  const int perm_base = lane * 4;
  float wrap_w[16];
#pragma unroll
  for (int q = 0; q < 16; q++) wrap_w[q] = col + 8 * (q >> 2) + (q & 3) >= 32 ? 1.0f : 0.0f;
  float* const ring_mine = sm.sRing[wave][half];
  const int d1_lane = 4 * half - col - 32 * wave;  // D1 = 32 u + d1_lane
  float carry = 0.0f;  // partner's crossing sum of the previous step
  // Candidate rows all sit at position n_h, so every candidate pair of the
  // lane's key j lands on one position entry, (N-1) - (n_h - p(j)): the
  // lane sums them over the item in its own LDS word (a register would
  // stay live through every step) and adds them once at its end.
  float* const cand_sum = &sm.sCand[wave][lane];
  *cand_sum = 0.0f;
  auto pos_step = [&](int u, const float (&ds)[16]) {
    float sum = 0.0f, wsum = 0.0f;
#pragma unroll
    for (int q = 0; q < 16; q++) {
      const float rv = __int_as_float(__builtin_amdgcn_ds_bpermute(
          perm_base + 4 * (8 * (q >> 2) + (q & 3)), __float_as_int(ds[q])));
      sum += rv;
      wsum = __builtin_fmaf(rv, wrap_w[q], wsum);
    }
    ring_mine[(32 * u + d1_lane) & (kRing - 1)] = (sum - wsum) + carry;
    carry = __int_as_float(__builtin_amdgcn_ds_bpermute(perm_base ^ 128, __float_as_int(wsum)));
  };
  // Diagonals [32c, 32c + 31] are complete after step c + 4; one wave sums
  // them over the rings, adds them to the table and clears them after the
  // next barrier.
  const int R = L - j0;  // p(i) - p(j) of kept history pairs lies in [0, R)
  auto ring_flush = [&](int c) {
    if (lane < 32) {
      const int k = 32 * c + lane, sl = k & (kRing - 1);
      float v = 0.0f;
#pragma unroll
      for (int w = 0; w < kBwdWaves; w++)
#pragma unroll
        for (int h = 0; h < 2; h++) {
          v += sm.sRing[w][h][sl];
          sm.sRing[w][h][sl] = 0.0f;
        }
      if (v != 0.0f && k < R) unsafeAtomicAdd(&A.d_rab_pos[(N - 1) - k], v * invN);
    }
  };

  auto grads = [&](int u, const Path& pth, const float (&ds)[16]) {
    const int i0 = row0(u);
    if (i0 + BM - 1 >= n_h && i0 < L) {
      // Candidate rows: into the lane's candidate sum, out of the
      // diagonal sums.
      float dh[16], cs = 0.0f;
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int i = i0 + 8 * (q >> 2) + 4 * half + (q & 3);
        dh[q] = i < n_h ? ds[q] : 0.0f;
        if (i >= n_h && i < L && key_ok && pair_valid(i, my_j, n_h)) cs += ds[q];
      }
      *cand_sum += cs;
      pos_step(u, dh);
    } else {
      pos_step(u, ds);
    }
    if (pth.kind() != kGeneral) {
      float tot = 0.0f;
#pragma unroll
      for (int q = 0; q < 16; q++) tot += ds[q];
      if (pth.kind() == kTwo) {
        uint32_t ti[16];
        row_ts(u, ti);
        const uint32_t lim = tjr + pth.thr();
        float far = 0.0f;
#pragma unroll
        for (int q = 0; q < 16; q++) far += ti[q] >= lim ? ds[q] : 0.0f;
        time_add(0, pth.slot(), tot - far);
        time_add(1, pth.slot_far(), far);
      } else {
        time_add(0, pth.slot(), tot);
      }
    } else {
      // Bucket by bucket over the slots of the tile's valid pairs.
      // Several buckets: a lane's 16 pairs (rows in order, its one key)
      // form runs of equal slot, each added once to the LDS table (masked
      // pairs carry dS = 0 and may sit in any run).
      int sl[16];
      pair_slots(u, sl);
      float run = ds[0];
#pragma unroll
      for (int q = 1; q < 16; q++) {
        if (sl[q] != sl[q - 1]) {
          atomicAdd(&sm.sTacc[sl[q - 1]], run);
          run = 0.0f;
        }
        run += ds[q];
      }
      atomicAdd(&sm.sTacc[sl[15]], run);
    }
  };

  // ---- pipelined steps ----
  // Step u: dQ(u-1); S, dP of step u+1 seeded and issued; SiLU' of step u;
  // dV, dK of step u; dS^T(u) to LDS; bias gradients of step u.
  Path path_cur, path_next, path_nn;
  auto step = [&](int u, f32x16& s_cur, f32x16& p_cur, f32x16& s_next, f32x16& p_next) {
    if (u >= 3)
      wait_vmcnt_lgkmcnt0<OPS_PER_STEP + 16>();
    else
      wait_vmcnt_lgkmcnt0<OPS_PER_STEP>();
    barrier_no_fence();
    if (u >= 5 && wave == (u & 3)) ring_flush(u - 5);
    issue_tiles(u + 3);
    issue_win(u + 3);
    issue_ts(u + 5);
    f32x16 qacc;
    if (u >= 1) dq_mfma(u - 1, qacc);
    if (u + 1 < nsteps) seed(u + 1, path_next, s_next);
    if (u >= 1) dq_atomics(u - 1, qacc);
    scores(u + 1, s_next, p_next);
    float pv[16], dsv[16];
#pragma unroll
    for (int q = 0; q < 16; q++) {
      const float x = s_cur[q];
      const float sg = silu_sigma(x);
      const float p = x * sg;
      pv[q] = p;
      dsv[q] = p_cur[q] * __builtin_fmaf(p, 1.0f - sg, sg);
    }
    u32x4 pa[2], da[2], pl[2], dl[2];
#pragma unroll
    for (int st = 0; st < 2; st++) {
      pa[st] = pack_bf16x8(pv + 8 * st);
      da[st] = pack_bf16x8(dsv + 8 * st);
      if constexpr (SPLIT) {
        // low terms: value - bf16(value), exact in fp32
#pragma unroll
        for (int e = 0; e < 4; e++) {
          const uint32_t h = pa[st][e], g = da[st][e];
          pl[st][e] = pack_bf16x2(pv[8 * st + 2 * e] - __uint_as_float(h << 16),
                                  pv[8 * st + 2 * e + 1] - __uint_as_float(h & 0xffff0000u));
          dl[st][e] = pack_bf16x2(dsv[8 * st + 2 * e] - __uint_as_float(g << 16),
                                  dsv[8 * st + 2 * e + 1] - __uint_as_float(g & 0xffff0000u));
        }
      }
    }
    key_grads(u, pa, da, pl, dl);
    store_dst(u, da, dl);
    grads(u, path_cur, dsv);
    path_nn = classify(u + 2);
    reduce_ts(u + 3);
    path_cur = path_next;
    path_next = path_nn;
  };

  // Prologue: timestamps of steps 0..4, tiles and windows of steps 0..2,
  // row ranges of steps 0..2; then step 0 is scored.
  for (int v = 0; v < 5; v++) issue_ts(v);
  for (int v = 0; v < 3; v++) {
    issue_tiles(v);
    issue_win(v);
  }
  wait_vmcnt_lgkmcnt0<0>();
  barrier_no_fence();
  for (int v = 0; v < 3; v++) reduce_ts(v);
  wait_vmcnt_lgkmcnt0<0>();
  barrier_no_fence();
  f32x16 sA, pA, sB, pB;
  path_cur = classify(0);
  path_next = classify(1);
  seed(0, path_cur, sA);
  scores(0, sA, pA);
  int u = 0;
  for (; u + 1 < nsteps; u += 2) {
    step(u, sA, pA, sB, pB);
    step(u + 1, sB, pB, sA, pA);
  }
  if (u < nsteps) step(u, sA, pA, sB, pB);
  // dS^T of the last step is visible after one more barrier; no LDS DMA
  // may be in flight when the workgroup ends.
  wait_vmcnt_lgkmcnt0<0>();
  barrier_no_fence();
  {
    f32x16 qacc;
    dq_mfma(nsteps - 1, qacc);
    dq_atomics(nsteps - 1, qacc);
  }
  time_flush(0);
  time_flush(1);
  if (const float cv = *cand_sum; cv != 0.0f)
    unsafeAtomicAdd(&A.d_rab_pos[(N - 1) - (n_h - pj)], cv * invN);
  // The last crossing sums belong to D1 of step nsteps; then the chunks
  // not flushed inside the loop, max(0, nsteps - 5) .. nsteps.
  ring_mine[(32 * nsteps + d1_lane) & (kRing - 1)] = carry;
  wait_vmcnt_lgkmcnt0<0>();
  barrier_no_fence();
  {
    const int c0 = max(0, nsteps - 5);
    for (int c = c0 + wave; c <= nsteps; c += kBwdWaves) ring_flush(c);
  }

  // dK, dV of the wave's keys: lane holds (key jw0 + 8g + 4*half + m, feature 32nb + col).
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
}

// ---------------------------------------------------------------------------
// Role-split backward: 8 waves, two per SIMD, no duplicated work.
//
// With one wave per SIMD the step above is bound by the latency of one
// instruction stream: its 40 MFMAs keep the matrix core busy for under a
// fifth of the step.  Here each SIMD runs two waves that own the same 32
// keys and divide a step between them:
//   role A (waves 0-3): S = Q K^T and dP = dO V^T (bias-seeded), SiLU and
//        SiLU', the bias gradients, and P, dS rounded to bf16 into LDS;
//   role B (waves 4-7), one step behind: dV += P^T dO, dK += dS^T Q (the
//        dK, dV accumulators live only here) and the dQ product.
// The dQ product of a step (32 rows x d_qk over the block's 128 keys) is
// not added to a shared accumulator with atomics: their memory-side rate
// would bind the kernel (one fp32 row per key block and visited row,
// 16x the algorithmic traffic).  It is stored in the step's own slot of a
// partial buffer as f16 scaled by a power of two that puts the block's
// largest magnitude in [2^13, 2^14) (half the bytes of fp32, 2^-11
// relative rounding, no overflow whatever the data), and dq_reduce_kernel
// sums the slots of every row in key-block order (deterministic).
// A holds K and V as MFMA operands, B the dK / dV accumulators and the dQ
// operand, so each role fits in half the register file.  One barrier per
// step orders the hand-over: A writes P and dS of step u into slot u & 1;
// B reads them, and the Q / dO tile of step u, after the next barrier.  B
// lags one step, so the Q / dO ring has five slots (DMA three ahead).
template <int DQK, int DV, bool SPLIT = false>
struct BwdSharedRS {
  using QT = StepTile<DQK>;
  using OT = StepTile<DV>;
  static constexpr int BN = kBwdBN, BM = kBwdBM;
  // Q / dO ring: at step u role A reads the tiles of step u + 1 and role B
  // those of u - 1 (and u at the next step), and LDS DMA fills kAhead steps
  // ahead, so kAhead + 2 slots.  SPLIT also stages the low dO terms and, to
  // fit LDS, fills two steps ahead instead of three.
  static constexpr int kAhead = SPLIT ? 2 : 3;
  static constexpr int kSlots = kAhead + 2;
  static constexpr int NLO = SPLIT ? kSlots : 1, LOB = SPLIT ? OT::BYTES : 16;
  // dS^T [128 keys][32 rows] bf16, pitch 72 bytes: role A's row-wise
  // 8-byte stores and role B's row-wise dK-operand reads of 32 keys then
  // spread over all banks (a 96-byte pitch put them on 8 of 32); the
  // transposing reads of the dQ step take a few more conflicts than at
  // 96 bytes (long workload: backward 1.412 -> 1.377 ms).
  static constexpr int DST_LD = 36;
  static constexpr int KB_LD = DQK + 16;
  static constexpr int kWinPad = 4, WIN_LD = 264;
  union Ring {
    struct {
      __align__(16) uint8_t q[kSlots][QT::BYTES];
      __align__(16) uint8_t dO[kSlots][OT::BYTES];
      __align__(16) uint8_t dOl[NLO][LOB];  // low terms of dO (SPLIT)
    } t;
    __align__(16) uint16_t kblk[BN * KB_LD];  // prologue only
  };
  Ring ring;
  __align__(16) uint16_t sdST[2][BN * DST_LD];
  // P as role A's MFMA operand registers: [slot][wave][k-step][lane].
  __align__(16) u32x4 sPA[2][4][2][64];
  __align__(16) float sWin[4][4][WIN_LD];
  __align__(16) uint32_t sT[8][64];
  __align__(16) uint32_t sTr[8][32];
  uint32_t sRr[4][2];
  float sTab[64];
  float sTacc[64];
  static constexpr int kRing = 256;
  float sRing[4][2][kRing];
  float sCand[4][64];  // per role-A lane: dS of candidate rows at its key
  // SPLIT: the low bf16 terms of dS^T and P, laid out as sdST and sPA.
  __align__(16) uint16_t sdSTl[SPLIT ? 2 : 1][SPLIT ? BN * DST_LD : 8];
  __align__(16) u32x4 sPAl[SPLIT ? 2 : 1][4][2][SPLIT ? 64 : 1];
};

// Everything both roles compute from the item (no per-role state).
struct RsItem {
  int64_t o;
  int seq, L, n_h, j0, head, nsteps;
};

// TGT: the batch may hold candidate rows (num_targets given); without
// them the candidate paths below are compiled out.  CF: candidate rows
// against history keys are full tiles (key-only position term, one-bucket
// time paths); the two-term instance leaves them on the general path,
// which timed faster there on batches without candidates.
template <int DQK, int DV, bool FAST, bool SPLIT, bool TGT>
__device__ __forceinline__ void bwd_role_a(BwdSharedRS<DQK, DV, SPLIT>& sm, const BwdArgs& A,
                                           const RsItem& it, int64_t tbase) {
  using Sh = BwdSharedRS<DQK, DV, SPLIT>;
  constexpr bool CF = TGT && !SPLIT;
  // Masked tiles of history rows read the position window as full tiles
  // do, where registers allow: at d_qk or d_v = 128 the other form spills.
  constexpr bool kMaskedWindowReads = DQK <= 64 && DV <= 64;
  using QT = typename Sh::QT;
  using OT = typename Sh::OT;
  constexpr int BN = Sh::BN, BM = Sh::BM, DST_LD = Sh::DST_LD, kSlots = Sh::kSlots;
  constexpr int kAhead = Sh::kAhead;
  const JaggedArgs& ja = A.ja;
  const int H = ja.num_heads, N = ja.max_seq_len;
  const int64_t o = it.o;
  const int L = it.L, n_h = it.n_h, j0 = it.j0, head = it.head, nsteps = it.nsteps;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // 0..3
  const int col = lane & 31, half = lane >> 5;
  const int jw0 = j0 + 32 * wave;
  const int my_j = jw0 + col;
  const bool key_ok = my_j < L;
  const int pj = bias_pos(my_j, n_h);
  const int64_t* __restrict__ ts = ja.timestamps + o;
  const uint16_t* __restrict__ kg = (const uint16_t*)A.t.k + o * A.t.k_stride + head * DQK;
  const uint16_t* __restrict__ vg = (const uint16_t*)A.t.v + o * A.t.v_stride + head * DV;
  const uint16_t* __restrict__ qg = (const uint16_t*)A.t.q + o * A.t.q_stride + head * DQK;
  const uint16_t* __restrict__ dog = A.dO + (o * H + head) * DV;
  const uint16_t* __restrict__ dogl = SPLIT ? A.dO_lo + (o * H + head) * DV : dog;
  const uint32_t kstride_b = (uint32_t)A.t.k_stride * 2u, vstride_b = (uint32_t)A.t.v_stride * 2u;
  const uint32_t qstride_b = (uint32_t)A.t.q_stride * 2u, dostride_b = (uint32_t)(H * DV) * 2u;
  const float invN = 1.0f / (float)N;
  auto row0 = [&](int u) { return j0 + BM * u; };

  // K, V of the wave's keys: B operands of S and dP (keys past the end read as zeros).
  const __amdgpu_buffer_rsrc_t krs = make_rsrc(kg, (uint32_t)(L * A.t.k_stride * 2));
  const __amdgpu_buffer_rsrc_t vrs = make_rsrc(vg, (uint32_t)(L * A.t.v_stride * 2));
  u32x4 kf[DQK / 16], vf[DV / 16];
#pragma unroll
  for (int s = 0; s < DQK / 16; s++)
    kf[s] = buffer_load16(krs, (uint32_t)my_j * kstride_b + (uint32_t)(16 * s + 8 * half) * 2u);
#pragma unroll
  for (int s = 0; s < DV / 16; s++)
    vf[s] = buffer_load16(vrs, (uint32_t)my_j * vstride_b + (uint32_t)(16 * s + 8 * half) * 2u);

  const int64_t tj64 = key_ok ? ts[my_j] : tbase;
  const uint32_t tjr = (uint32_t)(tj64 - tbase);
  const uint32_t klo32 =
      __builtin_amdgcn_readfirstlane((uint32_t)(wave_min_i64(key_ok ? tj64 : kI64Max) - tbase));
  const uint32_t khi32 =
      __builtin_amdgcn_readfirstlane((uint32_t)(wave_max_i64(key_ok ? tj64 : kI64Min) - tbase));

  // A-operand reads of row `col`, 16-byte chunk (2s + half) (as in bwd_item).
  auto a_base = [&](auto tile_tag, uint32_t (&ab)[4]) {
    using T = decltype(tile_tag);
    const int sw = T::swz(col);
#pragma unroll
    for (int k = 0; k < 4; k++)
      ab[k] = (uint32_t)(T::row_base(col) + 16 * (half ^ (sw & 1)) + 32 * (k ^ (sw >> 1)));
  };
  auto a_off = [&](auto tile_tag, const uint32_t (&ab)[4], int s) -> uint32_t {
    using T = decltype(tile_tag);
    if constexpr (T::SWZ)
      return ab[s & 3] + 128u * (uint32_t)(s >> 2);
    else
      return (uint32_t)(col * T::RB + 16 * (2 * s + half));
  };
  uint32_t qa[4], oa[4];
  a_base(QT{}, qa);
  a_base(OT{}, oa);

  // ---- staging by LDS DMA: Q and dO kAhead steps ahead (three, or two
  // with SPLIT's low dO terms), the rab_pos window three steps ahead, row
  // timestamps five.  Only role A issues DMA, in the order tiles, window,
  // timestamps.  Step u needs the tiles and window of step u + 1 and (for
  // role B's reduce_ts(u + 3), after the same barrier) the row timestamps
  // of step u + 3.  With kAhead = 3 all were issued at step u - 2 and only
  // step u - 1's operations follow them; with kAhead = 2 the tiles were
  // the first operations of step u - 1, followed by its window and
  // timestamps.  The wait at step u allows that many outstanding (later
  // atomics only make it stricter).
  constexpr int OPS_PER_STEP = kAhead == 3 ? QT::OPW + OT::OPW + 3 + 1 : 3 + 1;
  const u32x4 qrs = rsrc_words(qg, (uint32_t)(L * A.t.q_stride * 2));
  const u32x4 ors = rsrc_words(dog, (uint32_t)L * dostride_b);
  const u32x4 orsl = rsrc_words(dogl, (uint32_t)L * dostride_b);
  const u32x4 trs = rsrc_words(ts, (uint32_t)L * 8u);
  const u32x4 prs = rsrc_words(ja.rab_pos, (uint32_t)(2 * N - 1) * 4u);
  uint32_t qoffs[QT::OPW], ooffs[OT::OPW];
  auto tile_offs = [&](auto tile_tag, uint32_t* offs, uint32_t stride_b) {
    using T = decltype(tile_tag);
#pragma unroll
    for (int k = 0; k < T::OPW; k++) {
      const int op = min(wave * T::OPW + k, T::OPS - 1), g = 64 * op + lane;
      const int r = g / T::PC, p = g % T::PC;
      const int c = p < T::CPR ? (p ^ T::swz(r)) : 0;
      offs[k] = (uint32_t)r * stride_b + (uint32_t)c * 16u;
    }
  };
  tile_offs(QT{}, qoffs, qstride_b);
  tile_offs(OT{}, ooffs, dostride_b);
  auto issue_tiles = [&](int u) {
    const int i0 = row0(u), slot = u % kSlots;
#pragma unroll
    for (int k = 0; k < QT::OPW; k++)
      dma_to_lds16_asm(qrs, sm.ring.t.q[slot] + QT::op_base(min(wave * QT::OPW + k, QT::OPS - 1)),
                       qoffs[k] + (uint32_t)i0 * qstride_b);
#pragma unroll
    for (int k = 0; k < OT::OPW; k++)
      dma_to_lds16_asm(ors, sm.ring.t.dO[slot] + OT::op_base(min(wave * OT::OPW + k, OT::OPS - 1)),
                       ooffs[k] + (uint32_t)i0 * dostride_b);
    if constexpr (SPLIT) {
#pragma unroll
      for (int k = 0; k < OT::OPW; k++)
        dma_to_lds16_asm(orsl,
                         sm.ring.t.dOl[slot] + OT::op_base(min(wave * OT::OPW + k, OT::OPS - 1)),
                         ooffs[k] + (uint32_t)i0 * dostride_b);
    }
  };
  const int Pk = min(j0 + BN - 1, n_h);
  auto issue_win = [&](int u) {
    const int pb = (N - 1) + Pk - min(row0(u), n_h);
#pragma unroll
    for (int k = 0; k < 3; k++) {
      const int op = 3 * wave + k, c = op / 3, ch = op % 3;
      dma_to_lds4_asm(prs, &sm.sWin[u & 3][c][Sh::kWinPad + 64 * ch],
                      (uint32_t)(pb - 64 * ch - lane - c) * 4u);
    }
  };
  auto issue_ts = [&](int u) {
    dma_to_lds4_asm(trs, sm.sT[u & 7], (uint32_t)row0(u) * 8u + 4u * (uint32_t)lane);
  };

  // ---- bias path of a (wave, step) tile (as in bwd_item) ----
  enum { kUniform = 0, kTwo = 1, kGeneral = 2 };
  struct Path {
    int code;
    float cb, cb_far;
    __device__ int kind() const { return code & 3; }
    __device__ int slot() const { return (code >> 2) & 63; }
    __device__ int slot_far() const { return (code >> 8) & 63; }
    __device__ uint32_t thr() const { return 1u << ((code >> 14) & 31); }
  };
  // Full tile: every pair valid, either history rows after all of the
  // wave's keys, or candidate rows against history keys only.
  auto full_tile = [&](int i0) {
    return (i0 + BM - 1 < L) &&
           ((jw0 + 31 <= i0 && i0 + BM - 1 < n_h) || (CF && i0 >= n_h && jw0 + 31 < n_h));
  };
  auto classify = [&](int u) -> Path {
    Path r{kGeneral, 0.0f, 0.0f};
    if (u >= nsteps) {
      r.code = kUniform;
      return r;
    }
    if constexpr (FAST) {
      if (full_tile(row0(u))) {
        const uint32_t rlo = __builtin_amdgcn_readfirstlane(sm.sRr[u & 3][0]);
        const uint32_t rhi = __builtin_amdgcn_readfirstlane(sm.sRr[u & 3][1]);
        const bool ordered = rlo >= khi32;
        uint32_t dmin, dmax;
        if (ordered) {
          dmin = rlo - khi32;
          dmax = rhi - klo32;
        } else if (klo32 >= rhi) {
          dmin = klo32 - rhi;
          dmax = khi32 - rlo;
        } else {
          dmin = 0;
          dmax = max(rhi - klo32, khi32 - rlo);
        }
        const int bnear = 31 - __clz((int)(dmin | 1u)), bfar = 31 - __clz((int)(dmax | 1u));
        if (bnear == bfar) {
          r.code = kUniform | (63 - bnear) << 2;
          r.cb = sm.sTab[63 - bnear];
        } else if (ordered && bfar == bnear + 1) {
          r.code = kTwo | (63 - bnear) << 2 | (63 - bfar) << 8 | bfar << 14;
          r.cb = sm.sTab[63 - bnear];
          r.cb_far = sm.sTab[63 - bfar];
        }
      }
    }
    return r;
  };
  const int a_y = Pk - my_j + 4 * half;
  auto win_reads = [&](int u, float (&w)[16]) {
    const int c = a_y & 3;
    const float* wp = &sm.sWin[u & 3][c][Sh::kWinPad + a_y - c];
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(wp + 8 * g);
#pragma unroll
      for (int m = 0; m < 4; m++) w[4 * g + m] = v[m];
    }
  };
  auto row_ts = [&](int u, uint32_t (&ti)[16]) {
    const uint32_t* tp = sm.sTr[u & 7] + 4 * half;
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(tp + 8 * g);
#pragma unroll
      for (int m = 0; m < 4; m++) ti[4 * g + m] = v[m];
    }
  };
  auto pair_slots = [&](int u, int (&sl)[16]) {
    if constexpr (FAST) {
      uint32_t ti[16];
      row_ts(u, ti);
#pragma unroll
      for (int q = 0; q < 16; q++) {
        uint32_t d, z;
        asm("v_sad_u32 %0, %1, %2, 0" : "=v"(d) : "v"(ti[q]), "v"(tjr));
        asm("v_ffbh_u32 %0, %1" : "=v"(z) : "v"(d));
        sl[q] = 32 + (int)z;
      }
    } else {
      const uint32_t* tp = sm.sT[u & 7] + 2 * (4 * half);
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int r = 8 * (q >> 2) + (q & 3);
        const int64_t ti = (int64_t)(((uint64_t)tp[2 * r + 1] << 32) | tp[2 * r]);
        sl[q] = slot64(ti - tj64);
      }
    }
  };
  // Candidate rows all sit at position n_h: their position term depends
  // on the key alone.
  auto full_win = [&](int u, float (&w)[16]) {
    if (CF && row0(u) >= n_h) {
      const float wc = sm.sWin[u & 3][0][Sh::kWinPad + Pk - pj];
#pragma unroll
      for (int q = 0; q < 16; q++) w[q] = wc;
    } else {
      win_reads(u, w);
    }
  };
  auto seed = [&](int u, const Path& pth, f32x16& acc) {
    if (pth.kind() == kUniform) {
      float w[16];
      full_win(u, w);
#pragma unroll
      for (int q = 0; q < 16; q++) acc[q] = w[q] + pth.cb;
    } else if (pth.kind() == kTwo) {
      float w[16];
      uint32_t ti[16];
      full_win(u, w);
      row_ts(u, ti);
      const uint32_t lim = tjr + pth.thr();
#pragma unroll
      for (int q = 0; q < 16; q++) acc[q] = w[q] + (ti[q] >= lim ? pth.cb_far : pth.cb);
    } else if (kMaskedWindowReads && (!TGT || row0(u) + BM - 1 < n_h)) {
      // Masked or ragged pairs of history rows (position = index): the
      // window reads of full tiles, then the mask.
      const int i0 = row0(u);
      int sl[16];
      pair_slots(u, sl);
      float w[16], tv[16];
      win_reads(u, w);
#pragma unroll
      for (int q = 0; q < 16; q++) tv[q] = sm.sTab[sl[q]];
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int i = i0 + 8 * (q >> 2) + 4 * half + (q & 3);
        acc[q] = key_ok && i < L && pair_valid(i, my_j, n_h) ? w[q] + tv[q] : kMaskedBias;
      }
    } else {
      const int i0 = row0(u), pi0 = min(i0, n_h);
      int sl[16];
      pair_slots(u, sl);
      bool ok[16];
      int y[16];
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int i = i0 + 8 * (q >> 2) + 4 * half + (q & 3);
        ok[q] = key_ok && i < L && pair_valid(i, my_j, n_h);
        y[q] = ok[q] ? (Pk - pj) + (bias_pos(i, n_h) - pi0) : 0;
      }
      float w[16], tv[16];
#pragma unroll
      for (int q = 0; q < 16; q++) {
        w[q] = sm.sWin[u & 3][0][Sh::kWinPad + y[q]];
        tv[q] = sm.sTab[sl[q]];
      }
#pragma unroll
      for (int q = 0; q < 16; q++) acc[q] = ok[q] ? w[q] + tv[q] : kMaskedBias;
    }
  };
  auto scores = [&](int u, f32x16& sacc, f32x16& pacc) {
    const uint8_t* qb = sm.ring.t.q[u % kSlots];
    const uint8_t* ob = sm.ring.t.dO[u % kSlots];
    pacc = f32x16{};
    constexpr int SMAX = DQK > DV ? DQK / 16 : DV / 16;
#pragma unroll
    for (int s = 0; s < SMAX; s++) {
      if (s < DQK / 16) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(qb + a_off(QT{}, qa, s));
        sacc = mfma32x32x16(as_bf16x8(a), as_bf16x8(kf[s]), sacc);
      }
      if (s < DV / 16) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(ob + a_off(OT{}, oa, s));
        pacc = mfma32x32x16(as_bf16x8(a), as_bf16x8(vf[s]), pacc);
        if constexpr (SPLIT) {
          const u32x4 al =
              *reinterpret_cast<const u32x4*>(sm.ring.t.dOl[u % kSlots] + a_off(OT{}, oa, s));
          pacc = mfma32x32x16(as_bf16x8(al), as_bf16x8(vf[s]), pacc);
        }
      }
    }
  };
  // Hand-over to role B: dS^T in the dQ layout (role B reads its dK
  // operand from it too) and P as this lane's operand registers; with
  // SPLIT also their low terms (pl, dl), laid out the same way.
  auto store_step = [&](int u, const u32x4 (&pa)[2], const u32x4 (&da)[2], const u32x4 (&pl)[2],
                        const u32x4 (&dl)[2]) {
    uint16_t* dp = sm.sdST[u & 1] + (32 * wave + col) * DST_LD + 4 * half;
#pragma unroll
    for (int st = 0; st < 2; st++) {
      *reinterpret_cast<uint2*>(dp + 16 * st) = uint2{da[st][0], da[st][1]};
      *reinterpret_cast<uint2*>(dp + 16 * st + 8) = uint2{da[st][2], da[st][3]};
      sm.sPA[u & 1][wave][st][lane] = pa[st];
    }
    if constexpr (SPLIT) {
      uint16_t* dpl = sm.sdSTl[u & 1] + (32 * wave + col) * DST_LD + 4 * half;
#pragma unroll
      for (int st = 0; st < 2; st++) {
        *reinterpret_cast<uint2*>(dpl + 16 * st) = uint2{dl[st][0], dl[st][1]};
        *reinterpret_cast<uint2*>(dpl + 16 * st + 8) = uint2{dl[st][2], dl[st][3]};
        sm.sPAl[u & 1][wave][st][lane] = pl[st];
      }
    }
  };

  // ---- bias gradients (as in bwd_item) ----
  int run_slot[2] = {-1, -1};
  float run_acc[2] = {0.0f, 0.0f};
  auto time_flush = [&](int r) {
    if (run_slot[r] >= 0) {
      const float v = wave_sum_dpp(run_acc[r]);
      if (lane == 0) atomicAdd(&sm.sTacc[run_slot[r]], v);
    }
    run_acc[r] = 0.0f;
  };
  auto time_add = [&](int r, int slot, float v) {
    if (slot != run_slot[r]) {
      time_flush(r);
      run_slot[r] = slot;
    }
    run_acc[r] += v;
  };
  constexpr int kRing = Sh::kRing;
  const int perm_base = lane * 4;
  // Lane (col, half) reads register q = 4g + m from lane + r0(q), r0 =
  // 8g + m (mod 64); the value crossed into the other half-wave when
  // r0(q) >= 32 - col (a suffix of q, since r0 grows with q), so the
  // lane's own diagonal gets the prefix sum before that point.
  const int wrap_from = 32 - col;
  float* const ring_mine = sm.sRing[wave][half];
  const int d1_lane = 4 * half - col - 32 * wave;  // D1 = 32 u + d1_lane
  float carry = 0.0f;  // partner's crossing sum of the previous step
  // Candidate rows all sit at position n_h, so every candidate pair of the
  // lane's key j lands on one position entry, (N-1) - (n_h - p(j)): the
  // lane sums them over the item in its own LDS word (a register would
  // stay live through every step) and adds them once at its end.
  float* const cand_sum = &sm.sCand[wave][lane];
  if constexpr (TGT) *cand_sum = 0.0f;
  auto pos_step = [&](int u, const float (&ds)[16]) {
    float sum = 0.0f, nowrap = 0.0f;
#pragma unroll
    for (int q = 0; q < 16; q++) {
      const float rv = __int_as_float(__builtin_amdgcn_ds_bpermute(
          perm_base + 4 * (8 * (q >> 2) + (q & 3)), __float_as_int(ds[q])));
      sum += rv;
      if (8 * (q >> 2) + (q & 3) < wrap_from) nowrap = sum;
    }
    ring_mine[(32 * u + d1_lane) & (kRing - 1)] = nowrap + carry;
    carry = __int_as_float(
        __builtin_amdgcn_ds_bpermute(perm_base ^ 128, __float_as_int(sum - nowrap)));
  };
  const int R = L - j0;
  auto ring_flush = [&](int c) {
    if (lane < 32) {
      const int k = 32 * c + lane, sl = k & (kRing - 1);
      float v = 0.0f;
#pragma unroll
      for (int w = 0; w < 4; w++)
#pragma unroll
        for (int h = 0; h < 2; h++) {
          v += sm.sRing[w][h][sl];
          sm.sRing[w][h][sl] = 0.0f;
        }
      if (v != 0.0f && k < R) unsafeAtomicAdd(&A.d_rab_pos[(N - 1) - k], v * invN);
    }
  };
  auto grads = [&](int u, const Path& pth, const float (&ds)[16]) {
    const int i0 = row0(u);
    if (TGT && i0 + BM - 1 >= n_h && i0 < L) {
      float dh[16], cs = 0.0f;
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int i = i0 + 8 * (q >> 2) + 4 * half + (q & 3);
        dh[q] = i < n_h ? ds[q] : 0.0f;
        if (i >= n_h && i < L && key_ok && pair_valid(i, my_j, n_h)) cs += ds[q];
      }
      *cand_sum += cs;
      if (CF && i0 >= n_h) {
        // no history row: the step's diagonal sums are all zero
        ring_mine[(32 * u + d1_lane) & (kRing - 1)] = carry;
        carry = 0.0f;
      } else {
        pos_step(u, dh);
      }
    } else {
      pos_step(u, ds);
    }
    if (pth.kind() != kGeneral) {
      float tot = 0.0f;
#pragma unroll
      for (int q = 0; q < 16; q++) tot += ds[q];
      if (pth.kind() == kTwo) {
        uint32_t ti[16];
        row_ts(u, ti);
        const uint32_t lim = tjr + pth.thr();
        float far = 0.0f;
#pragma unroll
        for (int q = 0; q < 16; q++) far += ti[q] >= lim ? ds[q] : 0.0f;
        time_add(0, pth.slot(), tot - far);
        time_add(1, pth.slot_far(), far);
      } else {
        time_add(0, pth.slot(), tot);
      }
    } else {
      // Several buckets: a lane's 16 pairs (rows in order, its one key)
      // form runs of equal slot, each added once to the LDS table (masked
      // pairs carry dS = 0 and may sit in any run).
      int sl[16];
      pair_slots(u, sl);
      float run = ds[0];
#pragma unroll
      for (int q = 1; q < 16; q++) {
        if (sl[q] != sl[q - 1]) {
          atomicAdd(&sm.sTacc[sl[q - 1]], run);
          run = 0.0f;
        }
        run += ds[q];
      }
      atomicAdd(&sm.sTacc[sl[15]], run);
    }
  };

  // ---- pipelined steps: S, dP of step u+1 issued while step u goes
  // through SiLU'; one barrier per step (role B runs the same count).
  Path path_cur, path_next, path_nn;
  auto step = [&](int u, f32x16& s_cur, f32x16& p_cur, f32x16& s_next, f32x16& p_next) {
    wait_vmcnt_lgkmcnt0<OPS_PER_STEP>();
    barrier_no_fence();
    if (u >= 5 && wave == (u & 3)) ring_flush(u - 5);
    issue_tiles(u + kAhead);
    issue_win(u + 3);
    issue_ts(u + 5);
    if (u + 1 < nsteps) seed(u + 1, path_next, s_next);
    scores(u + 1, s_next, p_next);
    float pv[16], dsv[16];
#pragma unroll
    for (int q = 0; q < 16; q++) {
      const float x = s_cur[q];
      const float sg = silu_sigma(x);
      const float p = x * sg;
      pv[q] = p;
      dsv[q] = p_cur[q] * __builtin_fmaf(p, 1.0f - sg, sg);
    }
    u32x4 pa[2], da[2], pl[2], dl[2];
#pragma unroll
    for (int st = 0; st < 2; st++) {
      pa[st] = pack_bf16x8(pv + 8 * st);
      da[st] = pack_bf16x8(dsv + 8 * st);
      if constexpr (SPLIT) {
        // low terms: value - bf16(value), exact in fp32
#pragma unroll
        for (int e = 0; e < 4; e++) {
          const uint32_t h = pa[st][e], g = da[st][e];
          pl[st][e] = pack_bf16x2(pv[8 * st + 2 * e] - __uint_as_float(h << 16),
                                  pv[8 * st + 2 * e + 1] - __uint_as_float(h & 0xffff0000u));
          dl[st][e] = pack_bf16x2(dsv[8 * st + 2 * e] - __uint_as_float(g << 16),
                                  dsv[8 * st + 2 * e + 1] - __uint_as_float(g & 0xffff0000u));
        }
      }
    }
    store_step(u, pa, da, pl, dl);
    grads(u, path_cur, dsv);
    path_nn = classify(u + 2);
    path_cur = path_next;
    path_next = path_nn;
  };

  // Prologue: timestamps of steps 0..4, tiles and windows 0..2 (role B
  // reduces the row timestamps of steps 0..2 between the two barriers).
  for (int v = 0; v < 5; v++) issue_ts(v);
  for (int v = 0; v < 3; v++) {
    if (v < kAhead) issue_tiles(v);
    issue_win(v);
  }
  wait_vmcnt_lgkmcnt0<0>();
  barrier_no_fence();  // (P1)
  barrier_no_fence();  // (P2)
  f32x16 sA, pA, sB, pB;
  path_cur = classify(0);
  path_next = classify(1);
  seed(0, path_cur, sA);
  scores(0, sA, pA);
  int u = 0;
  for (; u + 1 < nsteps; u += 2) {
    step(u, sA, pA, sB, pB);
    step(u + 1, sB, pB, sA, pA);
  }
  if (u < nsteps) step(u, sA, pA, sB, pB);
  // Role B's last step.
  wait_vmcnt_lgkmcnt0<0>();
  barrier_no_fence();  // (L)
  time_flush(0);
  time_flush(1);
  if constexpr (TGT) {
    if (const float cv = *cand_sum; cv != 0.0f)
      unsafeAtomicAdd(&A.d_rab_pos[(N - 1) - (n_h - pj)], cv * invN);
  }
  ring_mine[(32 * nsteps + d1_lane) & (kRing - 1)] = carry;
  wait_vmcnt_lgkmcnt0<0>();
  barrier_no_fence();  // (E)
  {
    const int c0 = max(0, nsteps - 5);
    for (int c = c0 + wave; c <= nsteps; c += 4) ring_flush(c);
  }
}

template <int DQK, int DV, bool SPLIT>
__device__ __forceinline__ void bwd_role_b(BwdSharedRS<DQK, DV, SPLIT>& sm, const BwdArgs& A,
                                           const RsItem& it, const u32x4* kq, bool fast,
                                           int64_t tbase) {
  using Sh = BwdSharedRS<DQK, DV, SPLIT>;
  using QT = typename Sh::QT;
  using OT = typename Sh::OT;
  constexpr int BN = Sh::BN, BM = Sh::BM, DST_LD = Sh::DST_LD, kSlots = Sh::kSlots;
  const JaggedArgs& ja = A.ja;
  const int H = ja.num_heads, N = ja.max_seq_len;
  const int64_t o = it.o;
  const int L = it.L, j0 = it.j0, head = it.head, nsteps = it.nsteps;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane((tid >> 6) - 4);  // 0..3
  const int col = lane & 31, half = lane >> 5;
  const int jw0 = j0 + 32 * wave;
  const float invN = 1.0f / (float)N;
  // dQ: column block `wave` (waves past DQK / 32 have none) over all 128 keys.
  constexpr int NCB = DQK / 32, KSTEPS = BN / 16;
  const int tr_row = 4 * half + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  f32x16 dkacc[DQK / 32], dvacc[DV / 32];
#pragma unroll
  for (int nb = 0; nb < DQK / 32; nb++)
#pragma unroll
    for (int q = 0; q < 16; q++) dkacc[nb][q] = 0.0f;
#pragma unroll
  for (int nb = 0; nb < DV / 32; nb++)
#pragma unroll
    for (int q = 0; q < 16; q++) dvacc[nb][q] = 0.0f;

  // Transposing reads of the Q / dO tiles (as in bwd_item).
  auto tr_base = [&](auto tile_tag, uint32_t (&tb)[2]) {
    using T = decltype(tile_tag);
    const int sw = T::swz(tr_row);
    const int c1 = tr_col >> 3, off = (tr_col & 7) * 2;
    const int b = tr_row * T::RB + 16 * (c1 ^ (sw & 3)) + off;
    tb[0] = (uint32_t)(b + 64 * (sw >> 2));
    tb[1] = (uint32_t)(b - 64 * (sw >> 2));
  };
  auto tr_off = [&](auto tile_tag, const uint32_t (&tb)[2], int st, int hi, int nb) -> uint32_t {
    using T = decltype(tile_tag);
    const int rows = T::row_base(16 * st + 8 * hi);  // tr_row < 8: same row group
    if constexpr (T::SWZ)
      return tb[nb & 1] + (uint32_t)(rows + 64 * nb);
    else
      return (uint32_t)(tr_row * T::RB + rows + 64 * nb + tr_col * 2);
  };
  uint32_t qt[2], ot[2];
  tr_base(QT{}, qt);
  tr_base(OT{}, ot);

  // dV += P^T dO, dK += dS^T Q of step u: P as role A's operand registers,
  // dS read back from the dS^T tile in the same (accumulator-row) order.
  // SPLIT: dV += P_hi^T dO_hi + P_lo^T dO_hi + P_hi^T dO_lo and
  // dK += dS_hi^T Q + dS_lo^T Q.
  auto key_grads = [&](int u) {
    const uint8_t* qb = sm.ring.t.q[u % kSlots];
    const uint8_t* ob = sm.ring.t.dO[u % kSlots];
    const uint16_t* dp = sm.sdST[u & 1] + (32 * wave + col) * DST_LD + 4 * half;
    u32x4 pa[2], da[2], pl[2], dl[2];
#pragma unroll
    for (int st = 0; st < 2; st++) {
      pa[st] = sm.sPA[u & 1][wave][st][lane];
      const uint2 lo = *reinterpret_cast<const uint2*>(dp + 16 * st);
      const uint2 hi = *reinterpret_cast<const uint2*>(dp + 16 * st + 8);
      da[st] = u32x4{lo.x, lo.y, hi.x, hi.y};
      if constexpr (SPLIT) {
        const uint16_t* dpl = sm.sdSTl[u & 1] + (32 * wave + col) * DST_LD + 4 * half;
        pl[st] = sm.sPAl[u & 1][wave][st][lane];
        const uint2 l2 = *reinterpret_cast<const uint2*>(dpl + 16 * st);
        const uint2 h2 = *reinterpret_cast<const uint2*>(dpl + 16 * st + 8);
        dl[st] = u32x4{l2.x, l2.y, h2.x, h2.y};
      }
    }
#pragma unroll
    for (int st = 0; st < 2; st++) {
#pragma unroll
      for (int nb = 0; nb < DV / 32; nb++) {
        const uint2 lo = lds_read_tr16((const uint16_t*)(ob + tr_off(OT{}, ot, st, 0, nb)));
        const uint2 hi = lds_read_tr16((const uint16_t*)(ob + tr_off(OT{}, ot, st, 1, nb)));
        dvacc[nb] = mfma32x32x16(as_bf16x8(pa[st]),
                                 as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y}), dvacc[nb]);
        if constexpr (SPLIT) {
          dvacc[nb] = mfma32x32x16(as_bf16x8(pl[st]),
                                 as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y}), dvacc[nb]);
          const uint8_t* obl = sm.ring.t.dOl[u % kSlots];
          const uint2 l2 = lds_read_tr16((const uint16_t*)(obl + tr_off(OT{}, ot, st, 0, nb)));
          const uint2 h2 = lds_read_tr16((const uint16_t*)(obl + tr_off(OT{}, ot, st, 1, nb)));
          dvacc[nb] = mfma32x32x16(as_bf16x8(pa[st]),
                                 as_bf16x8(u32x4{l2.x, l2.y, h2.x, h2.y}), dvacc[nb]);
        }
      }
#pragma unroll
      for (int nb = 0; nb < DQK / 32; nb++) {
        const uint2 lo = lds_read_tr16((const uint16_t*)(qb + tr_off(QT{}, qt, st, 0, nb)));
        const uint2 hi = lds_read_tr16((const uint16_t*)(qb + tr_off(QT{}, qt, st, 1, nb)));
        dkacc[nb] = mfma32x32x16(as_bf16x8(da[st]),
                                 as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y}), dkacc[nb]);
        if constexpr (SPLIT)
          dkacc[nb] = mfma32x32x16(as_bf16x8(dl[st]),
                                 as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y}), dkacc[nb]);
      }
    }
  };
  // Partial slot of step u: slot0 + u, slot0 = pbase[seq] + kb S - 2 kb (kb - 1)
  // (the steps of the sequence's earlier key blocks); a slot holds h x NCB
  // blocks of 1024 f16, [head][column block], each block two halves of
  // [lane][8 accumulator registers] (registers 0-7, then 8-15), so that
  // every 16-byte store of a wave covers 1 KB; dq_scale one float per block.
  const int S_b = (L + BM - 1) / BM, kb = j0 / BN;
  const int64_t slot0 = A.pbase[it.seq] + (int64_t)kb * S_b - 2 * (int64_t)kb * (kb - 1);
  const int64_t blk0 = (slot0 * H + head) * NCB + wave;
  uint16_t* const part_lane = A.dq_part + blk0 * 1024 + (int64_t)lane * 8;
  const int64_t blk_stride = (int64_t)H * NCB;
  auto dq_step = [&](int u) {
    const uint16_t* dp = sm.sdST[u & 1] + tr_row * DST_LD + tr_col;
    f32x16 qacc = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ks++) {
      const uint2 lo = lds_read_tr16(dp + 16 * ks * DST_LD);
      const uint2 hi = lds_read_tr16(dp + (16 * ks + 8) * DST_LD);
      qacc = mfma32x32x16(as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y}), as_bf16x8(kq[ks]), qacc);
    }
    if constexpr (SPLIT) {
      const uint16_t* dpl = sm.sdSTl[u & 1] + tr_row * DST_LD + tr_col;
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ks++) {
        const uint2 lo = lds_read_tr16(dpl + 16 * ks * DST_LD);
        const uint2 hi = lds_read_tr16(dpl + (16 * ks + 8) * DST_LD);
        qacc = mfma32x32x16(as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y}), as_bf16x8(kq[ks]), qacc);
      }
    }
    // Block scale 2^(140 - e), e the biased exponent of the largest
    // magnitude (clamped so that it and its inverse are normal floats).
    float mx = 0.0f;
#pragma unroll
    for (int q = 0; q < 16; q++) mx = fmaxf(mx, fabsf(qacc[q]));
    const int e = (int)((wave_max_dpp(__float_as_uint(mx)) >> 23) & 0xffu);
    const uint32_t se = (uint32_t)min(max(267 - e, 1), 253);
    const float sc = __uint_as_float(se << 23);
    uint32_t h[8];
#pragma unroll
    for (int k = 0; k < 8; k++) h[k] = pack_f16x2(qacc[2 * k] * sc, qacc[2 * k + 1] * sc);
    if (slot0 + u >= A.dq_slots) return;
    uint16_t* dst = part_lane + (int64_t)u * blk_stride * 1024;
    __builtin_nontemporal_store(u32x4{h[0], h[1], h[2], h[3]}, reinterpret_cast<u32x4*>(dst));
    __builtin_nontemporal_store(u32x4{h[4], h[5], h[6], h[7]}, reinterpret_cast<u32x4*>(dst + 512));
    if (lane == 0) A.dq_scale[blk0 + (int64_t)u * blk_stride] = __uint_as_float((254u - se) << 23);
  };

  // Fast path: the row timestamps of step u rebased to 32 bits, and their
  // min / max, for role A's tile classification (one wave).  Role A's
  // staging wait at step u covers the timestamps of step u + 3.
  auto reduce_ts = [&](int u) {
    if (fast && wave == 0) {
      const uint32_t v = sm.sT[u & 7][2 * (lane & 31)] - (uint32_t)tbase;
      const uint32_t lo = wave_min_dpp(v), hi = wave_max_dpp(v);
      sm.sTr[u & 7][lane & 31] = v;
      if (lane < 2) sm.sRr[u & 3][lane] = lane ? hi : lo;
    }
  };
  // The same barriers as role A: two in its prologue, one per step, then
  // one for the last hand-over and one before its final flushes.
  barrier_no_fence();  // (P1)
  for (int v = 0; v < 3; v++) reduce_ts(v);
  wait_vmcnt_lgkmcnt0<63>();
  barrier_no_fence();  // (P2)
  for (int u = 0; u < nsteps; u++) {
    wait_vmcnt_lgkmcnt0<63>();
    barrier_no_fence();
    reduce_ts(u + 3);
    if (u >= 1) {
      key_grads(u - 1);
      if (wave < NCB) dq_step(u - 1);
    }
  }
  wait_vmcnt_lgkmcnt0<63>();
  barrier_no_fence();  // (L)
  key_grads(nsteps - 1);
  if (wave < NCB) dq_step(nsteps - 1);
  wait_vmcnt_lgkmcnt0<63>();
  barrier_no_fence();  // (E)

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
}

constexpr int kRsThreads = 512;

// One work item (a 128-key block of one sequence and head) of the
// two-role backward.  FAST: the sequence's timestamps span less than 2^31
// and are rebased to 32 bits; the 64-bit path is a kernel of its own, so
// that the code the common case runs does not carry it.
template <int DQK, int DV, bool SPLIT, bool TGT, bool FAST>
__device__ __forceinline__ void rs_item(BwdSharedRS<DQK, DV, SPLIT>& sm, const BwdArgs& A,
                                        const WorkItem wi, const int head) {
  using S = BwdSharedRS<DQK, DV, SPLIT>;
  constexpr int BN = S::BN, KB_LD = S::KB_LD;
  const JaggedArgs& ja = A.ja;
  const int N = ja.max_seq_len, NB = ja.num_buckets;
  RsItem it;
  it.o = ja.seq_offsets[wi.seq];
  it.seq = wi.seq;
  it.L = (int)(ja.seq_offsets[wi.seq + 1] - it.o);
  it.n_h = it.L - (ja.num_targets ? (int)ja.num_targets[wi.seq] : 0);
  it.j0 = wi.blk * BN;
  it.head = head;
  // Candidate keys see only themselves; otherwise every later row sees them.
  const int i_end = it.j0 >= it.n_h ? min(it.j0 + BN, it.L) : it.L;
  it.nsteps = (i_end - it.j0 + S::BM - 1) / S::BM;
  const int tid = threadIdx.x;
  const int64_t tlo = ja.seq_trange[2 * wi.seq];
  constexpr bool fast = FAST;
  for (int x = tid; x < 64; x += kRsThreads) {
    sm.sTab[x] = (fast && x == 31) ? ja.rab_time[0] : ja.rab_time[min(63 - x, NB - 1)];
    sm.sTacc[x] = 0.0f;
  }
  for (int x = tid; x < 4 * 2 * S::kRing; x += kRsThreads) (&sm.sRing[0][0][0])[x] = 0.0f;

  // The block's K, row-major in LDS, then role B's dQ operand down its rows.
  const int lane = tid & 63, wave = tid >> 6;
  constexpr int NCB = DQK / 32, KSTEPS = BN / 16;
  u32x4 kq[KSTEPS];
  {
    const uint16_t* kg = (const uint16_t*)A.t.k + it.o * A.t.k_stride + head * DQK;
    const __amdgpu_buffer_rsrc_t krs = make_rsrc(kg, (uint32_t)(it.L * A.t.k_stride * 2));
    const uint32_t kstride_b = (uint32_t)A.t.k_stride * 2u;
    constexpr int KCH = BN * DQK / 8;
    for (int c = tid; c < KCH; c += kRsThreads) {
      const int r = c / (DQK / 8), cc = c % (DQK / 8);
      *reinterpret_cast<u32x4*>(sm.ring.kblk + r * KB_LD + 8 * cc) =
          buffer_load16(krs, (uint32_t)(it.j0 + r) * kstride_b + (uint32_t)cc * 16u);
    }
    __syncthreads();
    if (wave >= 4 && wave < 4 + NCB) {
      const int cbw = wave - 4, half = lane >> 5;
      const int tr_row = 4 * half + ((lane & 15) >> 2);
      const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
      const uint16_t* kp = sm.ring.kblk + tr_row * KB_LD + 32 * cbw + tr_col;
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ks++) {
        const uint2 lo = lds_read_tr16(kp + 16 * ks * KB_LD);
        const uint2 hi = lds_read_tr16(kp + (16 * ks + 8) * KB_LD);
        kq[ks] = u32x4{lo.x, lo.y, hi.x, hi.y};
      }
    }
    __syncthreads();  // the ring may be overwritten from here on
  }

  if (wave < 4)
    bwd_role_a<DQK, DV, FAST, SPLIT, TGT>(sm, A, it, tlo);
  else
    bwd_role_b<DQK, DV, SPLIT>(sm, A, it, kq, FAST, tlo);

  __syncthreads();
  const float invN = 1.0f / (float)N;
  if (tid < 64) {
    const float v = sm.sTacc[tid];
    const int b = (fast && tid == 31) ? 0 : min(63 - tid, NB - 1);
    if (v != 0.0f) unsafeAtomicAdd(&A.d_rab_time[b], v * invN);
  }
}

__device__ __forceinline__ bool seq_fast(const JaggedArgs& ja, int seq) {
  return ja.seq_trange[2 * seq + 1] - ja.seq_trange[2 * seq] < ((int64_t)1 << 31);
}

// The items of sequences on the 32-bit timestamp path, one per workgroup
// (the others return at once).
template <int DQK, int DV, bool SPLIT, bool TGT>
__global__ __launch_bounds__(kRsThreads, 1) void attn_bwd_rs_kernel(
    BwdArgs A, const WorkItem* __restrict__ items, const int32_t* __restrict__ count) {
  __shared__ BwdSharedRS<DQK, DV, SPLIT> sm;
  const int H = A.ja.num_heads;
  const int item = (int)(blockIdx.x / (unsigned)H);
  const int head = (int)blockIdx.x - item * H;
  if (item >= *count) return;
  const WorkItem wi = items[item];
  if (!seq_fast(A.ja, wi.seq)) return;
  rs_item<DQK, DV, SPLIT, TGT, true>(sm, A, wi, head);
}

// The items of sequences whose timestamps span 2^31 or more, in a
// grid-stride loop over the work list; when there is no such sequence
// (the check reads every sequence's range once) the launch ends at once.
template <int DQK, int DV, bool SPLIT, bool TGT>
__global__ __launch_bounds__(kRsThreads, 1) void attn_bwd_rs_wide_kernel(
    BwdArgs A, const WorkItem* __restrict__ items, const int32_t* __restrict__ count) {
  __shared__ BwdSharedRS<DQK, DV, SPLIT> sm;
  const JaggedArgs& ja = A.ja;
  int wide = 0;
  for (int b = (int)threadIdx.x; b < ja.num_seqs; b += kRsThreads) wide |= !seq_fast(ja, b);
  if (!__syncthreads_or(wide)) return;
  const int H = ja.num_heads;
  const int total = *count * H;
  for (int w = (int)blockIdx.x; w < total; w += (int)gridDim.x) {
    const WorkItem wi = items[w / H];
    if (seq_fast(ja, wi.seq)) continue;
    __syncthreads();  // the previous item's last LDS reads are done
    rs_item<DQK, DV, SPLIT, TGT, false>(sm, A, wi, w - (w / H) * H);
  }
}

// dQ of the two-role kernel.  Workgroup = (row block of 32 rows of one
// sequence, head); wave = column block of 32.  It sums, in key-block
// order, the partial blocks (f16 times their block scale) of every key
// block that visits the row block
// (all history blocks up to it; a candidate block only its own rows),
// scales by 1/N and stores bf16 [T][h][d_qk].  Lane l holds column
// 32 cb + l % 32 and rows 8g + 4 (l / 32) + m, the MFMA accumulator layout
// the partials were stored in.
template <int NCB>
__global__ __launch_bounds__(64 * NCB) void dq_reduce_kernel(JaggedArgs ja,
                                                             const uint16_t* __restrict__ part,
                                                             const float* __restrict__ scale,
                                                             const int64_t* __restrict__ rbase,
                                                             const int64_t* __restrict__ pbase,
                                                             int64_t dq_slots,
                                                             uint16_t* __restrict__ dq) {
  constexpr int DQK = 32 * NCB;
  const int H = ja.num_heads, B = ja.num_seqs;
  const int64_t nrb = rbase[B];
  const int64_t gi = (int64_t)(blockIdx.x / (unsigned)H);
  const int head = (int)(blockIdx.x % (unsigned)H);
  if (gi >= nrb) return;
  // Last row blocks first: within a sequence the later rows have the most
  // key blocks to sum.
  const int64_t g = nrb - 1 - gi;
  // The sequence whose row blocks hold g: the last b with rbase[b] <= g
  // (empty sequences have no row blocks).
  int lo = 0, hi = B;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (rbase[mid] <= g) lo = mid; else hi = mid;
  }
  const int b = lo;
  const int64_t o = ja.seq_offsets[b];
  const int L = (int)(ja.seq_offsets[b + 1] - o);
  const int n_h = L - (ja.num_targets ? (int)ja.num_targets[b] : 0);
  const int i0 = (int)(g - rbase[b]) * kBwdBM;
  const int S_b = (L + kBwdBM - 1) / kBwdBM;
  const int lane = threadIdx.x & 63, cb = threadIdx.x >> 6;
  const int col = lane & 31, half = lane >> 5;
  float acc[16];
#pragma unroll
  for (int q = 0; q < 16; q++) acc[q] = 0.0f;
  const int kb_max = i0 / kBwdBN;  // every key block starts at or before i0
  const int64_t pb = pbase[b];
  // Sixteen key blocks per round (32 loads in flight per lane; four and
  // eight ran 7 % and 2 % slower): their loads are all issued before the
  // round's sums (kept in key-block order).  The partial blocks are read
  // once, so the loads are non-temporal (as are the backward's stores).
  constexpr int KR = 16;
  for (int kb0 = 0; kb0 <= kb_max; kb0 += KR) {
    u32x4 w0[KR], w1[KR];
    float inv[KR];
    bool ok[KR];
#pragma unroll
    for (int t = 0; t < KR; t++) {
      const int kb = kb0 + t, j0 = kb * kBwdBN;
      const int i_end = j0 >= n_h ? min(j0 + kBwdBN, L) : L;
      const int64_t slot =
          pb + (int64_t)kb * S_b - 2 * (int64_t)kb * (kb - 1) + (i0 - j0) / kBwdBM;
      ok[t] = kb <= kb_max && i0 < i_end && slot < dq_slots;
      if (ok[t]) {
        const int64_t blk = (slot * H + head) * NCB + cb;
        const uint16_t* src = part + blk * 1024 + (int64_t)lane * 8;
        w0[t] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src));
        w1[t] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + 512));
        inv[t] = scale[blk];
      }
    }
#pragma unroll
    for (int t = 0; t < KR; t++) {
      if (!ok[t]) continue;
      const uint32_t w[8] = {w0[t][0], w0[t][1], w0[t][2], w0[t][3],
                             w1[t][0], w1[t][1], w1[t][2], w1[t][3]};
#pragma unroll
      for (int k = 0; k < 8; k++) {
        const float flo = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[k] & 0xffffu));
        const float fhi = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[k] >> 16));
        acc[2 * k] = __builtin_fmaf(flo, inv[t], acc[2 * k]);
        acc[2 * k + 1] = __builtin_fmaf(fhi, inv[t], acc[2 * k + 1]);
      }
    }
  }
  const float invN = 1.0f / (float)ja.max_seq_len;
#pragma unroll
  for (int q = 0; q < 16; q++) {
    const int i = i0 + 8 * (q >> 2) + 4 * half + (q & 3);
    if (i < L) dq[((o + i) * H + head) * DQK + 32 * cb + col] = f32_to_bf16_bits(acc[q] * invN);
  }
}

template <int DQK, int DV, bool SPLIT>
__global__ __launch_bounds__(kBwdThreads, 1) void attn_bwd_bf16_kernel(
    BwdArgs A, const WorkItem* __restrict__ items, const int32_t* __restrict__ count) {
  using S = BwdShared<DQK, DV, SPLIT>;
  constexpr int BN = S::BN;
  __shared__ S sm;

  // Workgroup id = item * H + head: the dispatcher walks the (longest
  // first) work list with all heads of an item together, so the long items
  // of every head start early.
  const JaggedArgs& ja = A.ja;
  const int item = (int)(blockIdx.x / (unsigned)ja.num_heads);
  const int head = (int)blockIdx.x - item * ja.num_heads;
  if (item >= *count) return;
  const WorkItem it = items[item];
  const int N = ja.max_seq_len, NB = ja.num_buckets;
  const int64_t o = ja.seq_offsets[it.seq];
  const int L = (int)(ja.seq_offsets[it.seq + 1] - o);
  const int n_h = L - (ja.num_targets ? (int)ja.num_targets[it.seq] : 0);
  const int j0 = it.blk * BN;
  const int tid = threadIdx.x;

  // The 32-bit fast path applies when the sequence's timestamps span less
  // than 2^31; they are then rebased to its smallest one.
  const int64_t tlo = ja.seq_trange[2 * it.seq], thi = ja.seq_trange[2 * it.seq + 1];
  const bool fast = thi - tlo < ((int64_t)1 << 31);
  // Slots 0..32 are unreachable when every |dt| < 2^31; there slot 31
  // stands for dt = 0 (bucket 0).
  for (int x = tid; x < 64; x += kBwdThreads) {
    sm.sTab[x] = (fast && x == 31) ? ja.rab_time[0] : ja.rab_time[min(63 - x, NB - 1)];
    sm.sTacc[x] = 0.0f;
  }
  for (int x = tid; x < kBwdWaves * 2 * S::kRing; x += kBwdThreads) (&sm.sRing[0][0][0])[x] = 0.0f;
  __syncthreads();
  if (fast) {
    bwd_item<DQK, DV, true, SPLIT>(sm, A, o, L, n_h, j0, head, tlo);
  } else {
    bwd_item<DQK, DV, false, SPLIT>(sm, A, o, L, n_h, j0, head, tlo);
  }

  __syncthreads();
  const float invN = 1.0f / (float)N;
  if (tid < 64) {
    const float v = sm.sTacc[tid];
    const int b = (fast && tid == 31) ? 0 : min(63 - tid, NB - 1);
    if (v != 0.0f) unsafeAtomicAdd(&A.d_rab_time[b], v * invN);
  }
}

template <int DQK, int DV>
hipError_t launch_bwd(const JaggedArgs& ja, const Tensors& t, const void* d_out,
                      const void* d_out_lo, float* dq_acc, uint16_t* dq_part, float* dq_scale,
                      int64_t dq_slots, const int64_t* bases, void* dk, void* dv, float* d_rab_pos,
                      float* d_rab_time, const WorkItem* items, const int32_t* count,
                      int64_t max_items, hipStream_t s) {
  BwdArgs A;
  A.ja = ja;
  A.t = t;
  A.dO = (const uint16_t*)d_out;
  A.dO_lo = (const uint16_t*)d_out_lo;
  A.dq_acc = dq_acc;
  A.dq_part = dq_part;
  A.dq_scale = dq_scale;
  A.dq_slots = dq_slots;
  A.pbase = bases ? bases + (ja.num_seqs + 1) : nullptr;
  A.dK = (uint16_t*)dk;
  A.dV = (uint16_t*)dv;
  A.d_rab_pos = d_rab_pos;
  A.d_rab_time = d_rab_time;
  static_assert(sizeof(BwdShared<DQK, DV, true>) <= kLdsBytes, "LDS budget");
  static_assert(sizeof(BwdSharedRS<DQK, DV>) <= kLdsBytes, "LDS budget");
  dim3 grid((unsigned)(max_items * ja.num_heads));
  // The two-role kernel runs as two launches: the items on the 32-bit
  // timestamp path, then those of sequences spanning 2^31 or more, by at
  // most one workgroup per CU, each of which first reads every sequence's
  // range (fewer workgroups for many sequences, so that this check stays
  // within ~256 K ranges read in all) and ends when none is that wide.
  int64_t nwide = std::min<int64_t>(max_items * ja.num_heads, 256);
  nwide = std::max<int64_t>(1, std::min<int64_t>(nwide, 262144 / std::max(1, ja.num_seqs)));
  const dim3 wide_grid((unsigned)nwide);
  if (d_out_lo) {
    if constexpr (bwd_split_two_role(DQK, DV)) {
      static_assert(sizeof(BwdSharedRS<DQK, DV, true>) <= kLdsBytes, "LDS budget");
      // (One instance for the two-term form: without its candidate paths
      // it timed slower.)
      hipLaunchKernelGGL((attn_bwd_rs_kernel<DQK, DV, true, true>), grid, dim3(kRsThreads), 0,
                         s, A, items, count);
      hipLaunchKernelGGL((attn_bwd_rs_wide_kernel<DQK, DV, true, true>), wide_grid,
                         dim3(kRsThreads), 0, s, A, items, count);
    } else {
      hipLaunchKernelGGL((attn_bwd_bf16_kernel<DQK, DV, true>), grid, dim3(kBwdThreads), 0, s, A,
                         items, count);
    }
  } else {
    if (ja.num_targets) {
      hipLaunchKernelGGL((attn_bwd_rs_kernel<DQK, DV, false, true>), grid, dim3(kRsThreads), 0, s,
                         A, items, count);
      hipLaunchKernelGGL((attn_bwd_rs_wide_kernel<DQK, DV, false, true>), wide_grid,
                         dim3(kRsThreads), 0, s, A, items, count);
    } else {
      hipLaunchKernelGGL((attn_bwd_rs_kernel<DQK, DV, false, false>), grid, dim3(kRsThreads), 0, s,
                         A, items, count);
      hipLaunchKernelGGL((attn_bwd_rs_wide_kernel<DQK, DV, false, false>), wide_grid,
                         dim3(kRsThreads), 0, s, A, items, count);
    }
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bwd_bf16(const JaggedArgs& ja, const Tensors& t, int dqk, int dv,
                                const void* d_out, const void* d_out_lo, float* dq_acc,
                                uint16_t* dq_part, float* dq_scale, int64_t dq_slots,
                                const int64_t* bases, void* dk, void* dv_out, float* d_rab_pos,
                                float* d_rab_time,
                                const WorkItem* items, const int32_t* count, int64_t max_items,
                                hipStream_t s) {
#define HSTU_BWD_CASE(A, B)                                                                  \
  if (dqk == A && dv == B)                                                                   \
    return launch_bwd<A, B>(ja, t, d_out, d_out_lo, dq_acc, dq_part, dq_scale, dq_slots, bases,\
                            dk, dv_out, d_rab_pos, d_rab_time, items, count, max_items, s);
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

hipError_t launch_dq_reduce_bf16(const JaggedArgs& ja, int dqk, const uint16_t* dq_part,
                                 const float* dq_scale, int64_t dq_slots, const int64_t* bases,
                                 void* dq, hipStream_t s) {
  // Row blocks: at most ceil(T / 32) + B; workgroups past the true count return.
  const int64_t nrb = (ja.total_tokens + kBwdBM - 1) / kBwdBM + ja.num_seqs;
  const dim3 grid((unsigned)(nrb * ja.num_heads));
  const int64_t* rbase = bases;
  const int64_t* pbase = bases + ja.num_seqs + 1;
  if (dqk == 32)
    hipLaunchKernelGGL((dq_reduce_kernel<1>), grid, dim3(64), 0, s, ja, dq_part, dq_scale, rbase,
                       pbase, dq_slots, (uint16_t*)dq);
  else if (dqk == 64)
    hipLaunchKernelGGL((dq_reduce_kernel<2>), grid, dim3(128), 0, s, ja, dq_part, dq_scale, rbase,
                       pbase, dq_slots, (uint16_t*)dq);
  else if (dqk == 128)
    hipLaunchKernelGGL((dq_reduce_kernel<4>), grid, dim3(256), 0, s, ja, dq_part, dq_scale, rbase,
                       pbase, dq_slots, (uint16_t*)dq);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace hstu
