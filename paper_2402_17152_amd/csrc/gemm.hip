// Dense products of the layer's two linear maps: f_1 of Eq. 1 (with the
// SiLU of phi_1 and the bias in the epilogue, output split U|V|Q|K by
// columns) and f_2 of Eq. 3 (bias and the residual connection in the
// epilogue), with their input and weight gradients.
//
// All are C[m][n] = sum_k A(m, k) B(n, k) over bf16 operands with fp32
// accumulation on v_mfma_f32_32x32x16_bf16.  An operand is stored either
// k-contiguous (A[m][k], B[n][k]: activations and [out][in] weights in the
// forward) or k-major (A[k][m], B[k][n]: the transposed operands of the
// gradients).  A workgroup of 4 waves computes a 256 x 128 tile, each wave
// 128 x 64 (8 accumulator tiles), over k-steps of 32 staged in LDS (double
// buffered, one barrier per step; global loads run two steps ahead through
// two register sets); two workgroups share a CU, so one's epilogue and
// staging overlap the other's matrix-core work.  A k-contiguous tile gives a
// lane its 8 contraction elements in one 16-byte LDS read; a k-major tile
// is read with two transposing reads (ds_read_b64_tr_b16) that return the
// same 8 elements in the same order.  The products are computed
// transposed (B's fragment as the matrix core's first operand), so a lane
// owns one output row and 4 consecutive columns per register group.
// Weight gradients split the contraction over the tokens; each split
// writes an fp32 slab and an ordered reduction sums the slabs, so results
// do not depend on scheduling.
#include "bias.h"
#include "kernels.h"

namespace hstu {

namespace {

constexpr int kGBM = 256, kGBN = 128, kGBK = 32;
constexpr int kLdK = kGBK + 8;  // k-contiguous tile: row stride in elements (80 B)
// k-major tile of R rows of m / n: row stride R + 8 elements.
template <int R>
struct TileDims {
  static constexpr int kElemsK = R * kLdK;           // k-contiguous
  static constexpr int kElemsN = kGBK * (R + 8);     // k-major
  static constexpr int kElems = kElemsK > kElemsN ? kElemsK : kElemsN;
};

struct GemmShared {
  uint16_t a[2][TileDims<kGBM>::kElems];
  uint16_t b[2][TileDims<kGBN>::kElems];
};

__device__ __forceinline__ float silu_f(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x * -kLog2e));
}

// Staging of one operand tile (R rows of the m or n dimension x 32 of k)
// through registers: R * 4 chunks of 16 bytes, R / 64 per thread.
template <bool KMAJOR, int R>
struct Stager {
  static constexpr int kPer = R / 64;
  static constexpr int kLdN = R + 8;
  __amdgpu_buffer_rsrc_t rs;
  uint32_t ld_b;  // row stride in bytes
  __device__ __forceinline__ void load(u32x4 (&r)[kPer], int k0, int tid) const {
#pragma unroll
    for (int e = 0; e < kPer; e++) {
      const int c = tid + 256 * e;
      uint32_t off;
      if constexpr (KMAJOR)  // row k0 + c / (R/8), chunk c % (R/8)
        off = (uint32_t)(k0 + c / (R / 8)) * ld_b + (uint32_t)(c % (R / 8)) * 16u;
      else                   // row c / 4, k chunk c % 4
        off = (uint32_t)(c >> 2) * ld_b + (uint32_t)(k0 + 8 * (c & 3)) * 2u;
      r[e] = buffer_load16(rs, off);
    }
  }
  __device__ __forceinline__ static void store(uint16_t* t, const u32x4 (&r)[kPer], int tid) {
#pragma unroll
    for (int e = 0; e < kPer; e++) {
      const int c = tid + 256 * e;
      uint16_t* p = KMAJOR ? t + (c / (R / 8)) * kLdN + 8 * (c % (R / 8))
                           : t + (c >> 2) * kLdK + 8 * (c & 3);
      *reinterpret_cast<u32x4*>(p) = r[e];
    }
  }
  // MFMA operand of 32 rows (row0 .. row0+31 of the tile) for the 16-wide
  // contraction block s: lane -> row row0 + lane % 32, k = 16 s + 8 h .. +7.
  __device__ __forceinline__ static u32x4 frag(const uint16_t* t, int row0, int s, int lane) {
    const int h = lane >> 5;
    if constexpr (KMAJOR) {
      const uint16_t* p = t + (16 * s + 8 * h + ((lane & 15) >> 2)) * kLdN + row0 +
                          16 * ((lane >> 4) & 1) + 4 * (lane & 3);
      const uint2 lo = lds_read_tr16(p), hi = lds_read_tr16(p + 4 * kLdN);
      const u32x4 v = {lo.x, lo.y, hi.x, hi.y};
      return v;
    } else {
      return *reinterpret_cast<const u32x4*>(t + (row0 + (lane & 31)) * kLdK + 16 * s + 8 * h);
    }
  }
};

template <bool A_KM, bool B_KM, int EPI>
__global__ __launch_bounds__(256, 2) void gemm_bf16_kernel(GemmArgs g) {
  __shared__ GemmShared sm;
  using SA = Stager<A_KM, kGBM>;
  using SB = Stager<B_KM, kGBN>;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;  // wave tile: rows 128 wm .., columns 64 wn ..
  // Tile order: consecutive tiles (same row panel of A, n fastest) go to
  // one XCD (workgroup ids are dealt to the 8 XCDs round robin).
  const int tn = (g.N + kGBN - 1) / kGBN, nt = ((g.M + kGBM - 1) / kGBM) * tn;
  const int id = blockIdx.x, xcd = id & 7, per = nt >> 3, rem = nt & 7;
  const int tile = xcd * per + min(xcd, rem) + (id >> 3);
  const int m0 = (tile / tn) * kGBM, n0 = (tile % tn) * kGBN;
  const int kb = blockIdx.y * g.k_split;
  const int ke = min(g.K, kb + g.k_split);
  const int nk = (ke - kb + kGBK - 1) / kGBK;

  // Buffer ranges: rows past M / N (k-contiguous) and contraction rows at
  // or past ke (k-major) read as zeros; k-major columns past M / N read
  // neighbouring data that only reaches outputs that are not stored.
  SA sa;
  SB sb;
  if constexpr (A_KM) {
    sa.rs = make_rsrc(g.a + m0, (uint32_t)(((int64_t)(ke - 1) * g.lda + (g.M - m0)) * 2));
  } else {
    sa.rs = make_rsrc(g.a + (int64_t)m0 * g.lda, (uint32_t)((int64_t)(g.M - m0) * g.lda * 2));
  }
  if constexpr (B_KM) {
    sb.rs = make_rsrc(g.b + n0, (uint32_t)(((int64_t)(ke - 1) * g.ldb + (g.N - n0)) * 2));
  } else {
    sb.rs = make_rsrc(g.b + (int64_t)n0 * g.ldb, (uint32_t)((int64_t)(g.N - n0) * g.ldb * 2));
  }
  sa.ld_b = (uint32_t)g.lda * 2u;
  sb.ld_b = (uint32_t)g.ldb * 2u;

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; i++)
#pragma unroll
    for (int j = 0; j < 2; j++)
#pragma unroll
      for (int q = 0; q < 16; q++) acc[i][j][q] = 0.0f;

  // Two register sets stage k-steps two ahead: while step kt is computed
  // from LDS, the loads of step kt + 2 go into the set that step kt came
  // through, and the set holding step kt + 1 (loaded during step kt - 1)
  // is written to the other LDS buffer.
  u32x4 ra0[SA::kPer], rb0[SB::kPer], ra1[SA::kPer], rb1[SB::kPer];
  auto compute = [&](int cur) {
    const uint16_t* ta = sm.a[cur];
    const uint16_t* tb = sm.b[cur];
    // Both contraction blocks' operands are read before the first MFMA.
    u32x4 af[2][4], bf[2][2];
#pragma unroll
    for (int s = 0; s < 2; s++) {
#pragma unroll
      for (int i = 0; i < 4; i++) af[s][i] = SA::frag(ta, 128 * wm + 32 * i, s, lane);
#pragma unroll
      for (int j = 0; j < 2; j++) bf[s][j] = SB::frag(tb, 64 * wn + 32 * j, s, lane);
    }
#pragma unroll
    for (int s = 0; s < 2; s++)
#pragma unroll
      for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 2; j++)
          acc[i][j] = mfma32x32x16(as_bf16x8(bf[s][j]), as_bf16x8(af[s][i]), acc[i][j]);
  };
  // One k-step: ra/rb_free receive step kt + 2, ra/rb_next (step kt + 1)
  // go to LDS buffer (kt + 1) & 1.
  auto kstep = [&](int kt, u32x4 (&ra_free)[SA::kPer], u32x4 (&rb_free)[SB::kPer],
                   u32x4 (&ra_next)[SA::kPer], u32x4 (&rb_next)[SB::kPer]) {
    if (kt + 2 < nk) {
      sa.load(ra_free, kb + (kt + 2) * kGBK, tid);
      sb.load(rb_free, kb + (kt + 2) * kGBK, tid);
    }
    compute(kt & 1);
    if (kt + 1 < nk) {
      SA::store(sm.a[(kt + 1) & 1], ra_next, tid);
      SB::store(sm.b[(kt + 1) & 1], rb_next, tid);
    }
    __syncthreads();
  };
  if (nk > 0) {
    sa.load(ra0, kb, tid);
    sb.load(rb0, kb, tid);
    if (nk > 1) {
      sa.load(ra1, kb + kGBK, tid);
      sb.load(rb1, kb + kGBK, tid);
    }
    SA::store(sm.a[0], ra0, tid);
    SB::store(sm.b[0], rb0, tid);
  }
  __syncthreads();
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    kstep(kt, ra0, rb0, ra1, rb1);      // step kt came through set 0
    kstep(kt + 1, ra1, rb1, ra0, rb0);  // step kt + 1 through set 1
  }
  if (kt < nk) kstep(kt, ra0, rb0, ra1, rb1);

  // Epilogue, per group of 32 rows: the wave writes its 32 x 64 fp32 block
  // to a private LDS region (acc[i][j] register 4 g4 + e is row lane % 32,
  // column 32 j + 8 g4 + 4 h + e), then each lane takes 8 consecutive
  // columns of a row back, applies bias / SiLU / residual and stores 16
  // bytes: a store instruction covers 8 rows x 128 contiguous bytes.  (The
  // loop's last barrier has retired every read of the staging buffers; LDS
  // operations of one wave complete in order.)
  constexpr int kEpLd = 64 + 4;
  float* ep = reinterpret_cast<float*>(&sm) + wave * (32 * kEpLd);
  const int h = lane >> 5;
#pragma unroll
  for (int i = 0; i < 4; i++) {
#pragma unroll
    for (int j = 0; j < 2; j++)
#pragma unroll
      for (int g4 = 0; g4 < 4; g4++) {
        const f32x4 v = {acc[i][j][4 * g4], acc[i][j][4 * g4 + 1], acc[i][j][4 * g4 + 2],
                         acc[i][j][4 * g4 + 3]};
        *reinterpret_cast<f32x4*>(ep + (lane & 31) * kEpLd + 32 * j + 8 * g4 + 4 * h) = v;
      }
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int r = 0; r < 4; r++) {
      const int c = lane + 64 * r, row = c >> 3, cc = c & 7;
      const int m = m0 + 128 * wm + 32 * i + row, n = n0 + 64 * wn + 8 * cc;
      const f32x4 lo = *reinterpret_cast<const f32x4*>(ep + row * kEpLd + 8 * cc);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(ep + row * kEpLd + 8 * cc + 4);
      if (m >= g.M || n >= g.N) continue;
      float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      if constexpr (EPI == kEpiSlab) {
        float* o = g.slab + ((int64_t)blockIdx.y * g.M + m) * g.N + n;
        *reinterpret_cast<f32x4*>(o) = lo;
        *reinterpret_cast<f32x4*>(o + 4) = hi;
      } else {
        if (g.bias) {
          const f32x4 b0 = *reinterpret_cast<const f32x4*>(g.bias + n);
          const f32x4 b1 = *reinterpret_cast<const f32x4*>(g.bias + n + 4);
#pragma unroll
          for (int e = 0; e < 4; e++) {
            v[e] += b0[e];
            v[4 + e] += b1[e];
          }
        }
        if constexpr (EPI == kEpiSilu) {
          if (g.c2) {
            const u32x4 pre = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                               pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
            *reinterpret_cast<u32x4*>(g.c2 + (int64_t)m * g.ldc2 + n) = pre;
          }
#pragma unroll
          for (int e = 0; e < 8; e++) v[e] = silu_f(v[e]);
        } else if (g.res) {
          const u32x4 rv = *reinterpret_cast<const u32x4*>(g.res + (int64_t)m * g.ldr + n);
#pragma unroll
          for (int e = 0; e < 4; e++) {
            v[2 * e] += __uint_as_float(rv[e] << 16);
            v[2 * e + 1] += __uint_as_float(rv[e] & 0xffff0000u);
          }
        }
        const u32x4 o = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                         pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
        *reinterpret_cast<u32x4*>(g.c + (int64_t)m * g.ldc + n) = o;
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// fp32 problems (small shapes): a plain tiled product on the vector ALUs,
// 64 x 64 tile per workgroup, 4 x 4 outputs per thread, any strides.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgsF32 g) {
  __shared__ float As[16][65], Bs[16][65];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.x * 64, n0 = blockIdx.y * 64;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < g.K; k0 += 16) {
    for (int x = tid; x < 16 * 64; x += 256) {
      const int kk = x >> 6, r = x & 63;
      const int k = k0 + kk, m = m0 + r, n = n0 + r;
      As[kk][r] = (k < g.K && m < g.M) ? g.a[(int64_t)m * g.sam + (int64_t)k * g.sak] : 0.0f;
      Bs[kk][r] = (k < g.K && n < g.N) ? g.b[(int64_t)n * g.sbn + (int64_t)k * g.sbk] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; kk++)
#pragma unroll
      for (int a = 0; a < 4; a++)
#pragma unroll
        for (int b = 0; b < 4; b++) acc[a][b] += As[kk][ty + 16 * a] * Bs[kk][tx + 16 * b];
    __syncthreads();
  }
#pragma unroll
  for (int a = 0; a < 4; a++)
#pragma unroll
    for (int b = 0; b < 4; b++) {
      const int m = m0 + ty + 16 * a, n = n0 + tx + 16 * b;
      if (m >= g.M || n >= g.N) continue;
      float v = acc[a][b];
      if constexpr (EPI == kEpiSlab) {
        g.c[(int64_t)m * g.ldc + n] = v;
      } else {
        if (g.bias) v += g.bias[n];
        if constexpr (EPI == kEpiSilu) {
          if (g.c2) g.c2[(int64_t)m * g.ldc2 + n] = v;
          v = v / (1.0f + expf(-v));
        } else if (g.res) {
          v += g.res[(int64_t)m * g.ldr + n];
        }
        g.c[(int64_t)m * g.ldc + n] = v;
      }
    }
}

template <bool BF16>
__device__ __forceinline__ float ld_e(const void* p, int64_t i) {
  if constexpr (BF16)
    return bf16_bits_to_f32(((const uint16_t*)p)[i]);
  else
    return ((const float*)p)[i];
}

template <bool BF16>
__device__ __forceinline__ void st_e(void* p, int64_t i, float v) {
  if constexpr (BF16)
    ((uint16_t*)p)[i] = f32_to_bf16_bits(v);
  else
    ((float*)p)[i] = v;
}

// dpre = dZ * SiLU'(pre), dZ = [dU | dV | dQ | dK] from four dense
// [T][h][d] gradients, and partial column sums of the fp32 dpre for the
// bias gradient, one row of partials per block of kColRows token rows.  A
// thread owns 8 consecutive columns (16-byte accesses in bf16; the four
// sources meet at multiples of 64 columns, so 8 columns never straddle
// two) and walks the block's rows.  Blocks of 32 rows (eight in flight per
// thread) give the HBM-bound pass enough workgroups: 128-row blocks left
// it at ~3.7 TB/s (projection backward at the training shape 0.58 ->
// 0.55 ms).
constexpr int kColRows = 32;

template <bool BF16>
__device__ __forceinline__ void load8(const void* p, int64_t i, float (&v)[8]) {
  if constexpr (BF16) {
    const u32x4 r = *reinterpret_cast<const u32x4*>((const uint16_t*)p + i);
#pragma unroll
    for (int e = 0; e < 4; e++) {
      v[2 * e] = __uint_as_float(r[e] << 16);
      v[2 * e + 1] = __uint_as_float(r[e] & 0xffff0000u);
    }
  } else {
    const f32x4 a = *reinterpret_cast<const f32x4*>((const float*)p + i);
    const f32x4 b = *reinterpret_cast<const f32x4*>((const float*)p + i + 4);
#pragma unroll
    for (int e = 0; e < 4; e++) {
      v[e] = a[e];
      v[4 + e] = b[e];
    }
  }
}

template <bool BF16>
__device__ __forceinline__ void store8(void* p, int64_t i, const float (&v)[8]) {
  if constexpr (BF16) {
    const u32x4 r = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                     pack_bf16x2(v[6], v[7])};
    *reinterpret_cast<u32x4*>((uint16_t*)p + i) = r;
  } else {
    const f32x4 a = {v[0], v[1], v[2], v[3]}, b = {v[4], v[5], v[6], v[7]};
    *reinterpret_cast<f32x4*>((float*)p + i) = a;
    *reinterpret_cast<f32x4*>((float*)p + i + 4) = b;
  }
}

template <bool BF16>
__global__ __launch_bounds__(256) void silu_bwd_kernel(int64_t T, int F, int hv, int hq,
                                                       const void* __restrict__ pre,
                                                       const void* __restrict__ du,
                                                       const void* __restrict__ dv,
                                                       const void* __restrict__ dq,
                                                       const void* __restrict__ dk,
                                                       void* __restrict__ dpre,
                                                       float* __restrict__ partial) {
  const int c = 8 * (blockIdx.x * 256 + threadIdx.x);
  if (c >= F) return;
  const void* src;
  int w, cc;
  if (c < hv) {
    src = du, w = hv, cc = c;
  } else if (c < 2 * hv) {
    src = dv, w = hv, cc = c - hv;
  } else if (c < 2 * hv + hq) {
    src = dq, w = hq, cc = c - 2 * hv;
  } else {
    src = dk, w = hq, cc = c - 2 * hv - hq;
  }
  const int64_t r0 = (int64_t)blockIdx.y * kColRows;
  const int64_t r1 = min(T, r0 + kColRows);
  float sum[8] = {};
#pragma unroll 8
  for (int64_t r = r0; r < r1; r++) {
    float x[8], d[8];
    load8<BF16>(pre, r * F + c, x);
    load8<BF16>(src, r * w + cc, d);
#pragma unroll
    for (int e = 0; e < 8; e++) {
      const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x[e] * -kLog2e));
      d[e] *= sg * (1.0f + x[e] * (1.0f - sg));
      sum[e] += d[e];
    }
    store8<BF16>(dpre, r * F + c, d);
  }
  float* pp = partial + (int64_t)blockIdx.y * F + c;
  const f32x4 a = {sum[0], sum[1], sum[2], sum[3]}, b = {sum[4], sum[5], sum[6], sum[7]};
  *reinterpret_cast<f32x4*>(pp) = a;
  *reinterpret_cast<f32x4*>(pp + 4) = b;
}

// Partial column sums of x [T][N] (row stride ld, N and ld multiples of 8)
// per block of kColRows rows.
template <bool BF16>
__global__ __launch_bounds__(256) void colsum_kernel(int64_t T, int N, int64_t ld,
                                                     const void* __restrict__ x,
                                                     float* __restrict__ partial) {
  const int c = 8 * (blockIdx.x * 256 + threadIdx.x);
  if (c >= N) return;
  const int64_t r0 = (int64_t)blockIdx.y * kColRows;
  const int64_t r1 = min(T, r0 + kColRows);
  float sum[8] = {};
#pragma unroll 4
  for (int64_t r = r0; r < r1; r++) {
    float v[8];
    load8<BF16>(x, r * ld + c, v);
#pragma unroll
    for (int e = 0; e < 8; e++) sum[e] += v[e];
  }
  float* pp = partial + (int64_t)blockIdx.y * N + c;
  const f32x4 a = {sum[0], sum[1], sum[2], sum[3]}, b = {sum[4], sum[5], sum[6], sum[7]};
  *reinterpret_cast<f32x4*>(pp) = a;
  *reinterpret_cast<f32x4*>(pp + 4) = b;
}

// out[i] = sum over s of part[s][i], s in order (few rows, many columns:
// the split-K slabs).
__global__ __launch_bounds__(256) void reduce_slabs_kernel(int64_t n, int S,
                                                           const float* __restrict__ part,
                                                           float* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    float s = 0.0f;
    for (int k = 0; k < S; k++) s += part[(int64_t)k * n + i];
    out[i] = s;
  }
}

// The same sum for many rows and few columns (bias partials): a block owns
// 16 columns; its 16 row groups each sum every 16th row, then the group
// sums are added in group order.  The order is fixed, so the result is.
__global__ __launch_bounds__(256) void reduce_cols_kernel(int n, int S,
                                                          const float* __restrict__ part,
                                                          float* __restrict__ out) {
  __shared__ float red[16][17];
  const int col = threadIdx.x & 15, grp = threadIdx.x >> 4;
  const int i = blockIdx.x * 16 + col;
  float s = 0.0f;
  if (i < n) {
#pragma unroll 8
    for (int k = grp; k < S; k += 16) s += part[(int64_t)k * n + i];
  }
  red[grp][col] = s;
  __syncthreads();
  if (grp == 0 && i < n) {
    float t = 0.0f;
#pragma unroll
    for (int q = 0; q < 16; q++) t += red[q][col];
    out[i] = t;
  }
}

}  // namespace

int gemm_num_splits(int M, int N, int64_t K, int* k_split) {
  const int tiles = ((M + kGBM - 1) / kGBM) * ((N + kGBN - 1) / kGBN);
  int64_t want = (512 + tiles - 1) / tiles;
  // At least 256 contraction rows per split, and at least one split.
  const int64_t max_splits = K > 256 ? (K + 255) / 256 : 1;
  want = want < 1 ? 1 : want > max_splits ? max_splits : want;
  int64_t ks = (K + want - 1) / want;
  ks = (ks + kGBK - 1) / kGBK * kGBK;
  if (ks < kGBK) ks = kGBK;
  *k_split = (int)ks;
  return (int)((K + ks - 1) / ks);
}

hipError_t launch_gemm_bf16(const GemmArgs& g, int a_kmajor, int b_kmajor, int epi, int splits,
                            hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  const int nt = ((g.M + kGBM - 1) / kGBM) * ((g.N + kGBN - 1) / kGBN);
  const dim3 grid((unsigned)nt, (unsigned)splits);
#define HSTU_GEMM_CASE(AK, BK, E)                                                         \
  if (a_kmajor == AK && b_kmajor == BK && epi == E) {                                     \
    hipLaunchKernelGGL((gemm_bf16_kernel<AK, BK, E>), grid, dim3(256), 0, s, g);          \
    return hipGetLastError();                                                             \
  }
  HSTU_GEMM_CASE(0, 0, kEpiSilu)
  HSTU_GEMM_CASE(0, 0, kEpiAdd)
  HSTU_GEMM_CASE(0, 1, kEpiAdd)
  HSTU_GEMM_CASE(1, 1, kEpiSlab)
#undef HSTU_GEMM_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_gemm_f32(const GemmArgsF32& g, int epi, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  const dim3 grid((unsigned)((g.M + 63) / 64), (unsigned)((g.N + 63) / 64));
  if (epi == kEpiSilu)
    hipLaunchKernelGGL(gemm_f32_kernel<kEpiSilu>, grid, dim3(256), 0, s, g);
  else if (epi == kEpiAdd)
    hipLaunchKernelGGL(gemm_f32_kernel<kEpiAdd>, grid, dim3(256), 0, s, g);
  else
    hipLaunchKernelGGL(gemm_f32_kernel<kEpiSlab>, grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

int64_t colsum_blocks(int64_t T) { return (T + kColRows - 1) / kColRows; }

hipError_t launch_silu_bwd(int is_bf16, int64_t T, int F, int hv, int hq, const void* pre,
                           const void* du, const void* dv, const void* dq, const void* dk,
                           void* dpre, float* partial, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const dim3 grid((unsigned)((F / 8 + 255) / 256), (unsigned)colsum_blocks(T));
  if (is_bf16)
    hipLaunchKernelGGL(silu_bwd_kernel<true>, grid, dim3(256), 0, s, T, F, hv, hq, pre, du, dv,
                       dq, dk, dpre, partial);
  else
    hipLaunchKernelGGL(silu_bwd_kernel<false>, grid, dim3(256), 0, s, T, F, hv, hq, pre, du, dv,
                       dq, dk, dpre, partial);
  return hipGetLastError();
}

hipError_t launch_colsum(int is_bf16, int64_t T, int N, int64_t ld, const void* x, float* partial,
                         hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const dim3 grid((unsigned)((N / 8 + 255) / 256), (unsigned)colsum_blocks(T));
  if (is_bf16)
    hipLaunchKernelGGL(colsum_kernel<true>, grid, dim3(256), 0, s, T, N, ld, x, partial);
  else
    hipLaunchKernelGGL(colsum_kernel<false>, grid, dim3(256), 0, s, T, N, ld, x, partial);
  return hipGetLastError();
}

hipError_t launch_reduce_cols(int n, int S, const float* part, float* out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(reduce_cols_kernel, dim3((unsigned)((n + 15) / 16)), dim3(256), 0, s, n, S,
                     part, out);
  return hipGetLastError();
}

hipError_t launch_reduce_slabs(int64_t n, int S, const float* part, float* out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  const dim3 grid((unsigned)(blocks < 4096 ? blocks : 4096));
  hipLaunchKernelGGL(reduce_slabs_kernel, grid, dim3(256), 0, s, n, S, part, out);
  return hipGetLastError();
}

}  // namespace hstu
