// Device helpers shared by the libhstu kernels (gfx950 / CDNA4).
//
// Definitions restated from the paper (Zhai et al., ICML 2024):
//  - mask: causal with the diagonal; candidates (the last n_t tokens of a
//    sequence) see the history and themselves only (Algorithm 1);
//  - bias position: every candidate sits at position n_h = L - n_t;
//  - time bucket: min(B_t - 1, floor(log2(max(|t_i - t_j|, 1))))
//    (notation table, entry rab^{p,t});
//  - phi2 = SiLU (Eq. 2).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hstu {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;

// One work item of the jagged tile scheduler: (sequence, block index).
struct WorkItem {
  int32_t seq;
  int32_t blk;
};

__device__ __forceinline__ bool pair_valid(int i, int j, int n_h) {
  return j <= i && (j < n_h || j == i);
}

__device__ __forceinline__ int bias_pos(int x, int n_h) { return x < n_h ? x : n_h; }

// floor(log2(max(|dt|, 1))) clamped to nb-1, exact integer arithmetic.
__device__ __forceinline__ int time_bucket64(int64_t dt, int nb) {
  uint64_t a = dt < 0 ? (uint64_t)0 - (uint64_t)dt : (uint64_t)dt;
  a = a < 1 ? 1 : a;
  int b = 63 - __clzll((long long)a);
  return b < nb - 1 ? b : nb - 1;
}

// sigma(x) with one exp2 and one reciprocal (both hardware transcendentals).
__device__ __forceinline__ float sigmoid_fast(float x) {
  float e = __builtin_amdgcn_exp2f(-x * kLog2e);
  return __builtin_amdgcn_rcpf(1.0f + e);
}

__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ u32x4 zero_u32x4() {
  u32x4 z = {0u, 0u, 0u, 0u};
  return z;
}

// Packs two floats into two bf16 (round to nearest even) in one dword.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  bf16x2 r;
  r[0] = (__bf16)lo;
  r[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, r);
}

// Eight floats as eight bf16 (round to nearest even), low halves first.
__device__ __forceinline__ u32x4 pack_bf16x8(const float* v) {
  return u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
               pack_bf16x2(v[6], v[7])};
}

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// Packs two floats into two f16 (round to nearest even) in one dword.
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  f16x2 r;
  r[0] = (_Float16)lo;
  r[1] = (_Float16)hi;
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float x) {
  return __builtin_bit_cast(uint16_t, (__bf16)x);
}

// Raw buffer resource over `bytes` bytes from `base` (stride 0, 32-bit
// data format word of gfx9-family parts).  Loads whose byte offset lies at
// or past `bytes` return zeros instead of touching memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

__device__ __forceinline__ u32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0));
}

__device__ __forceinline__ uint64_t buffer_load8(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(uint64_t, __builtin_amdgcn_raw_buffer_load_b64(r, byte_off, 0, 0));
}

__device__ __forceinline__ uint32_t buffer_load4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 0);
}

// LDS DMA: each of the 64 lanes loads `size` bytes at byte offset `off`
// of the buffer and the wave writes them to LDS at lds + size * lane.
// Completion is counted by vmcnt, like any buffer load.
__device__ __forceinline__ void dma_to_lds16(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16,
                                           off, 0, 0, 0);
}

__device__ __forceinline__ void dma_to_lds4(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 4,
                                           off, 0, 0, 0);
}

// The same LDS DMA issued from inline assembly, on a resource given as its
// four descriptor words.  The compiler does not see these as pending LDS
// writes, so it does not make later LDS reads wait for every outstanding
// vector-memory operation (it cannot tell ring slots of one array apart);
// the caller orders the data with explicit vmcnt waits and barriers.  The
// statement sets M0, which the kernels using it keep no value in.
__device__ __forceinline__ u32x4 rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)base;
  return u32x4{(uint32_t)a, (uint32_t)(a >> 32) & 0xffffu, bytes, 0x00020000u};
}

__device__ __forceinline__ void dma_to_lds16_asm(u32x4 r, void* lds, uint32_t off) {
  const uint32_t l = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)lds;
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(l), "v"(off), "s"(r)
               : "memory");
}

__device__ __forceinline__ void dma_to_lds4_asm(u32x4 r, void* lds, uint32_t off) {
  const uint32_t l = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)lds;
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds"
               :
               : "s"(l), "v"(off), "s"(r)
               : "memory");
}

// s_waitcnt vmcnt(VM) lgkmcnt(0) (gfx9 encoding: vmcnt in bits 3:0 and
// 15:14, expcnt in 6:4, lgkmcnt in 11:8).
template <int VM>
__device__ __forceinline__ void wait_vmcnt_lgkmcnt0() {
  static_assert(VM >= 0 && VM < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4));
}

// Workgroup barrier without __syncthreads' memory fence (which would wait
// for every outstanding LDS-DMA load).  The caller waits for what must be
// visible; the empty asm statements keep the compiler from moving memory
// accesses across the barrier.
__device__ __forceinline__ void barrier_no_fence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Position of row index `r` (0..31) inside a 32-wide LDS strip whose
// contraction order matches the 32x32 MFMA accumulator layout: an
// accumulator lane holds rows 8*g + 4*half + m (g = 0..3, m = 0..3) and
// feeds them as the k-operand of the next contraction in the order
// (step = g/2, half, g%2, m).  Storing row r at swap_bits23(r) lets the
// other operand be read with one 16-byte LDS load.
__device__ __forceinline__ int swap_bits23(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

}  // namespace hstu
