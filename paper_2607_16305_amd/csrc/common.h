// Shared device helpers for the LookME gfx950 kernels.
//
// All contractions in the path are "NT" products over 16-byte chunks of
// K-contiguous rows: scores(key, token) = <key_row, q_row>.  One "chunk step"
// covers 64 bytes of a row: the four 16-lane groups of a wave each hold one
// 16-byte chunk.  For bf16 a step is one v_mfma_f32_16x16x32_bf16; for fp32
// it is four v_mfma_f32_16x16x4_f32 (one per 4-byte element of the chunk).
// Operand A and operand B always take the same chunk for the same lane group
// and element, so every product pairs equal k; the order in which k is
// visited is free because the result is a plain sum.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lookme {

enum : int { DT_F32 = 0, DT_BF16 = 1 };

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int WAVE = 64;

__device__ __forceinline__ u32x4_t ld16(const void* p) {
  return *reinterpret_cast<const u32x4_t*>(p);
}
__device__ __forceinline__ u32x4_t ld16_nt(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
}
__device__ __forceinline__ void st16(void* p, u32x4_t v) {
  *reinterpret_cast<u32x4_t*>(p) = v;
}

template <int DT>
__device__ __forceinline__ f32x4_t mfma_chunk(u32x4_t a, u32x4_t b, f32x4_t c);

template <>
__device__ __forceinline__ f32x4_t mfma_chunk<DT_BF16>(u32x4_t a, u32x4_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

template <>
__device__ __forceinline__ f32x4_t mfma_chunk<DT_F32>(u32x4_t a, u32x4_t b, f32x4_t c) {
  // Reinterpret the whole vector, then index it: this compiler folds
  // __builtin_bit_cast applied to a single vector element to element 0.
  const f32x4_t af = __builtin_bit_cast(f32x4_t, a);
  const f32x4_t bf = __builtin_bit_cast(f32x4_t, b);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(af[0], bf[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(af[1], bf[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(af[2], bf[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(af[3], bf[3], c, 0, 0, 0);
  return c;
}

// Scalar reinterpretation.  Always pass a scalar value (never a vector
// element expression) into __builtin_bit_cast; these helpers take it by value.
__device__ __forceinline__ float as_f32(uint32_t u) { return __uint_as_float(u); }
__device__ __forceinline__ uint32_t as_u32(float f) { return __float_as_uint(f); }

// bf16 <-> fp32.  bf16 is the upper half of a binary32; widening is exact.
__device__ __forceinline__ float bf16lo(uint32_t w) { return as_f32(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) {
  return as_f32(w & 0xFFFF0000u);
}

// Round a finite binary32 to the nearest bf16, ties to even: add half an
// ulp of the target minus one, plus the lowest kept bit, then truncate.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = as_u32(f);
  if ((u & 0x7F800000u) == 0x7F800000u) return (u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_rne(lo) | (f32_to_bf16_rne(hi) << 16);
}

// Ordering used by every selection: larger score first, equal scores by
// smaller index.  Index -1 marks an empty slot (score -inf).
// (bitwise operators: with || and && the compiler branches on the exec mask)
__device__ __forceinline__ bool beats(float s, int i, float t, int j) {
  return (s > t) | ((s == t) & ((unsigned)i < (unsigned)j));
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Blocks are dispatched round-robin over the 8 XCDs of the chip; this maps
// a launch index to a work index so that each XCD receives a contiguous
// range of work items (neighbouring items share that XCD's L2).  Returns -1
// for launch slots beyond `count` items.
__device__ __forceinline__ int xcd_remap(int b, int count) {
  const int per = (count + 7) >> 3;
  const int x = b & 7, j = b >> 3;
  if (j >= per) return -1;
  const int u = x * per + j;
  return u < count ? u : -1;
}

// Inclusive prefix sum over the threads of one wave.
__device__ __forceinline__ int wave_scan_incl(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int o = __shfl_up(v, d, 64);
    if (lane >= d) v += o;
  }
  return v;
}

// Inclusive prefix sum over the first `waves` waves of the block (all
// threads of the block must call it; threads beyond them pass 0).
template <int MAXW>
__device__ __forceinline__ int block_scan_incl(int v, int* wsum) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int incl = wave_scan_incl(v);
  if (lane == 63 && wv < MAXW) wsum[wv] = incl;
  __syncthreads();
  int off = 0;
  for (int w = 0; w < wv && w < MAXW; ++w) off += wsum[w];
  __syncthreads();
  return incl + off;
}

}  // namespace lookme
