// Per-lane top-k upkeep and list merging shared by the scoring kernels
// (Level-2 over primitive keys, score.hip; Level-2 over the relevance MLP's
// logits, relevance.hip) and their lane-group helpers.  The 16 x 16 score
// tile of a 16-key block has keys 4g..4g+3 of the block for query row n in
// lane (g, n); the four lanes n, n + 16, n + 32, n + 48 hold a row's lists.
#pragma once
#include "common.h"

namespace lookme {

// Both values of the lane pairs (L, L ^ 32) and (L, L ^ 16), from the
// gfx950 permlane swaps (vector instructions, no LDS round trip): with both
// operands equal to v, lane L gets {v[L], v[L ^ 32]} (resp. L ^ 16) as the
// two results, in an order that does not matter to a sum or a max.
__device__ __forceinline__ void pair32(float v, float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}
__device__ __forceinline__ void pair16(float v, float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}

// The sum over the 4 lane groups (lanes n, n + 16, n + 32, n + 48) that hold
// the chunks of one row (added in the order (L, L^16) then the pairs, the same
// in every lane of the group).
__device__ __forceinline__ float sum_lane_groups(float v) {
  float a, b;
  pair16(v, a, b);
  v = a + b;
  pair32(v, a, b);
  return a + b;
}

// The maximum over the same 4 lanes.
__device__ __forceinline__ float max_lane_groups(float v) {
  float a, b;
  pair16(v, a, b);
  v = fmaxf(a, b);
  pair32(v, a, b);
  return fmaxf(a, b);
}

// The minimum over the same 4 lanes.
__device__ __forceinline__ float min_lane_groups(float v) {
  float a, b;
  pair16(v, a, b);
  v = fminf(a, b);
  pair32(v, a, b);
  return fminf(a, b);
}

// The sum of squares of a 16-byte chunk's elements added to acc.
template <int DT>
__device__ __forceinline__ float chunk_sumsq(u32x4_t v, float acc) {
  if constexpr (DT == DT_BF16) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc = fmaf(bf16lo(v[e]), bf16lo(v[e]), acc);
      acc = fmaf(bf16hi(v[e]), bf16hi(v[e]), acc);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) acc = fmaf(as_f32(v[e]), as_f32(v[e]), acc);
  }
  return acc;
}

__device__ __forceinline__ float inv_norm(float sq) { return sq > 0.f ? rsqrtf(sq) : 0.f; }

// Cosine scaling of a tile's 4 scores (keys 4g + r of the block, query row
// n): knsq holds, in every lane of row n', the squared norm of key n'.
__device__ __forceinline__ f32x4_t cos_scale(f32x4_t acc, float qinv, float knsq, int g) {
#pragma unroll
  for (int r = 0; r < 4; ++r) acc[r] *= qinv * inv_norm(__shfl(knsq, 4 * g + r, 64));
  return acc;
}

// Scores of 4 keys (blk*16 + 4g + r) for one query row folded into the
// lane's running result: arg max (routing, with the scene bias) or a sorted
// list of the KL best (Level-2; with LBIAS, bias points at the 16 biases of
// this block in LDS, the relevance logits' b2, 0 for keys past kend, and
// each key's is added first).  `tight` (only when the lists are exactly k
// long) also drops values below the smallest KL/4-th entry of the row's
// four lists: those four lists hold k values at least that large.
template <bool LOOKUP, int KL, bool LBIAS = false>
__device__ __forceinline__ void fold_scores(f32x4_t acc, int blk, int g, int kend, const float* bias,
                                            float (&ls)[KL], int (&li)[KL], bool tight = false) {
  float v[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) v[r] = blk * 16 + 4 * g + r < kend ? acc[r] : -__builtin_inff();
  if constexpr (LOOKUP && LBIAS) {
    // one 16-byte read (keys past kend stay -inf: their bias is 0)
    const f32x4_t bv = *reinterpret_cast<const f32x4_t*>(bias + 4 * g);
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] += bv[r];
  }
  if constexpr (!LOOKUP) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int p = blk * 16 + 4 * g + r;
      float x = v[r];
      if (bias != nullptr && p < kend) x += bias[p];
      if (x > ls[0]) { ls[0] = x; li[0] = p; }
    }
  } else {
    // The 4 values go in largest first (the first of equal values, i.e. the
    // lowest key), one insertion round per value that still beats some
    // lane's list: the rounds are wave-wide (branch-free sorted insertion),
    // and after the first blocks a round is rarely needed by any lane, so
    // most blocks cost one vote instead of four insertions.  A value below
    // T, the largest last entry of the row's 4 lists in this wave, cannot
    // reach the row's top k (that list holds KL >= k keys at least as
    // large), so it is dropped; values equal to T stay, for the lower-index
    // rule.
    const int p0 = blk * 16 + 4 * g;
    float T = max_lane_groups(ls[KL - 1]);
    if (tight) T = fmaxf(T, min_lane_groups(ls[KL / 4 - 1]));
#pragma unroll
    for (int round = 0; round < 4; ++round) {
      float x = v[0];
      int w = 0;
#pragma unroll
      for (int r = 1; r < 4; ++r)
        if (v[r] > x) { x = v[r]; w = r; }
      if (!(x >= T)) x = -__builtin_inff();
      if (!__any(x > ls[KL - 1])) break;
      const int p = p0 + w;
      // sorted insertion, the list descending: entry e becomes ls[e-1] if x
      // beats it, else x if x beats ls[e], else stays: the median of the
      // three values (one instruction), and the index by the same two tests
      // as two plain selects (written as one nested conditional, the
      // compiler turns them into exec-mask branches, several scalar
      // instructions an entry)
#pragma unroll
      for (int e = KL - 1; e >= 1; --e) {
        const bool above_prev = x > ls[e - 1];
        const bool above_cur = x > ls[e];
        const int kept = above_cur ? p : li[e];
        li[e] = above_prev ? li[e - 1] : kept;
        ls[e] = __builtin_amdgcn_fmed3f(x, ls[e - 1], ls[e]);
      }
      li[0] = x > ls[0] ? p : li[0];
      ls[0] = fmaxf(x, ls[0]);
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (r == w) v[r] = -__builtin_inff();
    }
  }
}

// k rounds of a butterfly arg max over the 2^STEPS lanes that hold the
// candidate lists of one row (lane distance `stride`, doubling each step).
// Each lane passes its own sorted list; every lane receives the k winners.
template <int KL, int STEPS>
__device__ __forceinline__ void merge_lists(const float (&ls)[KL], const int (&li)[KL], int k,
                                            int stride, float (&top_s)[KL], int (&top_i)[KL]) {
  int head = 0;
  float hs = ls[0];
  int hi = li[0];
#pragma unroll
  for (int e = 0; e < KL; ++e) {
    if (e < k) {
      float bs = hs;
      int bi = hi;
#pragma unroll
      for (int d = 0; d < STEPS; ++d) {
        const float os = __shfl_xor(bs, stride << d, 64);
        const int oi = __shfl_xor(bi, stride << d, 64);
        if (beats(os, oi, bs, bi)) { bs = os; bi = oi; }
      }
      top_s[e] = bs;
      top_i[e] = bi;
      // the list that supplied the winner moves its head on (selects, not
      // branches)
      const bool won = (hi == bi) & (hs == bs);
      head += won ? 1 : 0;
      float ns = -__builtin_inff();
      int ni = -1;
#pragma unroll
      for (int x = 1; x < KL; ++x) {
        ns = x == head ? ls[x] : ns;
        ni = x == head ? li[x] : ni;
      }
      hs = won ? ns : hs;
      hi = won ? ni : hi;
    }
  }
}

// A 16-key block of a scene (16 consecutive key rows: 16 row_bytes contiguous
// bytes, row_bytes = 64 ks) is copied straight from global memory into an
// LDS image by ks load instructions of one KiB each: instruction i reads the
// block's bytes [1024 i, 1024 i + 1024), a whole contiguous KiB, with the
// nontemporal hint (every key is read once).  That form streams from HBM at
// ~7 TB/s on this chip, against ~6.1 TB/s for 16 rows x 64 bytes an
// instruction (the operand order), measured at the Zipf workload's shape.
// Lane L's 16 bytes land at image byte 1024 i + 16 L, i.e. row
// r = (64 i + L) / C, slot s = (64 i + L) % C (C = 4 ks chunks a row), and the
// lane reads chunk s ^ swz(r) of that row: the chunks of a row are permuted
// inside groups of G (16 when C is a multiple of 16), so that the fragment
// reads (16 rows, one chunk index) hit distinct banks.  The operand fragment
// of lane (g, n) at step j is row n, chunk 4 j + g, at image byte
// n row_bytes + ((4 j + g) ^ swz(n)) 16.
struct KeyImage {
  int C;         // chunks a row
  int G;         // swizzle group (a power of two dividing C, at most 16)
  int64_t rb;    // row bytes
  __device__ __forceinline__ int swz(int r) const { return r & (G - 1); }
  // byte of the block that lane L of load instruction i reads (row r of the
  // image; rr: the key row actually read, r unless clamped)
  __device__ __forceinline__ uint32_t src_off(int i, int L, int rr) const {
    const int e = 64 * i + L, r = e / C, sl = e - r * C;
    return (uint32_t)(rr * rb) + (uint32_t)((sl ^ swz(r)) * 16);
  }
  __device__ __forceinline__ int row_of(int i, int L) const { return (64 * i + L) / C; }
  __device__ __forceinline__ uint32_t frag_off(int j, int g, int n) const {
    return (uint32_t)(n * rb) + (uint32_t)((((4 * j + g) ^ swz(n))) * 16);
  }
};

}  // namespace lookme
