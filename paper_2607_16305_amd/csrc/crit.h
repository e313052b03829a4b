// Criticality, the top-n_keep select and the learned gate of the sparse
// injection (arXiv 2607.16305, Sec. 3.3, Eq. 9-10): the bodies shared by the stand-alone
// kernels (inject.hip) and by the launches that carry them beside the
// bucketing and the Level-2 scoring of small batches (bucket.hip, score.hip),
// so that all give the same bits.
//
//   row_sumsq    one wave streams a row of Delta once (NORM_UNROLL 16-byte
//                loads of a lane in flight) and returns its fp32 sum of
//                squares, accumulated in a fixed order; stored as its bit
//                pattern, it orders like the norm (non-negative floats order
//                like their bits, and the square root keeps the order);
//   select_layer one workgroup (1024 or 256 threads): 4-pass MSB-first radix
//                select of the n_keep-th largest key (keys cached in LDS when
//                they fit), then an order-preserving compaction (block prefix
//                sums) of the kept token ids;
//   row_dot, gate_compact_layer  the learned SKA gate's logit z = Delta_i W_g
//                and the ascending compaction of its open rows (Eq. 9).
#pragma once

#include "common.h"

namespace lookme {

constexpr int NORM_UNROLL = 4;
constexpr int SEL_THREADS = 1024;
constexpr int SEL_WAVES = SEL_THREADS / WAVE;

// CN > 0: a layer's keys (n <= CN) are first copied to LDS, so that the four
// passes and the compaction read them there instead of from L2 (one global
// round trip instead of five).  Element i sits at i + i / 32: the padding
// keeps threads that walk ranges of 32 keys on distinct banks.  Launchers
// take the smallest cache that holds n: the small one leaves room on the CU
// for the workgroups of a kernel that runs beside the select.
constexpr int SEL_CACHE_SMALL = 4096, SEL_CACHE_N = 32768;

template <int DT>
__device__ __forceinline__ float row_sumsq(const char* __restrict__ p, int chunks, int lane) {
  float acc0 = 0.f, acc1 = 0.f;
  // chunks past the row re-read its last chunk and are not summed (a
  // 4096-element bf16 row is two rounds)
  for (int c0 = lane; c0 < chunks; c0 += NORM_UNROLL * WAVE) {
    u32x4_t vv[NORM_UNROLL];
#pragma unroll
    for (int u = 0; u < NORM_UNROLL; ++u) {
      const int c = c0 + u * WAVE;
      vv[u] = ld16_nt(p + (int64_t)(c < chunks ? c : chunks - 1) * 16);
    }
#pragma unroll
    for (int u = 0; u < NORM_UNROLL; ++u) {
      if (c0 + u * WAVE >= chunks) continue;
      const u32x4_t v = vv[u];
      if constexpr (DT == DT_BF16) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = bf16lo(v[e]), hi = bf16hi(v[e]);
          acc0 = fmaf(lo, lo, acc0);
          acc1 = fmaf(hi, hi, acc1);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float f = as_f32(v[e]);
          if (e & 1) acc1 = fmaf(f, f, acc1);
          else acc0 = fmaf(f, f, acc0);
        }
      }
    }
  }
  float acc = acc0 + acc1;
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) acc += __shfl_xor(acc, d, 64);
  return acc;
}

// z = row . w (the SKA gate's logit of Eq. 9) by one wave: NORM_UNROLL 16-byte
// loads of the row and of w in flight per lane, fp32 fused multiply-adds in a
// fixed order, then the wave sum.
template <int DT>
__device__ __forceinline__ float row_dot(const char* __restrict__ p, const char* __restrict__ w,
                                         int chunks, int lane) {
  float acc = 0.f;
  for (int c0 = lane; c0 < chunks; c0 += NORM_UNROLL * WAVE) {
    u32x4_t dv[NORM_UNROLL], wv[NORM_UNROLL];
#pragma unroll
    for (int u = 0; u < NORM_UNROLL; ++u) {
      const int c = c0 + u * WAVE;
      const int cc = c < chunks ? c : chunks - 1;
      dv[u] = ld16_nt(p + (int64_t)cc * 16);
      wv[u] = ld16(w + (int64_t)cc * 16);
    }
#pragma unroll
    for (int u = 0; u < NORM_UNROLL; ++u) {
      if (c0 + u * WAVE >= chunks) continue;
      if constexpr (DT == DT_BF16) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc = fmaf(bf16lo(dv[u][e]), bf16lo(wv[u][e]), acc);
          acc = fmaf(bf16hi(dv[u][e]), bf16hi(wv[u][e]), acc);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) acc = fmaf(as_f32(dv[u][e]), as_f32(wv[u][e]), acc);
      }
    }
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) acc += __shfl_xor(acc, d, 64);
  return acc;
}

// The open gates of one layer in ascending order (Eq. 9-10: z > 0; z = 0
// stays closed): every thread owns GATE_PER_THREAD consecutive rows (their
// signs packed in one register), a block prefix sum of the per-thread counts
// places each open row; kept[count ..  n) = -1 and *count = the number open.
// Called by all THREADS threads of a workgroup.
constexpr int GATE_PER_THREAD = 32;

// LDS words the select and the gate compaction work in (counts, scan
// partials, the located prefix).  The caller passes them: a kernel that
// also stages operands by direct-to-LDS loads keeps all of its LDS in one
// object (with several, the compiler puts a load wait before every LDS read
// that follows those loads).
struct SelLds {
  int hist[256];
  int wsum[SEL_WAVES];
  uint32_t prefix;
  int need;
  int total;
};

template <int THREADS>
__device__ __forceinline__ void gate_compact_layer(const float* __restrict__ z, int64_t n,
                                                   int32_t* __restrict__ kept,
                                                   int32_t* __restrict__ count, SelLds& sl) {
  constexpr int SPAN = THREADS * GATE_PER_THREAD;   // rows a round
  static_assert(THREADS / WAVE <= SEL_WAVES, "scan partials");
  int* wsum = sl.wsum;
  int& s_total = sl.total;
  const int tid = threadIdx.x;
  int64_t base = 0;   // open rows in earlier rounds
  for (int64_t r0 = 0; r0 < n; r0 += SPAN) {
    const int64_t i0 = r0 + (int64_t)tid * GATE_PER_THREAD;
    uint32_t open = 0;
#pragma unroll
    for (int b = 0; b < GATE_PER_THREAD; ++b) {
      const int64_t i = i0 + b;
      const float v = z[i < n ? i : n - 1];   // every load issued, none under a branch
      if (i < n && v > 0.f) open |= 1u << b;
    }
    const int c = __popc(open);
    const int incl = block_scan_incl<THREADS / WAVE>(c, wsum);
    if (tid == THREADS - 1) s_total = incl;
    int64_t slot = base + incl - c;
    while (open != 0) {
      const int b = __ffs(open) - 1;
      open &= open - 1;
      kept[slot++] = (int32_t)(i0 + b);
    }
    __syncthreads();
    base += s_total;
    __syncthreads();   // s_total is rewritten by the next round
  }
  for (int64_t i = base + tid; i < n; i += THREADS) kept[i] = -1;
  if (tid == 0) *count = (int32_t)base;
}

// LDS words of select_layer's key cache for CN keys.
constexpr int sel_cache_words(int cn) { return cn > 0 ? cn + cn / 32 : 1; }

// The kept set of one layer: kept[0 .. n_keep) = the n_keep tokens of
// largest key (ties: lowest token), ascending.  Called by all THREADS (a
// multiple of 256) threads of a workgroup; cache: sel_cache_words(CN) words
// of LDS.
template <int CN, int THREADS = SEL_THREADS>
__device__ __forceinline__ void select_layer(const uint32_t* __restrict__ gkey, int64_t n,
                                             int64_t n_keep, int32_t* __restrict__ kept,
                                             uint32_t* cache, SelLds& sl) {
  constexpr bool CACHED = CN > 0;
  constexpr int WAVES = THREADS / WAVE;
  static_assert(THREADS % 256 == 0, "a thread per radix bin");
  static_assert(WAVES <= SEL_WAVES, "scan partials");
  int* hist = sl.hist;
  int* wsum = sl.wsum;
  uint32_t& s_prefix = sl.prefix;
  int& s_need = sl.need;
  if (n_keep == 0) return;
  const int tid = threadIdx.x;
  if constexpr (CACHED) {
    for (int i = tid; i < n; i += THREADS) cache[i + (i >> 5)] = gkey[i];
    __syncthreads();
  }
  auto key = [&](int64_t i) -> uint32_t {
    if constexpr (CACHED) return cache[i + (i >> 5)];
    else return gkey[i];
  };
  // every thread owns a contiguous range of tokens
  const int64_t per = (n + THREADS - 1) / THREADS;
  const int64_t i0 = min<int64_t>(n, tid * per), i1 = min<int64_t>(n, i0 + per);

  // ---- radix select (MSB first, 8 bits a pass): the n_keep-th largest T ----
  uint32_t prefix = 0, mask = 0;
  int need = (int)n_keep;   // rank from the top still to be located
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    for (int64_t i = i0; i < i1; ++i) {
      const uint32_t k = key(i);
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255], 1);
    }
    __syncthreads();
    // thread t looks at bin 255 - t: cum = keys in bins >= that bin
    const int b = 255 - tid;
    const int h = tid < 256 ? hist[b] : 0;
    const int cum = block_scan_incl<4>(h, wsum);
    if (tid < 256 && cum - h < need && need <= cum) {
      s_prefix = prefix | ((uint32_t)b << shift);
      s_need = need - (cum - h);
    }
    __syncthreads();
    prefix = s_prefix;
    need = s_need;
    mask |= 255u << shift;
  }
  const uint32_t T = prefix;   // kept: keys > T, plus the first `need` keys == T
  const int take_eq = need;

  // ---- order-preserving compaction: one block scan of per-thread counts ----
  int n_gt = 0, n_eq = 0;
  for (int64_t i = i0; i < i1; ++i) {
    const uint32_t k = key(i);
    n_gt += k > T;
    n_eq += k == T;
  }
  const int gt_before = block_scan_incl<WAVES>(n_gt, wsum) - n_gt;
  const int eq_before = block_scan_incl<WAVES>(n_eq, wsum) - n_eq;
  int g = gt_before, e = eq_before;
  for (int64_t i = i0; i < i1; ++i) {
    const uint32_t k = key(i);
    if (k > T) {
      const int pos = g + min(e, take_eq);
      if (pos < n_keep) kept[pos] = (int32_t)i;
      ++g;
    } else if (k == T) {
      if (e < take_eq) {
        const int pos = g + e;
        if (pos < n_keep) kept[pos] = (int32_t)i;
      }
      ++e;
    }
  }
}

}  // namespace lookme
