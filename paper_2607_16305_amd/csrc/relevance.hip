// Level-2 in the paper's own form (arXiv 2607.16305, Sec. 3.2, Eq. 6-7):
// a scene-shared two-layer MLP on [v_e, e_img[j]] gives one relevance logit
// per primitive, the top k primitives by logit are kept, and their weights
// are the softmax of cos(v_e, e_{j,p}) + tanh(r_j[p]).  Launches:
//
//   tile_gemm_kernel (hidden)  a = round(ReLU([q_t, K1[scene_t]] W1^T + b1)):
//                             64 x 64 output tiles on the matrix cores, the
//                             operand-A row of token t being its query
//                             followed by its scene's key (gathered per row,
//                             K stages of 128 bytes straight into LDS);
//   relevance_topk32_kernel / relevance_topk_fused_kernel
//                             r = a W2^T + b2 and its top k per row in one
//                             pass, the rows of W2 streamed through a ring of
//                             LDS block images as the Level-2 scoring kernel
//                             streams a scene's keys, each score + b2 folded
//                             into per-lane sorted lists, no logit written:
//                             bf16 batches of 4096 rows or more with k <= 16
//                             on 32 x 32 tiles (128 rows a unit, 32 a wave),
//                             the rest on 16 x 16 tiles (64 rows a unit);
//                             with few row blocks the rows of W2 are split
//                             over several units and relevance_merge_kernel
//                             merges their lists;
//   relevance_weights_kernel  one wave per row: the k cosines against the
//                             chosen primitive keys, + tanh of the logits,
//                             softmax over the k.
// Hidden widths the fused kernel does not take (rows other than 512 or 1024
// bytes) run the logits as a product into the workspace (float32) and
// relevance_topk_kernel (one wave per row) instead.
#include "common.h"
#include "dtl.h"
#include "kernels.h"
#include "tile_gemm.h"
#include "topk.h"

namespace lookme {

// One wave per row of logits [rows, P]: lane l keeps a sorted list of the
// KL largest of logits l, l + 64, ... (visited in increasing p, so a strict
// '>' keeps the lower p first among equal values), then k rounds of a
// butterfly arg max over the 64 lists give the row's top k in order.  A
// value below T, the largest KL-th entry of the 64 lists (refreshed every
// 4 values a lane), cannot reach the row's top KL and is skipped; values
// equal to T are kept for the lower-index rule.
template <int KL>
__global__ __launch_bounds__(256) void relevance_topk_kernel(const float* __restrict__ logits,
                                                             int64_t rows, int P, int k,
                                                             int32_t* __restrict__ prim,
                                                             float* __restrict__ top) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= rows) return;
  const float* r = logits + t * P;
  float ls[KL];
  int li[KL];
#pragma unroll
  for (int e = 0; e < KL; ++e) { ls[e] = -__builtin_inff(); li[e] = -1; }
  float T = -__builtin_inff();
  for (int p0 = 0; p0 < P; p0 += 4 * WAVE) {
    float x4[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int p = p0 + u * WAVE + lane;
      x4[u] = p < P ? r[p] : -__builtin_inff();
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float x = x4[u];
      const int p = p0 + u * WAVE + lane;
      if (x > ls[KL - 1] && x >= T) {
#pragma unroll
        for (int e = KL - 1; e >= 1; --e) {
          const bool above_prev = x > ls[e - 1];
          const bool above_cur = x > ls[e];
          const float s_keep = above_cur ? x : ls[e];
          const int i_keep = above_cur ? p : li[e];
          ls[e] = above_prev ? ls[e - 1] : s_keep;
          li[e] = above_prev ? li[e - 1] : i_keep;
        }
        if (x > ls[0]) { ls[0] = x; li[0] = p; }
      }
    }
    float m = ls[KL - 1];
#pragma unroll
    for (int d = 1; d < WAVE; d <<= 1) m = fmaxf(m, __shfl_xor(m, d, 64));
    T = m;
  }
  int head = 0;
  float hs = ls[0];
  int hi = li[0];
#pragma unroll
  for (int e = 0; e < KL; ++e) {
    if (e < k) {
      float bs = hs;
      int bi = hi;
#pragma unroll
      for (int d = 1; d < WAVE; d <<= 1) {
        const float os = __shfl_xor(bs, d, 64);
        const int oi = __shfl_xor(bi, d, 64);
        if (beats(os, oi, bs, bi)) { bs = os; bi = oi; }
      }
      if (lane == 0) {
        prim[t * k + e] = bi;
        top[t * k + e] = bs;
      }
      if (hi == bi && hs == bs) {   // this lane's list supplied the winner
        ++head;
        float ns = -__builtin_inff();
        int ni = -1;
#pragma unroll
        for (int x = 1; x < KL; ++x)
          if (x == head) { ns = ls[x]; ni = li[x]; }
        hs = ns;
        hi = ni;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Fused second layer and top-k
// ---------------------------------------------------------------------------
struct RelTopkParams {
  const char* act;      // [rows, hidden] hidden activations (storage dtype)
  const char* w2;       // [P, hidden]
  const float* b2;      // [P]
  int64_t rows;
  int64_t row_bytes;    // hidden * elem size: 64 KS
  int P, k;
  int splits;           // ranges of W2 rows per row block
  int kps;              // W2 rows per range (a multiple of 16)
  int units;            // row blocks * splits
  int32_t* prim;        // [rows, k] (splits == 1)
  float* top;           // [rows, k] the k logits, best first (splits == 1)
  uint64_t* part;       // [rows, splits, k] (idx << 32 | logit bits) (splits > 1)
};

constexpr int RT_WAVES = 4, RT_THREADS = RT_WAVES * WAVE, RT_ROWS = 16 * RT_WAVES;
constexpr int RT_NBUF = 4;       // block images in the ring: three in flight while one is used
constexpr int RT_MAX_KPS = 4096; // W2 rows of one range: their b2 is kept in LDS

// One unit: rows [64 b, 64 b + 64) of the batch against W2 rows [kps s,
// kps s + kps), split s.  Wave w holds the query fragments of rows
// 64 b + 16 w + n (lane (g, n): chunks 4 j + g) and scores each 16-key block
// (keys as MFMA operand A, rows as B), adds b2 and keeps per-lane sorted
// lists of the KL best (values below the bound of fold_scores dropped; keys
// arrive in increasing index, so equal logits keep the lower index first);
// the four lists of a row are merged inside the wave.  The blocks go
// straight from global memory into a ring of LDS images (contiguous KiB
// loads, the layout of KeyImage), every wave issuing its share of each
// block's loads; W2 is read by every row block, so the loads keep the
// temporal cache policy.  The range's b2 is copied to LDS first (zero past
// its end), so the loop's only global loads are the ring's, whose count the
// waits below name.  (float32, and lists longer than 16, and small batches;
// bf16 otherwise takes the 32 x 32 form below.)
template <int DT, int KS, int KL>
__global__ __launch_bounds__(RT_THREADS) void relevance_topk_fused_kernel(RelTopkParams a) {
  constexpr int BLOCK = KS * 1024;
  constexpr int PW = KS / RT_WAVES;   // load instructions a wave issues per block
  static_assert(KS % RT_WAVES == 0 && KS <= 16, "whole load shares, fragments in registers");
  // one LDS object (ring, then the range's b2): a second one would make the
  // compiler wait for every load into LDS before each read of the ring
  __shared__ __attribute__((aligned(1024))) char smem[RT_NBUF * BLOCK + RT_MAX_KPS * 4];
  float* bl = reinterpret_cast<float*>(smem + RT_NBUF * BLOCK);
  const int u = xcd_remap(blockIdx.x, a.units);
  if (u < 0) return;
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 15, g = lane >> 4;
  const int64_t rb = u / a.splits;
  const int split = u % a.splits;
  const int64_t r0 = rb * RT_ROWS;
  const int nr = (int)min<int64_t>(RT_ROWS, a.rows - r0);
  const bool has_rows = 16 * wv < nr;   // waves without rows only help to load
  const int k0 = split * a.kps, k1 = min(a.P, k0 + a.kps);
  const int b0 = k0 >> 4, b1 = (k1 + 15) >> 4;

  for (int i = threadIdx.x; i < (b1 - b0) * 16; i += RT_THREADS)
    bl[i] = k0 + i < k1 ? a.b2[k0 + i] : 0.f;
  __syncthreads();

  u32x4_t qf[KS];
  {
    const char* row = a.act + (r0 + min(16 * wv + n, nr - 1)) * a.row_bytes + g * 16;
#pragma unroll
    for (int j = 0; j < KS; ++j) qf[j] = ld16(row + j * 64);
  }
  KeyImage im;
  im.rb = a.row_bytes;
  im.C = 4 * KS;
  im.G = im.C < 16 ? im.C : 16;
  uint32_t off[PW];
#pragma unroll
  for (int t = 0; t < PW; ++t) {
    const int i = wv + RT_WAVES * t;
    off[t] = im.src_off(i, lane, im.row_of(i, lane));
  }
  uint32_t fbase[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) fbase[t] = im.frag_off(t, g, n);
  // the loads of block blk of W2 (rows from P on read row P - 1: they are
  // masked by index when folded)
  auto issue = [&](int blk) {
    if (blk >= b1) return;
    const int row0 = blk * 16;
    const bool ragged = row0 + 16 > a.P;   // uniform
    const char* src = a.w2 + (int64_t)row0 * a.row_bytes;
    char* img = smem + ((blk - b0) % RT_NBUF) * BLOCK;
#pragma unroll
    for (int t = 0; t < PW; ++t) {
      const int i = wv + RT_WAVES * t;
      uint32_t o = off[t];
      if (ragged) {
        const int r = im.row_of(i, lane);
        o = im.src_off(i, lane, row0 + r < a.P ? r : a.P - 1 - row0);
      }
      load_lds16(src + o, img + i * 1024);
    }
  };

  float ls[KL];
  int li[KL];
#pragma unroll
  for (int e = 0; e < KL; ++e) { ls[e] = -__builtin_inff(); li[e] = -1; }
  const bool tight = a.k == KL;

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // query fragments first
#pragma unroll
  for (int b = 0; b < RT_NBUF - 1; ++b) issue(b0 + b);
  for (int blk = b0; blk < b1; ++blk) {
    // this wave's loads of block blk have landed once at most those of the
    // RT_NBUF - 2 younger blocks are outstanding (near the end, once all
    // have); the barrier makes every wave's visible and ends every read of
    // block blk - 1, whose image the next loads overwrite (a plain
    // s_barrier: the fence of __syncthreads would wait for every load)
    if (blk + RT_NBUF - 2 < b1)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"((RT_NBUF - 2) * PW) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    issue(blk + RT_NBUF - 1);
    if (has_rows) {
      const char* img = smem + ((blk - b0) % RT_NBUF) * BLOCK;
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < KS; ++j) {
        const u32x4_t kf = *reinterpret_cast<const u32x4_t*>(img + fbase[j & 3] + 256 * (j >> 2));
        acc = mfma_chunk<DT>(kf, qf[j], acc);
      }
      fold_scores<true, KL, true>(acc, blk, g, k1, bl + (blk - b0) * 16, ls, li, tight);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // no load into LDS outlives the wave
  if (!has_rows) return;
  float top_s[KL];
  int top_i[KL];
  merge_lists<KL, 2>(ls, li, a.k, 16, top_s, top_i);
  const int slot = 16 * wv + n;
  if (g != 0 || slot >= nr) return;
  const int64_t t = r0 + slot;
#pragma unroll
  for (int e = 0; e < KL; ++e) {
    if (e < a.k) {
      if (a.splits == 1) {
        a.prim[t * a.k + e] = top_i[e];
        a.top[t * a.k + e] = top_s[e];
      } else {
        a.part[(t * a.splits + split) * a.k + e] =
            ((uint64_t)(uint32_t)top_i[e] << 32) | __float_as_uint(top_s[e]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// bf16: the second layer on 32 x 32 tiles
// ---------------------------------------------------------------------------
// A unit is 128 rows (32 a wave) against a range of W2 rows taken 32 at a
// time: v_mfma_f32_32x32x16_bf16 with the 32 keys as operand A and the
// wave's 32 rows as B leaves lane (h, n) = (L >> 5, L & 31) with the 16
// scores of keys 8 j + 4 h + r (j, r < 4) of the block for row n, so a row's
// candidates sit in two lanes (n, n + 32) instead of four, each lane folds 16
// values at a time, and every key fragment read from LDS feeds a 32-row
// product: per (row, key) pair about half the list upkeep and half the LDS
// reads of the 16 x 16 form.  The keys stream through the same ring of
// 16-row LDS block images (a 32-key block is two consecutive images: key m
// in image m >> 4, row m & 15); the B operand of step s is the 16 bytes
// [32 s + 16 h, +16) of the lane's row, A the same bytes of key n's row.
// 32 WAVES-row units and a ring of WAVES x 16 KiB of 16-row images (at most
// 16 images); the library runs WAVES = 4: 128-row units, a 64 KiB ring
// (4 images at 1 KiB rows: one 32-key block in flight while one is used; 8
// at 512 bytes: three) and two workgroups a CU.  (A 256-row form with a
// 128 KiB ring, one workgroup a CU, measured slower at the Zipf shape.)
template <int KS, int WAVES>
constexpr int r32_images() {
  return (WAVES * 16 * 1024) / (KS * 1024) > 16 ? 16 : (WAVES * 16 * 1024) / (KS * 1024);
}

// 16 scores of one row (keys pbase + 8 (i >> 2) + (i & 3)) folded into the
// lane's sorted list: the largest first, the first of equal values (the
// lower key) first, one wave-wide insertion round per value that still
// beats some lane's list; values below T (see fold_scores) are dropped.
template <int KL>
__device__ __forceinline__ void fold16(float (&v)[16], int pbase, float T, float (&ls)[KL],
                                       int (&li)[KL]) {
#pragma unroll 1
  for (int round = 0; round < 16; ++round) {
    float x = v[0];
    int w = 0;
#pragma unroll
    for (int i = 1; i < 16; ++i) {
      const bool gt = v[i] > x;
      x = gt ? v[i] : x;
      w = gt ? i : w;
    }
    if (!(x >= T)) x = -__builtin_inff();
    if (!__any(x > ls[KL - 1])) break;
    const int p = pbase + 8 * (w >> 2) + (w & 3);
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
    for (int i = 0; i < 16; ++i) v[i] = i == w ? -__builtin_inff() : v[i];
  }
}

// The maximum (minimum) over lanes L and L ^ 32.
__device__ __forceinline__ float max_half(float v) {
  float a, b;
  pair32(v, a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float min_half(float v) {
  float a, b;
  pair32(v, a, b);
  return fminf(a, b);
}

template <int KS, int KL, int WAVES>
__global__ __launch_bounds__(WAVES * WAVE) void relevance_topk32_kernel(RelTopkParams a) {
  constexpr int IMG = KS * 1024;                 // one 16-row image
  constexpr int NIMG = r32_images<KS, WAVES>();  // images in the ring (an even count)
  constexpr int NB = NIMG / 2;                   // 32-key blocks in the ring
  constexpr int NS = 2 * KS;                     // 32-byte K steps a row
  constexpr int PW = 2 * KS / WAVES;             // load instructions a wave issues per block
  constexpr int ROWS = 32 * WAVES;
  static_assert(NB >= 2 && (2 * KS) % WAVES == 0, "ring of at least two blocks, whole shares");
  // one LDS object (ring, then the range's b2)
  __shared__ __attribute__((aligned(1024))) char smem[NIMG * IMG + RT_MAX_KPS * 4];
  float* bl = reinterpret_cast<float*>(smem + NIMG * IMG);
  const int u = xcd_remap(blockIdx.x, a.units);
  if (u < 0) return;
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 31, h = lane >> 5;
  const int64_t rb = u / a.splits;
  const int split = u % a.splits;
  const int64_t r0 = rb * ROWS;
  const int nr = (int)min<int64_t>(ROWS, a.rows - r0);
  const bool has_rows = 32 * wv < nr;   // waves without rows only help to load
  const int k0 = split * a.kps, k1 = min(a.P, k0 + a.kps);
  const int b0 = k0 >> 5, b1 = (k1 + 31) >> 5;

  for (int i = threadIdx.x; i < (b1 - b0) * 32; i += WAVES * WAVE)
    bl[i] = k0 + i < k1 ? a.b2[k0 + i] : 0.f;
  __syncthreads();

  u32x4_t qf[NS];
  {
    const char* row = a.act + (r0 + min(32 * wv + n, nr - 1)) * a.row_bytes + h * 16;
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[s] = ld16(row + s * 32);
  }
  KeyImage im;
  im.rb = a.row_bytes;
  im.C = 4 * KS;
  im.G = 16;
  // load instruction t of a block (t < 2 KS): image t / KS, instruction
  // t % KS of it; wave w issues t = w + WAVES q.  off: the lane's byte in
  // the block (a block of 32 whole W2 rows is contiguous)
  uint32_t off[PW];
#pragma unroll
  for (int q = 0; q < PW; ++q) {
    const int t = wv + WAVES * q;
    const int img = t / KS, i = t % KS;
    off[q] = (uint32_t)(img * 16 * a.row_bytes) + im.src_off(i, lane, im.row_of(i, lane));
  }
  // fragment of step s = 8 m + t: key n (image n >> 4, row n & 15), chunk
  // 2 s + h, at fb[t] + 256 m of the block's first image
  uint32_t fb[8];
#pragma unroll
  for (int t = 0; t < 8; ++t)
    fb[t] = (uint32_t)((n >> 4) * IMG) + (uint32_t)((n & 15) * a.row_bytes) +
            (uint32_t)(((2 * t + h) ^ (n & 15)) * 16);
  auto issue = [&](int blk) {
    if (blk >= b1) return;
    char* ring = smem + ((blk - b0) % NB) * 2 * IMG;
    if ((blk + 1) * 32 <= a.P) {   // uniform: 32 whole rows of W2
      const char* src = a.w2 + (int64_t)blk * 32 * a.row_bytes;
#pragma unroll
      for (int q = 0; q < PW; ++q) {
        const int t = wv + WAVES * q;
        load_lds16(src + off[q], ring + (t / KS) * IMG + (t % KS) * 1024);
      }
      return;
    }
#pragma unroll
    for (int q = 0; q < PW; ++q) {
      // the last block: rows from P on read row P - 1 (masked by index when
      // folded); an image wholly past P reads row P - 1 throughout
      const int t = wv + WAVES * q;
      const int img = t / KS, i = t % KS;
      const int row0 = blk * 32 + img * 16;
      const int r = im.row_of(i, lane);
      const int base_row = min(row0, a.P - 1);
      const uint32_t o = im.src_off(i, lane, min(row0 + r, a.P - 1) - base_row);
      load_lds16(a.w2 + (int64_t)base_row * a.row_bytes + o, ring + img * IMG + i * 1024);
    }
  };

  float ls[KL];
  int li[KL];
#pragma unroll
  for (int e = 0; e < KL; ++e) { ls[e] = -__builtin_inff(); li[e] = -1; }
  const bool tight = a.k == KL;

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // query fragments first
#pragma unroll
  for (int b = 0; b < NB - 1; ++b) issue(b0 + b);
  for (int blk = b0; blk < b1; ++blk) {
    // this wave's loads of block blk have landed once at most those of the
    // NB - 2 younger blocks are outstanding (near the end, once all have);
    // the barrier makes every wave's visible and ends every read of block
    // blk - 1, whose images the next loads overwrite
    if (blk + NB - 2 < b1)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NB - 2) * PW) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    issue(blk + NB - 1);
    if (has_rows) {
      const char* ring = smem + ((blk - b0) % NB) * 2 * IMG;
      f32x16_t acc = {};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const u32x4_t kf = *reinterpret_cast<const u32x4_t*>(ring + fb[s & 7] + 256 * (s >> 3));
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kf),
                                                      __builtin_bit_cast(bf16x8_t, qf[s]), acc,
                                                      0, 0, 0);
      }
      // scores + b2 (keys past k1 at -inf), then the lists
      const int pbase = blk * 32 + 4 * h;
      const float* bb = bl + (blk - b0) * 32 + 4 * h;
      float v[16];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4_t bv = *reinterpret_cast<const f32x4_t*>(bb + 8 * j);
#pragma unroll
        for (int r = 0; r < 4; ++r)
          v[4 * j + r] = pbase + 8 * j + r < k1 ? acc[4 * j + r] + bv[r] : -__builtin_inff();
      }
      float T = max_half(ls[KL - 1]);
      if (tight) T = fmaxf(T, min_half(ls[KL / 2 - 1]));
      fold16<KL>(v, pbase, T, ls, li);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // no load into LDS outlives the wave
  if (!has_rows) return;
  float top_s[KL];
  int top_i[KL];
  merge_lists<KL, 1>(ls, li, a.k, 32, top_s, top_i);
  const int slot = 32 * wv + n;
  if (h != 0 || slot >= nr) return;
  const int64_t t = r0 + slot;
#pragma unroll
  for (int e = 0; e < KL; ++e) {
    if (e < a.k) {
      if (a.splits == 1) {
        a.prim[t * a.k + e] = top_i[e];
        a.top[t * a.k + e] = top_s[e];
      } else {
        a.part[(t * a.splits + split) * a.k + e] =
            ((uint64_t)(uint32_t)top_i[e] << 32) | __float_as_uint(top_s[e]);
      }
    }
  }
}

// The lists of the ranges of a split merged per row: SPL lanes a row (the
// next power of two >= splits), 64 / SPL rows a wave; lane j < splits of a
// row's group holds range j's list, the butterfly of merge_lists over the
// group orders their union by the rule of one unit over all of W2 (a range
// with fewer than k rows pads its list with -inf, which the P >= k real
// logits outrank).
template <int KL, int LOG>
__global__ __launch_bounds__(256) void relevance_merge_kernel(const uint64_t* __restrict__ part,
                                                              int64_t rows, int splits, int k,
                                                              int32_t* __restrict__ prim,
                                                              float* __restrict__ top) {
  constexpr int SPL = 1 << LOG;
  const int lane = threadIdx.x & 63;
  const int j = lane & (SPL - 1);
  const int64_t t = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> LOG;
  const bool live = t < rows;   // lanes past the last row join the shuffles with empty lists
  float ls[KL], ms[KL];
  int li[KL], mi[KL];
#pragma unroll
  for (int e = 0; e < KL; ++e) {
    ls[e] = -__builtin_inff();
    li[e] = -1;
    if (live && j < splits && e < k) {
      const uint64_t v = part[(t * splits + j) * k + e];
      ls[e] = __uint_as_float((uint32_t)v);
      li[e] = (int)(v >> 32);
    }
  }
  merge_lists<KL, LOG>(ls, li, k, 1, ms, mi);
  if (!live || j != 0) return;
#pragma unroll
  for (int e = 0; e < KL; ++e)
    if (e < k) {
      prim[t * k + e] = mi[e];
      top[t * k + e] = ms[e];
    }
}

// Ranges of W2 rows per row block: enough units to fill the chip's 512
// resident workgroups, each range at least 128 rows (and k), and as many as
// keep a range's b2 within its LDS space; 0 when that takes more than 16.
static int relevance_splits(int64_t row_blocks, int P, int k) {
  int splits = 1;
  while (splits < 16 && row_blocks * splits < 512 && P / (2 * splits) >= 128 &&
         P / (2 * splits) >= k)
    splits *= 2;
  while (splits <= 16 && (P + splits - 1) / splits > RT_MAX_KPS) splits *= 2;
  return splits <= 16 ? splits : 0;
}

// The split's lists merged per row (nothing to do for one range).
template <int KL>
static hipError_t launch_merge(const RelTopkParams& p, hipStream_t st) {
  if (p.splits > 1) {
    const int log = p.splits <= 2 ? 1 : p.splits <= 4 ? 2 : p.splits <= 8 ? 3 : 4;
    const dim3 grid((unsigned)(((p.rows << log) + 255) / 256));
    if (log == 1)
      hipLaunchKernelGGL((relevance_merge_kernel<KL, 1>), grid, dim3(256), 0, st, p.part, p.rows,
                         p.splits, p.k, p.prim, p.top);
    else if (log == 2)
      hipLaunchKernelGGL((relevance_merge_kernel<KL, 2>), grid, dim3(256), 0, st, p.part, p.rows,
                         p.splits, p.k, p.prim, p.top);
    else if (log == 3)
      hipLaunchKernelGGL((relevance_merge_kernel<KL, 3>), grid, dim3(256), 0, st, p.part, p.rows,
                         p.splits, p.k, p.prim, p.top);
    else
      hipLaunchKernelGGL((relevance_merge_kernel<KL, 4>), grid, dim3(256), 0, st, p.part, p.rows,
                         p.splits, p.k, p.prim, p.top);
  }
  return hipGetLastError();
}

template <int DT, int KS, int KL>
static hipError_t launch_topk16(const RelTopkParams& p0, float* part_ws, hipStream_t st) {
  RelTopkParams p = p0;
  const int64_t row_blocks = (p.rows + RT_ROWS - 1) / RT_ROWS;
  p.splits = relevance_splits(row_blocks, p.P, p.k);
  if (p.splits < 1) return hipErrorInvalidValue;
  p.kps = ((p.P + p.splits - 1) / p.splits + 15) / 16 * 16;
  p.splits = (p.P + p.kps - 1) / p.kps;   // no empty range
  // the lists of a split live in the logits' workspace ([rows, P] float32)
  if (p.splits > 1 && (int64_t)p.splits * p.k * 2 > p.P) return hipErrorInvalidValue;
  p.units = (int)(row_blocks * p.splits);
  p.part = reinterpret_cast<uint64_t*>(part_ws);
  hipLaunchKernelGGL((relevance_topk_fused_kernel<DT, KS, KL>),
                     dim3((unsigned)((p.units + 7) / 8 * 8)), dim3(RT_THREADS), 0, st, p);
  return launch_merge<KL>(p, st);
}

template <int KS, int KL, int WAVES>
static hipError_t launch_topk32(const RelTopkParams& p0, float* part_ws, hipStream_t st) {
  RelTopkParams p = p0;
  const int64_t row_blocks = (p.rows + 32 * WAVES - 1) / (32 * WAVES);
  p.splits = relevance_splits(row_blocks, p.P, p.k);
  if (p.splits < 1) return hipErrorInvalidValue;
  p.kps = ((p.P + p.splits - 1) / p.splits + 31) / 32 * 32;
  p.splits = (p.P + p.kps - 1) / p.kps;   // no empty range
  if (p.kps > RT_MAX_KPS) return hipErrorInvalidValue;
  if (p.splits > 1 && (int64_t)p.splits * p.k * 2 > p.P) return hipErrorInvalidValue;
  p.units = (int)(row_blocks * p.splits);
  p.part = reinterpret_cast<uint64_t*>(part_ws);
  hipLaunchKernelGGL((relevance_topk32_kernel<KS, KL, WAVES>),
                     dim3((unsigned)((p.units + 7) / 8 * 8)), dim3(WAVES * WAVE), 0, st, p);
  return launch_merge<KL>(p, st);
}

template <int DT, int KS, int KL>
static hipError_t launch_topk_fused(const RelTopkParams& p, float* part_ws, hipStream_t st) {
  if constexpr (DT == DT_BF16 && KL <= 16)
    if (p.rows >= 4096) return launch_topk32<KS, KL, 4>(p, part_ws, st);
  return launch_topk16<DT, KS, KL>(p, part_ws, st);
}

// One wave per row: cosines of q_t with its k chosen primitive keys, plus
// tanh of their logits (read from w), softmax over the k, written to w.
template <int DT, int K>
__global__ __launch_bounds__(256) void relevance_weights_kernel(
    const char* __restrict__ q, const int32_t* __restrict__ scene,
    const char* __restrict__ prim_keys, const int32_t* __restrict__ prim, float* __restrict__ w,
    int64_t rows, int S, int P, int k, int64_t q_bytes) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= rows) return;
  int s = scene[t];
  s = s < 0 ? 0 : (s >= S ? S - 1 : s);
  const char* rows_base[K];
#pragma unroll
  for (int e = 0; e < K; ++e) {
    int p = e < k ? prim[t * k + e] : 0;
    p = p < 0 ? 0 : (p >= P ? P - 1 : p);
    rows_base[e] = prim_keys + ((int64_t)s * P + p) * q_bytes;
  }
  float qq = 0.f, dot[K], ee[K];
#pragma unroll
  for (int e = 0; e < K; ++e) dot[e] = ee[e] = 0.f;
  const int chunks = (int)(q_bytes / 16);
  auto accum = [&](u32x4_t u, u32x4_t v, float& d, float& n) {
    if constexpr (DT == DT_BF16) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float a0 = bf16lo(u[c]), a1 = bf16hi(u[c]), b0 = bf16lo(v[c]), b1 = bf16hi(v[c]);
        d = fmaf(a0, b0, fmaf(a1, b1, d));
        n = fmaf(b0, b0, fmaf(b1, b1, n));
      }
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float a0 = as_f32(u[c]), b0 = as_f32(v[c]);
        d = fmaf(a0, b0, d);
        n = fmaf(b0, b0, n);
      }
    }
  };
  for (int c = lane; c < chunks; c += WAVE) {
    const u32x4_t qv = ld16(q + t * q_bytes + (int64_t)c * 16);
    float unused = 0.f;
    accum(qv, qv, unused, qq);
#pragma unroll
    for (int e = 0; e < K; ++e)
      if (e < k) accum(qv, ld16(rows_base[e] + (int64_t)c * 16), dot[e], ee[e]);
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    qq += __shfl_xor(qq, d, 64);
#pragma unroll
    for (int e = 0; e < K; ++e) {
      dot[e] += __shfl_xor(dot[e], d, 64);
      ee[e] += __shfl_xor(ee[e], d, 64);
    }
  }
  // lane e < k owns entry e
  float z = -__builtin_inff();
#pragma unroll
  for (int e = 0; e < K; ++e) {
    if (e < k && lane == e) {
      const float den = sqrtf(qq) * sqrtf(ee[e]);
      const float c = den > 0.f ? dot[e] / den : 0.f;
      z = c + tanhf(w[t * k + e]);
    }
  }
  float m = z;
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) m = fmaxf(m, __shfl_xor(m, d, 64));
  const float ex = lane < k ? expf(z - m) : 0.f;
  float sum = ex;
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) sum += __shfl_xor(sum, d, 64);
  if (lane < k) w[t * k + lane] = ex / sum;
}

// The same weights with the products on the matrix cores, for rows of
// 64 KS bytes and k < 32: one wave per row.  The row's k chosen keys and its
// query form the rows of 16-row operand tiles (key m at row m, the query at
// row k; NT = 1 tile when k < 16, else 2), gathered straight into MFMA
// fragments (lane (g, n): tile row n, chunks 4 j + g), and the products of
// the tiles with themselves give every number the weights need: a key's
// squared norm on the diagonal, key . q in the query's column, ||q||^2 at
// the query's diagonal entry.  One gather of k + 1 rows, no cross-lane sums;
// the vector form (below) covers the other widths and k = 32.  At k = 16
// (NT = 0) the keys fill one tile and every lane also loads its query
// fragments: key . q is the product with the query in every column, ||q||^2
// comes from the fragments (a second tile holding the query alone costs
// more load instructions than this).
template <int DT, int KS, int NT>
__global__ __launch_bounds__(256) void relevance_weights_mma_kernel(
    const char* __restrict__ q, const int32_t* __restrict__ scene,
    const char* __restrict__ prim_keys, const int32_t* __restrict__ prim, float* __restrict__ w,
    int64_t rows, int S, int P, int k) {
  constexpr int64_t RB = 64 * KS;
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= rows) return;
  const int n = lane & 15, g = lane >> 4;
  int s = scene[t];
  s = s < 0 ? 0 : (s >= S ? S - 1 : s);
  if constexpr (NT == 0) {
    u32x4_t kf[KS], qf[KS];
    int p = prim[t * k + n];
    p = p < 0 ? 0 : (p >= P ? P - 1 : p);
    const char* kr_ = prim_keys + ((int64_t)s * P + p) * RB + g * 16;
    const char* qr = q + t * RB + g * 16;
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      kf[j] = ld16(kr_ + j * 64);
      qf[j] = ld16(qr + j * 64);
    }
    float qq = 0.f;
#pragma unroll
    for (int j = 0; j < KS; ++j) qq = chunk_sumsq<DT>(qf[j], qq);
    qq = sum_lane_groups(qq);
    f32x4_t dq = {0.f, 0.f, 0.f, 0.f}, kk = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      dq = mfma_chunk<DT>(kf[j], qf[j], dq);   // [key 4g + r][any column] = key . q
      kk = mfma_chunk<DT>(kf[j], kf[j], kk);   // [key 4g + r][key n]
    }
    float z[4], mx = -__builtin_inff();
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float ee = __shfl(kk[r], 16 * g + 4 * g + r, 64);
      const float den = sqrtf(qq) * sqrtf(ee);
      const float c = den > 0.f ? dq[r] / den : 0.f;
      z[r] = c + tanhf(w[t * 16 + 4 * g + r]);
      mx = fmaxf(mx, z[r]);
    }
    mx = max_lane_groups(mx);
    float ex[4], sum = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      ex[r] = expf(z[r] - mx);
      sum += ex[r];
    }
    sum = sum_lane_groups(sum);
    if (n == 0)
#pragma unroll
      for (int r = 0; r < 4; ++r) w[t * 16 + 4 * g + r] = ex[r] / sum;
    return;
  }
  constexpr int NTT = NT > 0 ? NT : 1;
  // operand rows: m < k key prim[m], m == k the query, past it zero
  u32x4_t f[NTT][KS];
#pragma unroll
  for (int T = 0; T < NTT; ++T) {
    const int m = 16 * T + n;
    const char* src = q + t * RB;
    if (m < k) {
      int p = prim[t * k + m];
      p = p < 0 ? 0 : (p >= P ? P - 1 : p);
      src = prim_keys + ((int64_t)s * P + p) * RB;
    }
#pragma unroll
    for (int j = 0; j < KS; ++j)
      f[T][j] = m <= k ? ld16(src + g * 16 + j * 64) : u32x4_t{0, 0, 0, 0};
  }
  // products: G[T] = tile T x tile T^T, and with two tiles C = tile 0 x
  // tile 1^T (keys 0..15 against keys 16.. and the query); lane (g, n) holds
  // [row 4g + r][row n]
  const int kr = k & 15;   // the query's row in its tile (tile k >> 4)
  f32x4_t G[NTT], C = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int T = 0; T < NTT; ++T) {
    G[T] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < KS; ++j) G[T] = mfma_chunk<DT>(f[T][j], f[T][j], G[T]);
  }
  if constexpr (NT == 2) {
#pragma unroll
    for (int j = 0; j < KS; ++j) C = mfma_chunk<DT>(f[0][j], f[1][j], C);
  }
  // ||q||^2: the query's diagonal entry, in lane (kr >> 2, kr), element kr & 3
  float qq = 0.f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float v = __shfl(G[NTT - 1][r], 16 * (kr >> 2) + kr, 64);
    qq = (kr & 3) == r ? v : qq;
  }
  // lanes n == kr hold key (4g + r) . q of each tile: tile k >> 4 in its own
  // product, tile 0 (when the query is in tile 1) in C
  float z[NTT][4];
#pragma unroll
  for (int T = 0; T < NTT; ++T) {
    const f32x4_t dq = (NT == 2 && T == 0) ? C : G[T];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      // ||key 4g + r||^2 sits in lane (g, 4g + r), element r, of G[T]
      const float ee = __shfl(G[T][r], 16 * g + 4 * g + r, 64);
      const int m = 16 * T + 4 * g + r;
      const float den = sqrtf(qq) * sqrtf(ee);
      const float c = den > 0.f ? dq[r] / den : 0.f;
      z[T][r] = m < k ? c + tanhf(w[t * k + m]) : -__builtin_inff();
    }
  }
  float mx = -__builtin_inff();
#pragma unroll
  for (int T = 0; T < NTT; ++T)
#pragma unroll
    for (int r = 0; r < 4; ++r) mx = fmaxf(mx, z[T][r]);
  mx = max_lane_groups(mx);
  float ex[NTT][4], sum = 0.f;
#pragma unroll
  for (int T = 0; T < NTT; ++T)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      ex[T][r] = 16 * T + 4 * g + r < k ? expf(z[T][r] - mx) : 0.f;
      sum += ex[T][r];
    }
  sum = sum_lane_groups(sum);
  if (n != kr) return;
#pragma unroll
  for (int T = 0; T < NTT; ++T)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = 16 * T + 4 * g + r;
      if (m < k) w[t * k + m] = ex[T][r] / sum;
    }
}

static hipError_t launch_relevance_weights(int dt, const void* q, const int32_t* scene,
                                           const void* prim_keys, const int32_t* prim, float* w,
                                           int64_t rows, int S, int P, int k, int64_t q_bytes,
                                           hipStream_t st) {
  const dim3 wgrid((unsigned)((rows + 3) / 4));
  if ((q_bytes == 1024 || q_bytes == 512) && k < 32) {
#define LOOKME_RWM(DT_, KS_)                                                                     \
  do {                                                                                           \
    if (k < 16)                                                                                  \
      hipLaunchKernelGGL((relevance_weights_mma_kernel<DT_, KS_, 1>), wgrid, dim3(256), 0, st,   \
                         static_cast<const char*>(q), scene,                                     \
                         static_cast<const char*>(prim_keys), prim, w, rows, S, P, k);           \
    else if (k == 16)                                                                            \
      hipLaunchKernelGGL((relevance_weights_mma_kernel<DT_, KS_, 0>), wgrid, dim3(256), 0, st,   \
                         static_cast<const char*>(q), scene,                                     \
                         static_cast<const char*>(prim_keys), prim, w, rows, S, P, k);           \
    else                                                                                         \
      hipLaunchKernelGGL((relevance_weights_mma_kernel<DT_, KS_, 2>), wgrid, dim3(256), 0, st,   \
                         static_cast<const char*>(q), scene,                                     \
                         static_cast<const char*>(prim_keys), prim, w, rows, S, P, k);           \
  } while (0)
    if (dt == DT_BF16) {
      if (q_bytes == 1024) LOOKME_RWM(DT_BF16, 16);
      else LOOKME_RWM(DT_BF16, 8);
    } else {
      if (q_bytes == 1024) LOOKME_RWM(DT_F32, 16);
      else LOOKME_RWM(DT_F32, 8);
    }
#undef LOOKME_RWM
    return hipGetLastError();
  }
#define LOOKME_RW(DT_, K_)                                                                       \
  hipLaunchKernelGGL((relevance_weights_kernel<DT_, K_>), wgrid, dim3(256), 0, st,             \
                     static_cast<const char*>(q), scene, static_cast<const char*>(prim_keys), \
                     prim, w, rows, S, P, k, q_bytes)
  if (dt == DT_BF16) {
    if (k <= 4) LOOKME_RW(DT_BF16, 4);
    else if (k <= 8) LOOKME_RW(DT_BF16, 8);
    else if (k <= 16) LOOKME_RW(DT_BF16, 16);
    else LOOKME_RW(DT_BF16, 32);
  } else {
    if (k <= 4) LOOKME_RW(DT_F32, 4);
    else if (k <= 8) LOOKME_RW(DT_F32, 8);
    else if (k <= 16) LOOKME_RW(DT_F32, 16);
    else LOOKME_RW(DT_F32, 32);
  }
#undef LOOKME_RW
  return hipGetLastError();
}

hipError_t launch_relevance_table(int dt, const void* scene_keys, const RelevanceMlp& mlp, int S,
                                  int d_e, float* tab, hipStream_t st) {
  const int es = dt == DT_BF16 ? 2 : 4;
  // tab = K1 W1b^T + b1: W1 is [hidden, 2 d_e], W1b its last d_e columns
  TileGemmParams g{};
  g.a0 = static_cast<const char*>(scene_keys);
  g.b = static_cast<const char*>(mlp.w1) + (int64_t)d_e * es;
  g.b_ld = 2 * (int64_t)d_e * es;
  g.bias = mlp.b1;
  g.out = reinterpret_cast<char*>(tab);
  g.rows = S;
  g.a_bytes = (int64_t)d_e * es;
  g.k_bytes = g.a_bytes;
  g.cols = mlp.hidden;
  g.ksplit = (int)(g.a_bytes / TG_KB);
  g.tiles = (int)(((S + TgShape::BM - 1) / TgShape::BM) *
                  ((mlp.hidden + TgShape::BN - 1) / TgShape::BN));
  return launch_tile_gemm<EPI_LOGIT>(dt, g, 1, st);
}

hipError_t launch_relevance(int dt, const void* q, const int32_t* scene, const float* tab,
                            const void* prim_keys, const RelevanceMlp& mlp, int64_t rows, int d_e,
                            int S, int P, int k, void* act, int32_t* prim, float* w,
                            float* logits, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  const int es = dt == DT_BF16 ? 2 : 4;
  const int64_t rt = (rows + TgShape::BM - 1) / TgShape::BM;
  // hidden layer: ReLU(q W1a^T + tab[scene]), W1a the first d_e columns of W1
  // (the scene half and b1 are in the table: half the first layer's
  // products of the joint form, computed once per scene instead of per row)
  TileGemmParams g1{};
  g1.a0 = static_cast<const char*>(q);
  g1.sel = scene;
  g1.tab = tab;
  g1.b = static_cast<const char*>(mlp.w1);
  g1.b_ld = 2 * (int64_t)d_e * es;
  g1.out = static_cast<char*>(act);
  g1.rows = rows;
  g1.a_bytes = (int64_t)d_e * es;
  g1.k_bytes = g1.a_bytes;
  g1.sel_rows = S;
  g1.cols = mlp.hidden;
  g1.ksplit = (int)(g1.a_bytes / TG_KB);
  g1.tiles = (int)(rt * ((mlp.hidden + TgShape::BN - 1) / TgShape::BN));
  hipError_t e = launch_tile_gemm<EPI_ACT_TAB>(dt, g1, 1, st);
  if (e != hipSuccess) return e;
  const int64_t hb = (int64_t)mlp.hidden * es;
  if ((hb == 1024 || hb == 512) && relevance_splits((rows + 63) / 64, P, k) > 0) {
    // second layer and top-k fused (no float32 logits written); the ranges'
    // lists of a split go to the logits' workspace
    RelTopkParams p{};
    p.act = static_cast<const char*>(act);
    p.w2 = static_cast<const char*>(mlp.w2);
    p.b2 = mlp.b2;
    p.rows = rows;
    p.row_bytes = hb;
    p.P = P;
    p.k = k;
    p.prim = prim;
    p.top = w;
#define LOOKME_RT(KS_)                                                                 \
  do {                                                                                 \
    if (dt == DT_BF16) {                                                               \
      if (k <= 4) e = launch_topk_fused<DT_BF16, KS_, 4>(p, logits, st);               \
      else if (k <= 8) e = launch_topk_fused<DT_BF16, KS_, 8>(p, logits, st);          \
      else if (k <= 16) e = launch_topk_fused<DT_BF16, KS_, 16>(p, logits, st);        \
      else e = launch_topk_fused<DT_BF16, KS_, 32>(p, logits, st);                     \
    } else {                                                                           \
      if (k <= 4) e = launch_topk_fused<DT_F32, KS_, 4>(p, logits, st);                \
      else if (k <= 8) e = launch_topk_fused<DT_F32, KS_, 8>(p, logits, st);           \
      else if (k <= 16) e = launch_topk_fused<DT_F32, KS_, 16>(p, logits, st);         \
      else e = launch_topk_fused<DT_F32, KS_, 32>(p, logits, st);                      \
    }                                                                                  \
  } while (0)
    if (hb == 1024) LOOKME_RT(16);
    else LOOKME_RT(8);
#undef LOOKME_RT
    if (e != hipSuccess) return e;
    return launch_relevance_weights(dt, q, scene, prim_keys, prim, w, rows, S, P, k,
                                    (int64_t)d_e * es, st);
  }
  // logits: r = a W2^T + b2, float32
  TileGemmParams g2{};
  g2.a0 = static_cast<const char*>(act);
  g2.b = static_cast<const char*>(mlp.w2);
  g2.bias = mlp.b2;
  g2.out = reinterpret_cast<char*>(logits);
  g2.rows = rows;
  g2.a_bytes = (int64_t)mlp.hidden * es;
  g2.k_bytes = g2.a_bytes;
  g2.cols = P;
  g2.ksplit = (int)(g2.k_bytes / TG_KB);
  g2.tiles = (int)(rt * ((P + TgShape::BN - 1) / TgShape::BN));
  // large products on the projection's 256 x 256 tiles, small ones here
  if (!launch_logits_gemm(dt, act, mlp.w2, mlp.b2, logits, rows, P, g2.k_bytes, st))
    e = launch_tile_gemm<EPI_LOGIT>(dt, g2, 1, st);
  else
    e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 wgrid((unsigned)((rows + 3) / 4));
  if (k <= 4)
    hipLaunchKernelGGL(relevance_topk_kernel<4>, wgrid, dim3(256), 0, st, logits, rows, P, k, prim, w);
  else if (k <= 8)
    hipLaunchKernelGGL(relevance_topk_kernel<8>, wgrid, dim3(256), 0, st, logits, rows, P, k, prim, w);
  else if (k <= 16)
    hipLaunchKernelGGL(relevance_topk_kernel<16>, wgrid, dim3(256), 0, st, logits, rows, P, k, prim, w);
  else
    hipLaunchKernelGGL(relevance_topk_kernel<32>, wgrid, dim3(256), 0, st, logits, rows, P, k, prim, w);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_relevance_weights(dt, q, scene, prim_keys, prim, w, rows, S, P, k,
                                  (int64_t)d_e * es, st);
}

}  // namespace lookme
