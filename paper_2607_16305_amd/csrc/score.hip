// Streaming key-scoring kernels: Level-1 routing (Eq. 5, fused arg max) and
// Level-2 primitive scoring over scene buckets (Eq. 6-7 in the dot form,
// fused top-k and softmax).  arXiv 2607.16305, Sec. 3.2.
//
// Work unit = up to 16 query rows that share one key set (all rows for
// routing; one scene's bucket tile for Level-2).  The unit's key set is
// split over the NW waves of the workgroup; each wave streams 16-key blocks
// straight from HBM into registers (the next block's chunk is requested as
// soon as the current one has been consumed by the MFMA), computes a
// 16 keys x 16 rows score tile on the matrix cores with the keys as operand A
// and the queries as operand B, and keeps per-lane running results: lane
// (g, n) of the wave sees keys 4g..4g+3 of every block for query row n.
// At the end the 4*NW per-lane candidate lists of every query row are merged
// in parallel: one thread per list, k rounds of a butterfly arg max over the
// row's threads, the winning list advancing its head.  Score matrices are
// never written to memory.
#include "common.h"
#include "kernels.h"

namespace lookme {


struct ScoreParams {
  const char* q;            // [rows, d_e]
  const char* keys;         // routing: [S, d_e]; lookup: [S, P, d_e]
  const float* bias;        // routing only, may be null
  const int32_t* perm;      // lookup: bucketed row ids
  const int32_t* offsets;   // lookup: bucket offsets [S+1]
  const int32_t* unit_scene;
  const int32_t* unit_begin;
  const int32_t* unit_count;
  int64_t rows;             // routing: number of query rows
  int64_t row_bytes;        // d_e * elem size
  int ks;                   // chunk steps per row = row_bytes / 64
  int nkeys;                // routing: S; lookup: P
  int k;                    // lookup: top-k
  int32_t* out_idx;         // routing: scene[rows]; lookup: prim[rows, k]
  float* out_w;             // lookup: w[rows, k]
};

// KS: compile-time number of chunk steps; with MASKED, steps >= ks are
// skipped (row widths that are not a power-of-two multiple of 64 bytes).
// KL: per-lane candidate list length (>= k) for lookup; 1 for routing.
// NW: waves per workgroup (they split the unit's key blocks).
template <int DT, int KS, bool MASKED, bool LOOKUP, int KL, int NW>
__global__ __launch_bounds__(NW * WAVE) void score_kernel(ScoreParams a) {
  constexpr int NL = NW * 4;                 // candidate lists per query row
  __shared__ float cand_s[NL][16][KL];
  __shared__ int cand_i[NL][16][KL];

  const int lane = threadIdx.x & 63;
  // wave index as a scalar, so that the key range (and every branch on it)
  // is known to be uniform across the wave
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 15;     // A: key row in block; B: query row in tile
  const int g = lane >> 4;     // 16-lane group: chunk 4*j + g of each step

  // ---- the unit: rows [begin, begin + nr) and its key set -----------------
  int64_t begin;
  int nr;
  const char* keys;
  if constexpr (LOOKUP) {
    const int u = xcd_remap(blockIdx.x, *a.unit_count);
    if (u < 0) return;
    const int s = a.unit_scene[u];
    begin = a.unit_begin[u];
    nr = min(16, a.offsets[s + 1] - (int)begin);
    keys = a.keys + (int64_t)s * a.nkeys * a.row_bytes;
  } else {
    const int64_t tiles = (a.rows + 15) >> 4;
    const int u = xcd_remap(blockIdx.x, (int)tiles);
    if (u < 0) return;
    begin = (int64_t)u * 16;
    nr = (int)min<int64_t>(16, a.rows - begin);
    keys = a.keys;
  }
  const int nkeys = a.nkeys;

  // ---- query fragments (operand B), kept in registers for the whole unit --
  const int my_row_slot = n < nr ? n : nr - 1;
  int64_t my_row;
  if constexpr (LOOKUP) my_row = a.perm[begin + my_row_slot];
  else my_row = begin + my_row_slot;
  u32x4_t qb[KS];
  {
    const char* qp = a.q + my_row * a.row_bytes + g * 16;
#pragma unroll
    for (int j = 0; j < KS; ++j)
      qb[j] = (!MASKED || j < a.ks) ? ld16(qp + j * 64) : u32x4_t{0, 0, 0, 0};
  }

  // ---- this wave's share of the key blocks --------------------------------
  const int nblk = (nkeys + 15) >> 4;
  const int bpw = (nblk + NW - 1) / NW;
  const int kb0 = wv * bpw;
  const int kb1 = min(nblk, kb0 + bpw);
  const int kend = min(nkeys, kb1 * 16);

  float ls[KL];
  int li[KL];
#pragma unroll
  for (int e = 0; e < KL; ++e) { ls[e] = -__builtin_inff(); li[e] = -1; }

  // loads of one 16-key block: lane (n, g) takes chunk 4j + g of key row n
  auto load_block = [&](u32x4_t (&buf)[KS], int blk) {
    const int row = min(blk * 16 + n, kend - 1);
    const char* kp = keys + (int64_t)row * a.row_bytes + g * 16;
#pragma unroll
    for (int j = 0; j < KS; ++j)
      buf[j] = (!MASKED || j < a.ks) ? ld16(kp + j * 64) : u32x4_t{0, 0, 0, 0};
  };
  // scores of one block; the buffer is refilled with block `next` right
  // after the matrix cores have read it.  The refill is unconditional (past
  // the wave's range it re-reads the last block, an L2 hit): a conditional
  // load would make the compiler wait for every load before each block.
  auto score_block = [&](u32x4_t (&buf)[KS], int next) {
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < KS; ++j)
      if (!MASKED || j < a.ks) acc = mfma_chunk<DT>(buf[j], qb[j], acc);
    load_block(buf, min(next, kb1 - 1));
    return acc;
  };
  // lane holds scores of keys blk*16 + 4g + r (r = 0..3) for query row n
  auto update = [&](f32x4_t acc, int blk) {
    float v[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = blk * 16 + 4 * g + r < kend ? acc[r] : -__builtin_inff();
    if constexpr (!LOOKUP) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int p = blk * 16 + 4 * g + r;
        float x = v[r];
        if (a.bias != nullptr && p < kend) x += a.bias[p];
        if (x > ls[0]) { ls[0] = x; li[0] = p; }
      }
    } else {
      const float best = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
      if (best > ls[KL - 1]) {
        // keys reach a lane in increasing p: strict '>' keeps the lower p
        // ahead on exact ties
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int p = blk * 16 + 4 * g + r;
          const float x = v[r];
#pragma unroll
          for (int e = KL - 1; e >= 1; --e) {
            const bool above_prev = x > ls[e - 1];
            const bool above_cur = x > ls[e];
            const float s_keep = above_cur ? x : ls[e];
            const int i_keep = above_cur ? p : li[e];
            ls[e] = above_prev ? ls[e - 1] : s_keep;
            li[e] = above_prev ? li[e - 1] : i_keep;
          }
          const bool top = x > ls[0];
          ls[0] = top ? x : ls[0];
          li[0] = top ? p : li[0];
        }
      }
    }
  };

  // The query fragments must have landed before the key stream starts, so
  // that at the loop head only key loads are outstanding, oldest first, on
  // every path into it (otherwise the per-block waits become conservative).
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  if (kb0 < kb1) {
    // two register buffers: while one block is multiplied, the next two are
    // in flight (the single-buffer form keeps 64 more VGPRs free for very
    // wide keys)
    u32x4_t ka[KS];
    load_block(ka, kb0);
    if constexpr (KS <= 16) {
      u32x4_t kbuf[KS];
      asm volatile("" ::: "memory");   // keep the first block's loads the oldest
      load_block(kbuf, min(kb0 + 1, kb1 - 1));
      // full pairs only inside the loop: every path into the loop head then
      // has the same loads outstanding (an early exit in the middle would
      // make the compiler's wait counts conservative)
      int blk = kb0;
      for (; blk + 1 < kb1; blk += 2) {
        update(score_block(ka, blk + 2), blk);
        update(score_block(kbuf, blk + 3), blk + 1);
      }
      if (blk < kb1) update(score_block(ka, blk + 2), blk);
    } else {
      for (int blk = kb0; blk < kb1; ++blk) update(score_block(ka, blk + 1), blk);
    }
  }

  // ---- merge: thread (t, L) owns list L of query row t ---------------------
  const int list = wv * 4 + g;
#pragma unroll
  for (int e = 0; e < KL; ++e) {
    cand_s[list][n][e] = ls[e];
    cand_i[list][n][e] = li[e];
  }
  __syncthreads();
  const int t = threadIdx.x / NL;          // query row of this thread
  const int L = threadIdx.x % NL;          // its list
  int head = 0;
  float hs = cand_s[L][t][0];
  int hi = cand_i[L][t][0];
  const int k = LOOKUP ? a.k : 1;
  float top_s[KL];
  int top_i[KL];
#pragma unroll
  for (int e = 0; e < KL; ++e) {
    if (e < k) {
      float bs = hs;
      int bi = hi;
#pragma unroll
      for (int d = NL / 2; d >= 1; d >>= 1) {
        const float os = __shfl_xor(bs, d, NL);
        const int oi = __shfl_xor(bi, d, NL);
        if (beats(os, oi, bs, bi)) { bs = os; bi = oi; }
      }
      top_s[e] = bs;
      top_i[e] = bi;
      if (hi == bi && hs == bs) {      // this list supplied the winner
        ++head;
        hs = head < KL ? cand_s[L][t][head] : -__builtin_inff();
        hi = head < KL ? cand_i[L][t][head] : -1;
      }
    }
  }
  if (L != 0 || t >= nr) return;
  int64_t out_row;
  if constexpr (LOOKUP) out_row = a.perm[begin + t];
  else out_row = begin + t;
  if constexpr (!LOOKUP) {
    a.out_idx[out_row] = top_i[0];
  } else {
    float sum = 0.f;
#pragma unroll
    for (int e = 0; e < KL; ++e)
      if (e < k) sum += expf(top_s[e] - top_s[0]);
    const float inv = 1.0f / sum;
    int32_t* po = a.out_idx + out_row * k;
    float* wo = a.out_w + out_row * k;
#pragma unroll
    for (int e = 0; e < KL; ++e) {
      if (e < k) {
        po[e] = top_i[e];
        wo[e] = expf(top_s[e] - top_s[0]) * inv;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

template <int DT, bool LOOKUP, int KL, int NW>
static hipError_t launch_ks(int ks, int grid, const ScoreParams& p, hipStream_t st) {
#define LOOKME_SCORE_LAUNCH(KS_, M_)                                                     \
  hipLaunchKernelGGL((score_kernel<DT, KS_, M_, LOOKUP, KL, NW>), dim3(grid), dim3(NW * WAVE), \
                     0, st, p)
  switch (ks) {
    case 4: LOOKME_SCORE_LAUNCH(4, false); break;
    case 8: LOOKME_SCORE_LAUNCH(8, false); break;
    case 16: LOOKME_SCORE_LAUNCH(16, false); break;
    case 32: LOOKME_SCORE_LAUNCH(32, false); break;
    default: LOOKME_SCORE_LAUNCH(32, true);
  }
#undef LOOKME_SCORE_LAUNCH
  return hipGetLastError();
}

template <bool LOOKUP, int KL, int NW>
static hipError_t launch_dt(int dt, int ks, int grid, const ScoreParams& p, hipStream_t st) {
  return dt == DT_BF16 ? launch_ks<DT_BF16, LOOKUP, KL, NW>(ks, grid, p, st)
                       : launch_ks<DT_F32, LOOKUP, KL, NW>(ks, grid, p, st);
}

static inline int64_t round8(int64_t x) { return (x + 7) / 8 * 8; }

hipError_t launch_route(int dt, const void* q, const void* scene_keys, const float* bias,
                        int32_t* scene, int64_t rows, int d_e, int S, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  ScoreParams p{};
  p.q = static_cast<const char*>(q);
  p.keys = static_cast<const char*>(scene_keys);
  p.bias = bias;
  p.rows = rows;
  p.row_bytes = (int64_t)d_e * (dt == DT_BF16 ? 2 : 4);
  p.ks = (int)(p.row_bytes / 64);
  p.nkeys = S;
  p.k = 1;
  p.out_idx = scene;
  const int64_t tiles = (rows + 15) / 16;
  return launch_dt<false, 1, 4>(dt, p.ks, (int)round8(tiles), p, st);
}

hipError_t launch_lookup(int dt, const void* q, const void* prim_keys, const BucketWs& ws,
                         int d_e, int P, int k, int32_t* prim, float* w, hipStream_t st) {
  ScoreParams p{};
  p.q = static_cast<const char*>(q);
  p.keys = static_cast<const char*>(prim_keys);
  p.perm = ws.perm;
  p.offsets = ws.offsets;
  p.unit_scene = ws.unit_scene;
  p.unit_begin = ws.unit_begin;
  p.unit_count = ws.unit_count;
  p.row_bytes = (int64_t)d_e * (dt == DT_BF16 ? 2 : 4);
  p.ks = (int)(p.row_bytes / 64);
  p.nkeys = P;
  p.k = k;
  p.out_idx = prim;
  p.out_w = w;
  const int grid = (int)round8(ws.max_units);
  if (k <= 4) return launch_dt<true, 4, 4>(dt, p.ks, grid, p, st);
  if (k <= 8) return launch_dt<true, 8, 4>(dt, p.ks, grid, p, st);
  if (k <= 16) return launch_dt<true, 16, 4>(dt, p.ks, grid, p, st);
  return launch_dt<true, 32, 4>(dt, p.ks, grid, p, st);
}

}  // namespace lookme
