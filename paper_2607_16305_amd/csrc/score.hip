// Key-scoring kernels: Level-1 routing (Eq. 5, fused arg max) and Level-2
// primitive scoring over scene buckets (Eq. 6-7 in the dot form, fused
// top-k and softmax).  arXiv 2607.16305, Sec. 3.2.
//
// Every product is a 16 keys x 16 query rows tile on the matrix cores, the
// keys as MFMA operand A and the queries as operand B, so that lane (g, n)
// of a wave holds the scores of keys 4g..4g+3 of a block for query row n and
// keeps its own running arg max / sorted top-k list (keys reach a lane in
// increasing index, so a strict '>' keeps the lower index on exact ties).
// Score matrices are never written to memory.  A work unit is a set of query
// rows that share one key set (all rows for routing, one scene's bucket for
// Level-2); units come in two modes:
//
//  * streaming (up to 16 rows): the unit's key blocks are split over the 4
//    waves; each wave streams its 16-key blocks straight from HBM into
//    registers, two blocks in flight.  At the end the 16 per-lane lists of
//    every row are merged in parallel (one thread per list, k rounds of a
//    butterfly arg max).  Suits the many small buckets: all 4 waves compute.
//  * shared (64 rows for Level-2, 128 for routing): every 16-key block is
//    loaded once by the whole workgroup into an LDS tile (double-buffered,
//    two blocks in flight in registers) and read by every wave, each holding
//    one 16-row query tile (two for routing); the key stream is paid once for
//    up to 4 (8) tiles.  Lists are merged inside the wave (4 lanes per row).
//    Suits large buckets and routing of many rows.
//
// COS (the cosine of Eq. 5 and Eq. 7 instead of the dot product): each
// score is scaled by 1/||q|| 1/||k||, both norms taken from the fragments the
// matrix cores already read (a query row's once per unit, a key's once per
// 16-key block, over the 4 lane groups that hold its chunks); a zero vector
// gives 0.  No extra load, so the load pipelines are those of the dot form.
#include <hip/hip_ext.h>

#include "common.h"
#include "crit.h"
#include "dtl.h"
#include "kernels.h"
#include "route_merge.h"
#include "topk.h"

namespace lookme {

constexpr int SC_WAVES = 4;
constexpr int SH_LDS_BYTES = 48 * 1024;   // LDS for a shared unit's key block images
constexpr int SC_THREADS = SC_WAVES * WAVE;

struct ScoreParams {
  const char* q;            // [rows, d_e]
  const char* keys;         // routing: [S, d_e]; lookup: [S, P, d_e]
  const float* bias;        // routing only, may be null
  const int32_t* perm;      // lookup: bucketed row ids
  const int32_t* offsets;   // lookup: bucket offsets [S+1]
  const int32_t* unit_scene;
  const int32_t* unit_begin;
  int32_t* unit_count;      // lookup: [3] (kernels.h); [2] counts the parts taken
  uint64_t* split_part;     // lookup: the cut units' partial lists (SPLIT_PART_BYTES)
  int32_t* split_row;       // lookup: [SPLIT_UNITS, 16] output row + 1 of a cut unit's rows, else 0
  int64_t rows;             // routing: number of query rows
  int64_t row_bytes;        // d_e * elem size
  int ks;                   // chunk steps per row = row_bytes / 64
  int nkeys;                // routing: S; lookup: P
  int k;                    // lookup: top-k
  int route_rows;           // routing: rows per unit (16: streaming, else shared)
  int route_splits;         // routing, streaming: key ranges per 16-row tile
  int route_kps;            // routing, streaming: keys per range (multiple of 64)
  uint64_t* route_part;     // routing, splits > 1: [tiles, splits, 16] (idx, score)
  int32_t* route_count;     // routing, splits > 1: [tiles] arrivals, left at zero
  int shared_rows;          // lookup: rows of a shared unit (at most)
  int cos;                  // cosine scores (Eq. 5, Eq. 7) instead of dot products
  int32_t* out_idx;         // routing: scene[rows]; lookup: prim[rows, k]
  float* out_w;             // lookup: w[rows, k]
  // lookup with the select of the batch riding along (side0 > 0): launch
  // slot side0 + l selects layer l's kept set
  int side0;
  int64_t crit_n, n_keep;
  const uint32_t* crit_key; // [layers * crit_n] criticality keys (gate: logits)
  int32_t* kept;            // [layers, n_keep] (gate: [layers, crit_n])
  int32_t* gate_count;      // null: top-n_keep select; else the gate's counts [layers]
};

template <int KS, bool MASKED>
__device__ __forceinline__ void load_row_frags(u32x4_t (&f)[KS], const char* row_ptr, int g,
                                               int ks) {
  const char* p = row_ptr + g * 16;
#pragma unroll
  for (int j = 0; j < KS; ++j) f[j] = (!MASKED || j < ks) ? ld16(p + j * 64) : u32x4_t{0, 0, 0, 0};
}


template <bool LOOKUP, int KL>
__device__ __forceinline__ void write_row(const ScoreParams& a, int64_t out_row,
                                          const float (&top_s)[KL], const int (&top_i)[KL]) {
  if constexpr (!LOOKUP) {
    a.out_idx[out_row] = top_i[0];
  } else {
    const int k = a.k;
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

template <bool LOOKUP>
__device__ __forceinline__ int64_t row_id(const ScoreParams& a, int64_t begin, int slot) {
  if constexpr (LOOKUP) return a.perm[begin + slot];
  else return begin + slot;
}

// The partial list slot of row t of part `part` of cut unit `cut`: SPLIT_KMAX
// entries (index << 32 | score bits), sorted as the outputs.
__device__ __forceinline__ uint64_t* split_slot(const ScoreParams& a, int cut, int part, int t) {
  return a.split_part + ((int64_t)(cut * SPLIT_PARTS + part) * UNIT_STREAM_ROWS + t) * SPLIT_KMAX;
}


// ---------------------------------------------------------------------------
// Level-2 key blocks in LDS (the image layout: KeyImage, topk.h)
// ---------------------------------------------------------------------------

template <int KS, bool MASKED>
__device__ __forceinline__ KeyImage key_image(const ScoreParams& a) {
  KeyImage im;
  im.rb = a.row_bytes;
  im.C = MASKED ? 4 * a.ks : 4 * KS;
  const int low = im.C & -im.C;
  im.G = low < 16 ? low : 16;
  return im;
}

// Loads the block of key rows [row0, row0 + 16) (rows from kend on read row
// kend - 1: they are masked by index when scored) into `img`: instructions
// i = i0, i0 + istep, ... < ks.  off[t] holds src_off for instruction
// i0 + istep t of an unclamped block.  nt (uniform): the nontemporal hint,
// for keys no other unit reads; the units of a bucket cut into several read
// the same keys and keep the temporal policy, so the later ones find them
// in L2 (measured: 4-layer workload 318 -> 302 us; with the hint on every
// unit the single-unit buckets run faster, multi-scale 195 -> 174 us).
template <int KS, bool MASKED, int NT>
__device__ __forceinline__ void load_key_block(const KeyImage& im, const ScoreParams& a,
                                               const char* keys, int row0, int kend,
                                               const uint32_t (&off)[NT], int i0, int istep,
                                               char* img, int lane, bool nt = true) {
  const char* src = keys + (int64_t)row0 * im.rb;
  const bool ragged = row0 + 16 > kend;   // uniform
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int i = i0 + istep * t;
    if (MASKED && i >= a.ks) break;
    uint32_t o = off[t];
    if (ragged) {
      const int r = im.row_of(i, lane);
      const int rr = row0 + r < kend ? r : kend - 1 - row0;
      o = im.src_off(i, lane, rr);
    }
    if (nt) load_lds16_nt(src + o, img + i * 1024);
    else load_lds16(src + o, img + i * 1024);
  }
}

// ---------------------------------------------------------------------------
// Streaming mode: <= 16 rows, key blocks split over the waves
// ---------------------------------------------------------------------------
// key0, nkeys: the unit's key range (routing may split the keys; Level-2
// units take all P keys of their scene, key0 = 0).
template <int DT, int KS, bool MASKED, bool LOOKUP, int KL, bool COS>
__device__ __forceinline__ void stream_unit(const ScoreParams& a, char* smem, int64_t begin,
                                            int nr, const char* keys, int key0, int nkeys,
                                            int split) {
  constexpr int NL = SC_WAVES * 4;   // candidate lists per query row
  float (*cand_s)[16][KL] = reinterpret_cast<float (*)[16][KL]>(smem);
  int (*cand_i)[16][KL] = reinterpret_cast<int (*)[16][KL]>(smem + NL * 16 * KL * 4);
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 15, g = lane >> 4;
  const float* bias = a.bias != nullptr ? a.bias + key0 : nullptr;

  u32x4_t qb[KS];
  load_row_frags<KS, MASKED>(qb, a.q + row_id<LOOKUP>(a, begin, n < nr ? n : nr - 1) * a.row_bytes,
                             g, a.ks);

  const int nblk = (nkeys + 15) >> 4;
  const int bpw = (nblk + SC_WAVES - 1) / SC_WAVES;
  const int kb0 = wv * bpw;
  const int kb1 = min(nblk, kb0 + bpw);
  const int kend = min(nkeys, kb1 * 16);

  float ls[KL];
  int li[KL];
#pragma unroll
  for (int e = 0; e < KL; ++e) { ls[e] = -__builtin_inff(); li[e] = -1; }

  auto load_block = [&](u32x4_t (&buf)[KS], int blk) {
    const int row = min(blk * 16 + n, kend - 1);
    load_row_frags<KS, MASKED>(buf, keys + (int64_t)row * a.row_bytes, g, a.ks);
  };
  // The buffer is refilled with block `next` right after the matrix cores
  // have read it.  The refill is unconditional (past the wave's range it
  // re-reads the last block, an L2 hit): a conditional load would make the
  // compiler wait for every load before each block.
  float qinv = 0.f;   // COS: 1 / ||q|| of the lane's row (after the query landed)
  auto score_block = [&](u32x4_t (&buf)[KS], int next) {
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    float knsq = 0.f;
#pragma unroll
    for (int j = 0; j < KS; ++j)
      if (!MASKED || j < a.ks) {
        acc = mfma_chunk<DT>(buf[j], qb[j], acc);
        if constexpr (COS) knsq = chunk_sumsq<DT>(buf[j], knsq);
      }
    load_block(buf, min(next, kb1 - 1));
    if constexpr (COS) acc = cos_scale(acc, qinv, sum_lane_groups(knsq), g);
    return acc;
  };

  // The query fragments must have landed before the key stream starts, so
  // that at the loop head only key loads are outstanding, oldest first, on
  // every path into it (otherwise the per-block waits become conservative).
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  if constexpr (COS) {
    float qsq = 0.f;
#pragma unroll
    for (int j = 0; j < KS; ++j)
      if (!MASKED || j < a.ks) qsq = chunk_sumsq<DT>(qb[j], qsq);
    qinv = inv_norm(sum_lane_groups(qsq));
  }
  if (kb0 < kb1) {
    u32x4_t ka[KS];
    load_block(ka, kb0);
    if constexpr (KS <= 16) {
      u32x4_t kbuf[KS];
      asm volatile("" ::: "memory");   // keep the first block's loads the oldest
      load_block(kbuf, min(kb0 + 1, kb1 - 1));
      // full pairs only inside the loop: every path into the loop head then
      // has the same loads outstanding
      int blk = kb0;
      for (; blk + 1 < kb1; blk += 2) {
        fold_scores<LOOKUP, KL>(score_block(ka, blk + 2), blk, g, kend, bias, ls, li);
        fold_scores<LOOKUP, KL>(score_block(kbuf, blk + 3), blk + 1, g, kend, bias, ls, li);
      }
      if (blk < kb1) fold_scores<LOOKUP, KL>(score_block(ka, blk + 2), blk, g, kend, bias, ls, li);
    } else {
      for (int blk = kb0; blk < kb1; ++blk)
        fold_scores<LOOKUP, KL>(score_block(ka, blk + 1), blk, g, kend, bias, ls, li);
    }
  }

  // merge: thread (t, L) owns list L of query row t
  const int list = wv * 4 + g;
#pragma unroll
  for (int e = 0; e < KL; ++e) {
    cand_s[list][n][e] = ls[e];
    cand_i[list][n][e] = li[e];
  }
  __syncthreads();
  const int t = threadIdx.x / NL;
  const int L = threadIdx.x % NL;
  float ms[KL];
  int mi[KL];
#pragma unroll
  for (int e = 0; e < KL; ++e) { ms[e] = cand_s[L][t][e]; mi[e] = cand_i[L][t][e]; }
  float top_s[KL];
  int top_i[KL];
  merge_lists<KL, 4>(ms, mi, LOOKUP ? a.k : 1, 1, top_s, top_i);
  if constexpr (!LOOKUP) {
    top_i[0] += key0;
    if (a.route_splits > 1) {
      // the arrival flag sits past the candidate lists (the kernel's LDS is
      // one object; see score_kernel)
      int* s_last = reinterpret_cast<int*>(smem + NL * 16 * KL * 8);
      route_partial<UNIT_STREAM_ROWS>(a.route_part, a.route_count, a.route_splits, a.out_idx,
                                      begin / 16, split, L == 0 ? t : 16, nr, top_s[0], top_i[0],
                                      s_last);
      return;
    }
  }
  if (L == 0 && t < nr) write_row<LOOKUP, KL>(a, row_id<LOOKUP>(a, begin, t), top_s, top_i);
}

// Level-2 streaming units with the key blocks staged in LDS (KS <= 16): as
// stream_unit, each wave scores its quarter of the scene's keys against the
// unit's <= 16 query rows, but every block goes straight from global memory
// into the wave's LDS block image (load_key_block: contiguous KiB loads,
// nontemporal).  As soon as a block's fragments are in registers the next
// block's loads are issued into the image, so they fly while the block is
// multiplied and folded.  The waves never wait for each other until the
// merge.  LDS: 4 waves x KS KiB, so that two workgroups fit a CU.
// part (0 .. SPLIT_PARTS - 1, -1 for a whole unit): a part of a cut unit
// (kernels.h) takes blocks [part nblk / SPLIT_PARTS, (part + 1) nblk /
// SPLIT_PARTS) of the scene's keys and keeps the exact top k of its keys for
// each row in the partial list slot of cut unit `cut`, which
// split_merge_kernel merges after the launch.  (Merging in the last part to
// finish, after an agent-scope acquire-release arrival, cost more than the
// extra launch: each release writes back the XCD's L2 and each acquire
// invalidates it, 1861.7 against 1833 + 8 us on the Zipf workload with two
// parts.)
template <int DT, int KS, bool MASKED, int KL, bool COS>
__device__ __forceinline__ void stream_unit_lds(const ScoreParams& a, char* smem, int64_t begin,
                                                int nr, const char* keys, int part = -1,
                                                int cut = 0) {
  constexpr int NL = SC_WAVES * 4;   // candidate lists per query row
  constexpr int BLOCK = KS * 1024;
  static_assert(KS <= 16, "fragments of a block held in registers");
  float (*cand_s)[16][KL] = reinterpret_cast<float (*)[16][KL]>(smem);
  int (*cand_i)[16][KL] = reinterpret_cast<int (*)[16][KL]>(smem + NL * 16 * KL * 4);
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 15, g = lane >> 4;
  const int nkeys = a.nkeys;
  const KeyImage im = key_image<KS, MASKED>(a);
  char* img = smem + wv * BLOCK;

  u32x4_t qb[KS];
  load_row_frags<KS, MASKED>(qb, a.q + row_id<true>(a, begin, n < nr ? n : nr - 1) * a.row_bytes,
                             g, a.ks);

  const int nblk = (nkeys + 15) >> 4;
  // the unit's blocks
  const int rb0 = part < 0 ? 0 : part * nblk / SPLIT_PARTS;
  const int rb1 = part < 0 ? nblk : (part + 1) * nblk / SPLIT_PARTS;
  const int bpw = (rb1 - rb0 + SC_WAVES - 1) / SC_WAVES;
  const int kb0 = rb0 + wv * bpw;
  const int kb1 = min(rb1, kb0 + bpw);
  const int kend = min(nkeys, kb1 * 16);

  uint32_t off[KS];
#pragma unroll
  for (int i = 0; i < KS; ++i) off[i] = (!MASKED || i < a.ks) ? im.src_off(i, lane, im.row_of(i, lane)) : 0u;
  // fragment offsets inside the image: step j = 4 m + t at fbase[t] + 256 m
  // (C a multiple of 16: the swizzle only permutes the low two bits of j)
  uint32_t fbase[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) fbase[t] = im.frag_off(t, g, n);

  float ls[KL];
  int li[KL];
#pragma unroll
  for (int e = 0; e < KL; ++e) { ls[e] = -__builtin_inff(); li[e] = -1; }

  auto issue = [&](int blk) {
    load_key_block<KS, MASKED, KS>(im, a, keys, blk * 16, kend, off, 0, 1, img, lane);
  };

  // the first key block goes out with the query fragments (one memory round
  // trip at the unit's start instead of two); both land before the loop, so
  // that no load is outstanding at its head
  if (kb0 < kb1) issue(kb0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  float qinv = 0.f;
  if constexpr (COS) {
    float qsq = 0.f;
#pragma unroll
    for (int j = 0; j < KS; ++j)
      if (!MASKED || j < a.ks) qsq = chunk_sumsq<DT>(qb[j], qsq);
    qinv = inv_norm(sum_lane_groups(qsq));
  }
  for (int blk = kb0; blk < kb1; ++blk) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // block blk is in the image
    u32x4_t kf[KS];
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      if (!MASKED || j < a.ks) {
        const uint32_t fo = MASKED ? im.frag_off(j, g, n) : fbase[j & 3] + 256 * (j >> 2);
        kf[j] = *reinterpret_cast<const u32x4_t*>(img + fo);
      }
    }
    // every read of the image has returned: refill it with the next block
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if (blk + 1 < kb1) issue(blk + 1);
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    float knsq = 0.f;
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      if (!MASKED || j < a.ks) {
        acc = mfma_chunk<DT>(kf[j], qb[j], acc);
        if constexpr (COS) knsq = chunk_sumsq<DT>(kf[j], knsq);
      }
    }
    if constexpr (COS) acc = cos_scale(acc, qinv, sum_lane_groups(knsq), g);
    fold_scores<true, KL>(acc, blk, g, kend, nullptr, ls, li);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // no load into LDS outlives the wave

  // merge: thread (t, L) owns list L of query row t (the lists reuse the
  // images, so every wave must be done with its own first)
  __syncthreads();
  const int list = wv * 4 + g;
#pragma unroll
  for (int e = 0; e < KL; ++e) {
    cand_s[list][n][e] = ls[e];
    cand_i[list][n][e] = li[e];
  }
  __syncthreads();
  const int t = threadIdx.x / NL;
  const int L = threadIdx.x % NL;
  float ms[KL];
  int mi[KL];
#pragma unroll
  for (int e = 0; e < KL; ++e) { ms[e] = cand_s[L][t][e]; mi[e] = cand_i[L][t][e]; }
  float top_s[KL];
  int top_i[KL];
  merge_lists<KL, 4>(ms, mi, a.k, 1, top_s, top_i);
  if (part < 0) {
    if (L == 0 && t < nr) write_row<true, KL>(a, row_id<true>(a, begin, t), top_s, top_i);
    return;
  }
  if (L == 0 && t < nr) {
    uint64_t* o = split_slot(a, cut, part, t);
#pragma unroll
    for (int e = 0; e < KL; ++e)
      if (e < a.k) o[e] = ((uint64_t)(uint32_t)top_i[e] << 32) | __float_as_uint(top_s[e]);
    // the first part names the row's output row for the merge (plus one:
    // zero marks a slot row with nothing to merge)
    if (part == 0) a.split_row[cut * UNIT_STREAM_ROWS + t] = (int32_t)row_id<true>(a, begin, t) + 1;
  }
}

// The merge of the cut units' parts, after the Level-2 launch on the same
// stream: 2 KL lanes a row slot (cut unit, t).  Where the first part named an
// output row for it, lane e < KL holds the e-th entry of the merged lists so
// far and lane KL + e entry KL - 1 - e of the next part's list (a bitonic
// sequence, padded with -inf); the xor-partner compare-exchanges of a bitonic
// merge sort it by the order of the outputs (score descending, then index
// ascending), one part after another.  The row's outputs are then written as
// write_row writes them (the softmax sum in entry order, in every lane) and
// the name is cleared for the next launch.
template <int KL>
__global__ __launch_bounds__(256) void split_merge_kernel(ScoreParams a) {
  constexpr int LPR = 2 * KL;                    // lanes a row slot
  constexpr int RPW = WAVE / LPR;                // row slots a wave
  static_assert(RPW >= 1 && (SPLIT_UNITS * UNIT_STREAM_ROWS) % (4 * RPW) == 0, "whole waves");
  const int lane = threadIdx.x & 63;
  const int slot = (blockIdx.x * 4 + (threadIdx.x >> 6)) * RPW + lane / LPR;
  const int e = lane % LPR, base = lane - e;
  const int named = a.split_row[slot];
  if (!__any(named != 0)) return;                // nothing cut here (wave-uniform)
  const int cut = slot / UNIT_STREAM_ROWS, t = slot % UNIT_STREAM_ROWS;
  const int k = a.k;
  float s = -__builtin_inff();
  int i = 0x7fffffff;
  if (e < KL && e < k && named != 0) {
    const uint64_t v = split_slot(a, cut, 0, t)[e];
    s = __uint_as_float((uint32_t)v);
    i = (int)(v >> 32);
  }
#pragma unroll
  for (int q = 1; q < SPLIT_PARTS; ++q) {
    if (e >= KL) {
      const int r = LPR - 1 - e;
      s = -__builtin_inff();
      i = 0x7fffffff;
      if (r < k && named != 0) {
        const uint64_t v = split_slot(a, cut, q, t)[r];
        s = __uint_as_float((uint32_t)v);
        i = (int)(v >> 32);
      }
    }
#pragma unroll
    for (int d = KL; d >= 1; d >>= 1) {
      const float os = __shfl_xor(s, d, WAVE);
      const int oi = __shfl_xor(i, d, WAVE);
      // the lower lane of the pair keeps the winner, the upper the other
      const bool take = (e & d) == 0 ? beats(os, oi, s, i) : beats(s, i, os, oi);
      s = take ? os : s;
      i = take ? oi : i;
    }
  }
  if (named == 0) return;
  const float s0 = __shfl(s, base, WAVE);
  float sum = 0.f;
#pragma unroll
  for (int x = 0; x < KL; ++x) {
    const float sx = __shfl(s, base + x, WAVE);
    if (x < k) sum += expf(sx - s0);
  }
  const float inv = 1.0f / sum;
  if (e < k) {
    const int64_t row = named - 1;
    a.out_idx[row * k + e] = i;
    a.out_w[row * k + e] = expf(s - s0) * inv;
  }
  if (e == 0) a.split_row[slot] = 0;
}

// ---------------------------------------------------------------------------
// Shared mode: up to 128 rows, every key block staged once in LDS
// ---------------------------------------------------------------------------
// Key block images kept in LDS by a shared unit: as many as SH_LDS_BYTES
// hold, at least 2 and at most 8.
constexpr int shared_nbuf(int ks) {
  return SH_LDS_BYTES / (ks * 1024) < 2 ? 2
         : SH_LDS_BYTES / (ks * 1024) > 8 ? 8
                                          : SH_LDS_BYTES / (ks * 1024);
}
// Level-2: block images in the ring of a shared unit.  Up to 16 steps the
// kernel's LDS holds the streaming units' 4 images (one per wave), and the
// ring takes all 4 of them.
constexpr int lookup_ring(int ks) { return ks <= 16 ? 4 : shared_nbuf(ks); }

// multi (Level-2): the unit's bucket is cut into several units, which all
// read the scene's keys.
template <int DT, int KS, bool MASKED, bool LOOKUP, int KL, bool COS>
__device__ __forceinline__ void shared_unit(const ScoreParams& a, char* smem, int64_t begin,
                                            int nr, const char* keys, bool multi = false) {
  constexpr int BLOCK_BYTES = KS * 1024;
  constexpr int CPT = KS / 4;          // routing: 16-byte chunks per thread per key block
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, g = lane >> 4;
  const int nkeys = a.nkeys;
  // routing: a wave keeps two 16-row query tiles (rows 16 w.. and 16 (w+4)..)
  // when a key row is at most 1 KiB; Level-2: one (see shared_unit_rows)
  constexpr bool TWO_TILES = !LOOKUP && KS <= 16;
  const int tiles = (nr + 15) >> 4;
  const bool has0 = wv < tiles, has1 = TWO_TILES && wv + SC_WAVES < tiles;

  u32x4_t q0[KS], q1[KS];
  {
    const int s0 = min(16 * wv + n, nr - 1);
    load_row_frags<KS, MASKED>(q0, a.q + row_id<LOOKUP>(a, begin, s0) * a.row_bytes, g, a.ks);
    if constexpr (TWO_TILES) {
      const int s1 = min(16 * (wv + SC_WAVES) + n, nr - 1);
      load_row_frags<KS, MASKED>(q1, a.q + row_id<LOOKUP>(a, begin, s1) * a.row_bytes, g, a.ks);
    }
  }
  float qinv0 = 0.f, qinv1 = 0.f;   // COS: 1 / ||q|| of the lane's rows, once they landed
  auto qnorms = [&]() {
    if constexpr (COS) {
      float s0 = 0.f, s1 = 0.f;
#pragma unroll
      for (int j = 0; j < KS; ++j)
        if (!MASKED || j < a.ks) {
          s0 = chunk_sumsq<DT>(q0[j], s0);
          if constexpr (TWO_TILES) s1 = chunk_sumsq<DT>(q1[j], s1);
        }
      qinv0 = inv_norm(sum_lane_groups(s0));
      qinv1 = inv_norm(sum_lane_groups(s1));
    }
  };
  float ls0[KL], ls1[KL];
  int li0[KL], li1[KL];
#pragma unroll
  for (int e = 0; e < KL; ++e) {
    ls0[e] = ls1[e] = -__builtin_inff();
    li0[e] = li1[e] = -1;
  }

  const int nblk = (nkeys + 15) >> 4;
  // Level-2 block images (KeyImage): step j = 4 m + t at fbase[t] + 256 m
  const KeyImage im = key_image<KS, MASKED>(a);
  uint32_t fbase[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) fbase[t] = im.frag_off(t, g, n);
  auto compute = [&](int buf, int blk) {
    if (!has0) return;                 // a wave without rows only helps to load
    f32x4_t acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    const char* base = smem + buf * BLOCK_BYTES + lane * 16;
    const char* ibase = smem + buf * BLOCK_BYTES;
    float knsq = 0.f;
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      if (!MASKED || j < a.ks) {
        const uint32_t fo = MASKED ? im.frag_off(j, g, n) : fbase[j & 3] + 256 * (j >> 2);
        const u32x4_t kf = LOOKUP ? *reinterpret_cast<const u32x4_t*>(ibase + fo)
                                  : *reinterpret_cast<const u32x4_t*>(base + j * 1024);
        acc0 = mfma_chunk<DT>(kf, q0[j], acc0);
        if constexpr (TWO_TILES)
          if (has1) acc1 = mfma_chunk<DT>(kf, q1[j], acc1);
        if constexpr (COS) knsq = chunk_sumsq<DT>(kf, knsq);
      }
    }
    if constexpr (COS) {
      knsq = sum_lane_groups(knsq);
      acc0 = cos_scale(acc0, qinv0, knsq, g);
      acc1 = cos_scale(acc1, qinv1, knsq, g);
    }
    fold_scores<LOOKUP, KL>(acc0, blk, g, nkeys, a.bias, ls0, li0);
    if (has1) fold_scores<LOOKUP, KL>(acc1, blk, g, nkeys, a.bias, ls1, li1);
  };

  if constexpr (LOOKUP) {
    // The key blocks go straight from global memory into a ring of NBUF
    // block images (load_key_block: contiguous KiB loads, nontemporal; load
    // instruction i of a block by wave i % 4): NBUF - 1 blocks are in flight
    // while one is multiplied, and no register holds them on the way.
    constexpr int NBUF = lookup_ring(KS);
    constexpr int PW = (KS + SC_WAVES - 1) / SC_WAVES;   // load instructions per wave and block
    uint32_t off[PW];
#pragma unroll
    for (int t = 0; t < PW; ++t) {
      const int i = wv + SC_WAVES * t;
      off[t] = (i < (MASKED ? a.ks : KS)) ? im.src_off(i, lane, im.row_of(i, lane)) : 0u;
    }
    // only existing blocks are loaded (nothing is read twice from HBM); the
    // keys of a bucket cut into several units are read by each of them
    const bool nt = !multi;
    auto issue = [&](int blk) {
      if (blk < nblk)
        load_key_block<KS, MASKED, PW>(im, a, keys, blk * 16, nkeys, off, wv, SC_WAVES,
                                       smem + (blk % NBUF) * BLOCK_BYTES, lane, nt);
    };
    // the ring's first blocks go out with the query fragments (one memory
    // round trip at the unit's start instead of two); all land before the
    // loop, so that no load is outstanding at its head
#pragma unroll
    for (int b = 0; b < NBUF - 1; ++b) issue(b);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    qnorms();
    for (int blk = 0; blk < nblk; ++blk) {
      // this wave's loads of block blk have landed once at most those of the
      // NBUF - 2 younger blocks are outstanding (near the end, or with masked
      // steps, when fewer instructions are younger: once all have); the
      // barrier makes every wave's visible and ends every read of block
      // blk - 1, whose image the next loads overwrite (a plain s_barrier: the
      // fence of __syncthreads would wait for every load in flight)
      if (!MASKED && wv + SC_WAVES * (PW - 1) < KS && blk + NBUF - 2 < nblk)
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NBUF - 2) * PW) : "memory");
      else
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      issue(blk + NBUF - 1);
      compute(blk % NBUF, blk);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // no load into LDS outlives the wave
  } else {
    // routing: the same block images, staged through registers (two blocks
    // in flight; measured faster for routing than the direct-to-LDS ring).
    // Thread tid fills slots c = tid + 256 i.
    auto gload = [&](u32x4_t (&r)[CPT], int blk) {
      blk = min(blk, nblk - 1);          // unconditional: past the end, an L2 hit
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        const int c = tid + SC_THREADS * i;
        const int j = c >> 6, L = c & 63;
        const int row = min(blk * 16 + (L & 15), nkeys - 1);
        r[i] = (!MASKED || j < a.ks)
                   ? ld16(keys + (int64_t)row * a.row_bytes + (4 * j + (L >> 4)) * 16)
                   : u32x4_t{0, 0, 0, 0};
      }
    };
    auto lstore = [&](int buf, const u32x4_t (&r)[CPT]) {
#pragma unroll
      for (int i = 0; i < CPT; ++i) st16(smem + buf * BLOCK_BYTES + (tid + SC_THREADS * i) * 16, r[i]);
    };
    // Pipeline: at the top of step b the LDS buffer b%2 holds block b, the
    // register set for block b+1 and the one for block b+2 are in flight.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // query fragments first
    qnorms();
    u32x4_t r0[CPT], r1[CPT];
    gload(r0, 0);
    asm volatile("" ::: "memory");
    gload(r1, 1);
    lstore(0, r0);
    __syncthreads();
    gload(r0, 2);
    int blk = 0;
    for (; blk + 1 < nblk; blk += 2) {
      compute(0, blk);
      lstore(1, r1);          // block blk+1 (buffer 1 was last read two steps ago)
      __syncthreads();
      gload(r1, blk + 3);
      compute(1, blk + 1);
      lstore(0, r0);          // block blk+2
      __syncthreads();
      gload(r0, blk + 4);
    }
    if (blk < nblk) compute(0, blk);
  }

  // merge inside the wave: the 4 lists of row n sit in lanes n + 16 g
  const int k = LOOKUP ? a.k : 1;
  float top_s[KL];
  int top_i[KL];
  if (has0) {
    merge_lists<KL, 2>(ls0, li0, k, 16, top_s, top_i);
    const int slot = 16 * wv + n;
    if (g == 0 && slot < nr) write_row<LOOKUP, KL>(a, row_id<LOOKUP>(a, begin, slot), top_s, top_i);
  }
  if (has1) {
    merge_lists<KL, 2>(ls1, li1, k, 16, top_s, top_i);
    const int slot = 16 * (wv + SC_WAVES) + n;
    if (g == 0 && slot < nr) write_row<LOOKUP, KL>(a, row_id<LOOKUP>(a, begin, slot), top_s, top_i);
  }
}

// KS: compile-time number of chunk steps; with MASKED, steps >= ks are
// skipped (row widths that are not a power-of-two multiple of 64 bytes).
// The select of the batch carried by a Level-2 launch (Eq. 9-10): slot
// side0 + l selects layer l's kept set from its criticality keys (computed
// by an earlier launch), with the keys cached in `smem`: the body of
// crit_select_kernel on the launch's 256 threads, so the bits are its; or
// compacts layer l's open gates from their logits (gate_compact_kernel's
// body).
// The key cache takes the first SIDE_CACHE_BYTES of `smem`, the select's
// other words the SelLds after it.
constexpr int SIDE_CACHE_BYTES = (sel_cache_words(SEL_SIDE_MAX_N) * 4 + 15) / 16 * 16;

template <int KS>
__device__ __forceinline__ void side_select(const ScoreParams& a, char* smem) {
  const int layer = blockIdx.x - a.side0;
  SelLds& sl = *reinterpret_cast<SelLds*>(smem + SIDE_CACHE_BYTES);
  if (a.gate_count != nullptr) {
    gate_compact_layer<SC_THREADS>(
        reinterpret_cast<const float*>(a.crit_key) + (int64_t)layer * a.crit_n, a.crit_n,
        a.kept + (int64_t)layer * a.crit_n, a.gate_count + layer, sl);
    return;
  }
  select_layer<SEL_SIDE_MAX_N, SC_THREADS>(a.crit_key + (int64_t)layer * a.crit_n, a.crit_n,
                                           a.n_keep, a.kept + (int64_t)layer * a.n_keep,
                                           reinterpret_cast<uint32_t*>(smem), sl);
}

// KL: per-lane candidate list length (>= k) for lookup; 1 for routing.
// SIDE (lookup only): launch slots from a.side0 on run side_select; a
// separate instantiation, so that the kernels without it keep their code.
template <int DT, int KS, bool MASKED, bool LOOKUP, int KL, bool SIDE = false, bool COS = false>
__global__ __launch_bounds__(SC_THREADS) void score_kernel(ScoreParams a) {
  constexpr int MERGE_BYTES = SC_WAVES * 4 * 16 * KL * 8;
  constexpr int STAGE_BYTES = (LOOKUP ? lookup_ring(KS) : 2) * KS * 1024;
  constexpr int SIDE_BYTES = (LOOKUP && SIDE) ? SIDE_CACHE_BYTES + (int)sizeof(SelLds) : 0;
  constexpr int SMEM0 = MERGE_BYTES > STAGE_BYTES ? MERGE_BYTES : STAGE_BYTES;
  constexpr int SMEM = SMEM0 > SIDE_BYTES ? SMEM0 : SIDE_BYTES;
  // all of the kernel's LDS is this one object (with several, the compiler
  // puts a load wait before every LDS read that follows a direct-to-LDS
  // load); 16 bytes past the rest hold the split routing's arrival flag
  static_assert(SMEM >= MERGE_BYTES, "candidate lists");
  __shared__ __attribute__((aligned(1024))) char smem[SMEM + 16];
  if constexpr (LOOKUP && SIDE) {
    static_assert(SMEM >= SIDE_CACHE_BYTES + (int)sizeof(SelLds), "the side select's LDS");
    if ((int)blockIdx.x >= a.side0) {
      side_select<KS>(a, smem);
      return;
    }
  }

  int64_t begin;
  int nr;
  bool shared;
  const char* keys;
  int key0 = 0, nk = a.nkeys, split = 0;
  int part = -1, cut = 0;   // lookup: a part of a cut unit (kernels.h)
  bool multi = false;
  if constexpr (LOOKUP) {
    // units in list order (groups of one shared and three streaming units
    // while both kinds last), dealt to the XCDs in fours: each XCD takes a
    // whole group at a time, the same mix of the two kinds
    const int b = blockIdx.x, slot = b >> 3;
    int u = (slot >> 2) * 32 + (b & 7) * 4 + (slot & 3);
    const int total = a.unit_count[0], first_part = a.unit_count[1];
    if (u >= first_part) {
      // past the statically dealt units: the parts of the cut last round go
      // to whichever workgroups start first (those of the XCDs that are
      // through with their units), one fetch a workgroup; the slot past the
      // LDS's other uses carries the result to every wave
      if (KS > 16 || first_part == total) return;   // parts only with KS <= 16
      int* s_u = reinterpret_cast<int*>(smem + SMEM);
      if (threadIdx.x == 0) {
        int v = total;
        if (__hip_atomic_load(&a.unit_count[2], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <
            total - first_part)
          v = first_part + __hip_atomic_fetch_add(&a.unit_count[2], 1, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
        *s_u = v;
      }
      __syncthreads();
      u = *s_u;
      if (u >= total) return;
    }
    const int tag = a.unit_scene[u];
    const int s = tag & ~UNIT_SHARED;
    shared = (tag & UNIT_SHARED) != 0;
    begin = a.unit_begin[u];
    nr = min(shared ? a.shared_rows : UNIT_STREAM_ROWS, a.offsets[s + 1] - (int)begin);
    multi = a.offsets[s + 1] - a.offsets[s] > a.shared_rows;
    keys = a.keys + (int64_t)s * a.nkeys * a.row_bytes;
    if (u >= first_part) {
      part = (u - first_part) % SPLIT_PARTS;
      cut = (u - first_part) / SPLIT_PARTS;
    }
  } else {
    const int R = a.route_rows;
    const int splits = R > 16 ? 1 : a.route_splits;
    const int64_t units = (a.rows + R - 1) / R * splits;
    const int u = xcd_remap(blockIdx.x, (int)units);
    if (u < 0) return;
    begin = (int64_t)(u / splits) * R;
    nr = (int)min<int64_t>(R, a.rows - begin);
    shared = R > 16;
    split = u % splits;
    key0 = split * a.route_kps;
    nk = min(a.route_kps, a.nkeys - key0);
    keys = a.keys + (int64_t)key0 * a.row_bytes;
  }
  if (shared) shared_unit<DT, KS, MASKED, LOOKUP, KL, COS>(a, smem, begin, nr, keys, multi);
  else if constexpr (LOOKUP && KS <= 16) stream_unit_lds<DT, KS, MASKED, KL, COS>(a, smem, begin, nr, keys, part, cut);
  else stream_unit<DT, KS, MASKED, LOOKUP, KL, COS>(a, smem, begin, nr, keys, key0, nk, split);
}


// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

template <int DT, bool LOOKUP, int KL, bool SIDE = false, bool COS = false>
static hipError_t launch_ks(int ks, int grid, const ScoreParams& p, hipStream_t st,
                            const hipEvent_t* stamp) {
  // with a stamp pair, the launch itself records the kernel's start and end
  // in the two events (its own duration, without the gaps of recorded events)
#define LOOKME_SCORE_LAUNCH(KS_, M_)                                                         \
  do {                                                                                     \
    if (stamp != nullptr)                                                                  \
      hipExtLaunchKernelGGL((score_kernel<DT, KS_, M_, LOOKUP, KL, SIDE, COS>), dim3(grid),  \
                            dim3(SC_THREADS), 0, st, stamp[0], stamp[1], 0, p);           \
    else                                                                                   \
      hipLaunchKernelGGL((score_kernel<DT, KS_, M_, LOOKUP, KL, SIDE, COS>), dim3(grid),     \
                         dim3(SC_THREADS), 0, st, p);                                      \
  } while (0)
  // the compiled step count follows score_ks(), which also sizes the units
  switch (ks) {
    case 4: LOOKME_SCORE_LAUNCH(4, false); break;
    case 8: LOOKME_SCORE_LAUNCH(8, false); break;
    case 16: LOOKME_SCORE_LAUNCH(16, false); break;
    case 32: LOOKME_SCORE_LAUNCH(32, false); break;
    default:
      if (ks < 4) LOOKME_SCORE_LAUNCH(4, true);
      else LOOKME_SCORE_LAUNCH(32, true);
  }
#undef LOOKME_SCORE_LAUNCH
  return hipGetLastError();
}

template <bool LOOKUP, int KL>
static hipError_t launch_dt(int dt, int ks, int grid, const ScoreParams& p, hipStream_t st,
                            const hipEvent_t* stamp = nullptr) {
  if (p.cos)   // cosine scores (never with a carried select)
    return dt == DT_BF16 ? launch_ks<DT_BF16, LOOKUP, KL, false, true>(ks, grid, p, st, stamp)
                         : launch_ks<DT_F32, LOOKUP, KL, false, true>(ks, grid, p, st, stamp);
  if constexpr (LOOKUP) {
    if (p.side0 > 0)
      return dt == DT_BF16 ? launch_ks<DT_BF16, true, KL, true>(ks, grid, p, st, stamp)
                           : launch_ks<DT_F32, true, KL, true>(ks, grid, p, st, stamp);
  }
  return dt == DT_BF16 ? launch_ks<DT_BF16, LOOKUP, KL>(ks, grid, p, st, stamp)
                       : launch_ks<DT_F32, LOOKUP, KL>(ks, grid, p, st, stamp);
}

static inline int64_t round8(int64_t x) { return (x + 7) / 8 * 8; }

static int route_unit_rows(int64_t rows, int shared_rows) {
  // shared mode when there are enough rows to keep the chip busy with
  // 64- or 128-row units; small batches stream 16-row tiles
  if (shared_rows >= 128 && rows >= (int64_t)128 * 512) return 128;
  if (rows >= (int64_t)64 * 256) return 64;
  return UNIT_STREAM_ROWS;
}

static int cdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// Key ranges per row block of the tile kernel (at least `least`, so that a
// unit's bias table fits its LDS).  The kernel runs one workgroup a CU (its
// LDS): when the row blocks alone fill whole rounds of the 256 CUs to 90%,
// no split (each unit walks every key tile, no partial lists to merge;
// Zipf batch 176 -> 164 us against two splits); else about 512 workgroups
// (measured better than rounds filled with one-tile units, whose pipeline
// start and merge cost more than a partial round's idle CUs: multi-scale
// batch 51 us with 2 splits, 55 with 4).
static int route_splits(int64_t blocks, int tiles, int least) {
  const double fill = (double)blocks / (double)(cdiv(blocks, 256) * 256);
  if (least <= 1 && fill >= 0.9) return 1;
  int sp = blocks < 512 ? cdiv(512, blocks) : 1;
  sp = sp < tiles ? sp : tiles;
  return sp > least ? sp : least;
}

RoutePlan route_plan(int64_t rows, int S, int64_t row_bytes, bool cos) {
  RoutePlan p{ROUTE_SHARED, 1, S, 0};
  if (rows <= 0 || S <= 0) return p;
  const int64_t blocks = (rows + ROUTE_DTL_ROWS - 1) / ROUTE_DTL_ROWS;
  // the tile kernel scores dot products only
  if (!cos && rows >= ROUTE_DTL_MIN_ROWS && blocks < ROUTE_DTL_MAX_BLOCKS &&
      row_bytes % 128 == 0) {
    // enough 128-row blocks for the matrix-core kernel but too few to fill
    // the chip with the shared-mode units; split the key tiles until about
    // 512 workgroups run (and at most ROUTE_DTL_MAX_TPS tiles stay with one
    // workgroup, whose bias table lives in LDS)
    const int tiles = cdiv(S, ROUTE_DTL_KEYS);
    const int least = cdiv(tiles, ROUTE_DTL_MAX_TPS);
    int sp = route_splits(blocks, tiles, least);
    const int tps = cdiv(tiles, sp);
    sp = cdiv(tiles, tps);
    if (sp == 1 || blocks <= ROUTE_COUNTERS) {
      p.mode = ROUTE_DTL;
      p.splits = sp;
      p.per_split = tps;
      p.part_entries = sp > 1 ? blocks * sp * ROUTE_DTL_ROWS : 0;
      return p;
    }
  }
  if (route_unit_rows(rows, shared_unit_rows(row_bytes, 0)) == UNIT_STREAM_ROWS) {
    // small batch: split the keys of every 16-row tile (at least 64 keys a
    // workgroup) until about 512 workgroups run
    const int64_t tiles = (rows + 15) / 16;
    int sp = 1;
    if (tiles <= ROUTE_COUNTERS) {
      sp = tiles < 512 ? cdiv(512, tiles) : 1;
      const int most = cdiv(S, 64);
      sp = sp < most ? sp : most;
    }
    const int kps = cdiv(cdiv(S, sp), 64) * 64;
    p.mode = ROUTE_STREAM;
    p.splits = cdiv(S, kps);
    p.per_split = kps;
    p.part_entries = p.splits > 1 ? tiles * p.splits * UNIT_STREAM_ROWS : 0;
  }
  return p;
}

hipError_t launch_route(int dt, const void* q, const void* scene_keys, const float* bias,
                        int32_t* scene, int64_t rows, int d_e, int S, uint64_t* part,
                        int32_t* count, hipStream_t st, bool cos) {
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
  p.route_rows = route_unit_rows(rows, shared_unit_rows(p.row_bytes, 0));
  p.out_idx = scene;
  p.cos = cos ? 1 : 0;
  const RoutePlan plan = route_plan(rows, S, p.row_bytes, cos);
  if (plan.mode == ROUTE_DTL)
    return launch_route_dtl(dt, q, scene_keys, bias, scene, rows, d_e, S, plan, part, count, st);
  p.route_rows = plan.mode == ROUTE_STREAM ? UNIT_STREAM_ROWS : p.route_rows;
  p.route_splits = plan.mode == ROUTE_STREAM ? plan.splits : 1;
  p.route_kps = plan.mode == ROUTE_STREAM ? plan.per_split : S;
  p.route_part = part;
  p.route_count = count;
  const int64_t units = (rows + p.route_rows - 1) / p.route_rows * p.route_splits;
  return launch_dt<false, 1>(dt, p.ks, (int)round8(units), p, st);
}

// The Level-2 launch and, when the bucketing may cut the last round, the
// merge of the parts right after it on the same stream (its threads return
// at once where nothing was cut).  With stamps, the pair of events brackets
// both launches.
template <int KL>
static hipError_t launch_lookup_kl(int dt, int grid, const ScoreParams& p, bool split,
                                   hipStream_t st, const hipEvent_t* stamp) {
  if (!split) return launch_dt<true, KL>(dt, p.ks, grid, p, st, stamp);
  const hipEvent_t first[2] = {stamp != nullptr ? stamp[0] : nullptr, nullptr};
  const hipError_t e = launch_dt<true, KL>(dt, p.ks, grid, p, st, stamp != nullptr ? first : nullptr);
  if (e != hipSuccess) return e;
  // 2 KL lanes a row slot, four waves a workgroup
  const unsigned blocks = (unsigned)(SPLIT_UNITS * UNIT_STREAM_ROWS * 2 * KL / (4 * WAVE));
  hipExtLaunchKernelGGL((split_merge_kernel<KL>), dim3(blocks), dim3(256), 0, st, nullptr,
                        stamp != nullptr ? stamp[1] : nullptr, 0, p);
  return hipGetLastError();
}

hipError_t launch_lookup(int dt, const void* q, const void* prim_keys, const BucketWs& ws,
                         int d_e, int P, int k, int32_t* prim, float* w, hipStream_t st,
                         const SideSelect* side, bool cos, const hipEvent_t* stamp) {
  ScoreParams p{};
  p.cos = cos ? 1 : 0;
  p.q = static_cast<const char*>(q);
  p.keys = static_cast<const char*>(prim_keys);
  p.perm = ws.perm;
  p.offsets = ws.offsets;
  p.unit_scene = ws.unit_scene;
  p.unit_begin = ws.unit_begin;
  p.unit_count = ws.unit_count;
  p.row_bytes = (int64_t)d_e * (dt == DT_BF16 ? 2 : 4);
  p.ks = (int)(p.row_bytes / 64);
  p.shared_rows = shared_unit_rows(p.row_bytes, k);
  p.nkeys = P;
  p.k = k;
  p.out_idx = prim;
  p.out_w = w;
  p.split_part = ws.split_part;
  p.split_row = ws.split_row;
  int grid = (int)((ws.max_units + 31) / 32 * 32);   // whole fours on every XCD
  if (side != nullptr && (side->n_keep > 0 || side->count != nullptr) && side->n > 0) {
    p.side0 = grid;
    p.crit_n = side->n;
    p.n_keep = side->n_keep;
    p.crit_key = side->key;
    p.kept = side->kept;
    p.gate_count = side->count;
    grid += side->layers;
  }
  if (k <= 4) return launch_lookup_kl<4>(dt, grid, p, ws.split_max > 0, st, stamp);
  if (k <= 8) return launch_lookup_kl<8>(dt, grid, p, ws.split_max > 0, st, stamp);
  if (k <= 16) return launch_lookup_kl<16>(dt, grid, p, ws.split_max > 0, st, stamp);
  return launch_lookup_kl<32>(dt, grid, p, ws.split_max > 0, st, stamp);
}

}  // namespace lookme
