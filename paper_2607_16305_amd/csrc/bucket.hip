// Bucketing of query rows by their Level-1 scene (Sec. 3.2: rows routed to
// the same scene share that scene's primitive keys in Level-2).
//
// A stable counting sort in three passes, every step deterministic:
//   1. per 1024-row chunk: a histogram over scenes and, for every row, its
//      rank among equal-scene rows earlier in the chunk (wave match masks
//      built from ballots over the scene bits, then the 16 waves in order);
//   2. per scene (a thread each): prefix over chunks; then one workgroup:
//      exclusive scan over scenes (wavefront prefix sums) giving bucket
//      offsets, and the Level-2 work list (a bucket of <= 16 rows is one
//      streaming unit, a larger one is cut into shared units of <= 128 rows;
//      the two kinds alternate in the list);
//   3. per chunk: perm[offset + chunk prefix + rank] = row.
// Within a bucket rows keep ascending order.  Scene values outside [0, S)
// are clamped (results for such rows are undefined; memory stays in bounds).
#include "common.h"
#include "crit.h"
#include "kernels.h"

#include <algorithm>

namespace lookme {

constexpr int BK_THREADS = 1024;
constexpr int BK_WAVES = BK_THREADS / WAVE;
constexpr int TILE_ROWS = UNIT_STREAM_ROWS;

// Shared and streaming work units of a bucket of `size` rows.
__device__ __forceinline__ int shared_units(int size, int shared_rows) {
  return size > UNIT_STREAM_ROWS ? (size + shared_rows - 1) / shared_rows : 0;
}
__device__ __forceinline__ int stream_units(int size) {
  return (size > 0 && size <= UNIT_STREAM_ROWS) ? 1 : 0;
}

// List position of shared unit i and of streaming unit j (nb shared and ns
// streaming units in all): while both last, groups of one shared unit and
// ORDER_STREAM streaming units (c groups), then the rest of the shared units,
// then the rest of the streaming ones.  About a quarter of the resident
// units are then shared ones (matrix-core and vector work on keys mostly
// found in L2) and the rest stream keys from HBM.  With every shared unit
// first, the Zipf workload's 487 of them filled every slot for the first
// ~300 us while the key stream from HBM ran at about half its rate; with
// the kinds alternating one to one, the first ~550 us still had half of the
// slots on shared units and the stream at ~6.3 TB/s; one to three: 7.1-7.3
// TB/s there (Zipf Level-2 1836 -> 1829 us, multi-scale 186 -> 183 us).
constexpr int ORDER_STREAM = 3;
__device__ __forceinline__ int order_groups(int nb, int ns) { return min(nb, ns / ORDER_STREAM); }
__device__ __forceinline__ int shared_pos(int i, int nb, int ns) {
  const int c = order_groups(nb, ns);
  return i < c ? i * (ORDER_STREAM + 1) : c * (ORDER_STREAM + 1) + (i - c);
}
__device__ __forceinline__ int stream_pos(int j, int nb, int ns) {
  const int c = order_groups(nb, ns);
  return j < c * ORDER_STREAM ? (j / ORDER_STREAM) * (ORDER_STREAM + 1) + 1 + j % ORDER_STREAM
                              : nb + j;
}

// Writes the units of scene s: shared ones as shared units sh.., a streaming
// one as streaming unit st (list positions from shared_pos / stream_pos).  Of
// the last nsplit streaming units (all past the groups: ns - nsplit >=
// ORDER_STREAM c) each becomes SPLIT_PARTS entries, its parts, from position
// nb + ns - nsplit on.
__device__ __forceinline__ void write_units(int s, int offset, int size, int sh, int st, int nb,
                                            int ns, int nsplit, int shared_rows,
                                            int32_t* unit_scene, int32_t* unit_begin) {
  if (size == 0) return;
  if (size <= UNIT_STREAM_ROWS) {
    const int first = ns - nsplit;
    if (st >= first) {
      const int p = nb + first + SPLIT_PARTS * (st - first);
      for (int q = 0; q < SPLIT_PARTS; ++q) {
        unit_scene[p + q] = s;
        unit_begin[p + q] = offset;
      }
      return;
    }
    const int p = stream_pos(st, nb, ns);
    unit_scene[p] = s;
    unit_begin[p] = offset;
    return;
  }
  const int units = shared_units(size, shared_rows);
  for (int u = 0; u < units; ++u) {
    const int p = shared_pos(sh + u, nb, ns);
    unit_scene[p] = s | UNIT_SHARED;
    unit_begin[p] = offset + u * shared_rows;
  }
}

int64_t bucket_chunks(int64_t rows) { return (rows + BK_THREADS - 1) / BK_THREADS; }

int64_t bucket_max_units(int64_t rows, int S) {
  // the parts of a cut last round add at most (SPLIT_PARTS - 1) SPLIT_UNITS
  // entries
  return std::min<int64_t>(S, rows) + (rows + TILE_ROWS - 1) / TILE_ROWS +
         (int64_t)(SPLIT_PARTS - 1) * SPLIT_UNITS;
}

__device__ __forceinline__ int clamp_scene(int s, int S) { return s < 0 ? 0 : (s >= S ? S - 1 : s); }

__global__ __launch_bounds__(BK_THREADS) void bucket_hist_kernel(
    const int32_t* __restrict__ scene, int64_t rows, int S, int sbits,
    int32_t* __restrict__ chunk_hist, int32_t* __restrict__ local_rank) {
  extern __shared__ int hist[];
  for (int i = threadIdx.x; i < S; i += BK_THREADS) hist[i] = 0;
  __syncthreads();

  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * BK_THREADS + threadIdx.x;
  const bool valid = t < rows;
  const int s = valid ? clamp_scene(scene[t], S) : 0;

  // lanes of this wave holding the same scene
  uint64_t match = __ballot(valid);
  for (int b = 0; b < sbits; ++b) {
    const uint64_t ones = __ballot(valid && ((s >> b) & 1));
    match &= ((s >> b) & 1) ? ones : ~ones;
  }
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int rank_in_wave = __popcll(match & below);
  const int cnt = __popcll(match);

  int base = 0;
  for (int w = 0; w < BK_WAVES; ++w) {
    if (wv == w && valid) {
      base = hist[s];
      if (rank_in_wave == 0) hist[s] = base + cnt;
    }
    __syncthreads();
  }
  if (valid) local_rank[t] = base + rank_in_wave;
  int32_t* out = chunk_hist + (int64_t)blockIdx.x * S;
  for (int i = threadIdx.x; i < S; i += BK_THREADS) out[i] = hist[i];
}

// Inclusive wave prefix sum.
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int o = __shfl_up(v, d, 64);
    if (lane >= d) v += o;
  }
  return v;
}

// Exclusive block prefix of three counters over the block's threads; returns
// the totals through `tot`.
__device__ __forceinline__ void block_excl_scan3(int (&v)[3], int (&tot)[3]) {
  __shared__ int ws[3][BK_WAVES];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int inc[3];
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    inc[c] = wave_incl_scan(v[c]);
    if (lane == 63) ws[c][wv] = inc[c];
  }
  __syncthreads();
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    int pre = 0;
    tot[c] = 0;
    for (int w = 0; w < BK_WAVES; ++w) {
      if (w < wv) pre += ws[c][w];
      tot[c] += ws[c][w];
    }
    v[c] = pre + inc[c] - v[c];
  }
  __syncthreads();
}

// Offsets of the buckets [s0, s1) given their sizes in size_of(s), and the
// work list: the entry count, the first part's position and a zero fetch
// count into unit_count[0..2] (thread 0).  split_max: the number of last
// streaming units to cut in parts, when the streaming units outnumber the
// shared ones by that many and fill at least two rounds with them (else 0).
template <typename SizeOf, typename SetOffset>
__device__ __forceinline__ void offsets_and_units(int S, int shared_rows, SizeOf size_of,
                                                  SetOffset set_offset, int32_t* offsets,
                                                  int32_t* unit_scene, int32_t* unit_begin,
                                                  int32_t* unit_count, int split_max = 0) {
  const int ipt = (S + BK_THREADS - 1) / BK_THREADS;
  const int s0 = min(S, (int)threadIdx.x * ipt), s1 = min(S, s0 + ipt);
  int v[3] = {0, 0, 0};   // rows, shared units, streaming units
  for (int s = s0; s < s1; ++s) {
    const int size = size_of(s);
    v[0] += size;
    v[1] += shared_units(size, shared_rows);
    v[2] += stream_units(size);
  }
  int tot[3];
  block_excl_scan3(v, tot);
  const int nb = tot[1], ns = tot[2];
  const int nsplit = (split_max > 0 && ns - split_max >= ORDER_STREAM * order_groups(nb, ns) &&
                      ns - nb >= split_max && nb + ns >= 2 * split_max)
                         ? split_max
                         : 0;
  int row = v[0], sh = v[1], st = v[2];
  for (int s = s0; s < s1; ++s) {
    const int size = size_of(s);
    set_offset(s, row);
    write_units(s, row, size, sh, st, nb, ns, nsplit, shared_rows, unit_scene, unit_begin);
    row += size;
    sh += shared_units(size, shared_rows);
    st += stream_units(size);
  }
  if (threadIdx.x == 0) {
    offsets[S] = tot[0];
    unit_count[0] = nb + ns + (SPLIT_PARTS - 1) * nsplit;
    unit_count[1] = nb + ns - nsplit;
    unit_count[2] = 0;
  }
}

// Per-scene exclusive prefix of the chunk histograms over the chunks (in
// place), and the bucket sizes into offsets[] for bucket_scan_kernel: one
// thread a scene, CB chunk loads in flight (a single workgroup walking every
// scene took ~20 us on the Zipf workload, one dependent load round after
// another).
constexpr int COL_THREADS = 256;

__global__ __launch_bounds__(COL_THREADS) void bucket_colscan_kernel(
    int32_t* __restrict__ chunk_hist, int64_t chunks, int S, int32_t* __restrict__ offsets) {
  constexpr int CB = 32;
  const int s = blockIdx.x * COL_THREADS + threadIdx.x;
  if (s >= S) return;
  int run = 0;
  for (int64_t c0 = 0; c0 < chunks; c0 += CB) {
    int h[CB];
#pragma unroll
    for (int i = 0; i < CB; ++i) h[i] = c0 + i < chunks ? chunk_hist[(c0 + i) * S + s] : 0;
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      if (c0 + i < chunks) chunk_hist[(c0 + i) * S + s] = run;
      run += h[i];
    }
  }
  offsets[s] = run;
}

// COLS: the per-scene prefix over chunks ran in bucket_colscan_kernel (the
// bucket sizes are in offsets[]); otherwise this workgroup takes it first,
// eight chunk loads in flight a thread (few scenes and chunks: one launch
// less).
template <bool COLS>
__global__ __launch_bounds__(BK_THREADS) void bucket_scan_kernel(
    int32_t* __restrict__ chunk_hist, int64_t chunks, int S, int shared_rows,
    int32_t* __restrict__ offsets, int32_t* __restrict__ unit_scene,
    int32_t* __restrict__ unit_begin, int32_t* __restrict__ unit_count, int split_max) {
  if constexpr (!COLS) {
    for (int s = threadIdx.x; s < S; s += BK_THREADS) {
      int run = 0;
      for (int64_t c0 = 0; c0 < chunks; c0 += 8) {
        int h[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) h[i] = c0 + i < chunks ? chunk_hist[(c0 + i) * S + s] : 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if (c0 + i < chunks) chunk_hist[(c0 + i) * S + s] = run;
          run += h[i];
        }
      }
      offsets[s] = run;
    }
    __syncthreads();
  }
  // exclusive scan of the bucket sizes over scenes: offsets and the work list
  offsets_and_units(
      S, shared_rows, [&](int s) { return offsets[s]; },
      [&](int s, int off) { offsets[s] = off; }, offsets, unit_scene, unit_begin, unit_count,
      split_max);
}

__global__ __launch_bounds__(BK_THREADS) void bucket_scatter_kernel(
    const int32_t* __restrict__ scene, int64_t rows, int S, const int32_t* __restrict__ chunk_hist,
    const int32_t* __restrict__ local_rank, const int32_t* __restrict__ offsets,
    int32_t* __restrict__ perm) {
  const int64_t t = (int64_t)blockIdx.x * BK_THREADS + threadIdx.x;
  if (t >= rows) return;
  const int s = clamp_scene(scene[t], S);
  const int pos = offsets[s] + chunk_hist[(int64_t)blockIdx.x * S + s] + local_rank[t];
  perm[pos] = (int32_t)t;
}

// All three passes in one workgroup, for batches of at most one chunk
// (saves two launches where launch latency dominates); hist: S ints of LDS.
__device__ __forceinline__ void bucket_small_body(
    const int32_t* __restrict__ scene, int64_t rows, int S, int sbits, int shared_rows,
    int32_t* __restrict__ offsets, int32_t* __restrict__ perm, int32_t* __restrict__ unit_scene,
    int32_t* __restrict__ unit_begin, int32_t* __restrict__ unit_count, int* hist) {
  for (int i = threadIdx.x; i < S; i += BK_THREADS) hist[i] = 0;
  __syncthreads();
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int t = threadIdx.x;
  const bool valid = t < rows;
  const int s = valid ? clamp_scene(scene[t], S) : 0;
  uint64_t match = __ballot(valid);
  for (int b = 0; b < sbits; ++b) {
    const uint64_t ones = __ballot(valid && ((s >> b) & 1));
    match &= ((s >> b) & 1) ? ones : ~ones;
  }
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int rank_in_wave = __popcll(match & below);
  const int cnt = __popcll(match);
  int base = 0;
  for (int w = 0; w < BK_WAVES; ++w) {
    if (wv == w && valid) {
      base = hist[s];
      if (rank_in_wave == 0) hist[s] = base + cnt;
    }
    __syncthreads();
  }
  const int rank = base + rank_in_wave;
  // bucket offsets and the work list (hist[] becomes the offsets)
  offsets_and_units(
      S, shared_rows, [&](int x) { return hist[x]; },
      [&](int x, int off) {
        hist[x] = off;
        offsets[x] = off;
      },
      offsets, unit_scene, unit_begin, unit_count);
  __syncthreads();
  if (valid) perm[hist[s] + rank] = t;
}

__global__ __launch_bounds__(BK_THREADS) void bucket_small_kernel(
    const int32_t* __restrict__ scene, int64_t rows, int S, int sbits, int shared_rows,
    int32_t* __restrict__ offsets, int32_t* __restrict__ perm, int32_t* __restrict__ unit_scene,
    int32_t* __restrict__ unit_begin, int32_t* __restrict__ unit_count) {
  extern __shared__ int hist[];
  bucket_small_body(scene, rows, S, sbits, shared_rows, offsets, perm, unit_scene, unit_begin,
                    unit_count, hist);
}

// The bucketing of a small batch with the per-row signal of the sparse
// injection of the same rows (Eq. 9; independent of it) in the launch:
// workgroup 0 buckets, the others compute for BK_WAVES * NORM_ROWS_PER_WAVE
// rows each either the criticality norm (w_g null: the body of
// crit_norm_kernel) or the learned gate's logit Delta_r . W_g of the row's
// layer (n rows a layer: the body of gate_logit_kernel), the same bits.
constexpr int NORM_ROWS_PER_WAVE = 2;

template <int DT, bool GATE>
__global__ __launch_bounds__(BK_THREADS) void bucket_norm_kernel(
    const int32_t* __restrict__ scene, int64_t rows, int S, int sbits, int shared_rows,
    int32_t* __restrict__ offsets, int32_t* __restrict__ perm, int32_t* __restrict__ unit_scene,
    int32_t* __restrict__ unit_begin, int32_t* __restrict__ unit_count,
    const char* __restrict__ crit, int64_t row_bytes, uint32_t* __restrict__ key,
    const char* __restrict__ w_g, int64_t n) {
  extern __shared__ int hist[];
  if (blockIdx.x == 0) {
    bucket_small_body(scene, rows, S, sbits, shared_rows, offsets, perm, unit_scene, unit_begin,
                      unit_count, hist);
    return;
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t nwg = gridDim.x - 1;
  const int chunks = (int)(row_bytes / 16);
  for (int64_t r = (int64_t)(blockIdx.x - 1) * BK_WAVES + wv; r < rows; r += nwg * BK_WAVES) {
    float acc;
    if constexpr (GATE)
      acc = row_dot<DT>(crit + r * row_bytes, w_g + (r / n) * row_bytes, chunks, lane);
    else
      acc = row_sumsq<DT>(crit + r * row_bytes, chunks, lane);
    if (lane == 0) key[r] = as_u32(acc);
  }
}

bool launch_bucket_norms(int dt, const int32_t* scene, int64_t rows, int S, int shared_rows,
                         const BucketWs& ws, const void* crit, int d_c, uint32_t* key,
                         hipStream_t st, const void* w_g, int64_t n) {
  if (rows == 0 || bucket_chunks(rows) != 1) return false;
  int sbits = 0;
  while ((1 << sbits) < S) ++sbits;
  const int per_wg = BK_WAVES * NORM_ROWS_PER_WAVE;
  const dim3 grid((unsigned)(1 + (rows + per_wg - 1) / per_wg));
  const int64_t rb = (int64_t)d_c * (dt == DT_BF16 ? 2 : 4);
#define LOOKME_BUCKET_NORM(DT_, G_)                                                         \
  hipLaunchKernelGGL((bucket_norm_kernel<DT_, G_>), grid, dim3(BK_THREADS),                  \
                     (size_t)S * sizeof(int), st, scene, rows, S, sbits, shared_rows,          \
                     ws.offsets, ws.perm, ws.unit_scene, ws.unit_begin, ws.unit_count,         \
                     static_cast<const char*>(crit), rb, key, static_cast<const char*>(w_g), n)
  if (dt == DT_BF16) {
    if (w_g != nullptr) LOOKME_BUCKET_NORM(DT_BF16, true);
    else LOOKME_BUCKET_NORM(DT_BF16, false);
  } else {
    if (w_g != nullptr) LOOKME_BUCKET_NORM(DT_F32, true);
    else LOOKME_BUCKET_NORM(DT_F32, false);
  }
#undef LOOKME_BUCKET_NORM
  return true;
}

hipError_t launch_bucket(const int32_t* scene, int64_t rows, int S, int shared_rows,
                         const BucketWs& ws, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  int sbits = 0;
  while ((1 << sbits) < S) ++sbits;
  const int64_t chunks = bucket_chunks(rows);
  if (chunks == 1) {
    hipLaunchKernelGGL(bucket_small_kernel, dim3(1), dim3(BK_THREADS), (size_t)S * sizeof(int),
                       st, scene, rows, S, sbits, shared_rows, ws.offsets, ws.perm, ws.unit_scene,
                       ws.unit_begin, ws.unit_count);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(bucket_hist_kernel, dim3((unsigned)chunks), dim3(BK_THREADS),
                     (size_t)S * sizeof(int), st, scene, rows, S, sbits, ws.chunk_hist,
                     ws.local_rank);
  // the prefix over chunks in its own launch once the one workgroup would
  // need more than four dependent load rounds for it
  const int64_t rounds = ((S + BK_THREADS - 1) / BK_THREADS) * ((chunks + 7) / 8);
  if (rounds > 4) {
    hipLaunchKernelGGL(bucket_colscan_kernel,
                       dim3((unsigned)((S + COL_THREADS - 1) / COL_THREADS)), dim3(COL_THREADS), 0,
                       st, ws.chunk_hist, chunks, S, ws.offsets);
    hipLaunchKernelGGL(bucket_scan_kernel<true>, dim3(1), dim3(BK_THREADS), 0, st, ws.chunk_hist,
                       chunks, S, shared_rows, ws.offsets, ws.unit_scene, ws.unit_begin,
                       ws.unit_count, ws.split_max);
  } else {
    hipLaunchKernelGGL(bucket_scan_kernel<false>, dim3(1), dim3(BK_THREADS), 0, st, ws.chunk_hist,
                       chunks, S, shared_rows, ws.offsets, ws.unit_scene, ws.unit_begin,
                       ws.unit_count, ws.split_max);
  }
  hipLaunchKernelGGL(bucket_scatter_kernel, dim3((unsigned)chunks), dim3(BK_THREADS), 0, st,
                     scene, rows, S, ws.chunk_hist, ws.local_rank, ws.offsets, ws.perm);
  return hipGetLastError();
}

}  // namespace lookme
