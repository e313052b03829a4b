// Bucketing of query rows by their Level-1 scene (Sec. 3.2: rows routed to
// the same scene share that scene's primitive keys in Level-2).
//
// A stable counting sort in three passes, every step deterministic:
//   1. per 1024-row chunk: a histogram over scenes and, for every row, its
//      rank among equal-scene rows earlier in the chunk (wave match masks
//      built from ballots over the scene bits, then the 16 waves in order);
//   2. one workgroup: per-scene prefix over chunks, exclusive scan over
//      scenes (wavefront prefix sums) giving bucket offsets, and the work
//      list of 16-row tiles of every non-empty bucket;
//   3. per chunk: perm[offset + chunk prefix + rank] = row.
// Within a bucket rows keep ascending order.  Scene values outside [0, S)
// are clamped (results for such rows are undefined; memory stays in bounds).
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace lookme {

constexpr int BK_THREADS = 1024;
constexpr int BK_WAVES = BK_THREADS / WAVE;
constexpr int TILE_ROWS = 16;

int64_t bucket_chunks(int64_t rows) { return (rows + BK_THREADS - 1) / BK_THREADS; }

int64_t bucket_max_units(int64_t rows, int S) {
  return std::min<int64_t>(S, rows) + (rows + TILE_ROWS - 1) / TILE_ROWS;
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

// Exclusive block prefix of (a, b) pairs over the block's threads; returns
// the totals through the references.
__device__ __forceinline__ void block_excl_scan2(int& a, int& b, int& tot_a, int& tot_b) {
  __shared__ int wa[BK_WAVES], wb[BK_WAVES];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int ia = wave_incl_scan(a), ib = wave_incl_scan(b);
  if (lane == 63) { wa[wv] = ia; wb[wv] = ib; }
  __syncthreads();
  int pa = 0, pb = 0;
  tot_a = 0;
  tot_b = 0;
  for (int w = 0; w < BK_WAVES; ++w) {
    if (w < wv) { pa += wa[w]; pb += wb[w]; }
    tot_a += wa[w];
    tot_b += wb[w];
  }
  a = pa + ia - a;
  b = pb + ib - b;
  __syncthreads();
}

__global__ __launch_bounds__(BK_THREADS) void bucket_scan_kernel(
    int32_t* __restrict__ chunk_hist, int64_t chunks, int S, int32_t* __restrict__ offsets,
    int32_t* __restrict__ unit_scene, int32_t* __restrict__ unit_begin,
    int32_t* __restrict__ unit_count) {
  // 1. per-scene prefix over chunks; bucket sizes go to offsets[] for now
  // (loads are batched so that eight chunk reads are in flight at a time)
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
  // 2. exclusive scan of sizes and of tile counts over scenes
  const int ipt = (S + BK_THREADS - 1) / BK_THREADS;
  const int s0 = min(S, (int)threadIdx.x * ipt), s1 = min(S, s0 + ipt);
  int sum_rows = 0, sum_tiles = 0;
  for (int s = s0; s < s1; ++s) {
    sum_rows += offsets[s];
    sum_tiles += (offsets[s] + TILE_ROWS - 1) / TILE_ROWS;
  }
  int pre_rows = sum_rows, pre_tiles = sum_tiles, tot_rows, tot_tiles;
  block_excl_scan2(pre_rows, pre_tiles, tot_rows, tot_tiles);
  for (int s = s0; s < s1; ++s) {
    const int size = offsets[s];
    const int tiles = (size + TILE_ROWS - 1) / TILE_ROWS;
    offsets[s] = pre_rows;
    for (int t = 0; t < tiles; ++t) {
      unit_scene[pre_tiles + t] = s;
      unit_begin[pre_tiles + t] = pre_rows + t * TILE_ROWS;
    }
    pre_rows += size;
    pre_tiles += tiles;
  }
  if (threadIdx.x == 0) {
    offsets[S] = tot_rows;
    *unit_count = tot_tiles;
  }
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
// (saves two launches where launch latency dominates).
__global__ __launch_bounds__(BK_THREADS) void bucket_small_kernel(
    const int32_t* __restrict__ scene, int64_t rows, int S, int sbits,
    int32_t* __restrict__ offsets, int32_t* __restrict__ perm, int32_t* __restrict__ unit_scene,
    int32_t* __restrict__ unit_begin, int32_t* __restrict__ unit_count) {
  extern __shared__ int hist[];
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
  // bucket offsets and the tile work list (hist[] becomes the offsets)
  const int ipt = (S + BK_THREADS - 1) / BK_THREADS;
  const int s0 = min(S, (int)threadIdx.x * ipt), s1 = min(S, s0 + ipt);
  int sum_rows = 0, sum_tiles = 0;
  for (int x = s0; x < s1; ++x) {
    sum_rows += hist[x];
    sum_tiles += (hist[x] + TILE_ROWS - 1) / TILE_ROWS;
  }
  int pre_rows = sum_rows, pre_tiles = sum_tiles, tot_rows, tot_tiles;
  block_excl_scan2(pre_rows, pre_tiles, tot_rows, tot_tiles);
  for (int x = s0; x < s1; ++x) {
    const int size = hist[x];
    const int tiles = (size + TILE_ROWS - 1) / TILE_ROWS;
    hist[x] = pre_rows;
    offsets[x] = pre_rows;
    for (int u = 0; u < tiles; ++u) {
      unit_scene[pre_tiles + u] = x;
      unit_begin[pre_tiles + u] = pre_rows + u * TILE_ROWS;
    }
    pre_rows += size;
    pre_tiles += tiles;
  }
  if (threadIdx.x == 0) {
    offsets[S] = tot_rows;
    *unit_count = tot_tiles;
  }
  __syncthreads();
  if (valid) perm[hist[s] + rank] = t;
}

hipError_t launch_bucket(const int32_t* scene, int64_t rows, int S, const BucketWs& ws,
                         hipStream_t st) {
  if (rows == 0) return hipSuccess;
  int sbits = 0;
  while ((1 << sbits) < S) ++sbits;
  const int64_t chunks = bucket_chunks(rows);
  if (chunks == 1) {
    hipLaunchKernelGGL(bucket_small_kernel, dim3(1), dim3(BK_THREADS), (size_t)S * sizeof(int),
                       st, scene, rows, S, sbits, ws.offsets, ws.perm, ws.unit_scene,
                       ws.unit_begin, ws.unit_count);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(bucket_hist_kernel, dim3((unsigned)chunks), dim3(BK_THREADS),
                     (size_t)S * sizeof(int), st, scene, rows, S, sbits, ws.chunk_hist,
                     ws.local_rank);
  hipLaunchKernelGGL(bucket_scan_kernel, dim3(1), dim3(BK_THREADS), 0, st, ws.chunk_hist, chunks,
                     S, ws.offsets, ws.unit_scene, ws.unit_begin, ws.unit_count);
  hipLaunchKernelGGL(bucket_scatter_kernel, dim3((unsigned)chunks), dim3(BK_THREADS), 0, st,
                     scene, rows, S, ws.chunk_hist, ws.local_rank, ws.offsets, ws.perm);
  return hipGetLastError();
}

}  // namespace lookme
