// Sparse injection (arXiv 2607.16305, Sec. 3.3, Eq. 9-10) and the residual
// add of Eq. 2: the criticality of token t is ||Delta_t||_2 (the size of the
// attention update that drives the SKA gate); the n_keep most critical tokens
// of every layer receive H[t, :d_v] += sum_i w_i * V[scene_t * P + p_i, :].
//
//   crit_norm   one wave per row streams Delta once (HBM-bound) and stores
//               the fp32 sum of squares as its bit pattern (non-negative
//               floats order like their bits, and the square root keeps the
//               order, so selecting on it selects on the norm);
//   crit_select one workgroup per layer: 4-pass MSB-first radix select of
//               the n_keep-th largest key (keys cached in LDS when they
//               fit), then an order-preserving compaction (block prefix
//               sums) of the kept token ids;
//   inject      one workgroup per kept token (one thread per 16-byte chunk of
//               a row, up to 256): coalesced loads of its k table rows (all
//               in flight together), fp32 weighted sum in a fixed order, one
//               rounding of H + sum, in-place store.  The table rows are read
//               with the normal cache policy: tokens of one scene pick many of
//               the same primitives (the Zipf batch's 104864 gathered rows are
//               30680 distinct ones), and the caches serve the repeats (with
//               the nontemporal hint the kernel took 44.7 us there, without
//               27.4 us; multi-scale 23.2 -> 19.0, 4-layer 73.3 -> 65.5).
#include "common.h"
#include "crit.h"
#include "kernels.h"

namespace lookme {

constexpr int NORM_WAVES = 4;
constexpr int64_t NORM_BACKGROUND_WGS = 256;
constexpr int INJ_THREADS = 256;

template <int DT>
__global__ __launch_bounds__(NORM_WAVES * WAVE) void crit_norm_kernel(
    const char* __restrict__ crit, int64_t rows, int64_t row_bytes,
    uint32_t* __restrict__ key) {
  const int lane = threadIdx.x & 63;
  for (int64_t r = (int64_t)blockIdx.x * NORM_WAVES + (threadIdx.x >> 6); r < rows;
       r += (int64_t)gridDim.x * NORM_WAVES) {
    const float acc = row_sumsq<DT>(crit + r * row_bytes, (int)(row_bytes / 16), lane);
    if (lane == 0) key[r] = as_u32(acc);
  }
}

template <int CN>
__global__ __launch_bounds__(SEL_THREADS) void crit_select_kernel(
    const uint32_t* __restrict__ key_all, int64_t n, int64_t n_keep,
    int32_t* __restrict__ kept_all) {
  __shared__ uint32_t cache[sel_cache_words(CN)];
  __shared__ SelLds sl;
  const int layer = blockIdx.x;
  select_layer<CN>(key_all + (int64_t)layer * n, n, n_keep, kept_all + (int64_t)layer * n_keep,
                   cache, sl);
}

// Rows of the injections whose kept id, scene or primitive index lay outside
// its range since the counter was last read (lookme_index_errors): such a
// row is not injected (in TO_R form its R row is written as zeros), so a
// caller's bad index is counted instead of adding some other row into H.
__device__ unsigned long long g_index_errors;

// TO_R: the weighted row sum R of kept row j is rounded to the storage
// dtype and written to row j of `hidden` (the fusion's or the multi-scale
// router's input, [rows, d_v]) instead of being added into H.  Layer l reads
// its kept list at kept + l * kept_batch (0: one list for all layers) and
// its scenes (in [0, S)) from scene l * scene_step of the table (multi-scale:
// scale l's partition).  With a count array only the first count entries of
// a kept list are used (count[l], or count[0] for a list shared by all
// layers).
template <int DT, int K, bool TO_R = false>
__global__ __launch_bounds__(INJ_THREADS) void inject_kernel(
    int64_t n, int64_t n_keep, const int32_t* __restrict__ kept_all,
    const int32_t* __restrict__ scene_all, const int32_t* __restrict__ prim_all,
    const float* __restrict__ w_all, const char* __restrict__ values, int S, int P, int k,
    int64_t v_bytes, char* __restrict__ hidden, int64_t h_bytes, int64_t kept_batch,
    int scene_step, const int32_t* __restrict__ count) {
  const int64_t j = blockIdx.x;
  const int64_t layer = j / n_keep;
  // counted lists (the learned gate): entries past the list's count are unused
  if (count != nullptr && j - layer * n_keep >= count[kept_batch != 0 ? layer : 0]) return;
  const int chunks = (int)(v_bytes / 16);
  // an index out of range: count the row once and leave it out (every
  // index below is uniform over the workgroup)
  auto reject = [&]() {
    if (threadIdx.x == 0) atomicAdd(&g_index_errors, 1ull);
    if constexpr (TO_R)
      for (int c = threadIdx.x; c < chunks; c += blockDim.x)
        st16(hidden + j * v_bytes + (int64_t)c * 16, u32x4_t{0, 0, 0, 0});
  };
  const int64_t t = kept_all[layer * kept_batch + (j - layer * n_keep)];
  if (t < 0 || t >= n) return reject();
  const int64_t row = layer * n + t;
  const int s0 = scene_all[row];
  if (s0 < 0 || s0 >= S) return reject();
  const int s = s0 + (int)layer * scene_step;
  int64_t vrow[K];
  float wt[K];
  bool bad = false;
#pragma unroll
  for (int i = 0; i < K; ++i) {
    if (i < k) {
      const int p = prim_all[row * k + i];
      bad |= p < 0 || p >= P;
      vrow[i] = (int64_t)s * P + p;
      wt[i] = w_all[row * k + i];
    } else {
      vrow[i] = 0;
      wt[i] = 0.f;
    }
  }
  if (bad) return reject();
  char* h = TO_R ? hidden + j * v_bytes : hidden + row * h_bytes;
  for (int c = threadIdx.x; c < chunks; c += blockDim.x) {
    u32x4_t vv[K];
#pragma unroll
    for (int i = 0; i < K; ++i)
      if (i < k) vv[i] = ld16(values + vrow[i] * v_bytes + (int64_t)c * 16);
    const u32x4_t hv = TO_R ? u32x4_t{0, 0, 0, 0} : ld16(h + (int64_t)c * 16);
    u32x4_t out;
    if constexpr (DT == DT_BF16) {
      float acc[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll
      for (int i = 0; i < K; ++i) {
        if (i < k) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[2 * e] = fmaf(wt[i], bf16lo(vv[i][e]), acc[2 * e]);
            acc[2 * e + 1] = fmaf(wt[i], bf16hi(vv[i][e]), acc[2 * e + 1]);
          }
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e)
        out[e] = pack_bf16x2(bf16lo(hv[e]) + acc[2 * e], bf16hi(hv[e]) + acc[2 * e + 1]);
    } else {
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < K; ++i) {
        if (i < k) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc[e] = fmaf(wt[i], as_f32(vv[i][e]), acc[e]);
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e)
        out[e] = as_u32(as_f32(hv[e]) + acc[e]);
    }
    st16(h + (int64_t)c * 16, out);
  }
}

template <int DT, bool TO_R = false>
static void launch_inject_k(int kk, dim3 grid, hipStream_t st, int64_t n, int64_t n_keep,
                            const int32_t* kept, const int32_t* scene, const int32_t* prim,
                            const float* w, const char* values, int S, int P, int64_t vb,
                            char* hidden, int64_t hb, int64_t kept_batch, int scene_step,
                            const int32_t* count = nullptr) {
  // as many whole waves as the row has 16-byte chunks (up to 256 threads):
  // narrow rows leave no thread idle, and the CU holds more workgroups
  const int ch = (int)(vb / 16);
  const int bs = ch >= INJ_THREADS ? INJ_THREADS : (ch + 63) / 64 * 64;
#define LOOKME_INJ(K_)                                                                \
  hipLaunchKernelGGL((inject_kernel<DT, K_, TO_R>), grid, dim3(bs), 0, st, n, n_keep, kept, \
                     scene, prim, w, values, S, P, kk, vb, hidden, hb, kept_batch, scene_step, \
                     count)
  if (kk <= 4) LOOKME_INJ(4);
  else if (kk <= 8) LOOKME_INJ(8);
  else if (kk <= 16) LOOKME_INJ(16);
  else LOOKME_INJ(32);
#undef LOOKME_INJ
}

hipError_t launch_crit_norm(int dt, int64_t rows, const void* crit, int d_c, uint32_t* key,
                            hipStream_t st, bool background) {
  if (rows == 0) return hipSuccess;
  const int es = dt == DT_BF16 ? 2 : 4;
  // a wave a row; in the background form 256 workgroups walk the rows, one
  // per CU, so that the norms leave the projection and routing running
  // beside them most of every CU (Zipf batch: those two 312 -> 289 us, the
  // step 2.248 -> 2.216 ms median, while the norms stretch from 107 to
  // ~185 us behind them)
  const int64_t g0 = (rows + NORM_WAVES - 1) / NORM_WAVES;
  const dim3 grid((unsigned)(background && g0 > NORM_BACKGROUND_WGS ? NORM_BACKGROUND_WGS : g0));
  if (dt == DT_BF16)
    hipLaunchKernelGGL(crit_norm_kernel<DT_BF16>, grid, dim3(NORM_WAVES * WAVE), 0, st,
                       static_cast<const char*>(crit), rows, (int64_t)d_c * es, key);
  else
    hipLaunchKernelGGL(crit_norm_kernel<DT_F32>, grid, dim3(NORM_WAVES * WAVE), 0, st,
                       static_cast<const char*>(crit), rows, (int64_t)d_c * es, key);
  return hipGetLastError();
}

hipError_t launch_crit_select(int layers, int64_t n, int64_t n_keep, const uint32_t* key,
                              int32_t* kept, hipStream_t st) {
  if (n == 0 || n_keep == 0) return hipSuccess;
  if (n <= SEL_CACHE_SMALL)
    hipLaunchKernelGGL(crit_select_kernel<SEL_CACHE_SMALL>, dim3(layers), dim3(SEL_THREADS), 0, st,
                       key, n, n_keep, kept);
  else if (n <= SEL_CACHE_N)
    hipLaunchKernelGGL(crit_select_kernel<SEL_CACHE_N>, dim3(layers), dim3(SEL_THREADS), 0, st,
                       key, n, n_keep, kept);
  else
    hipLaunchKernelGGL(crit_select_kernel<0>, dim3(layers), dim3(SEL_THREADS), 0, st, key, n,
                       n_keep, kept);
  return hipGetLastError();
}

hipError_t take_index_errors(hipStream_t st, uint64_t* out) {
  static const unsigned long long zero = 0;
  unsigned long long v = 0;
  hipError_t e = hipMemcpyFromSymbolAsync(&v, HIP_SYMBOL(g_index_errors), sizeof(v), 0,
                                          hipMemcpyDeviceToHost, st);
  if (e == hipSuccess)
    e = hipMemcpyToSymbolAsync(HIP_SYMBOL(g_index_errors), &zero, sizeof(zero), 0,
                               hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e == hipSuccess) *out = v;
  return e;
}

hipError_t launch_inject_rows(int dt, int layers, int64_t n, int64_t n_keep, const int32_t* kept,
                              const int32_t* scene, const int32_t* prim, const float* w,
                              const void* values, int S, int P, int d_v, int k, void* hidden,
                              int d_h, hipStream_t st, const int32_t* count) {
  if (n == 0 || n_keep == 0) return hipSuccess;
  const int es = dt == DT_BF16 ? 2 : 4;
  const dim3 grid((unsigned)(layers * n_keep));
  if (dt == DT_BF16)
    launch_inject_k<DT_BF16>(k, grid, st, n, n_keep, kept, scene, prim, w,
                             static_cast<const char*>(values), S, P, (int64_t)d_v * es,
                             static_cast<char*>(hidden), (int64_t)d_h * es, n_keep, 0, count);
  else
    launch_inject_k<DT_F32>(k, grid, st, n, n_keep, kept, scene, prim, w,
                            static_cast<const char*>(values), S, P, (int64_t)d_v * es,
                            static_cast<char*>(hidden), (int64_t)d_h * es, n_keep, 0, count);
  return hipGetLastError();
}

hipError_t launch_gather_rows(int dt, int layers, int64_t n, int64_t n_keep, const int32_t* kept,
                              const int32_t* scene, const int32_t* prim, const float* w,
                              const void* values, int S, int P, int d_v, int k, void* r_out,
                              hipStream_t st, int64_t kept_batch, int scene_step,
                              const int32_t* count) {
  if (n == 0 || n_keep == 0) return hipSuccess;
  const int es = dt == DT_BF16 ? 2 : 4;
  const dim3 grid((unsigned)(layers * n_keep));
  if (dt == DT_BF16)
    launch_inject_k<DT_BF16, true>(k, grid, st, n, n_keep, kept, scene, prim, w,
                                   static_cast<const char*>(values), S, P, (int64_t)d_v * es,
                                   static_cast<char*>(r_out), 0, kept_batch, scene_step,
                                   count);
  else
    launch_inject_k<DT_F32, true>(k, grid, st, n, n_keep, kept, scene, prim, w,
                                  static_cast<const char*>(values), S, P, (int64_t)d_v * es,
                                  static_cast<char*>(r_out), 0, kept_batch, scene_step,
                                  count);
  return hipGetLastError();
}

}  // namespace lookme
