// Scene-centred keys (arXiv 2607.16305, Sec. 3.2, Eq. 4): a scene's key is
// the mean of its primitive embeddings, K1[s] = (1 / P) sum_p K2[s, p, :].
//
// One thread per (scene, 16-byte chunk of the key row): the P rows of the
// scene are walked in p order, SK_UNROLL of them in flight a thread, each
// element summed in float32 in that order; the sum is divided by P once and
// rounded once to the storage dtype.  The threads of a scene read one row's
// contiguous bytes at a time (coalesced); the 16 GiB of the largest
// workload's keys stream once.
#include "common.h"
#include "kernels.h"

namespace lookme {

constexpr int SK_THREADS = 256;
constexpr int SK_UNROLL = 8;

template <int DT>
__global__ __launch_bounds__(SK_THREADS) void scene_keys_kernel(const char* __restrict__ prim_keys,
                                                                int S, int P, int64_t row_bytes,
                                                                char* __restrict__ out) {
  const int chunks = (int)(row_bytes / 16);
  const int64_t tid = (int64_t)blockIdx.x * SK_THREADS + threadIdx.x;
  if (tid >= (int64_t)S * chunks) return;
  const int s = (int)(tid / chunks), c = (int)(tid % chunks);
  constexpr int NE = DT == DT_BF16 ? 8 : 4;
  float acc[NE];
#pragma unroll
  for (int e = 0; e < NE; ++e) acc[e] = 0.f;
  const char* base = prim_keys + (int64_t)s * P * row_bytes + (int64_t)c * 16;
  for (int p0 = 0; p0 < P; p0 += SK_UNROLL) {
    u32x4_t v[SK_UNROLL];
#pragma unroll
    for (int u = 0; u < SK_UNROLL; ++u)
      v[u] = p0 + u < P ? ld16_nt(base + (int64_t)(p0 + u) * row_bytes) : u32x4_t{0, 0, 0, 0};
#pragma unroll
    for (int u = 0; u < SK_UNROLL; ++u) {
      if (p0 + u >= P) break;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if constexpr (DT == DT_BF16) {
          acc[2 * e] += bf16lo(v[u][e]);
          acc[2 * e + 1] += bf16hi(v[u][e]);
        } else {
          acc[e] += as_f32(v[u][e]);
        }
      }
    }
  }
  const float fp = (float)P;
  u32x4_t o;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if constexpr (DT == DT_BF16)
      o[e] = pack_bf16x2(acc[2 * e] / fp, acc[2 * e + 1] / fp);
    else
      o[e] = as_u32(acc[e] / fp);
  }
  st16(out + (int64_t)s * row_bytes + (int64_t)c * 16, o);
}

hipError_t launch_scene_keys(int dt, const void* prim_keys, int S, int P, int d_e,
                             void* scene_keys, hipStream_t st) {
  const int64_t rb = (int64_t)d_e * (dt == DT_BF16 ? 2 : 4);
  const int64_t threads = (int64_t)S * (rb / 16);
  const dim3 grid((unsigned)((threads + SK_THREADS - 1) / SK_THREADS));
  if (dt == DT_BF16)
    hipLaunchKernelGGL(scene_keys_kernel<DT_BF16>, grid, dim3(SK_THREADS), 0, st,
                       static_cast<const char*>(prim_keys), S, P, rb,
                       static_cast<char*>(scene_keys));
  else
    hipLaunchKernelGGL(scene_keys_kernel<DT_F32>, grid, dim3(SK_THREADS), 0, st,
                       static_cast<const char*>(prim_keys), S, P, rb,
                       static_cast<char*>(scene_keys));
  return hipGetLastError();
}

}  // namespace lookme
