// Level-2 in the paper's own form (arXiv 2607.16305, Sec. 3.2, Eq. 6-7):
// a scene-shared two-layer MLP on [v_e, e_img[j]] gives one relevance logit
// per primitive, the top k primitives by logit are kept, and their weights
// are the softmax of cos(v_e, e_{j,p}) + tanh(r_j[p]).  Four launches:
//
//   tile_gemm_kernel (hidden)  a = round(ReLU([q_t, K1[scene_t]] W1^T + b1)):
//                             64 x 64 output tiles on the matrix cores, the
//                             operand-A row of token t being its query
//                             followed by its scene's key (gathered per row,
//                             K stages of 128 bytes straight into LDS);
//   tile_gemm_kernel (logits)  r = a W2^T + b2 in float32, to the workspace
//                             (large products: the projection's 256 x 256
//                             tile kernel with a float32 + bias epilogue);
//   relevance_topk_kernel     one wave per row: the k largest logits (lowest
//                             p on ties), each lane keeping a sorted list of
//                             its strided share, merged across the wave;
//   relevance_weights_kernel  one wave per row: the k cosines against the
//                             chosen primitive keys, + tanh of the logits,
//                             softmax over the k.
#include "common.h"
#include "kernels.h"
#include "tile_gemm.h"

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

hipError_t launch_relevance(int dt, const void* q, const int32_t* scene, const void* scene_keys,
                            const void* prim_keys, const RelevanceMlp& mlp, int64_t rows, int d_e,
                            int S, int P, int k, void* act, int32_t* prim, float* w,
                            float* logits, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  const int es = dt == DT_BF16 ? 2 : 4;
  const int64_t rt = (rows + TgShape::BM - 1) / TgShape::BM;
  // hidden layer: K = [query ; scene key]
  TileGemmParams g1{};
  g1.a0 = static_cast<const char*>(q);
  g1.a1 = static_cast<const char*>(scene_keys);
  g1.sel = scene;
  g1.b = static_cast<const char*>(mlp.w1);
  g1.bias = mlp.b1;
  g1.out = static_cast<char*>(act);
  g1.rows = rows;
  g1.a_bytes = (int64_t)d_e * es;
  g1.k_bytes = 2 * g1.a_bytes;
  g1.sel_rows = S;
  g1.cols = mlp.hidden;
  g1.ksplit = (int)(g1.a_bytes / TG_KB);
  g1.tiles = (int)(rt * ((mlp.hidden + TgShape::BN - 1) / TgShape::BN));
  hipError_t e = launch_tile_gemm<EPI_ACT>(dt, g1, 1, st);
  if (e != hipSuccess) return e;
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
#define LOOKME_RW(DT_, K_)                                                                       \
  hipLaunchKernelGGL((relevance_weights_kernel<DT_, K_>), wgrid, dim3(256), 0, st,             \
                     static_cast<const char*>(q), scene, static_cast<const char*>(prim_keys), \
                     prim, w, rows, S, P, k, (int64_t)d_e * es)
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

}  // namespace lookme
