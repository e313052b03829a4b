// Multi-scale image retrieval with the token-wise router (arXiv 2607.16305,
// Sec. 3.2, Eq. 8).  Each of the M scales was routed and looked up in its
// own scene partition of the table (scenes [m S/M, (m+1) S/M)); for every kept
// token t this file combines the M retrieved rows:
//
//   gather     R^m_t = round(sum_i w^m[t,i] V[partition m, scene^m_t, prim^m[t,i]])
//              for all scales at once (inject_kernel in gather mode, the kept
//              list shared by the scales, scene ids offset per scale);
//   query      q_t = round(H[t] W_{h->e}) on the matrix cores (tile_gemm.h; the
//              A rows are the kept tokens' hidden states, gathered per row);
//   router     alpha = softmax_m(q_t . R^m_t / sqrt(d_v)), then
//              H[t, :d_v] = round(H[t, :d_v] + sum_m alpha_m R^m_t):
//              ms_router_kernel, one workgroup per kept token.
#include "common.h"
#include "kernels.h"
#include "tile_gemm.h"

namespace lookme {

constexpr int MS_THREADS = 256;

// One workgroup per kept row j: the M dot products over d_v (16-byte chunks
// strided over the threads, float32, then a wave and a workgroup sum in a
// fixed order), the softmax over the scales, and the weighted sum added into
// the token's hidden row with one rounding.
template <int DT>
__global__ __launch_bounds__(MS_THREADS) void ms_router_kernel(
    int64_t n, int64_t n_keep, const int32_t* __restrict__ kept, int M,
    const char* __restrict__ q, const char* __restrict__ r, char* __restrict__ hidden,
    int64_t h_bytes, int64_t v_bytes, float inv_sqrt_d, const int32_t* __restrict__ count) {
  __shared__ float red[MS_MAX_SCALES][MS_THREADS / WAVE];
  const int64_t j = blockIdx.x;
  if (count != nullptr && j >= *count) return;   // past a counted list's end
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int nw = (int)(blockDim.x / WAVE);
  int64_t t = kept[j];
  t = t < 0 ? 0 : (t >= n ? n - 1 : t);
  const int chunks = (int)(v_bytes / 16);
  const char* qrow = q + j * v_bytes;

  float dot[MS_MAX_SCALES];
#pragma unroll
  for (int m = 0; m < MS_MAX_SCALES; ++m) dot[m] = 0.f;
  for (int c = tid; c < chunks; c += blockDim.x) {
    const u32x4_t qv = ld16(qrow + (int64_t)c * 16);
#pragma unroll
    for (int m = 0; m < MS_MAX_SCALES; ++m) {
      if (m < M) {
        const u32x4_t rv = ld16(r + ((int64_t)m * n_keep + j) * v_bytes + (int64_t)c * 16);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if constexpr (DT == DT_BF16) {
            dot[m] = fmaf(bf16lo(qv[e]), bf16lo(rv[e]), dot[m]);
            dot[m] = fmaf(bf16hi(qv[e]), bf16hi(rv[e]), dot[m]);
          } else {
            dot[m] = fmaf(as_f32(qv[e]), as_f32(rv[e]), dot[m]);
          }
        }
      }
    }
  }
#pragma unroll
  for (int m = 0; m < MS_MAX_SCALES; ++m) {
    if (m < M) {
      float v = dot[m];
#pragma unroll
      for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
      if (lane == 0) red[m][wv] = v;
    }
  }
  __syncthreads();
  float alpha[MS_MAX_SCALES];
  float top = -__builtin_inff();
#pragma unroll
  for (int m = 0; m < MS_MAX_SCALES; ++m) {
    alpha[m] = 0.f;
    if (m < M) {
      float v = 0.f;
      for (int w = 0; w < nw; ++w) v += red[m][w];
      alpha[m] = v * inv_sqrt_d;
      top = fmaxf(top, alpha[m]);
    }
  }
  float sum = 0.f;
#pragma unroll
  for (int m = 0; m < MS_MAX_SCALES; ++m) {
    if (m < M) {
      alpha[m] = expf(alpha[m] - top);
      sum += alpha[m];
    }
  }
#pragma unroll
  for (int m = 0; m < MS_MAX_SCALES; ++m) alpha[m] = alpha[m] / sum;

  char* h = hidden + t * h_bytes;
  for (int c = tid; c < chunks; c += blockDim.x) {
    const u32x4_t hv = ld16(h + (int64_t)c * 16);
    u32x4_t out;
    if constexpr (DT == DT_BF16) {
      float acc[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll
      for (int m = 0; m < MS_MAX_SCALES; ++m) {
        if (m < M) {
          const u32x4_t rv = ld16(r + ((int64_t)m * n_keep + j) * v_bytes + (int64_t)c * 16);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[2 * e] = fmaf(alpha[m], bf16lo(rv[e]), acc[2 * e]);
            acc[2 * e + 1] = fmaf(alpha[m], bf16hi(rv[e]), acc[2 * e + 1]);
          }
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e)
        out[e] = pack_bf16x2(bf16lo(hv[e]) + acc[2 * e], bf16hi(hv[e]) + acc[2 * e + 1]);
    } else {
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int m = 0; m < MS_MAX_SCALES; ++m) {
        if (m < M) {
          const u32x4_t rv = ld16(r + ((int64_t)m * n_keep + j) * v_bytes + (int64_t)c * 16);
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] = fmaf(alpha[m], as_f32(rv[e]), acc[e]);
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) out[e] = as_u32(as_f32(hv[e]) + acc[e]);
    }
    st16(h + (int64_t)c * 16, out);
  }
}

hipError_t launch_multiscale(int dt, int scales, int64_t n, int64_t n_keep, const int32_t* kept,
                             const int32_t* scene, const int32_t* prim, const float* w,
                             const void* values, int S, int P, int d_v, int k,
                             const void* w_he_t, int d_h, void* hidden, void* r, void* q,
                             hipStream_t st, const int32_t* count) {
  if (n == 0 || n_keep == 0) return hipSuccess;
  const int es = dt == DT_BF16 ? 2 : 4;
  const int Sm = S / scales;
  hipError_t e = launch_gather_rows(dt, scales, n, n_keep, kept, scene, prim, w, values, Sm, P,
                                    d_v, k, r, st, 0, Sm, count);
  if (e != hipSuccess) return e;

  // q = round(H[kept] W_he): every K stage of an A row comes from the kept
  // token's hidden row (a1 gathered by sel = kept)
  TileGemmParams g{};
  g.a0 = static_cast<const char*>(hidden);
  g.a1 = static_cast<const char*>(hidden);
  g.sel = kept;
  g.sel_rows = (int)n;
  g.b = static_cast<const char*>(w_he_t);
  g.out = static_cast<char*>(q);
  g.rows = n_keep;
  g.a_bytes = (int64_t)d_h * es;
  g.k_bytes = g.a_bytes;
  g.cols = d_v;
  g.ksplit = 0;
  g.count = count;   // a counted list: rows past count[0] are skipped
  g.count_step = 0;
  g.tiles = (int)(((n_keep + TgShape::BM - 1) / TgShape::BM) *
                  ((d_v + TgShape::BN - 1) / TgShape::BN));
  e = launch_tile_gemm<EPI_STORE>(dt, g, 1, st);
  if (e != hipSuccess) return e;

  const int64_t vb = (int64_t)d_v * es;
  const int ch = (int)(vb / 16);
  const int bs = ch >= MS_THREADS ? MS_THREADS : (ch + 63) / 64 * 64;
  const float inv_sqrt_d = 1.0f / sqrtf((float)d_v);
  if (dt == DT_BF16)
    hipLaunchKernelGGL(ms_router_kernel<DT_BF16>, dim3((unsigned)n_keep), dim3(bs), 0, st, n,
                       n_keep, kept, scales, static_cast<const char*>(q),
                       static_cast<const char*>(r), static_cast<char*>(hidden),
                       (int64_t)d_h * es, vb, inv_sqrt_d, count);
  else
    hipLaunchKernelGGL(ms_router_kernel<DT_F32>, dim3((unsigned)n_keep), dim3(bs), 0, st, n,
                       n_keep, kept, scales, static_cast<const char*>(q),
                       static_cast<const char*>(r), static_cast<char*>(hidden),
                       (int64_t)d_h * es, vb, inv_sqrt_d, count);
  return hipGetLastError();
}

}  // namespace lookme
