// Sparse injection through the SwiGLU fusion of Eq. 10 (arXiv 2607.16305,
// Sec. 3.3): for the kept tokens of layer l, H <- round(H + f_l(R)) with
// f_l(R) = W_down (silu(W_gate R) * (W_up R)).  R (the weighted row sums,
// rounded) comes from launch_gather_rows; two products on the matrix cores
// (tile_gemm.h), batched over the layers (blockIdx.y):
//
//   gate/up   U = round(silu(R W_gate^T) * (R W_up^T)): every tile computes
//             32 columns of both products for the same rows and combines
//             them in its epilogue;
//   down      H[kept] = round(H[kept] + U W_down^T), written in place (the
//             kept list of the layer maps a product row to its token).
//
// The inter-layer propagation of Eq. 11 (launch_propagate) carries R from a
// LookME layer to the layers after it: R_j = round(R_{j-1} W_p^j + R_{j-1}),
// one product per layer (each needs the previous one), the residual added in
// the epilogue.
#include "common.h"
#include "kernels.h"
#include "tile_gemm.h"

namespace lookme {

hipError_t launch_fusion(int dt, const FusionFfn& f, int layers, int64_t n, int64_t n_keep,
                         const int32_t* kept, int64_t kept_batch, int d_v, const void* r, void* u,
                         void* hidden, hipStream_t st, const int32_t* count) {
  if (n == 0 || n_keep == 0) return hipSuccess;
  const int es = dt == DT_BF16 ? 2 : 4;
  const int64_t rt = (n_keep + TgShape::BM - 1) / TgShape::BM;

  TileGemmParams g1{};
  g1.a0 = static_cast<const char*>(r);
  g1.b = static_cast<const char*>(f.w_gate);
  g1.b2 = static_cast<const char*>(f.w_up);
  g1.out = static_cast<char*>(u);
  g1.rows = n_keep;
  g1.a_bytes = (int64_t)d_v * es;
  g1.k_bytes = g1.a_bytes;
  g1.a_batch = n_keep * g1.a_bytes;
  g1.b_batch = (int64_t)f.d_ff * g1.k_bytes;
  g1.out_batch = n_keep * (int64_t)f.d_ff * es;
  g1.cols = f.d_ff;
  g1.ksplit = (int)(g1.k_bytes / TG_KB);
  g1.tiles = (int)(rt * ((f.d_ff + TgShape::BN / 2 - 1) / (TgShape::BN / 2)));
  g1.count = count;
  g1.count_step = kept_batch != 0 ? 1 : 0;
  hipError_t e = launch_tile_gemm<EPI_SWIGLU>(dt, g1, layers, st);
  if (e != hipSuccess) return e;

  TileGemmParams g2{};
  g2.a0 = static_cast<const char*>(u);
  g2.b = static_cast<const char*>(f.w_down);
  g2.out = static_cast<char*>(hidden);
  g2.kept = kept;
  g2.rows = n_keep;
  g2.a_bytes = (int64_t)f.d_ff * es;
  g2.k_bytes = g2.a_bytes;
  g2.a_batch = n_keep * g2.a_bytes;
  g2.b_batch = (int64_t)f.d_h * g2.k_bytes;
  g2.n = n;
  g2.kept_batch = kept_batch;
  g2.out_ld = (int64_t)f.d_h * es;
  g2.cols = f.d_h;
  g2.ksplit = (int)(g2.k_bytes / TG_KB);
  g2.tiles = (int)(rt * ((f.d_h + TgShape::BN - 1) / TgShape::BN));
  g2.count = count;
  g2.count_step = g1.count_step;
  return launch_tile_gemm<EPI_RESID>(dt, g2, layers, st);
}

hipError_t launch_propagate(int dt, const void* w_p_t, int steps, int64_t n_keep, int d_v,
                            void* r, hipStream_t st, const int32_t* count) {
  if (n_keep == 0) return hipSuccess;
  const int64_t es = dt == DT_BF16 ? 2 : 4;
  const int64_t slice = n_keep * d_v * es;
  const int64_t rt = (n_keep + TgShape::BM - 1) / TgShape::BM;
  for (int j = 1; j <= steps; ++j) {
    TileGemmParams g{};
    g.a0 = static_cast<const char*>(r) + (j - 1) * slice;
    g.res = g.a0;
    g.b = static_cast<const char*>(w_p_t) + (int64_t)(j - 1) * d_v * d_v * es;
    g.out = static_cast<char*>(r) + j * slice;
    g.rows = n_keep;
    g.a_bytes = (int64_t)d_v * es;
    g.k_bytes = g.a_bytes;
    g.cols = d_v;
    g.ksplit = (int)(g.k_bytes / TG_KB);
    g.tiles = (int)(rt * ((d_v + TgShape::BN - 1) / TgShape::BN));
    g.count = count;
    g.count_step = 0;
    const hipError_t e = launch_tile_gemm<EPI_ADD>(dt, g, 1, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace lookme
