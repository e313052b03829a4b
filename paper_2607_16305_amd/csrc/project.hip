// Query projection v_e = v W_{v->e} (arXiv 2607.16305, Sec. 3.2, Level-1),
// for all layers at once: the per-layer matrices are stacked along the
// output dimension, so x is read once for every layer.
//
// C[M, N] = A[M, K] . B[N, K]^T with A = x [n, d_in], B = W^T stacked
// [layers * d_e, d_in]; C is rounded once to the storage dtype and scattered
// to q[layer, token, :].  Tiled on LDS for the matrix cores: a BM x BN output
// tile per workgroup of 4 waves in a 2 x 2 grid (128 x 128, each wave 4 x 4
// MFMA tiles, when that gives enough tiles to fill the chip; 64 x 64 else),
// 128-byte K stages double-buffered in LDS (rows padded by 16 bytes so the
// 16-byte fragment reads of 8 consecutive rows hit distinct banks), the next
// stage's global loads in flight while the current one is multiplied.
#include "common.h"
#include "kernels.h"

namespace lookme {

constexpr int PJ_STAGE = 128;                // bytes of K per stage and row
constexpr int PJ_LD = PJ_STAGE + 16;         // padded LDS row pitch
constexpr int PJ_THREADS = 256;
constexpr int PJ_CPR = PJ_STAGE / 16;        // 16-byte chunks per row per stage

template <int DT, int BM, int BN>
__global__ __launch_bounds__(PJ_THREADS) void project_kernel(
    const char* __restrict__ A, const char* __restrict__ B, char* __restrict__ Q, int64_t M,
    int N, int64_t k_bytes, int d_e) {
  constexpr int MI = BM / 32, NJ = BN / 32;  // 16 x 16 MFMA tiles per wave
  constexpr int LA = BM * PJ_CPR / PJ_THREADS, LB = BN * PJ_CPR / PJ_THREADS;
  __shared__ __attribute__((aligned(16))) char lds_a[2][BM * PJ_LD];
  __shared__ __attribute__((aligned(16))) char lds_b[2][BN * PJ_LD];
  constexpr int ES = DT == DT_BF16 ? 2 : 4;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wv = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int wm = (wv >> 1) * (BM / 2), wn = (wv & 1) * (BN / 2);

  const int64_t tiles_n = (N + BN - 1) / BN;
  const int64_t m0 = (int64_t)(blockIdx.x / tiles_n) * BM;
  const int n0 = (int)(blockIdx.x % tiles_n) * BN;
  const int kchunks = (int)(k_bytes / 16);
  const int nstages = (int)((k_bytes + PJ_STAGE - 1) / PJ_STAGE);

  u32x4_t ra[LA], rb[LB];
  auto gload = [&](int stage) {
#pragma unroll
    for (int r = 0; r < LA; ++r) {
      const int ci = tid + r * PJ_THREADS;
      const int kc = stage * PJ_CPR + ci % PJ_CPR;
      const int64_t am = m0 + ci / PJ_CPR;
      ra[r] = (am < M && kc < kchunks) ? ld16(A + am * k_bytes + (int64_t)kc * 16)
                                       : u32x4_t{0, 0, 0, 0};
    }
#pragma unroll
    for (int r = 0; r < LB; ++r) {
      const int ci = tid + r * PJ_THREADS;
      const int kc = stage * PJ_CPR + ci % PJ_CPR;
      const int bn = n0 + ci / PJ_CPR;
      rb[r] = (bn < N && kc < kchunks) ? ld16(B + (int64_t)bn * k_bytes + (int64_t)kc * 16)
                                       : u32x4_t{0, 0, 0, 0};
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int r = 0; r < LA; ++r) {
      const int ci = tid + r * PJ_THREADS;
      st16(&lds_a[buf][(ci / PJ_CPR) * PJ_LD + (ci % PJ_CPR) * 16], ra[r]);
    }
#pragma unroll
    for (int r = 0; r < LB; ++r) {
      const int ci = tid + r * PJ_THREADS;
      st16(&lds_b[buf][(ci / PJ_CPR) * PJ_LD + (ci % PJ_CPR) * 16], rb[r]);
    }
  };

  f32x4_t acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  gload(0);
  lstore(0);
  __syncthreads();
  for (int st = 0; st < nstages; ++st) {
    const int buf = st & 1;
    if (st + 1 < nstages) gload(st + 1);
#pragma unroll
    for (int s = 0; s < PJ_STAGE / 64; ++s) {
      u32x4_t fa[MI], fb[NJ];
#pragma unroll
      for (int i = 0; i < MI; ++i)
        fa[i] = *reinterpret_cast<const u32x4_t*>(
            &lds_a[buf][(wm + 16 * i + n16) * PJ_LD + (4 * s + g) * 16]);
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        fb[j] = *reinterpret_cast<const u32x4_t*>(
            &lds_b[buf][(wn + 16 * j + n16) * PJ_LD + (4 * s + g) * 16]);
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = mfma_chunk<DT>(fa[i], fb[j], acc[i][j]);
    }
    if (st + 1 < nstages) {
      // the other buffer was last read in the previous stage, which every
      // wave finished before the barrier that ended it
      lstore(buf ^ 1);
      __syncthreads();
    }
  }

  // lane holds C[m0 + wm + 16i + 4g + r][n0 + wn + 16j + n16]
  const int64_t layer_stride = M * d_e;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int col = n0 + wn + 16 * j + n16;
    if (col >= N) continue;
    const int layer = col / d_e, jj = col % d_e;
    char* qcol = Q + ((int64_t)layer * layer_stride + jj) * ES;
#pragma unroll
    for (int i = 0; i < MI; ++i) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = m0 + wm + 16 * i + 4 * g + r;
        if (row < M) {
          if constexpr (DT == DT_BF16)
            *reinterpret_cast<uint16_t*>(qcol + row * d_e * ES) =
                (uint16_t)f32_to_bf16_rne(acc[i][j][r]);
          else
            *reinterpret_cast<float*>(qcol + row * d_e * ES) = acc[i][j][r];
        }
      }
    }
  }
}

template <int DT, int BM, int BN>
static void launch_tiles(const void* x, const void* wt, void* q, int64_t n, int N, int64_t kb,
                         int d_e, hipStream_t st) {
  const int64_t tiles = ((n + BM - 1) / BM) * ((N + BN - 1) / BN);
  hipLaunchKernelGGL((project_kernel<DT, BM, BN>), dim3((unsigned)tiles), dim3(PJ_THREADS), 0,
                     st, static_cast<const char*>(x), static_cast<const char*>(wt),
                     static_cast<char*>(q), n, N, kb, d_e);
}

hipError_t launch_project(int dt, const void* x, const void* wt, void* q, int64_t n, int d_in,
                          int d_e, int layers, hipStream_t st) {
  if (n == 0) return hipSuccess;
  const int es = dt == DT_BF16 ? 2 : 4;
  const int N = layers * d_e;
  const int64_t kb = (int64_t)d_in * es;
  // 128 x 128 tiles when there are enough of them to occupy every CU twice
  const bool big = ((n + 127) / 128) * ((N + 127) / 128) >= 512;
  if (dt == DT_BF16) {
    if (big) launch_tiles<DT_BF16, 128, 128>(x, wt, q, n, N, kb, d_e, st);
    else launch_tiles<DT_BF16, 64, 64>(x, wt, q, n, N, kb, d_e, st);
  } else {
    if (big) launch_tiles<DT_F32, 128, 128>(x, wt, q, n, N, kb, d_e, st);
    else launch_tiles<DT_F32, 64, 64>(x, wt, q, n, N, kb, d_e, st);
  }
  return hipGetLastError();
}

}  // namespace lookme
