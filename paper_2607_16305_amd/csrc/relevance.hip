// Level-2 in the paper's own form (arXiv 2607.16305, Sec. 3.2, Eq. 6-7):
// a scene-shared two-layer MLP on [v_e, e_img[j]] gives one relevance logit
// per primitive, the top k primitives by logit are kept, and their weights
// are the softmax of cos(v_e, e_{j,p}) + tanh(r_j[p]).  Three launches:
//
//   relevance_hidden_kernel   a = round(ReLU([q_t, K1[scene_t]] W1^T + b1)):
//                             64 x 64 output tiles on the matrix cores, the
//                             operand-A row of token t being its query
//                             followed by its scene's key (gathered per row,
//                             K stages of 128 bytes straight into LDS);
//   score_kernel (dense)      r = a W2^T + b2 with a fused top-k over the N_p
//                             logits (the Level-2 scoring kernel's shared
//                             units, every row against the one key set W2);
//                             writes the k logits, not weights;
//   relevance_weights_kernel  one wave per row: the k cosines against the
//                             chosen primitive keys, + tanh of the logits,
//                             softmax over the k (in place of the logits).
#include "common.h"
#include "dtl.h"
#include "kernels.h"

namespace lookme {

// 4 waves in 2 x 2, each 32 x 32 (2 x 2 MFMA tiles): 64 x 64 tiles, 128-byte
// K stages, two of them
using RhShape = DtlShape<2, 2, 2, 2, 128>;
constexpr int RH_KB = 128;

struct RelHiddenParams {
  const char* q;            // [rows, d_e]
  const int32_t* scene;     // [rows]
  const char* keys;         // [S, d_e] scene keys
  const char* w1;           // [h, 2 d_e]
  const float* b1;          // [h] or null
  char* act;                // [rows, h]
  int64_t rows;
  int64_t q_bytes;          // d_e * elem size, a multiple of 128
  int S, h, tiles;
};

template <int DT>
__global__ __launch_bounds__(256) void relevance_hidden_kernel(RelHiddenParams a) {
  using S = RhShape;
  constexpr int MI = 2, NJ = 2, KB = RH_KB, KSL = KB / 64, WN = 2;
  constexpr int ES = DT == DT_BF16 ? 2 : 4;
  __shared__ __attribute__((aligned(1024))) char lds[2][S::STAGE];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15, g = lane >> 4;
  const int wm = (wv / WN) * 16 * MI, wn = (wv % WN) * 16 * NJ;

  const int tiles_n = (a.h + S::BN - 1) / S::BN;
  const int tile = xcd_remap(blockIdx.x, a.tiles);
  if (tile < 0) return;
  const int64_t m0 = (int64_t)(tile / tiles_n) * S::BM;
  const int n0 = (tile % tiles_n) * S::BN;
  const int nq = (int)(a.q_bytes / KB);   // stages of the query half of K
  const int nst = 2 * nq;

  // load b covers tile row trow (A rows first, then B rows); p0 serves the
  // stages of the first half of K, p1 those of the second: for an A row the
  // token's query and its scene's key, for a B row the two halves of the
  // W1 row.  Rows past the edge are clamped (their outputs are not stored).
  const char* p0[S::PER_WAVE];
  const char* p1[S::PER_WAVE];
#pragma unroll
  for (int b = 0; b < S::PER_WAVE; ++b) {
    const int trow = (wv * S::PER_WAVE + b) * S::RPI + lane / S::LPR;
    const int chunk = (lane % S::LPR) ^ blk_swz<KB>(trow & 15);
    if (trow < S::BM) {
      int64_t r = m0 + trow;
      r = r < a.rows ? r : a.rows - 1;
      int s = a.scene[r];
      s = s < 0 ? 0 : (s >= a.S ? a.S - 1 : s);
      p0[b] = a.q + r * a.q_bytes + chunk * 16;
      p1[b] = a.keys + (int64_t)s * a.q_bytes + chunk * 16;
    } else {
      int r = n0 + trow - S::BM;
      r = r < a.h ? r : a.h - 1;
      p0[b] = a.w1 + (int64_t)r * 2 * a.q_bytes + chunk * 16;
      p1[b] = p0[b] + a.q_bytes;
    }
  }
  auto issue = [&](int stage) {
    const int s = stage < nst ? stage : nst - 1;   // past the end: a harmless reload
    char* dst = lds[stage & 1];
#pragma unroll
    for (int b = 0; b < S::PER_WAVE; ++b) {
      const char* src = s < nq ? p0[b] + (int64_t)s * KB : p1[b] + (int64_t)(s - nq) * KB;
      load_lds16(src, dst + (wv * S::PER_WAVE + b) * 1024);
    }
  };

  f32x4_t acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  issue(0);
  for (int s = 0; s < nst; ++s) {
    // stage s has landed everywhere and every read of stage s - 1 (the other
    // buffer) has ended: load stage s + 1 there, multiply stage s (a plain
    // s_barrier: the fence of __syncthreads would wait for every load)
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    issue(s + 1);
    const char* buf = lds[s & 1];
#pragma unroll
    for (int ks = 0; ks < KSL; ++ks) {
      u32x4_t fa[MI], fb[NJ];
#pragma unroll
      for (int i = 0; i < MI; ++i) fa[i] = read_frag<KB>(buf, wm + 16 * i, ks, n16, g);
#pragma unroll
      for (int j = 0; j < NJ; ++j) fb[j] = read_frag<KB>(buf, S::BM + wn + 16 * j, ks, n16, g);
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = mfma_chunk<DT>(fa[i], fb[j], acc[i][j]);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // no load into LDS outlives the wave

  // the lane holds rows m0 + wm + 16 i + 4 g + r and hidden unit
  // n0 + wn + 16 j + n16: + b1, ReLU, one rounding to the storage dtype
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int col = n0 + wn + 16 * j + n16;
    if (col >= a.h) continue;
    const float bias = a.b1 != nullptr ? a.b1[col] : 0.f;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = m0 + wm + 16 * i + 4 * g + r;
        if (row >= a.rows) continue;
        const float z = fmaxf(acc[i][j][r] + bias, 0.f);
        char* dst = a.act + (row * a.h + col) * ES;
        if constexpr (DT == DT_BF16)
          *reinterpret_cast<uint16_t*>(dst) = (uint16_t)f32_to_bf16_rne(z);
        else
          *reinterpret_cast<float*>(dst) = z;
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
                            hipStream_t st) {
  if (rows == 0) return hipSuccess;
  const int es = dt == DT_BF16 ? 2 : 4;
  RelHiddenParams hp{};
  hp.q = static_cast<const char*>(q);
  hp.scene = scene;
  hp.keys = static_cast<const char*>(scene_keys);
  hp.w1 = static_cast<const char*>(mlp.w1);
  hp.b1 = mlp.b1;
  hp.act = static_cast<char*>(act);
  hp.rows = rows;
  hp.q_bytes = (int64_t)d_e * es;
  hp.S = S;
  hp.h = mlp.hidden;
  hp.tiles = (int)(((rows + RhShape::BM - 1) / RhShape::BM) *
                   ((mlp.hidden + RhShape::BN - 1) / RhShape::BN));
  const unsigned grid = (unsigned)((hp.tiles + 7) / 8 * 8);
  if (dt == DT_BF16)
    hipLaunchKernelGGL(relevance_hidden_kernel<DT_BF16>, dim3(grid), dim3(256), 0, st, hp);
  else
    hipLaunchKernelGGL(relevance_hidden_kernel<DT_F32>, dim3(grid), dim3(256), 0, st, hp);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_relevance_topk(dt, act, mlp.w2, mlp.b2, rows, mlp.hidden, P, k, prim, w, st);
  if (e != hipSuccess) return e;
  const dim3 wgrid((unsigned)((rows + 3) / 4));
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
