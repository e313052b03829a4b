// Small-tile product C = A B^T on the matrix cores for the MLP-shaped steps
// (the relevance MLP of Eq. 6, the SwiGLU fusion of Eq. 10 and the
// propagation of Eq. 11): 64 x 64
// output tiles, 4 waves in 2 x 2 (each 2 x 2 MFMA tiles), K in 128-byte
// stages loaded straight into LDS (dtl.h), a ring of NS stages, NS - 1 in
// flight while one is multiplied.  These products have few rows and long K,
// so the loads' latency, not the matrix cores, sets the pace: a small grid
// takes a ring of 4 (64 KB of LDS, 2 workgroups a CU), a grid that would not
// fit the chip at that occupancy a ring of 2 (32 KB, up to 5 a CU); see
// launch_tile_gemm.
// blockIdx.y selects a batch (a layer) whose A, B and output start a fixed
// stride further.  Epilogues:
//
//   EPI_ACT     C + bias, ReLU, one rounding to the storage dtype, [rows, cols];
//   EPI_LOGIT   C + bias as float32, [rows, cols];
//   EPI_SWIGLU  the tile's B rows are 32 rows of B (gate) and the same 32 rows
//               of B2 (up): u = silu(gate) * up, rounded, [rows, cols] with
//               32 output columns a tile;
//   EPI_RESID   H[out_row(r), c] = round(H + C) with out_row(r) = z * n +
//               kept[z * kept_batch + r] (the kept token of row r of layer z);
//   EPI_ADD     round(C + res) with res [rows, cols], [rows, cols].
//
// An A row may take its first `ksplit` stages from a0 and the rest from a
// gathered row of a1 (the relevance MLP's [query ; scene key] input).
#pragma once

#include "common.h"
#include "dtl.h"

namespace lookme {

using TgShape = DtlShape<2, 2, 2, 2, 128>;
constexpr int TG_KB = 128;

enum : int { EPI_ACT = 0, EPI_LOGIT = 1, EPI_SWIGLU = 2, EPI_RESID = 3, EPI_ADD = 4 };

struct TileGemmParams {
  const char* a0;           // [rows, K] (or the first ksplit stages of a row)
  const char* a1;           // gathered second part of A rows, or null
  const int32_t* sel;       // [rows] row of a1 for each A row (clamped to [0, sel_rows))
  const char* b;            // [cols, K] (EPI_SWIGLU: gate rows)
  const char* b2;           // EPI_SWIGLU: up rows [cols, K]
  const float* bias;        // [cols] or null (EPI_ACT, EPI_LOGIT)
  char* out;
  const int32_t* kept;      // EPI_RESID: kept list of batch z at kept + z * kept_batch
  const char* res;          // EPI_ADD: [rows, cols]
  int64_t rows;
  int64_t a_bytes;          // bytes of an A row (of each part, when split)
  int64_t k_bytes;          // K in bytes, a multiple of 128
  int64_t a_batch, b_batch, out_batch;   // byte strides between batches
  int64_t n, kept_batch;    // EPI_RESID: tokens per layer, stride of the kept lists
  int64_t out_ld;           // EPI_RESID: bytes of an H row
  int sel_rows, cols, ksplit, tiles;
};

__device__ __forceinline__ float silu_f(float x) { return x / (1.f + expf(-x)); }

template <int DT, int EPI, int NS>
__global__ __launch_bounds__(256) void tile_gemm_kernel(TileGemmParams a) {
  using S = TgShape;
  constexpr int MI = 2, NJ = 2, KB = TG_KB, KSL = KB / 64, WN = 2;
  constexpr int ES = DT == DT_BF16 ? 2 : 4;
  constexpr int TCOLS = EPI == EPI_SWIGLU ? S::BN / 2 : S::BN;   // output columns a tile
  static_assert(NS >= 2, "a stage in flight while one is multiplied");
  __shared__ __attribute__((aligned(1024))) char lds[NS][S::STAGE];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15, g = lane >> 4;
  const int wm = (wv / WN) * 16 * MI, wn = (wv % WN) * 16 * NJ;
  const int64_t z = blockIdx.y;

  const int tiles_n = (a.cols + TCOLS - 1) / TCOLS;
  const int tile = xcd_remap(blockIdx.x, a.tiles);
  if (tile < 0) return;
  const int64_t m0 = (int64_t)(tile / tiles_n) * S::BM;
  const int n0 = (tile % tiles_n) * TCOLS;
  const int nst = (int)(a.k_bytes / KB);
  const char* A0 = a.a0 + z * a.a_batch;
  const char* B0 = a.b + z * a.b_batch;

  // load b covers tile row trow (A rows first, then B rows); an A row takes
  // its first ksplit stages from p0 and the rest from p1; a B row is
  // contiguous.  Rows past the edge are clamped (their outputs are not
  // stored).
  const char* p0[S::PER_WAVE];
  const char* p1[S::PER_WAVE];
  int split[S::PER_WAVE];
#pragma unroll
  for (int b = 0; b < S::PER_WAVE; ++b) {
    const int trow = (wv * S::PER_WAVE + b) * S::RPI + lane / S::LPR;
    const int chunk = (lane % S::LPR) ^ blk_swz<KB>(trow & 15);
    if (trow < S::BM) {
      int64_t r = m0 + trow;
      r = r < a.rows ? r : a.rows - 1;
      p0[b] = A0 + r * a.a_bytes + chunk * 16;
      if (a.a1 != nullptr) {
        int s = a.sel[r];
        s = s < 0 ? 0 : (s >= a.sel_rows ? a.sel_rows - 1 : s);
        p1[b] = a.a1 + (int64_t)s * a.a_bytes + chunk * 16;
      } else {
        p1[b] = p0[b] + (int64_t)a.ksplit * KB;
      }
      split[b] = a.ksplit;
    } else {
      int c = trow - S::BM;
      const char* base = B0;
      if constexpr (EPI == EPI_SWIGLU) {
        // rows 0..31 of the B part: gate rows, 32..63: the same up rows
        if (c >= TCOLS) {
          base = a.b2 + z * a.b_batch;
          c -= TCOLS;
        }
      }
      int r = n0 + c;
      r = r < a.cols ? r : a.cols - 1;
      p0[b] = base + (int64_t)r * a.k_bytes + chunk * 16;
      p1[b] = p0[b];
      split[b] = nst;
    }
  }
  auto issue = [&](int stage) {
    const int s = stage < nst ? stage : nst - 1;   // past the end: a harmless reload
    char* dst = lds[stage % NS];
#pragma unroll
    for (int b = 0; b < S::PER_WAVE; ++b) {
      const char* src =
          s < split[b] ? p0[b] + (int64_t)s * KB : p1[b] + (int64_t)(s - split[b]) * KB;
      load_lds16(src, dst + (wv * S::PER_WAVE + b) * 1024);
    }
  };

  f32x4_t acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int i = 0; i < NS - 1; ++i) issue(i);
  for (int s = 0; s < nst; ++s) {
    // this wave's loads of stage s have landed once at most those of the
    // NS - 2 younger stages are outstanding; the barrier makes every wave's
    // visible and ends every read of stage s - 1, whose buffer the next
    // loads fill (a plain s_barrier: the fence of __syncthreads would wait
    // for every load in flight)
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NS - 2) * S::PER_WAVE) : "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    issue(s + NS - 1);
    const char* buf = lds[s % NS];
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

  // the lane holds rows m0 + wm + 16 i + 4 g + r and tile column wn + 16 j +
  // n16
  if constexpr (EPI == EPI_SWIGLU) {
    // the up half (waves with wn = 32) passes its tile through the idle
    // stage buffer to the gate half (wn = 0) of the same rows
    float* xch = reinterpret_cast<float*>(&lds[0][0]);
    __syncthreads();   // every wave is done with the stage buffers
    if (wn != 0) {
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            xch[(((wv / WN) * MI * NJ + i * NJ + j) * 4 + r) * WAVE + lane] = acc[i][j][r];
    }
    __syncthreads();
    if (wn != 0) return;
    char* U = a.out + z * a.out_batch;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int col = n0 + 16 * j + n16;
      if (col >= a.cols) continue;
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = m0 + wm + 16 * i + 4 * g + r;
          if (row >= a.rows) continue;
          const float up = xch[(((wv / WN) * MI * NJ + i * NJ + j) * 4 + r) * WAVE + lane];
          const float u = silu_f(acc[i][j][r]) * up;
          char* dst = U + (row * a.cols + col) * ES;
          if constexpr (DT == DT_BF16)
            *reinterpret_cast<uint16_t*>(dst) = (uint16_t)f32_to_bf16_rne(u);
          else
            *reinterpret_cast<float*>(dst) = u;
        }
    }
  } else {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int col = n0 + wn + 16 * j + n16;
      if (col >= a.cols) continue;
      const float bias =
          (EPI == EPI_ACT || EPI == EPI_LOGIT) && a.bias != nullptr ? a.bias[col] : 0.f;
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = m0 + wm + 16 * i + 4 * g + r;
          if (row >= a.rows) continue;
          const float c = acc[i][j][r] + bias;
          if constexpr (EPI == EPI_LOGIT) {
            reinterpret_cast<float*>(a.out)[row * a.cols + col] = c;
          } else if constexpr (EPI == EPI_ACT) {
            char* dst = a.out + (row * a.cols + col) * ES;
            if constexpr (DT == DT_BF16)
              *reinterpret_cast<uint16_t*>(dst) = (uint16_t)f32_to_bf16_rne(fmaxf(c, 0.f));
            else
              *reinterpret_cast<float*>(dst) = fmaxf(c, 0.f);
          } else if constexpr (EPI == EPI_ADD) {
            const int64_t at = (row * a.cols + col) * ES;
            if constexpr (DT == DT_BF16)
              *reinterpret_cast<uint16_t*>(a.out + at) = (uint16_t)f32_to_bf16_rne(
                  bf16lo(*reinterpret_cast<const uint16_t*>(a.res + at)) + c);
            else
              *reinterpret_cast<float*>(a.out + at) = *reinterpret_cast<const float*>(a.res + at) + c;
          } else {   // EPI_RESID
            int64_t t = a.kept[z * a.kept_batch + row];
            t = t < 0 ? 0 : (t >= a.n ? a.n - 1 : t);
            char* dst = a.out + (z * a.n + t) * a.out_ld + (int64_t)col * ES;
            if constexpr (DT == DT_BF16) {
              uint16_t* h = reinterpret_cast<uint16_t*>(dst);
              *h = (uint16_t)f32_to_bf16_rne(bf16lo(*h) + c);
            } else {
              float* h = reinterpret_cast<float*>(dst);
              *h = *h + c;
            }
          }
        }
    }
  }
}

// Launches the product over `batches` batches (blockIdx.y) with the ring
// depth for its grid: 4 stages while every workgroup is resident at 2 a CU
// (at most 512 over the chip's 256 CUs), else 2.
template <int EPI>
hipError_t launch_tile_gemm(int dt, const TileGemmParams& p, int batches, hipStream_t st) {
  const unsigned gx = (unsigned)((p.tiles + 7) / 8 * 8);
  const dim3 grid(gx, (unsigned)batches);
  const bool deep = (int64_t)gx * batches <= 512;
  if (dt == DT_BF16) {
    if (deep)
      hipLaunchKernelGGL((tile_gemm_kernel<DT_BF16, EPI, 4>), grid, dim3(256), 0, st, p);
    else
      hipLaunchKernelGGL((tile_gemm_kernel<DT_BF16, EPI, 2>), grid, dim3(256), 0, st, p);
  } else {
    if (deep)
      hipLaunchKernelGGL((tile_gemm_kernel<DT_F32, EPI, 4>), grid, dim3(256), 0, st, p);
    else
      hipLaunchKernelGGL((tile_gemm_kernel<DT_F32, EPI, 2>), grid, dim3(256), 0, st, p);
  }
  return hipGetLastError();
}

}  // namespace lookme
