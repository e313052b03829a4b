// Small-tile product C = A B^T on the matrix cores for the MLP-shaped steps
// (the relevance MLP of Eq. 6, the SwiGLU fusion of Eq. 10 and the
// propagation of Eq. 11): 64 x 64
// output tiles, 4 waves in 2 x 2 (each 2 x 2 MFMA tiles), K in 128-byte
// stages loaded straight into LDS (dtl.h), a ring of NS stages, NS - 1 in
// flight while one is multiplied.  These products have few rows and long K,
// so the bytes in flight per CU over the loads' latency, not the matrix
// cores, set the pace: the ring is as deep as the grid's occupancy allows
// (launch_tile_gemm).
// blockIdx.y selects a batch (a layer) whose A, B and output start a fixed
// stride further.  With a count array, batch z has count[z] live rows (at
// most `rows`, which sizes the grid); the tiles beyond them do nothing.  Epilogues:
//
//   EPI_ACT     C + bias, ReLU, one rounding to the storage dtype, [rows, cols];
//   EPI_LOGIT   C + bias as float32, [rows, cols];
//   EPI_SWIGLU  the tile's B rows are 32 rows of B (gate) and the same 32 rows
//               of B2 (up): u = silu(gate) * up, rounded, [rows, cols] with
//               32 output columns a tile;
//   EPI_RESID   H[out_row(r), c] = round(H + C) with out_row(r) = z * n +
//               kept[z * kept_batch + r] (the kept token of row r of layer z);
//   EPI_ADD     round(C + res) with res [rows, cols], [rows, cols];
//   EPI_STORE   round(C), [rows, cols];
//   EPI_ACT_TAB C + tab[sel[row]] (a float32 row of [sel_rows, cols]: the
//               relevance MLP's per-scene half of the first layer, b1
//               included), ReLU, one rounding, [rows, cols].
//
// An A row may take its first `ksplit` stages from a0 and the rest from a
// gathered row of a1 (the relevance MLP's [query ; scene key] input).

#pragma once

#include "common.h"
#include "dtl.h"

namespace lookme {

// BIG: 128 x 128 output tiles (each wave 4 x 4 MFMA tiles), for products with
// enough rows to fill the chip with them (the relevance MLP's first layer of
// large batches): a quarter of the tiles, half the operand bytes into LDS.
template <bool BIG>
using TgShapeT = DtlShape<2, 2, BIG ? 4 : 2, BIG ? 4 : 2, 128>;
using TgShape = TgShapeT<false>;
constexpr int TG_KB = 128;

enum : int {
  EPI_ACT = 0, EPI_LOGIT = 1, EPI_SWIGLU = 2, EPI_RESID = 3, EPI_ADD = 4, EPI_STORE = 5,
  EPI_ACT_TAB = 6
};

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
  const float* tab;         // EPI_ACT_TAB: [sel_rows, cols], row sel[r] added to row r
  const int32_t* count;     // or null: batch z uses only its first count[z * count_step]
                            // rows (a gate's counted kept list); tiles past them end at once
  int64_t rows;
  int64_t a_bytes;          // bytes of an A row (of each part, when split)
  int64_t k_bytes;          // K in bytes, a multiple of 128
  int64_t b_ld;             // bytes between B rows (0: k_bytes; a column slice of a wider B)
  int64_t a_batch, b_batch, out_batch;   // byte strides between batches
  int64_t n, kept_batch;    // EPI_RESID: tokens per layer, stride of the kept lists
  int64_t out_ld;           // EPI_RESID: bytes of an H row
  int sel_rows, cols, ksplit, tiles;
  int col_major;            // tile ids run down the row tiles of a column block first
  int count_step;           // 1: a count per batch, 0: one count for all
};

// Origin of tile `tile`: row tiles of one column block are consecutive ids
// when col_major (so they land on one XCD and share its L2 copy of the B
// rows, which the larger operand then crosses HBM once), else the column
// tiles of one row block.
template <bool BIG = false>
__device__ __forceinline__ void tile_origin(const TileGemmParams& a, int tile, int tcols,
                                            int64_t* m0, int* n0) {
  constexpr int BM = TgShapeT<BIG>::BM;
  if (a.col_major) {
    const int tiles_m = (int)((a.rows + BM - 1) / BM);
    *m0 = (int64_t)(tile % tiles_m) * BM;
    *n0 = (tile / tiles_m) * tcols;
  } else {
    const int tiles_n = (a.cols + tcols - 1) / tcols;
    *m0 = (int64_t)(tile / tiles_n) * BM;
    *n0 = (tile % tiles_n) * tcols;
  }
}

__device__ __forceinline__ float silu_f(float x) { return x / (1.f + expf(-x)); }

// Epilogue of a tile (tile index `tile` of batch z) from the accumulators of
// thread tid: the lane holds rows m0 + wm + 16 i + 4 g + r and tile columns
// wn + 16 j + n16.  xch: 4096 floats of LDS (EPI_SWIGLU only, small tiles).
template <int DT, int EPI, bool BIG = false>
__device__ __forceinline__ void tile_epilogue(const TileGemmParams& a,
                                              f32x4_t (&acc)[BIG ? 4 : 2][BIG ? 4 : 2],
                                              int64_t z, int tile, int tid, float* xch,
                                              int64_t rows) {
  using S = TgShapeT<BIG>;
  constexpr int MI = BIG ? 4 : 2, NJ = BIG ? 4 : 2, WN = 2;
  static_assert(!BIG || EPI != EPI_SWIGLU, "the SwiGLU exchange is laid out for small tiles");
  constexpr int ES = DT == DT_BF16 ? 2 : 4;
  constexpr int TCOLS = EPI == EPI_SWIGLU ? S::BN / 2 : S::BN;
  const int lane = tid & 63, wv = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int wm = (wv / WN) * 16 * MI, wn = (wv % WN) * 16 * NJ;
  int64_t m0;
  int n0;
  tile_origin<BIG>(a, tile, TCOLS, &m0, &n0);
  if constexpr (BIG && EPI == EPI_ACT_TAB) {
    if (a.cols % 8 == 0 &&
        ((reinterpret_cast<uintptr_t>(a.out) | reinterpret_cast<uintptr_t>(a.tab)) & 15) == 0) {
      // through LDS, 64 rows at a time (xch: the stage ring, free once every
      // wave is past its last loads): the waves of those rows write their
      // sums, then every thread takes 8-column pieces of a row, whose table
      // part and output are 16-byte loads and stores (the lane layout of the
      // accumulators gave 2-byte stores and 4-byte table loads, ~25 us of
      // the Zipf batch's ~57)
      constexpr int LD = S::BN + 4;   // padded row: the four row groups of a write on distinct banks
#pragma unroll 1
      for (int half = 0; half < 2; ++half) {
        __syncthreads();
        if (wv / WN == half) {
#pragma unroll
          for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
              for (int r = 0; r < 4; ++r)
                xch[(16 * i + 4 * g + r) * LD + wn + 16 * j + n16] = acc[i][j][r];
        }
        __syncthreads();
#pragma unroll
        for (int c = 0; c < 64 * S::BN / 8 / 256; ++c) {
          const int id = tid + 256 * c;
          const int lr = id / (S::BN / 8), cc = (id % (S::BN / 8)) * 8;
          const int64_t row = m0 + 64 * half + lr;
          const int col = n0 + cc;
          if (row >= rows || col >= a.cols) continue;
          int sc = a.sel[row];
          sc = sc < 0 ? 0 : (sc >= a.sel_rows ? a.sel_rows - 1 : sc);
          const f32x4_t* tp = reinterpret_cast<const f32x4_t*>(a.tab + (int64_t)sc * a.cols + col);
          const f32x4_t t0 = tp[0], t1 = tp[1];
          const f32x4_t* xp = reinterpret_cast<const f32x4_t*>(xch + lr * LD + cc);
          const f32x4_t x0 = xp[0], x1 = xp[1];
          float v[8];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[e] = fmaxf(x0[e] + t0[e], 0.f);
            v[4 + e] = fmaxf(x1[e] + t1[e], 0.f);
          }
          char* dst = a.out + (row * a.cols + col) * ES;
          if constexpr (DT == DT_BF16) {
            u32x4_t o;
#pragma unroll
            for (int e = 0; e < 4; ++e) o[e] = pack_bf16x2(v[2 * e], v[2 * e + 1]);
            *reinterpret_cast<u32x4_t*>(dst) = o;
          } else {
            *reinterpret_cast<f32x4_t*>(dst) = f32x4_t{v[0], v[1], v[2], v[3]};
            *reinterpret_cast<f32x4_t*>(dst + 16) = f32x4_t{v[4], v[5], v[6], v[7]};
          }
        }
      }
      return;
    }
    // 32-bit row and table indices (rows of a product and scenes stay far
    // below 2^31) keep the big tile's epilogue within the registers of two
    // waves a SIMD; every table load still precedes the first store
    int orow[MI][4], trow[MI][4];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = m0 + wm + 16 * i + 4 * g + r;
        orow[i][r] = (int)(row < rows ? row : rows - 1);
        const int sc = a.sel[orow[i][r]];
        trow[i][r] = sc < 0 ? 0 : (sc >= a.sel_rows ? a.sel_rows - 1 : sc);
      }
    int col[NJ];
    float old[NJ][MI][4];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      col[j] = n0 + wn + 16 * j + n16;
      const int cc = col[j] < a.cols ? col[j] : a.cols - 1;
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) old[j][i][r] = a.tab[(int64_t)trow[i][r] * a.cols + cc];
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      if (col[j] >= a.cols) continue;
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          if (m0 + wm + 16 * i + 4 * g + r >= rows) continue;
          const float v = fmaxf(acc[i][j][r] + old[j][i][r], 0.f);
          char* dst = a.out + ((int64_t)orow[i][r] * a.cols + col[j]) * ES;
          if constexpr (DT == DT_BF16)
            *reinterpret_cast<uint16_t*>(dst) = (uint16_t)f32_to_bf16_rne(v);
          else
            *reinterpret_cast<float*>(dst) = v;
        }
    }
    return;
  }
  if constexpr (EPI == EPI_SWIGLU) {
    // the up half (waves with wn = 32) passes its tile through LDS to the
    // gate half (wn = 0) of the same rows
    __syncthreads();   // every wave is done with the LDS the exchange reuses
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
          if (row >= rows) continue;
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
    // every load (biases, kept rows, H or residual values) is issued before
    // the first store: as far as the compiler knows a store may alias a later
    // load, which would otherwise serialise the elements one round trip each.
    // The loads are unconditional, from addresses clamped into the operands
    // (a load under a branch gets a wait of its own where the paths meet).
    int col[NJ], ccol[NJ];
    float bias[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      col[j] = n0 + wn + 16 * j + n16;
      ccol[j] = col[j] < a.cols ? col[j] : a.cols - 1;
      bias[j] = 0.f;
      if constexpr (EPI == EPI_ACT || EPI == EPI_LOGIT)
        if (a.bias != nullptr) bias[j] = a.bias[ccol[j]];
    }
    int64_t orow[MI][4];   // output row: the tile row, or (EPI_RESID) its H row
    int64_t trow[MI][4];   // EPI_ACT_TAB: the row's table row
    bool rok[MI][4];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = m0 + wm + 16 * i + 4 * g + r;
        rok[i][r] = row < rows;
        orow[i][r] = rok[i][r] ? row : rows - 1;
        if constexpr (EPI == EPI_RESID) {
          int64_t t = a.kept[z * a.kept_batch + orow[i][r]];
          t = t < 0 ? 0 : (t >= a.n ? a.n - 1 : t);
          orow[i][r] = z * a.n + t;
        }
        if constexpr (EPI == EPI_ACT_TAB) {
          const int s = a.sel[orow[i][r]];
          trow[i][r] = s < 0 ? 0 : (s >= a.sel_rows ? a.sel_rows - 1 : s);
        }
      }
    float old[NJ][MI][4];   // EPI_RESID: H, EPI_ADD: the residual, EPI_ACT_TAB: the table
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          old[j][i][r] = 0.f;
          if constexpr (EPI == EPI_ACT_TAB)
            old[j][i][r] = a.tab[trow[i][r] * a.cols + ccol[j]];
          if constexpr (EPI == EPI_RESID || EPI == EPI_ADD) {
            const char* src = EPI == EPI_RESID
                                  ? a.out + orow[i][r] * a.out_ld + (int64_t)ccol[j] * ES
                                  : a.res + (orow[i][r] * a.cols + ccol[j]) * ES;
            if constexpr (DT == DT_BF16)
              old[j][i][r] = bf16lo(*reinterpret_cast<const uint16_t*>(src));
            else
              old[j][i][r] = *reinterpret_cast<const float*>(src);
          }
        }
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      if (col[j] >= a.cols) continue;
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          if (!rok[i][r]) continue;
          const float c = acc[i][j][r] + bias[j];
          if constexpr (EPI == EPI_LOGIT) {
            reinterpret_cast<float*>(a.out)[orow[i][r] * a.cols + col[j]] = c;
            continue;
          }
          float v;
          char* dst;
          if constexpr (EPI == EPI_ACT || EPI == EPI_STORE) {
            v = EPI == EPI_ACT ? fmaxf(c, 0.f) : c;
            dst = a.out + (orow[i][r] * a.cols + col[j]) * ES;
          } else if constexpr (EPI == EPI_ACT_TAB) {
            v = fmaxf(c + old[j][i][r], 0.f);
            dst = a.out + (orow[i][r] * a.cols + col[j]) * ES;
          } else if constexpr (EPI == EPI_ADD) {
            v = old[j][i][r] + c;
            dst = a.out + (orow[i][r] * a.cols + col[j]) * ES;
          } else {   // EPI_RESID
            v = old[j][i][r] + c;
            dst = a.out + orow[i][r] * a.out_ld + (int64_t)col[j] * ES;
          }
          if constexpr (DT == DT_BF16)
            *reinterpret_cast<uint16_t*>(dst) = (uint16_t)f32_to_bf16_rne(v);
          else
            *reinterpret_cast<float*>(dst) = v;
        }
    }
  }
}

template <int DT, int EPI, int NS, bool BIG = false>
__global__ __launch_bounds__(256, BIG ? 2 : 1) void tile_gemm_kernel(TileGemmParams a) {
  using S = TgShapeT<BIG>;
  constexpr int MI = BIG ? 4 : 2, NJ = BIG ? 4 : 2, KB = TG_KB, KSL = KB / 64, WN = 2;
  constexpr int TCOLS = EPI == EPI_SWIGLU ? S::BN / 2 : S::BN;   // output columns a tile
  static_assert(NS >= 2, "a stage in flight while one is multiplied");
  static_assert(!BIG || NS * S::STAGE >= 64 * (S::BN + 4) * 4, "room for the epilogue's 64 rows");
  __shared__ __attribute__((aligned(1024))) char lds[NS][S::STAGE];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15, g = lane >> 4;
  const int wm = (wv / WN) * 16 * MI, wn = (wv % WN) * 16 * NJ;
  const int64_t z = blockIdx.y;

  const int tile = xcd_remap(blockIdx.x, a.tiles);
  if (tile < 0) return;
  int64_t m0;
  int n0;
  tile_origin<BIG>(a, tile, TCOLS, &m0, &n0);
  int64_t rows = a.rows;   // live rows of this batch
  if (a.count != nullptr) {
    const int64_t c = a.count[z * a.count_step];
    rows = c < rows ? c : rows;
    if (m0 >= rows) return;   // the whole workgroup: no barrier is left waiting
  }
  const int nst = (int)(a.k_bytes / KB);
  const char* A0 = a.a0 + z * a.a_batch;
  const char* B0 = a.b + z * a.b_batch;

  // load b covers tile row trow (A rows first, then B rows); an A row takes
  // its first ksplit stages from p0 and the rest from p1; a B row is
  // contiguous.  Rows past the edge are clamped (their outputs are not
  // stored).
  const char* p0[S::PER_WAVE];
  const char* p1[S::PER_WAVE];
  int split_at[S::PER_WAVE];
  int sel[S::PER_WAVE];   // gathered a1 rows, loaded together (one branch, no wait each)
  if (a.a1 != nullptr) {
#pragma unroll
    for (int b = 0; b < S::PER_WAVE; ++b) {
      const int trow = (wv * S::PER_WAVE + b) * S::RPI + lane / S::LPR;
      int64_t r = m0 + (trow < S::BM ? trow : 0);
      r = r < rows ? r : rows - 1;
      sel[b] = a.sel[r];
    }
  }
#pragma unroll
  for (int b = 0; b < S::PER_WAVE; ++b) {
    const int trow = (wv * S::PER_WAVE + b) * S::RPI + lane / S::LPR;
    const int chunk = (lane % S::LPR) ^ blk_swz<KB>(trow & 15);
    if (trow < S::BM) {
      int64_t r = m0 + trow;
      r = r < rows ? r : rows - 1;
      p0[b] = A0 + r * a.a_bytes + chunk * 16;
      if (a.a1 != nullptr) {
        int s = sel[b];
        s = s < 0 ? 0 : (s >= a.sel_rows ? a.sel_rows - 1 : s);
        p1[b] = a.a1 + (int64_t)s * a.a_bytes + chunk * 16;
      } else {
        p1[b] = p0[b] + (int64_t)a.ksplit * KB;
      }
      split_at[b] = a.ksplit;
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
      p0[b] = base + (int64_t)r * (a.b_ld != 0 ? a.b_ld : a.k_bytes) + chunk * 16;
      p1[b] = p0[b];
      split_at[b] = nst;
    }
  }
  auto issue = [&](int i) {
    const int s = i < nst ? i : nst - 1;   // past the end: a harmless reload
    char* dst = lds[i % NS];
#pragma unroll
    for (int b = 0; b < S::PER_WAVE; ++b) {
      const char* src = s < split_at[b] ? p0[b] + (int64_t)s * KB
                                        : p1[b] + (int64_t)(s - split_at[b]) * KB;
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
  for (int i = 0; i < nst; ++i) {
    // this wave's loads of stage i have landed once at most those of the
    // NS - 2 younger stages are outstanding; the barrier makes every wave's
    // visible and ends every read of stage i - 1, whose buffer the next
    // loads fill (a plain s_barrier: the fence of __syncthreads would wait
    // for every load in flight)
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NS - 2) * S::PER_WAVE) : "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    issue(i + NS - 1);
    const char* buf = lds[i % NS];
#pragma unroll
    for (int ks = 0; ks < KSL; ++ks) {
      u32x4_t fa[MI], fb[NJ];
#pragma unroll
      for (int ii = 0; ii < MI; ++ii) fa[ii] = read_frag<KB>(buf, wm + 16 * ii, ks, n16, g);
#pragma unroll
      for (int j = 0; j < NJ; ++j) fb[j] = read_frag<KB>(buf, S::BM + wn + 16 * j, ks, n16, g);
#pragma unroll
      for (int ii = 0; ii < MI; ++ii)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[ii][j] = mfma_chunk<DT>(fa[ii], fb[j], acc[ii][j]);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // no load into LDS outlives the wave

  tile_epilogue<DT, EPI, BIG>(a, acc, z, tile, tid, reinterpret_cast<float*>(&lds[0][0]), rows);
}

// Launches the product over `batches` batches (blockIdx.y), tiles in the
// order that keeps the larger operand's rows on one XCD, with the deepest
// ring its grid's occupancy allows: 8 stages (128 KB of LDS) while every
// workgroup has a CU of its own (at most 256), 4 (64 KB) while all are
// resident at 2 a CU (at most 512), else 2 (32 KB, up to 5 a CU).
template <int EPI>
hipError_t launch_tile_gemm(int dt, TileGemmParams p, int batches, hipStream_t st) {
  // column-major tile order when B has at least as many rows as A
  p.col_major = (int64_t)p.cols * (EPI == EPI_SWIGLU ? 2 : 1) >= p.rows;
  if constexpr (EPI == EPI_ACT_TAB) {
    // 128 x 128 tiles once they alone fill two whole rounds of the CUs at
    // two a CU (relevance first layer, Zipf batch: 1024 tiles, 51.0 -> 44.5
    // us; the multi-scale batch's 720 took 37.4 against 35.4 us on 64 x 64)
    constexpr int BB = TgShapeT<true>::BM;
    const int64_t big = ((p.rows + BB - 1) / BB) * ((p.cols + BB - 1) / BB);
    if (big * batches >= 1024) {
      p.tiles = (int)big;
      const unsigned gx = (unsigned)((p.tiles + 7) / 8 * 8);
      const dim3 grid(gx, (unsigned)batches);
      // two 32 KiB stages: two workgroups a CU
      if (dt == DT_BF16)
        hipLaunchKernelGGL((tile_gemm_kernel<DT_BF16, EPI, 2, true>), grid, dim3(256), 0, st, p);
      else
        hipLaunchKernelGGL((tile_gemm_kernel<DT_F32, EPI, 2, true>), grid, dim3(256), 0, st, p);
      return hipGetLastError();
    }
  }
  const unsigned gx = (unsigned)((p.tiles + 7) / 8 * 8);
  const dim3 grid(gx, (unsigned)batches);
  const int64_t wgs = (int64_t)gx * batches;
  const int ns = wgs <= 256 ? 8 : (wgs <= 512 ? 4 : 2);
  if (dt == DT_BF16) {
    if (ns == 8)
      hipLaunchKernelGGL((tile_gemm_kernel<DT_BF16, EPI, 8>), grid, dim3(256), 0, st, p);
    else if (ns == 4)
      hipLaunchKernelGGL((tile_gemm_kernel<DT_BF16, EPI, 4>), grid, dim3(256), 0, st, p);
    else
      hipLaunchKernelGGL((tile_gemm_kernel<DT_BF16, EPI, 2>), grid, dim3(256), 0, st, p);
  } else {
    if (ns == 8)
      hipLaunchKernelGGL((tile_gemm_kernel<DT_F32, EPI, 8>), grid, dim3(256), 0, st, p);
    else if (ns == 4)
      hipLaunchKernelGGL((tile_gemm_kernel<DT_F32, EPI, 4>), grid, dim3(256), 0, st, p);
    else
      hipLaunchKernelGGL((tile_gemm_kernel<DT_F32, EPI, 2>), grid, dim3(256), 0, st, p);
  }
  return hipGetLastError();
}

}  // namespace lookme
