// Level-1 scene routing of large batches (arXiv 2607.16305, Sec. 3.2, Eq. 5)
// as a tiled product on the matrix cores with a fused arg max: scene[r] =
// argmax_s <q_r, K1[s]> + b[s], lowest s on exact ties; the scores are never
// written to memory.
//
// A workgroup owns 128 query rows and a range of 256-key tiles; 8 waves in a
// 2 x 4 grid each compute a 64 x 64 block of every tile.  The queries and the
// keys of a tile stream through LDS in 128-byte K stages by direct global-to-
// LDS loads (dtl.h), one stream of stages across all of the workgroup's key
// tiles, the next stages in flight while one is multiplied; the operand
// fragments are read from LDS half a stage ahead of their products.  After a tile's
// last stage every lane folds its scores (plus the bias, staged in LDS) into
// a running best per row; at the end the 16 lanes and then the 4 waves that
// share a row are merged in key order.  When a batch has few row blocks the
// key tiles are split over several workgroups and the partial arg maxima
// meet in route_partial (route_merge.h).
#include <type_traits>

#include "common.h"
#include "dtl.h"
#include "kernels.h"
#include "route_merge.h"

namespace lookme {

// WM x WN waves, each MI x NJ MFMA tiles; K stages of KB bytes
constexpr int RT_WM = 2, RT_WN = 4, RT_MI = 4, RT_NJ = 4, RT_KB = 128;
using RtShape = DtlShape<RT_WM, RT_WN, RT_MI, RT_NJ, RT_KB>;
static_assert(RtShape::BM == ROUTE_DTL_ROWS && RtShape::BN == ROUTE_DTL_KEYS, "tile shape");
// Stage buffers: three (two in flight while one is multiplied), or two when
// a bias table must fit beside them (16 KiB for the largest key range).
constexpr int rt_stages(bool bias) { return bias ? 2 : 3; }

struct RouteDtlParams {
  const char* q;         // [rows, d_e]
  const char* keys;      // [S, d_e]
  const float* bias;     // [S] (the BIAS instantiation only)
  int64_t rows;
  int64_t k_bytes;       // d_e * elem size, a multiple of 128
  int S;
  int splits;            // key ranges per row block
  int tps;               // 256-key tiles per range
  int units;             // row blocks * splits
  int32_t* scene;
  uint64_t* part;
  int32_t* count;
};

template <int DT, bool BIAS>
__global__ __launch_bounds__(64 * RT_WM * RT_WN) void route_dtl_kernel(RouteDtlParams a) {
  using S = RtShape;
  constexpr int MI = RT_MI, NJ = RT_NJ, KB = RT_KB, KSL = KB / 64, NS = rt_stages(BIAS);
  constexpr int THREADS = 64 * RT_WM * RT_WN;
  static_assert(NS >= 2, "a stage in flight while one is multiplied");
  static_assert(KSL == 2, "a stage is two 64-byte halves");
  // All of the kernel's LDS is one object.  With several __shared__ objects
  // the compiler tags their accesses with alias scopes and then, finding the
  // stage buffers' direct-to-LDS loads and fragment reads in one scope, puts
  // a vmcnt(0) wait after every stage's loads, before the first fragment
  // read: the next stage's loads then never overlap this stage's products.
  // Without scopes it leaves the ordering to the explicit waits below.  The
  // merge arrays and the arrival flag reuse the stage buffers (after the
  // last stage); the bias table has its own words.
  constexpr int BIAS_OFF = NS * S::STAGE;
  constexpr int BIAS_BYTES = BIAS ? ROUTE_DTL_MAX_TPS * S::BN * 4 : 0;
  static_assert(RT_WN * S::BM * 8 + 16 <= NS * S::STAGE, "merge arrays in the stage buffers");
  __shared__ __attribute__((aligned(1024))) char smem[BIAS_OFF + BIAS_BYTES];
  char (*lds)[S::STAGE] = reinterpret_cast<char (*)[S::STAGE]>(smem);
  float* s_bias = reinterpret_cast<float*>(smem + BIAS_OFF);
  float (*m_s)[S::BM] = reinterpret_cast<float (*)[S::BM]>(smem);
  int (*m_i)[S::BM] = reinterpret_cast<int (*)[S::BM]>(smem + RT_WN * S::BM * 4);
  int* s_last = reinterpret_cast<int*>(smem + RT_WN * S::BM * 8);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15, g = lane >> 4;
  const int wni = wv % RT_WN;
  const int wm = (wv / RT_WN) * 16 * MI, wn = wni * 16 * NJ;

  const int u = xcd_remap(blockIdx.x, a.units);
  if (u < 0) return;
  const int64_t rb = u / a.splits;
  const int split = u % a.splits;
  const int64_t m0 = rb * S::BM;
  const int ntiles = (a.S + S::BN - 1) / S::BN;
  const int kt0 = split * a.tps, kt1 = min(ntiles, kt0 + a.tps);
  const int nt = kt1 - kt0;              // key tiles of this unit
  const int nst = (int)(a.k_bytes / KB);
  const int total = nt * nst;            // K stages of this unit, tile by tile

  if constexpr (BIAS) {
    // the bias of the unit's keys (0 past the last scene: those keys are
    // masked by index anyway)
    for (int i = tid; i < nt * S::BN; i += THREADS) {
      const int key = kt0 * S::BN + i;
      s_bias[i] = key < a.S ? a.bias[key] : 0.f;
    }
  }

  // First key of tile t: a ragged last tile is moved back to end at the
  // last scene, so every key row it reads exists; its keys below t * 256
  // repeat the previous tile's and are masked in the epilogue.  With fewer
  // scenes than a tile there is one tile, at 0.
  auto tile_start = [&](int t) { return a.S < S::BN ? 0 : min(t * S::BN, a.S - S::BN); };
  // load b of a stage covers tile rows [(wv PER_WAVE + b) RPI, + RPI): the
  // query rows come first, then the 256 key rows of the stage's tile.  RPI
  // divides BM, so a load reads either query rows or key rows: the choice is
  // uniform over the wave, and the address is a uniform base (operand, row
  // block or key tile, K stage) plus a 32-bit lane offset fixed for the
  // launch (both operands are far below 4 GiB).  Rows past either operand
  // are clamped into it (they feed no stored result).
  // lane offset of load b from its base: the row block's first query row
  // (query loads) or the key tile's first key row (key loads)
  uint32_t off[S::PER_WAVE];
#pragma unroll
  for (int b = 0; b < S::PER_WAVE; ++b) {
    const int row0 = (wv * S::PER_WAVE + b) * S::RPI;       // uniform
    const int trow = row0 + lane / S::LPR;
    const uint32_t chunk = (uint32_t)(((lane % S::LPR) ^ blk_swz<KB>(trow & 15)) * 16);
    if (row0 < S::BM) {
      const int64_t r = min<int64_t>(m0 + trow, a.rows - 1) - m0;   // >= 0: m0 < rows
      off[b] = (uint32_t)(r * a.k_bytes) + chunk;
    } else {
      // fewer scenes than a tile: one tile, rows past the last scene read it
      const int kr = a.S < S::BN ? min(trow - S::BM, a.S - 1) : trow - S::BM;
      off[b] = (uint32_t)(kr * a.k_bytes) + chunk;
    }
  }
  const char* q_base = a.q + m0 * a.k_bytes;
  // the producer's position (tile within the unit, K stage, buffer), kept
  // as wave-uniform counters; past the unit's last stage it stays there (a
  // harmless reload keeps every wave's count of loads in flight the same)
  int p_tile = 0, p_stage = 0, p_buf = 0;
  auto issue = [&]() {
    char* dst = lds[p_buf];
    const char* k_base = a.keys + (int64_t)tile_start(kt0 + p_tile) * a.k_bytes + p_stage * KB;
    const char* qs_base = q_base + p_stage * KB;
#pragma unroll
    for (int b = 0; b < S::PER_WAVE; ++b) {
      const bool is_q = (wv * S::PER_WAVE + b) * S::RPI < S::BM;   // uniform
      load_lds16((is_q ? qs_base : k_base) + off[b], dst + (wv * S::PER_WAVE + b) * 1024);
    }
    p_buf = p_buf == NS - 1 ? 0 : p_buf + 1;
    if (++p_stage == nst) {
      if (p_tile + 1 < nt) {
        p_stage = 0;
        ++p_tile;
      } else {
        p_stage = nst - 1;
      }
    }
  };

  f32x4_t acc[MI][NJ];
  float bs[MI][4];
  int bi[MI][4];
#pragma unroll
  for (int i = 0; i < MI; ++i) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      bs[i][r] = -__builtin_inff();
      bi[i][r] = -1;
    }
  }

  // Fragments are read one half-stage (a 64-byte K slice) ahead of the
  // products that use them: f0 holds the first half of a stage, f1 the
  // second.  The second half's reads are issued before the first half's
  // products, the next stage's first half after the barrier that makes it
  // visible, so the products of each half run while the next half's reads
  // are in flight.
  u32x4_t f0a[MI], f0b[NJ], f1a[MI], f1b[NJ];
  auto read_half = [&](const char* buf, int ks, u32x4_t (&fa)[MI], u32x4_t (&fb)[NJ]) {
#pragma unroll
    for (int i = 0; i < MI; ++i) fa[i] = read_frag<KB>(buf, wm + 16 * i, ks, n16, g);
#pragma unroll
    for (int j = 0; j < NJ; ++j) fb[j] = read_frag<KB>(buf, S::BM + wn + 16 * j, ks, n16, g);
  };
  auto products = [&](const u32x4_t (&fa)[MI], const u32x4_t (&fb)[NJ]) {
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) acc[i][j] = mfma_chunk<DT>(fa[i], fb[j], acc[i][j]);
  };
  // matrix-core instructions per fragment pair, fragment reads per half-stage
  constexpr int MPC = DT == DT_BF16 ? 1 : 4, READS = MI + NJ;

  // every buffer of the ring filled: stages 0 .. NS - 1 in flight
#pragma unroll
  for (int i = 0; i < NS; ++i) issue();
  // stage 0 has landed (the NS - 1 younger stages may be outstanding) and
  // the barrier makes every wave's part visible (and the bias table)
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NS - 1) * S::PER_WAVE) : "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  read_half(lds[0], 0, f0a, f0b);
  // the consumer's position: tile within the unit, K stage, buffer
  int c_tile = 0, c_stage = 0, c_buf = 0;
  for (int sigma = 0; sigma < total; ++sigma) {
    const char* buf = lds[c_buf];
    const char* nbuf = lds[c_buf == NS - 1 ? 0 : c_buf + 1];
    // the first product waits for f0 (read during the previous half-stage's
    // products); the second half's reads go out behind it, so that at most
    // one half-stage of reads is outstanding (the LDS counter holds 15)
    read_half(buf, 1, f1a, f1b);
    products(f0a, f0b);
    __builtin_amdgcn_sched_group_barrier(0x008, MPC, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, READS, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, MPC * (MI * NJ - 1), 0);
    // stage sigma + 1 has landed once at most the loads of the NS - 2
    // younger stages are outstanding; after the barrier it is visible and
    // no wave reads this stage's buffer any more, so the loads of stage
    // sigma + NS refill it (a plain s_barrier: the fence of __syncthreads
    // would wait for every load in flight; the scheduling barriers keep the
    // products on their side of it)
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"((NS - 2) * S::PER_WAVE) : "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    issue();
    read_half(nbuf, 0, f0a, f0b);
    products(f1a, f1b);
    c_buf = c_buf == NS - 1 ? 0 : c_buf + 1;
    if (c_stage == nst - 1) {
      // the tile is complete: the lane holds rows wm + 16 i + 4 g + r and
      // keys key0 + 16 j (increasing in j, and above every earlier tile's,
      // so a strict '>' keeps the lowest key on exact ties).  Keys past the
      // last scene (a ragged last tile) get a bias of -inf.
      const int tile = kt0 + c_tile;
      const int key0 = tile_start(tile) + wn + n16;   // key of j = 0
      float bj[NJ];
      int kj[NJ];
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        kj[j] = key0 + 16 * j;
        bj[j] = BIAS ? s_bias[max(kj[j] - kt0 * S::BN, 0)] : 0.f;
      }
      if ((tile + 1) * S::BN > a.S) {
        // ragged last tile: keys already scored by the previous tile, and
        // with fewer scenes than a tile the rows past the last scene
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          if (kj[j] < tile * S::BN || kj[j] >= a.S) bj[j] = -__builtin_inff();
      }
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            const float v = acc[i][j][r] + bj[j];
            bi[i][r] = v > bs[i][r] ? kj[j] : bi[i][r];
            bs[i][r] = fmaxf(bs[i][r], v);
          }
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      c_stage = 0;
      ++c_tile;
    } else {
      ++c_stage;
    }
  }
  // no load into LDS outlives the wave, and every wave is done with the
  // stage buffers before the merge arrays overwrite them
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // merge the 16 lanes of a row group (keys n16 + 16 j of every tile), then
  // the 4 waves that share rows, in key order
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
#pragma unroll
      for (int d = 1; d < 16; d <<= 1) {
        const float os = __shfl_xor(bs[i][r], d, 64);
        const int oi = __shfl_xor(bi[i][r], d, 64);
        if (beats(os, oi, bs[i][r], bi[i][r])) {
          bs[i][r] = os;
          bi[i][r] = oi;
        }
      }
      if (n16 == 0) {
        m_s[wni][wm + 16 * i + 4 * g + r] = bs[i][r];
        m_i[wni][wm + 16 * i + 4 * g + r] = bi[i][r];
      }
    }
  __syncthreads();
  const int nr = (int)min<int64_t>(S::BM, a.rows - m0);
  float best_s = -__builtin_inff();
  int best_i = -1;
  if (tid < S::BM) {
#pragma unroll
    for (int w = 0; w < RT_WN; ++w)
      if (beats(m_s[w][tid], m_i[w][tid], best_s, best_i)) {
        best_s = m_s[w][tid];
        best_i = m_i[w][tid];
      }
  }
  if (a.splits == 1) {
    if (tid < nr) a.scene[m0 + tid] = best_i;
    return;
  }
  route_partial<S::BM>(a.part, a.count, a.splits, a.scene, rb, split, tid < S::BM ? tid : S::BM,
                       nr, best_s, best_i, s_last);
}

hipError_t launch_route_dtl(int dt, const void* q, const void* scene_keys, const float* bias,
                            int32_t* scene, int64_t rows, int d_e, int S, const RoutePlan& plan,
                            uint64_t* part, int32_t* count, hipStream_t st) {
  RouteDtlParams p{};
  p.q = static_cast<const char*>(q);
  p.keys = static_cast<const char*>(scene_keys);
  p.bias = bias;
  p.rows = rows;
  p.k_bytes = (int64_t)d_e * (dt == DT_BF16 ? 2 : 4);
  p.S = S;
  p.splits = plan.splits;
  p.tps = plan.per_split;
  p.units = (int)(((rows + RtShape::BM - 1) / RtShape::BM) * plan.splits);
  p.scene = scene;
  p.part = part;
  p.count = count;
  const unsigned grid = (unsigned)((p.units + 7) / 8 * 8);
  const dim3 block(64 * RT_WM * RT_WN);
  if (dt == DT_BF16) {
    if (bias != nullptr) hipLaunchKernelGGL((route_dtl_kernel<DT_BF16, true>), dim3(grid), block, 0, st, p);
    else hipLaunchKernelGGL((route_dtl_kernel<DT_BF16, false>), dim3(grid), block, 0, st, p);
  } else {
    if (bias != nullptr) hipLaunchKernelGGL((route_dtl_kernel<DT_F32, true>), dim3(grid), block, 0, st, p);
    else hipLaunchKernelGGL((route_dtl_kernel<DT_F32, false>), dim3(grid), block, 0, st, p);
  }
  return hipGetLastError();
}

}  // namespace lookme
