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
// 16-byte fragment reads of 8 consecutive rows hit distinct banks), the
// global loads of the next D stages in flight while one is multiplied.
#include <type_traits>

#include "common.h"
#include "dtl.h"
#include "kernels.h"

namespace lookme {

constexpr int PJ_STAGE = 128;                // bytes of K per stage and row
constexpr int PJ_LD = PJ_STAGE + 16;         // padded LDS row pitch
constexpr int PJ_THREADS = 256;
constexpr int PJ_CPR = PJ_STAGE / 16;        // 16-byte chunks per row per stage

// Rounds a wave's accumulators once to the storage dtype and scatters them
// to q[layer, token, :]: the lane holds C[r0 + 16i + 4g + r][c0 + 16j + n16].
template <int DT, int MI, int NJ>
__device__ __forceinline__ void store_tile(const f32x4_t (&acc)[MI][NJ], char* __restrict__ Q,
                                           int64_t M, int N, int d_e, int64_t r0, int c0,
                                           int n16, int g) {
  constexpr int ES = DT == DT_BF16 ? 2 : 4;
  const int64_t layer_stride = M * d_e;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int col = c0 + 16 * j + n16;
    if (col >= N) continue;
    const int layer = col / d_e, jj = col % d_e;
    char* qcol = Q + ((int64_t)layer * layer_stride + jj) * ES;
#pragma unroll
    for (int i = 0; i < MI; ++i) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = r0 + 16 * i + 4 * g + r;
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

// D: K stages whose global loads are in flight while one stage is multiplied
// (a ring of D register sets; every load is issued unconditionally, with
// its address clamped and its value zeroed when it lies outside the operand,
// so that the compiler's wait counts stay exact).  KG: groups of 4 waves that
// split K between them (group g takes stages g, g + KG, ...), each with its
// own LDS buffers; their partial tiles are summed through LDS in group order
// at the end, so a small M x N still keeps many loads in flight per tile.
template <int DT, int BM, int BN, int D, int KG>
__global__ __launch_bounds__(PJ_THREADS * KG) void project_kernel(
    const char* __restrict__ A, const char* __restrict__ B, char* __restrict__ Q, int64_t M,
    int N, int64_t k_bytes, int d_e, int tiles) {
  static_assert(D % 2 == 0, "the LDS buffer of a step is its parity");
  constexpr int MI = BM / 32, NJ = BN / 32;  // 16 x 16 MFMA tiles per wave
  constexpr int LA = BM * PJ_CPR / PJ_THREADS, LB = BN * PJ_CPR / PJ_THREADS;
  static_assert(LA >= 1 && LB >= 1, "a stage must cover every thread");
  __shared__ __attribute__((aligned(16))) char lds_a[KG][2][BM * PJ_LD];
  __shared__ __attribute__((aligned(16))) char lds_b[KG][2][BN * PJ_LD];
  const int tid = threadIdx.x & (PJ_THREADS - 1);
  const int kg = __builtin_amdgcn_readfirstlane(threadIdx.x / PJ_THREADS);
  const int lane = tid & 63, wv = tid >> 6;
  const int n16 = lane & 15, g = lane >> 4;
  const int wm = (wv >> 1) * (BM / 2), wn = (wv & 1) * (BN / 2);

  // tiles of one row block are neighbours in the work order and run on one
  // XCD, so their shared A rows come from that XCD's L2
  const int tiles_n = (N + BN - 1) / BN;
  const int tile = xcd_remap(blockIdx.x, tiles);
  if (tile < 0) return;
  const int64_t m0 = (int64_t)(tile / tiles_n) * BM;
  const int n0 = (tile % tiles_n) * BN;
  const int kchunks = (int)(k_bytes / 16);
  const int nstages = (int)((k_bytes + PJ_STAGE - 1) / PJ_STAGE);
  const int per_group = (nstages + KG - 1) / KG;
  const int nsteps = (per_group + D - 1) / D * D;   // padded: stages past K are zero

  u32x4_t ra[D][LA], rb[D][LB];
  auto gload = [&](u32x4_t (&a)[LA], u32x4_t (&b)[LB], int step) {
    const int stage = step * KG + kg;
#pragma unroll
    for (int r = 0; r < LA; ++r) {
      const int ci = tid + r * PJ_THREADS;
      const int kc = stage * PJ_CPR + ci % PJ_CPR;
      const int64_t am = m0 + ci / PJ_CPR;
      const bool ok = am < M && kc < kchunks;
      const u32x4_t v = ld16(A + (ok ? am * k_bytes + (int64_t)kc * 16 : 0));
      a[r] = ok ? v : u32x4_t{0, 0, 0, 0};
    }
#pragma unroll
    for (int r = 0; r < LB; ++r) {
      const int ci = tid + r * PJ_THREADS;
      const int kc = stage * PJ_CPR + ci % PJ_CPR;
      const int bn = n0 + ci / PJ_CPR;
      const bool ok = bn < N && kc < kchunks;
      const u32x4_t v = ld16(B + (ok ? (int64_t)bn * k_bytes + (int64_t)kc * 16 : 0));
      b[r] = ok ? v : u32x4_t{0, 0, 0, 0};
    }
  };
  auto lstore = [&](int buf, const u32x4_t (&a)[LA], const u32x4_t (&b)[LB]) {
#pragma unroll
    for (int r = 0; r < LA; ++r) {
      const int ci = tid + r * PJ_THREADS;
      st16(&lds_a[kg][buf][(ci / PJ_CPR) * PJ_LD + (ci % PJ_CPR) * 16], a[r]);
    }
#pragma unroll
    for (int r = 0; r < LB; ++r) {
      const int ci = tid + r * PJ_THREADS;
      st16(&lds_b[kg][buf][(ci / PJ_CPR) * PJ_LD + (ci % PJ_CPR) * 16], b[r]);
    }
  };

  f32x4_t acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int buf) {
#pragma unroll
    for (int s = 0; s < PJ_STAGE / 64; ++s) {
      u32x4_t fa[MI], fb[NJ];
#pragma unroll
      for (int i = 0; i < MI; ++i)
        fa[i] = *reinterpret_cast<const u32x4_t*>(
            &lds_a[kg][buf][(wm + 16 * i + n16) * PJ_LD + (4 * s + g) * 16]);
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        fb[j] = *reinterpret_cast<const u32x4_t*>(
            &lds_b[kg][buf][(wn + 16 * j + n16) * PJ_LD + (4 * s + g) * 16]);
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = mfma_chunk<DT>(fa[i], fb[j], acc[i][j]);
    }
  };

  // prologue: steps 0..D-1 in flight, step 0 in LDS buffer 0
#pragma unroll
  for (int d = 0; d < D; ++d) {
    gload(ra[d], rb[d], d);
    asm volatile("" ::: "memory");   // keep the issue order: older steps first
  }
  lstore(0, ra[0], rb[0]);
  __syncthreads();
  for (int st = 0; st < nsteps; st += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      // set d held step st+d, already in LDS: refill it with step st+d+D
      gload(ra[d], rb[d], st + d + D);
      compute(d & 1);
      // step st+d+1 (register set (d+1)%D) into the other buffer, which was
      // last read in the previous step, finished by every wave before the
      // barrier that ended it
      lstore((d + 1) & 1, ra[(d + 1) % D], rb[(d + 1) % D]);
      __syncthreads();
    }
  }

  if constexpr (KG > 1) {
    // partial tiles of groups 1..KG-1 through their (now idle) LDS buffers,
    // added by group 0 in group order; lane-private slots, no bank pattern
    // matters for this one pass
    static_assert(MI * NJ * PJ_THREADS * 16 <= 2 * (BM + BN) * PJ_LD,
                  "partial tile fits the buffers");
    // the buffers of one group are lds_a[g] (both halves) then lds_b[g]:
    // not contiguous, so the partial tile is split over lds_a[g] and lds_b[g]
    auto slot = [&](int grp, int idx) -> f32x4_t* {
      constexpr int IN_A = 2 * BM * PJ_LD / 16;   // f32x4 slots in lds_a[grp]
      const int e = idx * 256 + tid;               // wave-interleaved, 16 B per lane
      return e < IN_A ? reinterpret_cast<f32x4_t*>(&lds_a[grp][0][0]) + e
                      : reinterpret_cast<f32x4_t*>(&lds_b[grp][0][0]) + (e - IN_A);
    };
    if (kg > 0) {
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) *slot(kg, i * NJ + j) = acc[i][j];
    }
    __syncthreads();
    if (kg > 0) return;
#pragma unroll
    for (int o = 1; o < KG; ++o)
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const f32x4_t p = *slot(o, i * NJ + j);
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[i][j][r] += p[r];
        }
  }

  store_tile<DT, MI, NJ>(acc, Q, M, N, d_e, m0 + wm, n0 + wn, n16, g);
}

// Large problems: tiles fed by direct global-to-LDS loads, so no registers
// stage the operands; a ring of NS stages of KB bytes of K (64 or 128) per
// row.  WM x WN waves, each owning MI x NJ MFMA tiles of 16 x 16.  A stage
// holds blocks of 16 rows x KB bytes, row r at KB * r.  A load instruction
// fills 1 KB of a block: neighbouring lanes read one row's contiguous bytes
// (KB / 16 lanes per row, so the address unit coalesces them) and lane i's
// bytes land at 16 i; the row's 16-byte chunks are permuted by blk_swz so
// that the fragment reads of 8 or 16 lanes (rows) hit distinct LDS banks.
// With NS >= 3 the fragments of stage s + 1 are read while the matrix cores
// work on stage s; with NS = 2 the loads of stage s + 1 fly during stage s.
// Needs K in whole KB-byte steps.
// EPI_F32_BIAS epilogue: C + bias[col] stored as float32 [M, N] (the relevance
// MLP's logits), instead of the rounded, layer-scattered q.
constexpr int EPI_Q = 0, EPI_F32_BIAS = 1;

template <int MI, int NJ>
__device__ __forceinline__ void store_f32_bias(const f32x4_t (&acc)[MI][NJ], float* __restrict__ C,
                                               const float* __restrict__ bias, int64_t M, int N,
                                               int64_t r0, int c0, int n16, int g) {
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int col = c0 + 16 * j + n16;
    if (col >= N) continue;
    const float b = bias != nullptr ? bias[col] : 0.f;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = r0 + 16 * i + 4 * g + r;
        if (row < M) C[row * N + col] = acc[i][j][r] + b;
      }
  }
}

template <int DT, int WM, int WN, int MI, int NJ, int KB, int NS, int EPI = EPI_Q>
__global__ __launch_bounds__(64 * WM * WN) void project_dtl_kernel(
    const char* __restrict__ A, const char* __restrict__ B, char* __restrict__ Q, int64_t M,
    int N, int64_t k_bytes, int d_e, int tiles, const float* __restrict__ bias) {
  using S = DtlShape<WM, WN, MI, NJ, KB>;
  static_assert(NS >= 2, "a stage in flight while one is used");
  __shared__ __attribute__((aligned(1024))) char lds[NS][S::STAGE];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15, g = lane >> 4;
  const int wm = (wv / WN) * 16 * MI, wn = (wv % WN) * 16 * NJ;

  const int tiles_n = (N + S::BN - 1) / S::BN;
  const int tile = xcd_remap(blockIdx.x, tiles);
  if (tile < 0) return;
  const int64_t m0 = (int64_t)(tile / tiles_n) * S::BM;
  const int n0 = (tile % tiles_n) * S::BN;
  const int nst = (int)(k_bytes / KB);

  // this lane's source for each load it issues: load q of the stage covers
  // tile rows [q * RPI, q * RPI + RPI) (A rows first, then B rows); the lane
  // reads row q * RPI + lane / LPR, the chunk that belongs in slot lane % LPR.
  // Rows past the edge are clamped into the operand and feed only outputs
  // that are never stored.
  const char* src[S::PER_WAVE];
#pragma unroll
  for (int b = 0; b < S::PER_WAVE; ++b) {
    const int trow = (wv * S::PER_WAVE + b) * S::RPI + lane / S::LPR;
    const int chunk = (lane % S::LPR) ^ blk_swz<KB>(trow & 15);
    if (trow < S::BM) {
      int64_t r = m0 + trow;
      r = r < M ? r : M - 1;
      src[b] = A + r * k_bytes + chunk * 16;
    } else {
      int r = n0 + trow - S::BM;
      r = r < N ? r : N - 1;
      src[b] = B + (int64_t)r * k_bytes + chunk * 16;
    }
  }
  auto issue = [&](int stage) {
    const int s = stage < nst ? stage : nst - 1;   // past the end: a harmless reload
    char* dst = lds[stage % NS];
#pragma unroll
    for (int b = 0; b < S::PER_WAVE; ++b)
      load_lds16(src[b] + (int64_t)s * KB, dst + (wv * S::PER_WAVE + b) * 1024);
  };
  constexpr int KSL = KB / 64;   // MFMA k-steps per stage
  auto read = [&](int stage, u32x4_t (&fa)[KSL][MI], u32x4_t (&fb)[KSL][NJ]) {
    const char* buf = lds[stage % NS];
#pragma unroll
    for (int ks = 0; ks < KSL; ++ks) {
      const int off = n16 * KB + (((4 * ks + g) ^ blk_swz<KB>(n16)) << 4);
#pragma unroll
      for (int i = 0; i < MI; ++i)
        fa[ks][i] = *reinterpret_cast<const u32x4_t*>(buf + (wm + 16 * i) * KB + off);
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        fb[ks][j] = *reinterpret_cast<const u32x4_t*>(buf + (S::BM + wn + 16 * j) * KB + off);
    }
  };
  // wait until this wave's loads of all but the `younger` most recent stages
  // have landed, then a plain s_barrier (the fence of __syncthreads would
  // wait for every load in flight; the empty asm statements keep the compiler
  // from moving LDS accesses across it)
  auto sync = [&](auto younger) {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(decltype(younger)::value * S::PER_WAVE) : "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  f32x4_t acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  auto mma = [&](const u32x4_t (&fa)[KSL][MI], const u32x4_t (&fb)[KSL][NJ]) {
#pragma unroll
    for (int ks = 0; ks < KSL; ++ks)
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = mfma_chunk<DT>(fa[ks][i], fb[ks][j], acc[i][j]);
  };

  if constexpr (NS == 2) {
    issue(0);
    for (int s = 0; s < nst; ++s) {
      // stage s has landed everywhere and every read of stage s - 1 (the
      // other buffer) has ended: load stage s + 1 there, multiply stage s
      sync(std::integral_constant<int, 0>{});
      issue(s + 1);
      u32x4_t fa[KSL][MI], fb[KSL][NJ];
      read(s, fa, fb);
      mma(fa, fb);
    }
  } else {
    // step s: stage s + 1 has landed and every read of stage s - 1 has ended
    // (its fragments fed the previous step's products), so stage s + NS - 1
    // can go to the buffer of stage s - 1 while the fragments of stage s + 1
    // are read and the products of stage s run
    auto step = [&](int s, const u32x4_t (&ca)[KSL][MI], const u32x4_t (&cb)[KSL][NJ],
                    u32x4_t (&na)[KSL][MI], u32x4_t (&nb)[KSL][NJ]) {
      sync(std::integral_constant<int, NS - 3>{});
      issue(s + NS - 1);
      read(s + 1 < nst ? s + 1 : s, na, nb);
      mma(ca, cb);
    };
    u32x4_t fa0[KSL][MI], fb0[KSL][NJ], fa1[KSL][MI], fb1[KSL][NJ];
#pragma unroll
    for (int s = 0; s < NS - 1; ++s) issue(s);
    sync(std::integral_constant<int, NS - 2>{});
    read(0, fa0, fb0);
    int s = 0;
    for (; s + 1 < nst; s += 2) {
      step(s, fa0, fb0, fa1, fb1);
      step(s + 1, fa1, fb1, fa0, fb0);
    }
    if (s < nst) step(s, fa0, fb0, fa1, fb1);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // no load into LDS outlives the wave
  if constexpr (EPI == EPI_F32_BIAS)
    store_f32_bias<MI, NJ>(acc, reinterpret_cast<float*>(Q), bias, M, N, m0 + wm, n0 + wn, n16, g);
  else
    store_tile<DT, MI, NJ>(acc, Q, M, N, d_e, m0 + wm, n0 + wn, n16, g);
}

// 16 waves in 4 x 4, each 64 x 64: 256 x 256 tiles, one workgroup per CU,
// 128-byte stages, two of them
constexpr int PD_WM = 4, PD_WN = 4, PD_MI = 4, PD_NJ = 4, PD_KB = 128, PD_STAGES = 2;

template <int DT, int WM, int WN, int MI, int NJ, int KB, int NS>
static void launch_dtl(const void* x, const void* wt, void* q, int64_t n, int N, int64_t kb,
                       int d_e, hipStream_t st) {
  using S = DtlShape<WM, WN, MI, NJ, KB>;
  const int64_t tiles = ((n + S::BM - 1) / S::BM) * ((N + S::BN - 1) / S::BN);
  const int64_t slots = (tiles + 7) / 8 * 8;
  hipLaunchKernelGGL((project_dtl_kernel<DT, WM, WN, MI, NJ, KB, NS>), dim3((unsigned)slots),
                     dim3(64 * WM * WN), 0, st, static_cast<const char*>(x),
                     static_cast<const char*>(wt), static_cast<char*>(q), n, N, kb, d_e,
                     (int)tiles, nullptr);
}

template <int DT, int BM, int BN, int D, int KG>
static void launch_tiles(const void* x, const void* wt, void* q, int64_t n, int N, int64_t kb,
                         int d_e, hipStream_t st) {
  const int64_t tiles = ((n + BM - 1) / BM) * ((N + BN - 1) / BN);
  const int64_t slots = (tiles + 7) / 8 * 8;
  hipLaunchKernelGGL((project_kernel<DT, BM, BN, D, KG>), dim3((unsigned)slots),
                     dim3(PJ_THREADS * KG), 0,
                     st, static_cast<const char*>(x), static_cast<const char*>(wt),
                     static_cast<char*>(q), n, N, kb, d_e, (int)tiles);
}

hipError_t launch_project(int dt, const void* x, const void* wt, void* q, int64_t n, int d_in,
                          int d_e, int layers, hipStream_t st) {
  if (n == 0) return hipSuccess;
  const int es = dt == DT_BF16 ? 2 : 4;
  const int N = layers * d_e;
  const int64_t kb = (int64_t)d_in * es;
  const int64_t tiles128 = ((n + 127) / 128) * ((N + 127) / 128);
  if (tiles128 >= 256 && kb % PD_KB == 0) {
    // enough large tiles to fill the chip: direct-to-LDS pipeline
    if (dt == DT_BF16) launch_dtl<DT_BF16, PD_WM, PD_WN, PD_MI, PD_NJ, PD_KB, PD_STAGES>(x, wt, q, n, N, kb, d_e, st);
    else launch_dtl<DT_F32, PD_WM, PD_WN, PD_MI, PD_NJ, PD_KB, PD_STAGES>(x, wt, q, n, N, kb, d_e, st);
    return hipGetLastError();
  }
  // else 32 x 64 tiles with K split over 4 wave groups
  if (dt == DT_BF16) launch_tiles<DT_BF16, 32, 64, 4, 4>(x, wt, q, n, N, kb, d_e, st);
  else launch_tiles<DT_F32, 32, 64, 4, 4>(x, wt, q, n, N, kb, d_e, st);
  return hipGetLastError();
}

bool launch_logits_gemm(int dt, const void* a, const void* w, const float* bias, float* out,
                        int64_t rows, int N, int64_t kb, hipStream_t st) {
  const int64_t tiles128 = ((rows + 127) / 128) * ((N + 127) / 128);
  if (tiles128 < 256 || kb % PD_KB != 0) return false;
  using S = DtlShape<PD_WM, PD_WN, PD_MI, PD_NJ, PD_KB>;
  const int64_t tiles = ((rows + S::BM - 1) / S::BM) * ((N + S::BN - 1) / S::BN);
  const unsigned grid = (unsigned)((tiles + 7) / 8 * 8);
  if (dt == DT_BF16)
    hipLaunchKernelGGL((project_dtl_kernel<DT_BF16, PD_WM, PD_WN, PD_MI, PD_NJ, PD_KB, PD_STAGES,
                                           EPI_F32_BIAS>),
                       dim3(grid), dim3(64 * PD_WM * PD_WN), 0, st, static_cast<const char*>(a),
                       static_cast<const char*>(w), reinterpret_cast<char*>(out), rows, N, kb, N,
                       (int)tiles, bias);
  else
    hipLaunchKernelGGL((project_dtl_kernel<DT_F32, PD_WM, PD_WN, PD_MI, PD_NJ, PD_KB, PD_STAGES,
                                           EPI_F32_BIAS>),
                       dim3(grid), dim3(64 * PD_WM * PD_WN), 0, st, static_cast<const char*>(a),
                       static_cast<const char*>(w), reinterpret_cast<char*>(out), rows, N, kb, N,
                       (int)tiles, bias);
  return true;
}

}  // namespace lookme
