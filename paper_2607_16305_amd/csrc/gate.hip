// The learned SKA gate of the intra-layer sparse activation (arXiv
// 2607.16305, Sec. 3.3, Eq. 9) as it acts at inference: the Gumbel-Sigmoid
// is hard and noise-free, so position i opens when z_i = Delta_i W_g > 0.
// The open positions of a layer, in ascending order, are the rows R[g] that
// Eq. 10 injects; their number varies from batch to batch and stays on the
// device (a count per layer that the injection kernels read).
//
//   gate_logit    one wave per gated row: streams the row of Delta once
//                 (HBM-bound; four 16-byte loads in flight per lane) against
//                 the layer's W_g column (L2-resident), fp32 fused
//                 multiply-adds in a fixed order, one float z per row;
//   gate_compact  one workgroup per layer: every thread owns 32 consecutive
//                 rows (their signs packed in one register), a block prefix
//                 sum of the per-thread counts gives each open row its slot,
//                 so the list comes out ascending without sorting; the tail
//                 of the list is filled with -1 and the count stored.
#include "common.h"
#include "kernels.h"

namespace lookme {

constexpr int GATE_WAVES = 4;
constexpr int GATE_THREADS = 1024;
constexpr int GATE_PER_THREAD = 32;
constexpr int GATE_SPAN = GATE_THREADS * GATE_PER_THREAD;   // rows per compaction round

template <int DT>
__device__ __forceinline__ float dot16(u32x4_t a, u32x4_t b, float acc) {
  if constexpr (DT == DT_BF16) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc = fmaf(bf16lo(a[e]), bf16lo(b[e]), acc);
      acc = fmaf(bf16hi(a[e]), bf16hi(b[e]), acc);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) acc = fmaf(as_f32(a[e]), as_f32(b[e]), acc);
  }
  return acc;
}

// Row r of the launch is entry i = r mod n of layer l = r / n; it reads row
// pos[i] (clamped into [0, delta_rows)) of the layer's block of Delta, or row
// i when pos is null.
template <int DT>
__global__ __launch_bounds__(GATE_WAVES * WAVE) void gate_logit_kernel(
    const char* __restrict__ delta, int64_t n, int64_t delta_rows, int64_t row_bytes,
    const int32_t* __restrict__ pos, const char* __restrict__ w_g, int64_t rows,
    float* __restrict__ z_out) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * GATE_WAVES + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int64_t layer = r / n, i = r - layer * n;
  int64_t src = i;
  if (pos != nullptr) {
    src = pos[i];
    src = src < 0 ? 0 : (src >= delta_rows ? delta_rows - 1 : src);
  }
  const char* p = delta + (layer * delta_rows + src) * row_bytes;
  const char* w = w_g + layer * row_bytes;
  const int chunks = (int)(row_bytes / 16);
  float acc = 0.f;
  for (int c0 = lane; c0 < chunks; c0 += 4 * WAVE) {
    u32x4_t dv[4], wv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = c0 + u * WAVE;
      const int cc = c < chunks ? c : chunks - 1;
      dv[u] = ld16_nt(p + (int64_t)cc * 16);
      wv[u] = ld16(w + (int64_t)cc * 16);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (c0 + u * WAVE < chunks) acc = dot16<DT>(dv[u], wv[u], acc);
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) acc += __shfl_xor(acc, d, 64);
  if (lane == 0) z_out[r] = acc;
}

__global__ __launch_bounds__(GATE_THREADS) void gate_compact_kernel(
    const float* __restrict__ z_all, int64_t n, int32_t* __restrict__ kept_all,
    int32_t* __restrict__ count) {
  __shared__ int wsum[GATE_THREADS / WAVE];
  __shared__ int s_total;
  const int layer = blockIdx.x;
  const float* z = z_all + (int64_t)layer * n;
  int32_t* kept = kept_all + (int64_t)layer * n;
  const int tid = threadIdx.x;
  int64_t base = 0;   // open rows in earlier rounds
  for (int64_t r0 = 0; r0 < n; r0 += GATE_SPAN) {
    const int64_t i0 = r0 + (int64_t)tid * GATE_PER_THREAD;
    uint32_t open = 0;
#pragma unroll
    for (int b = 0; b < GATE_PER_THREAD; ++b) {
      const int64_t i = i0 + b;
      const float v = z[i < n ? i : n - 1];   // every load issued, none under a branch
      if (i < n && v > 0.f) open |= 1u << b;
    }
    const int c = __popc(open);
    const int incl = block_scan_incl<GATE_THREADS / WAVE>(c, wsum);
    if (tid == GATE_THREADS - 1) s_total = incl;
    int64_t slot = base + incl - c;
    while (open != 0) {
      const int b = __ffs(open) - 1;
      open &= open - 1;
      kept[slot++] = (int32_t)(i0 + b);
    }
    __syncthreads();
    base += s_total;
    __syncthreads();   // s_total is rewritten by the next round
  }
  for (int64_t i = base + tid; i < n; i += GATE_THREADS) kept[i] = -1;
  if (tid == 0) count[layer] = (int32_t)base;
}

hipError_t launch_gate(int dt, int layers, int64_t n, const void* delta, int64_t delta_rows,
                       int d_c, const int32_t* pos, const void* w_g, float* z, int32_t* kept,
                       int32_t* count, hipStream_t st) {
  const int64_t rows = (int64_t)layers * n;
  const int64_t rb = (int64_t)d_c * (dt == DT_BF16 ? 2 : 4);
  if (rows > 0) {
    const dim3 grid((unsigned)((rows + GATE_WAVES - 1) / GATE_WAVES));
    if (dt == DT_BF16)
      hipLaunchKernelGGL(gate_logit_kernel<DT_BF16>, grid, dim3(GATE_WAVES * WAVE), 0, st,
                         static_cast<const char*>(delta), n, delta_rows, rb, pos,
                         static_cast<const char*>(w_g), rows, z);
    else
      hipLaunchKernelGGL(gate_logit_kernel<DT_F32>, grid, dim3(GATE_WAVES * WAVE), 0, st,
                         static_cast<const char*>(delta), n, delta_rows, rb, pos,
                         static_cast<const char*>(w_g), rows, z);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(gate_compact_kernel, dim3((unsigned)layers), dim3(GATE_THREADS), 0, st, z,
                     n, kept, count);
  return hipGetLastError();
}

}  // namespace lookme
