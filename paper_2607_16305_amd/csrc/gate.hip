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
#include "crit.h"
#include "kernels.h"

namespace lookme {

constexpr int GATE_WAVES = 4;
constexpr int GATE_THREADS = 1024;

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
  const float acc = row_dot<DT>(delta + (layer * delta_rows + src) * row_bytes,
                                w_g + layer * row_bytes, (int)(row_bytes / 16), lane);
  if (lane == 0) z_out[r] = acc;
}

__global__ __launch_bounds__(GATE_THREADS) void gate_compact_kernel(
    const float* __restrict__ z_all, int64_t n, int32_t* __restrict__ kept_all,
    int32_t* __restrict__ count) {
  __shared__ SelLds sl;
  const int layer = blockIdx.x;
  gate_compact_layer<GATE_THREADS>(z_all + (int64_t)layer * n, n, kept_all + (int64_t)layer * n,
                                   count + layer, sl);
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
