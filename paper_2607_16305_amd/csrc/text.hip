// Text pathway of a LookME layer (arXiv 2607.16305, Sec. 3.2 "Text
// embedding index-based lookup", Eq. 1): a text position's token id indexes
// its layer's text table directly, R_text = E_text[u], and the open gates of
// the pathway (Eq. 9-10) add that row into the position's hidden state.
//
//   text_inject  one workgroup per gated entry (one thread per 16-byte chunk
//                of the row, up to 256): the table row and the hidden row are
//                read once with coalesced 16-byte loads, summed in fp32 and
//                rounded once into H in place.  HBM-bound: 2 row reads and
//                one row write per open entry.
#include "common.h"
#include "kernels.h"

namespace lookme {

constexpr int TXT_THREADS = 256;

template <int DT>
__global__ __launch_bounds__(TXT_THREADS) void text_inject_kernel(
    int64_t n_text, const int32_t* __restrict__ kept, const int32_t* __restrict__ count,
    const int32_t* __restrict__ pos, const int32_t* __restrict__ ids,
    const char* __restrict__ table, int64_t vocab, int64_t t_bytes, char* __restrict__ hidden,
    int64_t n, int64_t h_bytes) {
  const int64_t j = blockIdx.x;
  if (count != nullptr && j >= count[0]) return;
  int64_t i = kept != nullptr ? kept[j] : j;
  i = i < 0 ? 0 : (i >= n_text ? n_text - 1 : i);
  int64_t t = pos[i], u = ids[i];
  t = t < 0 ? 0 : (t >= n ? n - 1 : t);
  u = u < 0 ? 0 : (u >= vocab ? vocab - 1 : u);
  const char* e = table + u * t_bytes;
  char* h = hidden + t * h_bytes;
  const int chunks = (int)(t_bytes / 16);
  for (int c = threadIdx.x; c < chunks; c += blockDim.x) {
    const u32x4_t ev = ld16_nt(e + (int64_t)c * 16);
    const u32x4_t hv = ld16(h + (int64_t)c * 16);
    u32x4_t out;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if constexpr (DT == DT_BF16)
        out[k] = pack_bf16x2(bf16lo(hv[k]) + bf16lo(ev[k]), bf16hi(hv[k]) + bf16hi(ev[k]));
      else
        out[k] = as_u32(as_f32(hv[k]) + as_f32(ev[k]));
    }
    st16(h + (int64_t)c * 16, out);
  }
}

hipError_t launch_text_inject(int dt, int64_t n_text, const int32_t* kept, const int32_t* count,
                              const int32_t* pos, const int32_t* ids, const void* table,
                              int64_t vocab, int d_t, void* hidden, int64_t n, int d_h,
                              hipStream_t st) {
  if (n_text == 0) return hipSuccess;
  const int64_t es = dt == DT_BF16 ? 2 : 4;
  const int ch = (int)((int64_t)d_t * es / 16);
  const int bs = ch >= TXT_THREADS ? TXT_THREADS : (ch + 63) / 64 * 64;
  const dim3 grid((unsigned)n_text);
  if (dt == DT_BF16)
    hipLaunchKernelGGL(text_inject_kernel<DT_BF16>, grid, dim3(bs), 0, st, n_text, kept, count,
                       pos, ids, static_cast<const char*>(table), vocab, (int64_t)d_t * es,
                       static_cast<char*>(hidden), n, (int64_t)d_h * es);
  else
    hipLaunchKernelGGL(text_inject_kernel<DT_F32>, grid, dim3(bs), 0, st, n_text, kept, count,
                       pos, ids, static_cast<const char*>(table), vocab, (int64_t)d_t * es,
                       static_cast<char*>(hidden), n, (int64_t)d_h * es);
  return hipGetLastError();
}

}  // namespace lookme
