// Direct global-to-LDS operand staging for the tiled matrix-core kernels
// (projection and large-batch routing).  A stage holds blocks of 16 rows x
// KB bytes of K (KB = 64 or 128), row r at KB * r.  A load instruction fills
// 1 KB of a block: neighbouring lanes read one row's contiguous bytes (KB / 16
// lanes per row, so the address unit coalesces them) and lane i's bytes land
// at 16 i; the row's 16-byte chunks are permuted by blk_swz so that the
// fragment reads of 8 or 16 lanes (rows) hit distinct LDS banks.
#pragma once
#include "common.h"

namespace lookme {

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// One direct global-to-LDS load of 16 bytes per lane: lane i's bytes land at
// lds_dst + 16 i (lds_dst is the same for the whole wave).  A plain function,
// so that the builtin is never looked at in a dependent context.
__device__ __forceinline__ void load_lds16(const void* src, char* lds_dst) {
  __builtin_amdgcn_global_load_lds(src, (lds_ptr_t)lds_dst, 16, 0, 0);
}
// The same with the nontemporal hint (data read once: the Level-2 keys).
__device__ __forceinline__ void load_lds16_nt(const void* src, char* lds_dst) {
  __builtin_amdgcn_global_load_lds(src, (lds_ptr_t)lds_dst, 16, 0, 2);
}

// chunk c of row r of a block sits in slot c ^ blk_swz(r): rows that share a
// bank window get distinct slots for one chunk index.  For 128-byte rows,
// r & 7 lets a fragment read (16 rows, one chunk index) run at ~210 bytes
// per clock per CU on gfx950; adding (r >> 3) & 1, as a 128-byte bank
// window would suggest, halves that (measured with a read-only probe)
template <int KB>
__device__ __forceinline__ int blk_swz(int r) {
  if constexpr (KB == 64) return ((r >> 1) & 3) ^ ((r >> 3) & 1);
  else return r & 7;
}

template <int WM, int WN, int MI, int NJ, int KB>
struct DtlShape {
  static_assert(KB == 64 || KB == 128, "stage width");
  static constexpr int BM = 16 * MI * WM, BN = 16 * NJ * WN;
  static constexpr int STAGE = (BM + BN) * KB;               // bytes per stage
  static constexpr int INSTR = STAGE / 1024;                 // load instructions per stage
  static constexpr int PER_WAVE = INSTR / (WM * WN);
  static_assert(PER_WAVE * WM * WN == INSTR, "loads split evenly over the waves");
  static constexpr int LPR = KB / 16, RPI = 64 / LPR;        // lanes per row, rows per load
};

// Reads the MFMA operand fragment of 16 rows starting at LDS row `row0` of a
// stage buffer, k-step ks: lane (g, n16) gets chunk 4 ks + g of row row0 + n16.
template <int KB>
__device__ __forceinline__ u32x4_t read_frag(const char* buf, int row0, int ks, int n16, int g) {
  return *reinterpret_cast<const u32x4_t*>(buf + (row0 + n16) * KB +
                                           (((4 * ks + g) ^ blk_swz<KB>(n16)) << 4));
}

}  // namespace lookme
