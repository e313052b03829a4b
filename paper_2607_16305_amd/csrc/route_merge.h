// Routing with the scene keys split over several workgroups (Eq. 5, arg max
// over all scenes): each workgroup's best (score, scene) of every row of its
// R-row tile goes to a partial table; the last of the tile's workgroups to
// arrive (device-scope counter) reduces the tile's partials in key-range
// order with the lowest-index tie rule, writes the scenes and resets the
// counter to zero for the next call.
//
// Every access to the partial table is a device-scope atomic (stores and
// loads), and each writer waits for its own stores to complete before the
// workgroup's arrival is counted; so the last workgroup's loads, made after
// it has seen every arrival, return the final partials.  No release or
// acquire fence is needed for the table, and none is issued: on this chip
// they write back and invalidate the whole L2 of the workgroup's XCD, which
// cost the image workload's routing 3 us (15.0 -> 11.9 us a launch).
#pragma once
#include "common.h"

namespace lookme {

// Called by every thread of the workgroup; thread t < nr carries row t.
// part: [tiles, splits, R] of (scene << 32 | score bits); count: [tiles].
template <int R>
__device__ __forceinline__ void route_partial(uint64_t* part_all, int32_t* count, int splits,
                                              int32_t* scene_out, int64_t tile, int split, int t,
                                              int nr, float best_s, int best_i, int* s_last) {
  uint64_t* part = part_all + (tile * splits) * R;
  if (t < nr)
    __hip_atomic_store(&part[split * R + t],
                       ((uint64_t)(uint32_t)best_i << 32) | __float_as_uint(best_s),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // this thread's partial has reached the device's coherence point ...
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  // ... and, after the barrier, every thread's has, before the arrival
  __syncthreads();
  if (threadIdx.x == 0)
    *s_last = __hip_atomic_fetch_add(&count[tile], 1, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT) == splits - 1;
  __syncthreads();
  if (!*s_last) return;
  if (t < nr) {
    float bs = -__builtin_inff();
    int bi = -1;
    for (int sp = 0; sp < splits; ++sp) {
      const uint64_t v = __hip_atomic_load(&part[sp * R + t], __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
      const float vs = __uint_as_float((uint32_t)v);
      const int vi = (int)(v >> 32);
      if (beats(vs, vi, bs, bi)) { bs = vs; bi = vi; }
    }
    scene_out[tile * R + t] = bi;
  }
  if (threadIdx.x == 0) count[tile] = 0;
}

}  // namespace lookme
