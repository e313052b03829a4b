// Routing with the scene keys split over several workgroups (Eq. 5, arg max
// over all scenes): each workgroup's best (score, scene) of every row of its
// R-row tile goes to a partial table; the last of the tile's workgroups to
// arrive (device-scope counter) reduces the tile's partials in key-range
// order with the lowest-index tie rule, writes the scenes and resets the
// counter to zero for the next call.
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
    part[split * R + t] = ((uint64_t)(uint32_t)best_i << 32) | __float_as_uint(best_s);
  // the barrier orders every thread's store before thread 0's release; the
  // acquire half makes the other workgroups' partials visible to the last
  __syncthreads();
  if (threadIdx.x == 0)
    *s_last = __hip_atomic_fetch_add(&count[tile], 1, __ATOMIC_ACQ_REL,
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
