// Routing with the scene keys split over several workgroups (Eq. 5, arg max
// over all scenes): each workgroup's best (score, scene) of every row of its
// R-row tile goes to a partial table; the last of the tile's workgroups to
// arrive (device-scope counter) reduces the tile's partials in key-range
// order with the lowest-index tie rule, writes the scenes and resets the
// counter to zero for the next call.
//
// Ordering, in the terms of the scoped (HSA / LLVM AMDGPU) memory model: a
// thread's partial store is sequenced before the workgroup barrier, whose
// release/acquire fences (workgroup scope) order it before thread 0's arrival;
// the arrival is an agent-scope acquire-release read-modify-write, so every
// earlier arrival (a release at agent scope) synchronises with the last one,
// whose barrier then orders its threads' partial loads after all of them.
// Happens-before is transitive across these scope-inclusive pairs, so the
// last workgroup reads the final partials.  Relaxed atomics alone (an earlier
// form) give no order between the partial table and the counter in that
// model; they relied on the store acknowledgement that s_waitcnt vmcnt(0)
// waits for, a property of the hardware the model does not state.  The
// release costs one L2 write-back per arriving workgroup (only thread 0
// performs it), the acquire one invalidation in the last workgroup.
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
  __syncthreads();   // every thread's partial is ordered before the arrival
  if (threadIdx.x == 0)
    *s_last = __hip_atomic_fetch_add(&count[tile], 1, __ATOMIC_ACQ_REL,
                                     __HIP_MEMORY_SCOPE_AGENT) == splits - 1;
  __syncthreads();   // ... and the last arrival before every thread's loads
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
