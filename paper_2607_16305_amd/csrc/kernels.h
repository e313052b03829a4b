// Host-side launchers of the gfx950 kernels.  Each returns the HIP status of
// its launches; shapes are validated by the caller (lookme_abi.cpp) before
// any launcher runs.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "lookme.h"

namespace lookme {

// ---- projection: q[l, t, :] = round(x[t, :] . Wt[l]^T) --------------------
hipError_t launch_project(int dt, const void* x, const void* wt, void* q, int64_t n, int d_in,
                          int d_e, int layers, hipStream_t st);
// out[rows, N] = a w^T + bias (float32) on the projection's 256 x 256 tiles,
// when the product has enough of them (at least 256 of 128 x 128) and K is
// whole 128-byte stages; returns false (nothing launched) otherwise.
bool launch_logits_gemm(int dt, const void* a, const void* w, const float* bias, float* out,
                        int64_t rows, int N, int64_t kb, hipStream_t st);

// ---- library-owned scratch (noalloc.hip) ---------------------------------
// lookme_inject_noalloc keeps the criticality keys of up to
// LOOKME_NOALLOC_MAX_ROWS rows and, when the caller passes no kept_out, the
// kept lists in a static device array of NOALLOC_SCRATCH_BYTES; this returns
// its device address on the current device (looked up once per device).
constexpr size_t NOALLOC_KEYS_BYTES = (size_t)LOOKME_NOALLOC_MAX_ROWS * 4;
constexpr size_t NOALLOC_SCRATCH_BYTES = 2 * NOALLOC_KEYS_BYTES;
hipError_t noalloc_scratch(void** out);

// ---- routing: scene[r] = argmax_s <q_r, K1[s]> + bias[s] over rows r -------
// Three kernels, by batch size (route_plan):
//  * ROUTE_DTL: batches of ROUTE_DTL_MIN_ROWS to 128 * ROUTE_DTL_MAX_BLOCKS rows
//    whose key rows are whole 128-byte steps (larger batches run faster in
//    the shared mode): 128-row blocks x 256-key tiles on the matrix cores
//    (route.hip), the key tiles of a block split over up to `splits`
//    workgroups of `per_split` tiles when there are few blocks;
//  * ROUTE_STREAM: small batches, 16-row tiles in the scoring kernel's
//    streaming mode, the keys split over `splits` workgroups of `per_split`
//    keys;
//  * ROUTE_SHARED: the scoring kernel's shared mode (64- or 128-row units).
// Split work meets in route_partial: `part` holds part_entries (scene, score)
// pairs, `count` ROUTE_COUNTERS arrival counters that are zero before the
// first call and left at zero by every call.
constexpr int ROUTE_STREAM = 0, ROUTE_SHARED = 1, ROUTE_DTL = 2;
constexpr int ROUTE_DTL_ROWS = 128, ROUTE_DTL_KEYS = 256, ROUTE_DTL_MAX_TPS = 16;
constexpr int64_t ROUTE_DTL_MIN_ROWS = 4096, ROUTE_DTL_MAX_BLOCKS = 512;
constexpr int ROUTE_COUNTERS = 4096;
struct RoutePlan {
  int mode;
  int splits;
  int per_split;          // DTL: 256-key tiles; STREAM: keys (a multiple of 64)
  int64_t part_entries;
};
// cos: cosine scores, which only the scoring kernel's modes implement
RoutePlan route_plan(int64_t rows, int S, int64_t row_bytes, bool cos = false);
hipError_t launch_route(int dt, const void* q, const void* scene_keys, const float* bias,
                        int32_t* scene, int64_t rows, int d_e, int S, uint64_t* part,
                        int32_t* count, hipStream_t st, bool cos = false);
hipError_t launch_route_dtl(int dt, const void* q, const void* scene_keys, const float* bias,
                            int32_t* scene, int64_t rows, int d_e, int S, const RoutePlan& plan,
                            uint64_t* part, int32_t* count, hipStream_t st);

// ---- bucketing of rows by scene -----------------------------------------
// Level-2 work units: a bucket of at most UNIT_STREAM_ROWS rows is one
// streaming unit; a larger bucket is cut into shared units of at most
// shared_unit_rows() rows, tagged with UNIT_SHARED in unit_scene.  In the
// work list the two kinds alternate (shared first) while both last, then the
// rest of the longer kind follows; each kind keeps scene order.
//
// The launch's last round: when the streaming units outnumber the shared ones
// by at least SPLIT_UNITS (and the caller allows it), the last SPLIT_UNITS
// streaming units of the list are each cut into SPLIT_PARTS parts, equal
// ranges of the scene's key blocks, listed as consecutive entries at the end.
// Each part keeps the exact top k of its keys as a partial list; a small
// launch after the Level-2 launch merges a unit's lists (the results are
// those of the whole unit, bit for bit).  unit_count holds [0] the number of
// list entries, [1] the position of the first part (= [0] without parts),
// [2] the count of parts taken so far by the Level-2 launch's workgroups past
// the statically dealt units (zeroed by the bucketing).
constexpr int UNIT_STREAM_ROWS = 16;
constexpr int32_t UNIT_SHARED = 1 << 30;
constexpr int SPLIT_UNITS = 512;
constexpr int SPLIT_PARTS = 2;
constexpr int SPLIT_KMAX = 32;   // entries of a partial list slot (k <= 32)
// partial lists: [SPLIT_UNITS units][SPLIT_PARTS parts][16 rows][SPLIT_KMAX]
// of (index << 32 | score bits)
constexpr size_t SPLIT_PART_BYTES =
    (size_t)SPLIT_UNITS * SPLIT_PARTS * UNIT_STREAM_ROWS * SPLIT_KMAX * 8;
// Chunk steps (64 bytes of a key row each) the scoring kernel is compiled
// for, given the row width: 4, 8, 16 or 32 exactly; narrower rows run the
// 4-step kernel and other widths the 32-step kernel, with the steps past the
// row masked off.
inline int score_ks(int64_t row_bytes) {
  const int64_t ks = row_bytes / 64;
  if (ks == 4 || ks == 8 || ks == 16 || ks == 32) return (int)ks;
  return ks < 4 ? 4 : 32;
}
// Rows of a shared unit.  Level-2 (k > 0): 64, one 16-row query tile per
// wave (the per-lane top-k upkeep of a second tile would double each wave's
// serial vector work and its registers, one workgroup per CU instead of two).
// Routing (k = 0): two tiles per wave, 128 rows, when the kernel runs at most
// 16 chunk steps (two 32-step tiles would need 64 fragment loads in flight,
// more than the 6-bit vector-memory counter of a wave can track).
inline int shared_unit_rows(int64_t row_bytes, int k) {
  if (k > 0) return 64;
  return score_ks(row_bytes) <= 16 ? 128 : 64;
}
struct BucketWs {
  int32_t* chunk_hist;   // [chunks, S]
  int32_t* local_rank;   // [rows]
  int32_t* offsets;      // [S + 1]
  int32_t* perm;         // [rows]
  int32_t* unit_scene;   // [max_units]
  int32_t* unit_begin;   // [max_units]
  int32_t* unit_count;   // [3]: entries, first part, parts taken
  int64_t chunks;
  int64_t max_units;
  int split_max;         // SPLIT_UNITS or 0: whether the last round may be cut
  uint64_t* split_part;  // [SPLIT_PART_BYTES] partial lists of the parts
  int32_t* split_row;    // [SPLIT_UNITS, 16] output row + 1 of a cut unit's rows, zero between launches
};
int64_t bucket_chunks(int64_t rows);
int64_t bucket_max_units(int64_t rows, int S);
hipError_t launch_bucket(const int32_t* scene, int64_t rows, int S, int shared_rows,
                         const BucketWs& ws, hipStream_t st);
// launch_bucket for a batch of at most one chunk with the per-row signal of
// the sparse injection computed by extra workgroups of the same launch: the
// criticality norms of Eq. 9 (w_g null: crit [rows, d_c] -> key [rows], the
// bits of launch_crit_norm) or the learned gate's logits (w_g [rows / n, d_c]
// per layer of n rows -> key as float z, the bits of launch_gate's); false
// (nothing launched) when the batch is larger.
bool launch_bucket_norms(int dt, const int32_t* scene, int64_t rows, int S, int shared_rows,
                         const BucketWs& ws, const void* crit, int d_c, uint32_t* key,
                         hipStream_t st, const void* w_g = nullptr, int64_t n = 0);

// ---- Level-2 in the paper's form (Eq. 6-7): relevance MLP ----------------
// The MLP's tensors are borrowed from the caller: w1 [hidden, 2 d_e] and
// w2 [P, hidden] in the table's dtype, b1 [hidden] and b2 [P] float32 (or
// null).  launch_relevance writes act [rows, hidden], prim [rows, k] and
// w [rows, k], with logits [rows, P] float32 as scratch (workspace).
struct RelevanceMlp {
  int hidden;
  const void* w1;
  const float* b1;
  const void* w2;
  const float* b2;
};
// The per-scene half of the MLP's first layer, tab[s] = K1[s] W1b^T + b1
// ([S, hidden] float32; W1b the columns of W1 that multiply the scene key).
hipError_t launch_relevance_table(int dt, const void* scene_keys, const RelevanceMlp& mlp, int S,
                                  int d_e, float* tab, hipStream_t st);
// Level-2 in the paper's form for `rows` rows; tab from launch_relevance_table.
hipError_t launch_relevance(int dt, const void* q, const int32_t* scene, const float* tab,
                            const void* prim_keys, const RelevanceMlp& mlp, int64_t rows, int d_e,
                            int S, int P, int k, void* act, int32_t* prim, float* w,
                            float* logits, hipStream_t st);

// ---- sparse injection through the SwiGLU fusion (Eq. 10) ----------------
// Per layer l (tensors borrowed): w_gate, w_up [layers, d_ff, d_v] and
// w_down [layers, d_h, d_ff] in the table's dtype.  launch_gather_rows
// writes R [layers * n_keep, d_v] (rounded); launch_fusion then writes
// U [layers * n_keep, d_ff] and adds W_down U into the kept rows of H, the
// kept list of layer l at kept + l * kept_batch (0: one list for all).
struct FusionFfn {
  int layers, d_ff, d_h;
  const void* w_gate;
  const void* w_up;
  const void* w_down;
};
// kept_batch: stride between the layers' kept lists (0: one list for all);
// scene_step: scene offset of each layer in the table (multi-scale
// partitions; the layer's own scene ids are clamped into [0, S)).
hipError_t launch_gather_rows(int dt, int layers, int64_t n, int64_t n_keep, const int32_t* kept,
                              const int32_t* scene, const int32_t* prim, const float* w,
                              const void* values, int S, int P, int d_v, int k, void* r_out,
                              hipStream_t st, int64_t kept_batch, int scene_step,
                              const int32_t* count = nullptr);
// count (or null): the kept lists are counted (the learned gate), layer l
// using its first count[l] entries (count[0] when kept_batch is 0); n_keep
// is then the lists' capacity.
hipError_t launch_fusion(int dt, const FusionFfn& f, int layers, int64_t n, int64_t n_keep,
                         const int32_t* kept, int64_t kept_batch, int d_v, const void* r, void* u,
                         void* hidden, hipStream_t st, const int32_t* count = nullptr);
// Propagation of Eq. 11 over `steps` layers: r holds [steps + 1, n_keep, d_v]
// (slice 0 given); slice j = round(slice j-1 W_p^j + slice j-1), with
// w_p_t [steps, d_v, d_v] holding each W_p transposed (output-row-major).
// count (or null): only the first count[0] rows of each slice are live.
hipError_t launch_propagate(int dt, const void* w_p_t, int steps, int64_t n_keep, int d_v,
                            void* r, hipStream_t st, const int32_t* count = nullptr);

// ---- multi-scale retrieval with the token-wise router (Eq. 8) -------------
// Scale m's lookup (scene [M, n] local to partition m of S / M scenes, prim
// and w [M, n, k]) gives R^m of every kept token, gathered and rounded into
// r [M, n_keep, d_v]; q = round(H[kept] W_he) into q [n_keep, d_v] (w_he_t
// [d_v, d_h], output-row-major); then H[t, :d_v] = round(H + sum_m alpha_m
// R^m) with alpha = softmax_m(q . R^m / sqrt(d_v)).
constexpr int MS_MAX_SCALES = 8;
hipError_t launch_multiscale(int dt, int scales, int64_t n, int64_t n_keep, const int32_t* kept,
                             const int32_t* scene, const int32_t* prim, const float* w,
                             const void* values, int S, int P, int d_v, int k,
                             const void* w_he_t, int d_h, void* hidden, void* r, void* q,
                             hipStream_t st, const int32_t* count = nullptr);

// ---- Level-2 scoring of bucketed rows, fused top-k + softmax --------------
// The sparse-injection select (Eq. 9-10) of the same batch carried by the
// Level-2 launch: one extra workgroup per layer selects that layer's kept set
// [n_keep] (kept + l * n_keep) from its criticality keys (key + l * n, from
// an earlier launch); or, with `count` set, compacts the open rows of the
// learned gate from its logits (key + l * n as float) into kept + l * n
// (ascending, -1 tail) and count[l].  Needs n <= SEL_SIDE_MAX_N.
constexpr int SEL_SIDE_MAX_N = 4096;
struct SideSelect {
  int layers;
  int64_t n, n_keep;
  const uint32_t* key;
  int32_t* kept;
  int32_t* count = nullptr;
};
hipError_t launch_lookup(int dt, const void* q, const void* prim_keys, const BucketWs& ws,
                         int d_e, int P, int k, int32_t* prim, float* w, hipStream_t st,
                         const SideSelect* side = nullptr, bool cos = false,
                         const hipEvent_t* stamp = nullptr);

// ---- criticality, select and injection ------------------------------------
// background: a grid of one workgroup a CU walking the rows, for norms that
// run on a second stream beside the projection and routing (slower alone,
// but they take less of each CU from the kernels beside them)
hipError_t launch_crit_norm(int dt, int64_t rows, const void* crit, int d_c, uint32_t* key,
                            hipStream_t st, bool background = false);
hipError_t launch_crit_select(int layers, int64_t n, int64_t n_keep, const uint32_t* key,
                              int32_t* kept, hipStream_t st);
// The injections' count of rows with an index out of range (see
// inject_kernel), read and reset on `st` (synchronising it).
hipError_t take_index_errors(hipStream_t st, uint64_t* out);
hipError_t launch_inject_rows(int dt, int layers, int64_t n, int64_t n_keep, const int32_t* kept,
                              const int32_t* scene, const int32_t* prim, const float* w,
                              const void* values, int S, int P, int d_v, int k, void* hidden,
                              int d_h, hipStream_t st, const int32_t* count = nullptr);

// ---- learned SKA gate (Eq. 9) ---------------------------------------------
// z [layers * n] float32 scratch; kept [layers, n] gets each layer's open
// entries ascending, then -1; count [layers] their number.  Entry i of layer
// l reads row pos[i] (or i) of delta + l * delta_rows * d_c.
hipError_t launch_gate(int dt, int layers, int64_t n, const void* delta, int64_t delta_rows,
                       int d_c, const int32_t* pos, const void* w_g, float* z, int32_t* kept,
                       int32_t* count, hipStream_t st);

// ---- text pathway (Eq. 1) -------------------------------------------------
// For the first count[0] entries j of kept (all n_text entries when kept is
// null; count null: all of kept's n_text): i = kept[j],
// hidden[pos[i], :d_t] = round(hidden[pos[i], :d_t] + table[ids[i]]).
// Scene-centred keys of Eq. 4 (scene_keys.hip): scene_keys[s] = round(sum_p
// prim_keys[s, p] / P), float32 sum in p order.
hipError_t launch_scene_keys(int dt, const void* prim_keys, int S, int P, int d_e,
                             void* scene_keys, hipStream_t st);
hipError_t launch_text_inject(int dt, int64_t n_text, const int32_t* kept, const int32_t* count,
                              const int32_t* pos, const int32_t* ids, const void* table,
                              int64_t vocab, int d_t, void* hidden, int64_t n, int d_h,
                              hipStream_t st);

}  // namespace lookme
