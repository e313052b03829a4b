// C ABI of the LookME hot path: argument validation, workspace layout and
// launch sequencing.  All arithmetic happens in the gfx950 kernels; this file
// only checks arguments (before anything is launched) and enqueues kernels.
#include "lookme.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "kernels.h"

// Timing events of one kernel group launch (measurement support only).
struct TimedLaunch {
  int group;
  hipEvent_t start, stop;
};

struct lookme_s {
  lookme_desc_t d;
  const void* scene_keys;
  const void* prim_keys;
  const void* values;
  const float* bias;
  void* ws;
  size_t ws_bytes;
  bool profiling;
  std::vector<TimedLaunch> pending;        // recorded, not yet read
  std::vector<hipEvent_t> spare;           // event pool
  int64_t prof_count[LOOKME_GROUP_COUNT];
  double prof_ms[LOOKME_GROUP_COUNT];
  lookme::RelevanceMlp rel;                // hidden == 0: none registered
  bool rel_tab_ready = false;              // the workspace holds rel's per-scene table
  lookme::FusionFfn fus;                   // d_ff == 0: none registered
  int32_t prop_steps = 0;                  // Eq. 11 projections; 0: none registered
  const void* prop_w = nullptr;            // [prop_steps, value_dim, value_dim], transposed
  int32_t ms_scales = 0;                   // Eq. 8 router; 0: none registered
  int32_t ms_dh = 0;
  const void* ms_w = nullptr;              // W_{h->e} transposed, [value_dim, ms_dh]
};

namespace {

thread_local std::string g_err;

lookme_status_t fail(lookme_status_t st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
lookme_status_t fail(lookme_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

lookme_status_t hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return LOOKME_OK;
  return fail(LOOKME_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

inline int elem_size(int32_t dt) { return dt == LOOKME_BF16 ? 2 : 4; }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline size_t up256(size_t x) { return (x + 255) & ~size_t(255); }

constexpr int32_t MAX_SCENES = 16384;   // bucketing keeps one histogram per chunk in LDS

// Workspace layout for `layers` x `n` rows.
struct Layout {
  size_t chunk_hist, local_rank, offsets, perm, unit_scene, unit_begin, unit_count, route_count,
      route_part, split_row, split_part, crit_key, kept, rel_tab, rel_logits, fus_r, fus_u, ms_r,
      ms_q, total;
};

// The leading bytes of the workspace hold counters that start at zero; they
// are zero-filled once when the workspace is attached and every call leaves
// them at zero.
constexpr size_t ZEROED_BYTES =
    256 + lookme::ROUTE_COUNTERS * 4 + (size_t)lookme::SPLIT_UNITS * lookme::UNIT_STREAM_ROWS * 4;

Layout layout(const lookme_desc_t& d, int32_t layers, int64_t n, int32_t relevance,
              int32_t fusion_dff, int32_t scales) {
  const int64_t rows = (int64_t)layers * n;
  const int64_t chunks = lookme::bucket_chunks(rows);
  const int64_t units = lookme::bucket_max_units(rows, d.num_scenes);
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += up256(bytes);
    return at;
  };
  L.unit_count = take(256);   // counters first: the region zeroed at set-up
  L.route_count = take((size_t)lookme::ROUTE_COUNTERS * 4);
  L.split_row = take((size_t)lookme::SPLIT_UNITS * lookme::UNIT_STREAM_ROWS * 4);
  // the relevance MLP's per-scene table [S, hidden] float32, kept across
  // calls: at an offset that does not depend on the batch
  L.rel_tab = take(relevance ? (size_t)d.num_scenes * relevance * 4 : 0);
  const lookme::RoutePlan plan =
      lookme::route_plan(rows, d.num_scenes, (int64_t)d.key_dim * elem_size(d.dtype),
                         d.score == LOOKME_SCORE_COS);
  L.route_part = take((size_t)plan.part_entries * 8);
  L.chunk_hist = take((size_t)chunks * d.num_scenes * 4);
  L.local_rank = take((size_t)rows * 4);
  L.offsets = take(((size_t)d.num_scenes + 1) * 4);
  L.perm = take((size_t)rows * 4);
  L.unit_scene = take((size_t)units * 4);
  L.unit_begin = take((size_t)units * 4);
  // the partial lists of a Level-2 launch's cut last round (batches of at
  // least two rounds of units)
  L.split_part = take(rows >= 2 * lookme::SPLIT_UNITS ? lookme::SPLIT_PART_BYTES : 0);
  L.crit_key = take((size_t)rows * 4);
  L.kept = take((size_t)rows * 4);
  // relevance logits [rows, P] float32, when an MLP is registered (the
  // lists of a split second layer, or the logits of the unfused widths)
  L.rel_logits = take(relevance ? (size_t)rows * d.prims_per_scene * 4 : 0);
  // the fusion's R and inner activations of the kept rows (at most all rows)
  const size_t es = (size_t)elem_size(d.dtype);
  L.fus_r = take(fusion_dff > 0 ? (size_t)rows * d.value_dim * es : 0);
  L.fus_u = take(fusion_dff > 0 ? (size_t)rows * fusion_dff * es : 0);
  // the multi-scale router's retrieved rows [scales, rows, d_v] and queries
  L.ms_r = take(scales > 0 ? (size_t)scales * rows * d.value_dim * es : 0);
  L.ms_q = take(scales > 0 ? (size_t)rows * d.value_dim * es : 0);
  L.total = off;
  return L;
}

lookme_status_t check_handle(lookme_t h) {
  if (h == nullptr) return fail(LOOKME_ERR_INVALID, "null handle");
  return LOOKME_OK;
}

lookme_status_t check_ptr(const void* p, const char* name) {
  if (p == nullptr) return fail(LOOKME_ERR_INVALID, "%s is NULL", name);
  if (!aligned16(p)) return fail(LOOKME_ERR_INVALID, "%s is not 16-byte aligned", name);
  return LOOKME_OK;
}

lookme_status_t check_layers_n(int32_t layers, int64_t n) {
  if (layers < 1) return fail(LOOKME_ERR_INVALID, "layers must be >= 1 (got %d)", layers);
  if (n < 0) return fail(LOOKME_ERR_INVALID, "n must be >= 0 (got %lld)", (long long)n);
  if ((int64_t)layers * n > (int64_t)INT32_MAX / 2)
    return fail(LOOKME_ERR_UNSUPPORTED, "layers * n = %lld exceeds 2^30 rows",
                (long long)((int64_t)layers * n));
  return LOOKME_OK;
}

lookme_status_t check_workspace(lookme_t h, int32_t layers, int64_t n, Layout* L) {
  *L = layout(h->d, layers, n, h->rel.hidden, h->fus.d_ff, h->ms_scales);
  if (h->ws == nullptr) return fail(LOOKME_ERR_WORKSPACE, "no workspace set");
  if (h->ws_bytes < L->total)
    return fail(LOOKME_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed for %d x %lld rows",
                h->ws_bytes, L->total, layers, (long long)n);
  return LOOKME_OK;
}

lookme_status_t check_keep(int64_t n, int64_t n_keep) {
  if (n_keep < 0 || n_keep > n)
    return fail(LOOKME_ERR_INVALID, "n_keep %lld outside [0, n=%lld]", (long long)n_keep,
                (long long)n);
  return LOOKME_OK;
}

lookme_status_t check_crit_dim(const lookme_desc_t& d, int32_t d_c) {
  if (d_c < 1) return fail(LOOKME_ERR_INVALID, "d_c must be positive");
  if (((int64_t)d_c * elem_size(d.dtype)) % 16 != 0)
    return fail(LOOKME_ERR_UNSUPPORTED, "d_c times elem_size must be a multiple of 16");
  return LOOKME_OK;
}

lookme_status_t check_hidden_dim(const lookme_desc_t& d, int32_t d_h) {
  if (d_h < 1) return fail(LOOKME_ERR_INVALID, "d_h must be positive");
  if (d.value_dim > d_h)
    return fail(LOOKME_ERR_INVALID, "value_dim %d exceeds d_h %d", d.value_dim, d_h);
  if (((int64_t)d_h * elem_size(d.dtype)) % 16 != 0)
    return fail(LOOKME_ERR_UNSUPPORTED, "d_h times elem_size must be a multiple of 16");
  return LOOKME_OK;
}

hipError_t take_event(lookme_t h, hipEvent_t* ev) {
  if (!h->spare.empty()) {
    *ev = h->spare.back();
    h->spare.pop_back();
    return hipSuccess;
  }
  return hipEventCreate(ev);
}

// Brackets one kernel group with timing events when profiling is on.
class Timed {
 public:
  Timed(lookme_t h, int group, hipStream_t st) : h_(h), st_(st) {
    if (!h->profiling) return;
    t_.group = group;
    if (take_event(h, &t_.start) != hipSuccess) return;
    if (take_event(h, &t_.stop) != hipSuccess) {
      h->spare.push_back(t_.start);
      return;
    }
    armed_ = hipEventRecord(t_.start, st) == hipSuccess;
    if (!armed_) {
      h->spare.push_back(t_.start);
      h->spare.push_back(t_.stop);
    }
  }
  ~Timed() {
    if (!armed_) return;
    if (hipEventRecord(t_.stop, st_) == hipSuccess) {
      h_->pending.push_back(t_);
    } else {
      h_->spare.push_back(t_.start);
      h_->spare.push_back(t_.stop);
    }
  }

 private:
  lookme_t h_;
  hipStream_t st_;
  TimedLaunch t_{};
  bool armed_ = false;
};

// Hands a pair of timing events, when profiling is on, to a launch of one
// kernel that records its own start and end in them (hipExtLaunchKernelGGL):
// the kernel's duration, without the gaps that recorded events add.
class Stamped {
 public:
  Stamped(lookme_t h, int group) : h_(h) {
    if (!h->profiling) return;
    t_.group = group;
    if (take_event(h, &ev_[0]) != hipSuccess) return;
    if (take_event(h, &ev_[1]) != hipSuccess) {
      h->spare.push_back(ev_[0]);
      return;
    }
    armed_ = true;
  }
  const hipEvent_t* events() const { return armed_ ? ev_ : nullptr; }
  // ok: the launch went in, so it records both events
  void done(bool ok) {
    if (!armed_) return;
    armed_ = false;
    if (ok) {
      t_.start = ev_[0];
      t_.stop = ev_[1];
      h_->pending.push_back(t_);
    } else {
      h_->spare.push_back(ev_[0]);
      h_->spare.push_back(ev_[1]);
    }
  }
  ~Stamped() { done(false); }

 private:
  lookme_t h_;
  TimedLaunch t_{};
  hipEvent_t ev_[2] = {nullptr, nullptr};
  bool armed_ = false;
};

#define LOOKME_TRY(expr)                    \
  do {                                      \
    lookme_status_t st_ = (expr);           \
    if (st_ != LOOKME_OK) return st_;       \
  } while (0)

// criticality norms and, when n_keep > 0, the top-n_keep select (Eq. 9)
lookme_status_t run_select(lookme_t h, const Layout& L, int32_t layers, int64_t n,
                           int64_t n_keep, const void* crit, int32_t d_c, int32_t* kept,
                           hipStream_t st, bool background = false) {
  uint32_t* key = reinterpret_cast<uint32_t*>(static_cast<char*>(h->ws) + L.crit_key);
  {
    Timed tm(h, LOOKME_GROUP_NORM, st);
    LOOKME_TRY(hip_status(lookme::launch_crit_norm(h->d.dtype, (int64_t)layers * n, crit, d_c,
                                                   key, st, background),
                          "criticality launch"));
  }
  if (n_keep == 0) return LOOKME_OK;
  Timed tm(h, LOOKME_GROUP_SELECT, st);
  return hip_status(lookme::launch_crit_select(layers, n, n_keep, key, kept, st),
                    "select launch");
}

// row gather + residual add of the kept tokens (Eq. 10, Eq. 2)
lookme_status_t run_inject(lookme_t h, int32_t layers, int64_t n, int64_t n_keep,
                           const int32_t* kept, const int32_t* scene, const int32_t* prim,
                           const float* w, void* hidden, int32_t d_h, hipStream_t st) {
  const lookme_desc_t& d = h->d;
  Timed tm(h, LOOKME_GROUP_INJECT, st);
  return hip_status(lookme::launch_inject_rows(d.dtype, layers, n, n_keep, kept, scene, prim, w,
                                               h->values, d.num_scenes, d.prims_per_scene,
                                               d.value_dim, d.top_k, hidden, d_h, st),
                    "inject launch");
}

lookme_status_t check_lookup_out(const void* q, const int32_t* scene, int32_t* prim_out,
                                 float* w_out) {
  LOOKME_TRY(check_ptr(q, "q"));
  LOOKME_TRY(check_ptr(scene, "scene"));
  LOOKME_TRY(check_ptr(prim_out, "prim_out"));
  return check_ptr(w_out, "w_out");
}

// The sparse-injection select carried by a lookup: the top n_keep by
// criticality (lookme_lookup_select), or the learned gate when w_g is set
// (lookme_lookup_gate: kept [layers, n] and count [layers]).
struct SelectArgs {
  const void* crit;
  int32_t d_c;
  int64_t n_keep;
  int32_t* kept;
  const void* w_g = nullptr;
  int32_t* count = nullptr;
};

// bucketing and Level-2 scoring, with the select of `sel` carried along:
// its norms in the bucketing launch (small batches) and its select in the
// Level-2 launch (n <= SEL_SIDE_MAX_N); what does not fit runs as its own
// kernels after the bucketing
lookme_status_t run_lookup(lookme_t h, const Layout& L, int32_t layers, int64_t n, const void* q,
                           const int32_t* scene, int32_t* prim_out, float* w_out,
                           const SelectArgs* sel, hipStream_t st) {
  const lookme_desc_t& d = h->d;
  const int64_t rows = (int64_t)layers * n;
  char* ws = static_cast<char*>(h->ws);
  lookme::BucketWs b{};
  b.chunk_hist = reinterpret_cast<int32_t*>(ws + L.chunk_hist);
  b.local_rank = reinterpret_cast<int32_t*>(ws + L.local_rank);
  b.offsets = reinterpret_cast<int32_t*>(ws + L.offsets);
  b.perm = reinterpret_cast<int32_t*>(ws + L.perm);
  b.unit_scene = reinterpret_cast<int32_t*>(ws + L.unit_scene);
  b.unit_begin = reinterpret_cast<int32_t*>(ws + L.unit_begin);
  b.unit_count = reinterpret_cast<int32_t*>(ws + L.unit_count);
  b.chunks = lookme::bucket_chunks(rows);
  b.max_units = lookme::bucket_max_units(rows, d.num_scenes);
  uint32_t* key = reinterpret_cast<uint32_t*>(ws + L.crit_key);
  const bool gate = sel != nullptr && sel->w_g != nullptr;
  const bool select = sel != nullptr && (sel->n_keep > 0 || gate);
  // the Level-2 kernels that carry a select score dot products only
  const bool cos = d.score == LOOKME_SCORE_COS;
  // the last round of streaming units may be cut in halves (kernels.h) where
  // the streaming units keep their key blocks in LDS, each half holds at
  // least k keys, no select rides in the Level-2 launch (one-chunk batches
  // with a select, below), and the batch averages at most one streaming
  // unit's rows a scene (with more, few buckets are streaming units; the
  // merge's launch, ~4 us, would then be spent on nothing: multi-scale and
  // 4-layer workloads)
  const int64_t key_bytes = (int64_t)d.key_dim * elem_size(d.dtype);
  const bool cut = rows >= 2 * lookme::SPLIT_UNITS &&
                   rows <= (int64_t)lookme::UNIT_STREAM_ROWS * d.num_scenes &&
                   lookme::score_ks(key_bytes) <= 16 && d.prims_per_scene >= 512 &&
                   d.top_k <= lookme::SPLIT_KMAX && !(select && !cos && b.chunks == 1);
  b.split_max = cut ? lookme::SPLIT_UNITS : 0;
  b.split_part = reinterpret_cast<uint64_t*>(ws + L.split_part);
  b.split_row = reinterpret_cast<int32_t*>(ws + L.split_row);
  bool normed = false;
  {
    Timed tm(h, LOOKME_GROUP_BUCKET, st);
    const int shared_rows =
        lookme::shared_unit_rows((int64_t)d.key_dim * elem_size(d.dtype), d.top_k);
    if (select && !cos)
      normed = lookme::launch_bucket_norms(d.dtype, scene, rows, d.num_scenes, shared_rows, b,
                                           sel->crit, sel->d_c, key, st,
                                           gate ? sel->w_g : nullptr, n);
    if (normed) {
      LOOKME_TRY(hip_status(hipGetLastError(), "bucketing + norms launch"));
    } else {
      LOOKME_TRY(hip_status(lookme::launch_bucket(scene, rows, d.num_scenes, shared_rows, b, st),
                            "bucketing launch"));
    }
  }
  const bool ride = select && normed && n <= lookme::SEL_SIDE_MAX_N;
  if (select && !ride) {
    // the select's (or gate's) own kernels, after the bucketing
    if (gate)
      LOOKME_TRY(hip_status(lookme::launch_gate(d.dtype, layers, n, sel->crit, n, sel->d_c,
                                                nullptr, sel->w_g,
                                                reinterpret_cast<float*>(key), sel->kept,
                                                sel->count, st),
                            "gate launch"));
    else
      LOOKME_TRY(run_select(h, L, layers, n, sel->n_keep, sel->crit, sel->d_c, sel->kept, st));
  }
  lookme::SideSelect side{layers, n, select ? sel->n_keep : 0, key,
                          select ? sel->kept : nullptr};
  if (gate) side.count = sel->count;
  Stamped tm(h, LOOKME_GROUP_SCORE);
  const hipError_t e = lookme::launch_lookup(d.dtype, q, h->prim_keys, b, d.key_dim,
                                             d.prims_per_scene, d.top_k, prim_out, w_out, st,
                                             ride ? &side : nullptr, cos, tm.events());
  tm.done(e == hipSuccess);
  return hip_status(e, "lookup launch");
}

}  // namespace

extern "C" {

const char* lookme_last_error(void) { return g_err.c_str(); }

lookme_status_t lookme_create(const lookme_desc_t* desc, const void* scene_keys,
                              const void* prim_keys, const void* values, const float* scene_bias,
                              lookme_t* out) {
  if (out == nullptr) return fail(LOOKME_ERR_INVALID, "out is NULL");
  *out = nullptr;
  if (desc == nullptr) return fail(LOOKME_ERR_INVALID, "desc is NULL");
  const lookme_desc_t d = *desc;
  if (d.dtype != LOOKME_F32 && d.dtype != LOOKME_BF16)
    return fail(LOOKME_ERR_INVALID, "unknown dtype %d", d.dtype);
  if (d.score != LOOKME_SCORE_DOT && d.score != LOOKME_SCORE_COS)
    return fail(LOOKME_ERR_INVALID, "unknown score %d", d.score);
  if (d.num_scenes < 1 || d.prims_per_scene < 1 || d.key_dim < 1 || d.value_dim < 1)
    return fail(LOOKME_ERR_INVALID, "table sizes must be positive");
  if (d.top_k < 1 || d.top_k > d.prims_per_scene)
    return fail(LOOKME_ERR_INVALID, "top_k %d outside [1, prims_per_scene=%d]", d.top_k,
                d.prims_per_scene);
  if (d.top_k > LOOKME_KMAX)
    return fail(LOOKME_ERR_UNSUPPORTED, "top_k %d above LOOKME_KMAX=%d", d.top_k, LOOKME_KMAX);
  const int es = elem_size(d.dtype);
  const int64_t kb = (int64_t)d.key_dim * es;
  if (kb % 64 != 0 || kb > 2048)
    return fail(LOOKME_ERR_UNSUPPORTED,
                "key_dim * elem_size = %lld bytes; must be a multiple of 64 and <= 2048",
                (long long)kb);
  if (((int64_t)d.value_dim * es) % 16 != 0)
    return fail(LOOKME_ERR_UNSUPPORTED, "value_dim * elem_size must be a multiple of 16 bytes");
  if (d.num_scenes > MAX_SCENES)
    return fail(LOOKME_ERR_UNSUPPORTED, "num_scenes %d above %d", d.num_scenes, MAX_SCENES);
  if ((int64_t)d.num_scenes * d.prims_per_scene > (int64_t)INT32_MAX)
    return fail(LOOKME_ERR_UNSUPPORTED, "num_scenes * prims_per_scene exceeds 2^31 - 1 rows");
  LOOKME_TRY(check_ptr(scene_keys, "scene_keys"));
  LOOKME_TRY(check_ptr(prim_keys, "prim_keys"));
  LOOKME_TRY(check_ptr(values, "values"));
  if (scene_bias != nullptr && (reinterpret_cast<uintptr_t>(scene_bias) & 3u))
    return fail(LOOKME_ERR_INVALID, "scene_bias is not 4-byte aligned");
  lookme_s* h = new (std::nothrow) lookme_s{};
  if (h == nullptr) return fail(LOOKME_ERR_INVALID, "out of host memory");
  h->d = d;
  h->scene_keys = scene_keys;
  h->prim_keys = prim_keys;
  h->values = values;
  h->bias = scene_bias;
  *out = h;
  return LOOKME_OK;
}

lookme_status_t lookme_destroy(lookme_t h) {
  if (h == nullptr) return LOOKME_OK;
  for (auto& t : h->pending) {
    (void)hipEventSynchronize(t.stop);
    (void)hipEventDestroy(t.start);
    (void)hipEventDestroy(t.stop);
  }
  for (auto e : h->spare) (void)hipEventDestroy(e);
  delete h;
  return LOOKME_OK;
}

lookme_status_t lookme_profile_enable(lookme_t h, int32_t enabled) {
  LOOKME_TRY(check_handle(h));
  h->profiling = enabled != 0;
  return LOOKME_OK;
}

lookme_status_t lookme_profile_read(lookme_t h, int32_t group, int64_t* count, double* total_ms,
                                    int32_t reset) {
  LOOKME_TRY(check_handle(h));
  if (group < 0 || group >= LOOKME_GROUP_COUNT)
    return fail(LOOKME_ERR_INVALID, "unknown kernel group %d", group);
  // an entry leaves `pending` exactly when it is counted and its events go
  // back to the pool: a read that fails part way leaves the unread entries
  // pending and no entry both counted and still referenced
  size_t done = 0;
  lookme_status_t st = LOOKME_OK;
  for (; done < h->pending.size(); ++done) {
    const TimedLaunch& t = h->pending[done];
    float ms = 0.f;
    st = hip_status(hipEventSynchronize(t.stop), "hipEventSynchronize");
    if (st == LOOKME_OK)
      st = hip_status(hipEventElapsedTime(&ms, t.start, t.stop), "hipEventElapsedTime");
    if (st != LOOKME_OK) break;
    h->prof_count[t.group] += 1;
    h->prof_ms[t.group] += ms;
    h->spare.push_back(t.start);
    h->spare.push_back(t.stop);
  }
  h->pending.erase(h->pending.begin(), h->pending.begin() + done);
  if (st != LOOKME_OK) return st;
  if (count) *count = h->prof_count[group];
  if (total_ms) *total_ms = h->prof_ms[group];
  if (reset) {
    for (int g = 0; g < LOOKME_GROUP_COUNT; ++g) {
      h->prof_count[g] = 0;
      h->prof_ms[g] = 0.0;
    }
  }
  return LOOKME_OK;
}

lookme_status_t lookme_workspace_size(lookme_t h, int32_t layers, int64_t n_tokens,
                                      size_t* bytes) {
  LOOKME_TRY(check_handle(h));
  if (bytes == nullptr) return fail(LOOKME_ERR_INVALID, "bytes is NULL");
  LOOKME_TRY(check_layers_n(layers, n_tokens));
  *bytes = layout(h->d, layers, n_tokens, h->rel.hidden, h->fus.d_ff, h->ms_scales).total;
  return LOOKME_OK;
}

lookme_status_t lookme_set_workspace(lookme_t h, void* dev_ptr, size_t bytes) {
  LOOKME_TRY(check_handle(h));
  if (dev_ptr == nullptr) return fail(LOOKME_ERR_INVALID, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(dev_ptr) & 255u)
    return fail(LOOKME_ERR_INVALID, "workspace is not 256-byte aligned");
  if (bytes < ZEROED_BYTES)
    return fail(LOOKME_ERR_WORKSPACE, "workspace below %zu bytes", ZEROED_BYTES);
  LOOKME_TRY(hip_status(hipMemset(dev_ptr, 0, ZEROED_BYTES), "hipMemset(workspace counters)"));
  h->ws = dev_ptr;
  h->ws_bytes = bytes;
  h->rel_tab_ready = false;
  return LOOKME_OK;
}

lookme_status_t lookme_route(lookme_t h, int32_t layers, int64_t n, int32_t d_in, const void* x,
                             const void* w_proj, void* q_out, int32_t* scene_out, void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  const lookme_desc_t& d = h->d;
  const int es = elem_size(d.dtype);
  if (d_in < 1) return fail(LOOKME_ERR_INVALID, "d_in must be positive");
  if (((int64_t)d_in * es) % 16 != 0)
    return fail(LOOKME_ERR_UNSUPPORTED, "d_in * elem_size must be a multiple of 16 bytes");
  if (w_proj == nullptr && d_in != d.key_dim)
    return fail(LOOKME_ERR_INVALID, "w_proj is NULL but d_in (%d) != key_dim (%d)", d_in,
                d.key_dim);
  if (w_proj == nullptr && layers > 1 && q_out == x)
    return fail(LOOKME_ERR_INVALID, "q_out may alias x only for one layer");
  if ((int64_t)layers * d.key_dim > (int64_t)INT32_MAX / 2)
    return fail(LOOKME_ERR_UNSUPPORTED, "layers * key_dim too large");
  if (n == 0) return LOOKME_OK;
  LOOKME_TRY(check_ptr(x, "x"));
  if (w_proj) LOOKME_TRY(check_ptr(w_proj, "w_proj"));
  LOOKME_TRY(check_ptr(q_out, "q_out"));
  LOOKME_TRY(check_ptr(scene_out, "scene_out"));
  Layout L;
  LOOKME_TRY(check_workspace(h, layers, n, &L));
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t rows = (int64_t)layers * n;
  char* ws = static_cast<char*>(h->ws);
  if (w_proj) {
    Timed tm(h, LOOKME_GROUP_PROJECT, st);
    LOOKME_TRY(hip_status(
        lookme::launch_project(d.dtype, x, w_proj, q_out, n, d_in, d.key_dim, layers, st),
        "projection launch"));
  } else {
    // the tokens are the queries of every layer
    const size_t bytes = (size_t)n * d.key_dim * es;
    for (int32_t l = 0; l < layers; ++l) {
      char* dst = static_cast<char*>(q_out) + (size_t)l * bytes;
      if (dst == x) continue;
      LOOKME_TRY(hip_status(hipMemcpyAsync(dst, x, bytes, hipMemcpyDeviceToDevice, st),
                            "copy of queries"));
    }
  }
  Timed tm(h, LOOKME_GROUP_ROUTE, st);
  return hip_status(
      lookme::launch_route(d.dtype, q_out, h->scene_keys, h->bias, scene_out, rows, d.key_dim,
                           d.num_scenes, reinterpret_cast<uint64_t*>(ws + L.route_part),
                           reinterpret_cast<int32_t*>(ws + L.route_count), st,
                           d.score == LOOKME_SCORE_COS),
      "routing launch");
}

lookme_status_t lookme_lookup(lookme_t h, int32_t layers, int64_t n, const void* q,
                              const int32_t* scene, int32_t* prim_out, float* w_out,
                              void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  if (n == 0) return LOOKME_OK;
  LOOKME_TRY(check_lookup_out(q, scene, prim_out, w_out));
  Layout L;
  LOOKME_TRY(check_workspace(h, layers, n, &L));
  return run_lookup(h, L, layers, n, q, scene, prim_out, w_out, nullptr,
                    static_cast<hipStream_t>(stream));
}

lookme_status_t lookme_lookup_select(lookme_t h, int32_t layers, int64_t n, const void* q,
                                     const int32_t* scene, int32_t* prim_out, float* w_out,
                                     int64_t n_keep, const void* crit, int32_t d_c,
                                     int32_t* kept_out, void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  LOOKME_TRY(check_keep(n, n_keep));
  LOOKME_TRY(check_crit_dim(h->d, d_c));
  if (n == 0) return LOOKME_OK;
  LOOKME_TRY(check_lookup_out(q, scene, prim_out, w_out));
  if (n_keep > 0) {
    LOOKME_TRY(check_ptr(crit, "crit"));
    LOOKME_TRY(check_ptr(kept_out, "kept_out"));
  }
  Layout L;
  LOOKME_TRY(check_workspace(h, layers, n, &L));
  const SelectArgs sel{crit, d_c, n_keep, kept_out};
  return run_lookup(h, L, layers, n, q, scene, prim_out, w_out, n_keep > 0 ? &sel : nullptr,
                    static_cast<hipStream_t>(stream));
}

lookme_status_t lookme_lookup_gate(lookme_t h, int32_t layers, int64_t n, const void* q,
                                   const int32_t* scene, int32_t* prim_out, float* w_out,
                                   const void* delta, int32_t d_c, const void* w_g,
                                   int32_t* kept_out, int32_t* count_out, void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  LOOKME_TRY(check_crit_dim(h->d, d_c));
  if (n == 0) return LOOKME_OK;
  LOOKME_TRY(check_lookup_out(q, scene, prim_out, w_out));
  LOOKME_TRY(check_ptr(delta, "delta"));
  LOOKME_TRY(check_ptr(w_g, "w_g"));
  LOOKME_TRY(check_ptr(kept_out, "kept_out"));
  LOOKME_TRY(check_ptr(count_out, "count_out"));
  Layout L;
  LOOKME_TRY(check_workspace(h, layers, n, &L));
  SelectArgs sel{delta, d_c, 0, kept_out};
  sel.w_g = w_g;
  sel.count = count_out;
  return run_lookup(h, L, layers, n, q, scene, prim_out, w_out, &sel,
                    static_cast<hipStream_t>(stream));
}

lookme_status_t lookme_inject(lookme_t h, int32_t layers, int64_t n, int64_t n_keep,
                              const void* crit, int32_t d_c, const int32_t* scene,
                              const int32_t* prim, const float* w, void* hidden, int32_t d_h,
                              int32_t* kept_out, void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  LOOKME_TRY(check_keep(n, n_keep));
  LOOKME_TRY(check_crit_dim(h->d, d_c));
  LOOKME_TRY(check_hidden_dim(h->d, d_h));
  if (n == 0) return LOOKME_OK;
  LOOKME_TRY(check_ptr(crit, "crit"));
  LOOKME_TRY(check_ptr(scene, "scene"));
  LOOKME_TRY(check_ptr(prim, "prim"));
  LOOKME_TRY(check_ptr(w, "w"));
  LOOKME_TRY(check_ptr(hidden, "hidden"));
  if (kept_out) LOOKME_TRY(check_ptr(kept_out, "kept_out"));
  Layout L;
  LOOKME_TRY(check_workspace(h, layers, n, &L));
  int32_t* kept = kept_out ? kept_out : reinterpret_cast<int32_t*>(static_cast<char*>(h->ws) + L.kept);
  hipStream_t st = static_cast<hipStream_t>(stream);
  LOOKME_TRY(run_select(h, L, layers, n, n_keep, crit, d_c, kept, st));
  if (n_keep == 0) return LOOKME_OK;
  return run_inject(h, layers, n, n_keep, kept, scene, prim, w, hidden, d_h, st);
}

lookme_status_t lookme_inject_noalloc(lookme_t h, int32_t layers, int64_t n, int64_t n_keep,
                                      const void* crit, int32_t d_c, const int32_t* scene,
                                      const int32_t* prim, const float* w, void* hidden,
                                      int32_t d_h, int32_t* kept_out, void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  LOOKME_TRY(check_keep(n, n_keep));
  LOOKME_TRY(check_crit_dim(h->d, d_c));
  LOOKME_TRY(check_hidden_dim(h->d, d_h));
  if ((int64_t)layers * n > LOOKME_NOALLOC_MAX_ROWS)
    return fail(LOOKME_ERR_UNSUPPORTED, "layers * n = %lld rows exceeds the %d of the scratch",
                (long long)((int64_t)layers * n), LOOKME_NOALLOC_MAX_ROWS);
  if (n == 0) return LOOKME_OK;
  LOOKME_TRY(check_ptr(crit, "crit"));
  LOOKME_TRY(check_ptr(scene, "scene"));
  LOOKME_TRY(check_ptr(prim, "prim"));
  LOOKME_TRY(check_ptr(w, "w"));
  LOOKME_TRY(check_ptr(hidden, "hidden"));
  if (kept_out) LOOKME_TRY(check_ptr(kept_out, "kept_out"));
  void* scratch = nullptr;
  LOOKME_TRY(hip_status(lookme::noalloc_scratch(&scratch), "scratch address"));
  uint32_t* key = static_cast<uint32_t*>(scratch);
  int32_t* kept = kept_out ? kept_out
                           : reinterpret_cast<int32_t*>(static_cast<char*>(scratch) +
                                                        lookme::NOALLOC_KEYS_BYTES);
  const lookme_desc_t& d = h->d;
  hipStream_t st = static_cast<hipStream_t>(stream);
  // the kernels of lookme_inject (run_select, run_inject) without the timing
  // hooks, whose events would be created on first use
  LOOKME_TRY(hip_status(lookme::launch_crit_norm(d.dtype, (int64_t)layers * n, crit, d_c, key, st),
                        "criticality launch"));
  if (n_keep == 0) return LOOKME_OK;
  LOOKME_TRY(hip_status(lookme::launch_crit_select(layers, n, n_keep, key, kept, st),
                        "select launch"));
  return hip_status(lookme::launch_inject_rows(d.dtype, layers, n, n_keep, kept, scene, prim, w,
                                               h->values, d.num_scenes, d.prims_per_scene,
                                               d.value_dim, d.top_k, hidden, d_h, st),
                    "inject launch");
}

lookme_status_t lookme_select(lookme_t h, int32_t layers, int64_t n, int64_t n_keep,
                              const void* crit, int32_t d_c, int32_t* kept_out, void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  LOOKME_TRY(check_keep(n, n_keep));
  LOOKME_TRY(check_crit_dim(h->d, d_c));
  if (n == 0 || n_keep == 0) return LOOKME_OK;
  LOOKME_TRY(check_ptr(crit, "crit"));
  LOOKME_TRY(check_ptr(kept_out, "kept_out"));
  Layout L;
  LOOKME_TRY(check_workspace(h, layers, n, &L));
  // the norms in their background form: lookme_select is the call that runs
  // beside lookme_route / lookme_lookup on a second stream
  return run_select(h, L, layers, n, n_keep, crit, d_c, kept_out, static_cast<hipStream_t>(stream),
                    true);
}

lookme_status_t lookme_inject_kept(lookme_t h, int32_t layers, int64_t n, int64_t n_keep,
                                   const int32_t* kept, const int32_t* scene, const int32_t* prim,
                                   const float* w, void* hidden, int32_t d_h, void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  LOOKME_TRY(check_keep(n, n_keep));
  LOOKME_TRY(check_hidden_dim(h->d, d_h));
  if (n == 0 || n_keep == 0) return LOOKME_OK;
  LOOKME_TRY(check_ptr(kept, "kept"));
  LOOKME_TRY(check_ptr(scene, "scene"));
  LOOKME_TRY(check_ptr(prim, "prim"));
  LOOKME_TRY(check_ptr(w, "w"));
  LOOKME_TRY(check_ptr(hidden, "hidden"));
  return run_inject(h, layers, n, n_keep, kept, scene, prim, w, hidden, d_h,
                    static_cast<hipStream_t>(stream));
}

lookme_status_t lookme_set_relevance(lookme_t h, int32_t hidden, const void* w1,
                                     const float* b1, const void* w2, const float* b2) {
  LOOKME_TRY(check_handle(h));
  const int es = elem_size(h->d.dtype);
  if (hidden < 1) return fail(LOOKME_ERR_INVALID, "hidden must be positive (got %d)", hidden);
  if (((int64_t)hidden * es) % 128 != 0)
    return fail(LOOKME_ERR_UNSUPPORTED, "hidden * elem_size must be a multiple of 128 bytes");
  if (((int64_t)h->d.key_dim * es) % 128 != 0)
    return fail(LOOKME_ERR_UNSUPPORTED, "key_dim * elem_size must be a multiple of 128 bytes");
  LOOKME_TRY(check_ptr(w1, "w1"));
  LOOKME_TRY(check_ptr(w2, "w2"));
  if ((b1 != nullptr && (reinterpret_cast<uintptr_t>(b1) & 3u)) ||
      (b2 != nullptr && (reinterpret_cast<uintptr_t>(b2) & 3u)))
    return fail(LOOKME_ERR_INVALID, "b1 and b2 must be 4-byte aligned");
  h->rel = lookme::RelevanceMlp{hidden, w1, b1, w2, b2};
  h->rel_tab_ready = false;
  return LOOKME_OK;
}

lookme_status_t lookme_lookup_relevance(lookme_t h, int32_t layers, int64_t n, const void* q,
                                        const int32_t* scene, void* act_out, int32_t* prim_out,
                                        float* w_out, void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  if (h->rel.hidden < 1)
    return fail(LOOKME_ERR_INVALID, "no relevance MLP registered (lookme_set_relevance)");
  if (n == 0) return LOOKME_OK;
  LOOKME_TRY(check_ptr(q, "q"));
  LOOKME_TRY(check_ptr(scene, "scene"));
  LOOKME_TRY(check_ptr(act_out, "act_out"));
  LOOKME_TRY(check_ptr(prim_out, "prim_out"));
  LOOKME_TRY(check_ptr(w_out, "w_out"));
  Layout L;
  LOOKME_TRY(check_workspace(h, layers, n, &L));
  const lookme_desc_t& d = h->d;
  hipStream_t st = static_cast<hipStream_t>(stream);
  Timed tm(h, LOOKME_GROUP_SCORE, st);
  float* tab = reinterpret_cast<float*>(static_cast<char*>(h->ws) + L.rel_tab);
  if (!h->rel_tab_ready) {
    // the per-scene half of the first layer, once per MLP and workspace
    LOOKME_TRY(hip_status(lookme::launch_relevance_table(d.dtype, h->scene_keys, h->rel,
                                                         d.num_scenes, d.key_dim, tab, st),
                          "relevance table launch"));
    h->rel_tab_ready = true;
  }
  return hip_status(
      lookme::launch_relevance(d.dtype, q, scene, tab, h->prim_keys, h->rel,
                               (int64_t)layers * n, d.key_dim, d.num_scenes, d.prims_per_scene,
                               d.top_k, act_out, prim_out, w_out,
                               reinterpret_cast<float*>(static_cast<char*>(h->ws) + L.rel_logits),
                               st),
      "relevance lookup launch");
}

lookme_status_t lookme_set_fusion(lookme_t h, int32_t layers, int32_t d_ff, int32_t d_h,
                                  const void* w_gate, const void* w_up, const void* w_down) {
  LOOKME_TRY(check_handle(h));
  const int es = elem_size(h->d.dtype);
  if (layers < 1 || d_ff < 1 || d_h < 1)
    return fail(LOOKME_ERR_INVALID, "layers, d_ff and d_h must be positive");
  if (((int64_t)d_ff * es) % 128 != 0 || ((int64_t)h->d.value_dim * es) % 128 != 0)
    return fail(LOOKME_ERR_UNSUPPORTED,
                "d_ff * elem_size and value_dim * elem_size must be multiples of 128 bytes");
  LOOKME_TRY(check_ptr(w_gate, "w_gate"));
  LOOKME_TRY(check_ptr(w_up, "w_up"));
  LOOKME_TRY(check_ptr(w_down, "w_down"));
  h->fus = lookme::FusionFfn{layers, d_ff, d_h, w_gate, w_up, w_down};
  return LOOKME_OK;
}

// Checks shared by the fused injections: a fusion of at least `layers`
// layers writing rows of width d_h.
lookme_status_t check_fusion(lookme_t h, int32_t layers, int32_t d_h) {
  if (h->fus.d_ff < 1)
    return fail(LOOKME_ERR_INVALID, "no fusion registered (lookme_set_fusion)");
  if (layers > h->fus.layers)
    return fail(LOOKME_ERR_INVALID, "%d layers, the fusion has %d", layers, h->fus.layers);
  if (d_h != h->fus.d_h)
    return fail(LOOKME_ERR_INVALID, "d_h %d, the fusion writes %d", d_h, h->fus.d_h);
  return LOOKME_OK;
}

lookme_status_t check_lookup_ptrs(const int32_t* kept, const int32_t* scene, const int32_t* prim,
                                  const float* w, void* hidden) {
  LOOKME_TRY(check_ptr(kept, "kept"));
  LOOKME_TRY(check_ptr(scene, "scene"));
  LOOKME_TRY(check_ptr(prim, "prim"));
  LOOKME_TRY(check_ptr(w, "w"));
  return check_ptr(hidden, "hidden");
}

lookme_status_t lookme_inject_fused(lookme_t h, int32_t layers, int64_t n, int64_t n_keep,
                                    const int32_t* kept, const int32_t* scene,
                                    const int32_t* prim, const float* w, void* hidden,
                                    int32_t d_h, void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  LOOKME_TRY(check_keep(n, n_keep));
  LOOKME_TRY(check_fusion(h, layers, d_h));
  if (n == 0 || n_keep == 0) return LOOKME_OK;
  LOOKME_TRY(check_lookup_ptrs(kept, scene, prim, w, hidden));
  Layout L;
  LOOKME_TRY(check_workspace(h, layers, n, &L));
  const lookme_desc_t& d = h->d;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(h->ws);
  Timed tm(h, LOOKME_GROUP_INJECT, st);
  LOOKME_TRY(hip_status(lookme::launch_gather_rows(d.dtype, layers, n, n_keep, kept, scene, prim,
                                                   w, h->values, d.num_scenes, d.prims_per_scene,
                                                   d.value_dim, d.top_k, ws + L.fus_r, st,
                                                   n_keep, 0),
                        "fusion gather launch"));
  return hip_status(lookme::launch_fusion(d.dtype, h->fus, layers, n, n_keep, kept, n_keep,
                                          d.value_dim, ws + L.fus_r, ws + L.fus_u, hidden, st),
                    "fusion launch");
}

lookme_status_t lookme_set_propagation(lookme_t h, int32_t steps, const void* w_p_t) {
  LOOKME_TRY(check_handle(h));
  if (steps < 1) return fail(LOOKME_ERR_INVALID, "steps must be positive");
  if (((int64_t)h->d.value_dim * elem_size(h->d.dtype)) % 128 != 0)
    return fail(LOOKME_ERR_UNSUPPORTED, "value_dim * elem_size must be a multiple of 128 bytes");
  LOOKME_TRY(check_ptr(w_p_t, "w_p_t"));
  h->prop_steps = steps;
  h->prop_w = w_p_t;
  return LOOKME_OK;
}

lookme_status_t lookme_inject_propagated(lookme_t h, int32_t steps, int64_t n, int64_t n_keep,
                                         const int32_t* kept, const int32_t* scene,
                                         const int32_t* prim, const float* w, void* hidden,
                                         int32_t d_h, void* stream) {
  LOOKME_TRY(check_handle(h));
  if (steps < 0) return fail(LOOKME_ERR_INVALID, "steps must be >= 0 (got %d)", steps);
  if (steps >= INT32_MAX) return fail(LOOKME_ERR_INVALID, "steps too large");
  const int32_t layers = steps + 1;
  LOOKME_TRY(check_layers_n(layers, n));
  LOOKME_TRY(check_keep(n, n_keep));
  LOOKME_TRY(check_fusion(h, layers, d_h));
  if (steps > h->prop_steps)
    return fail(LOOKME_ERR_INVALID, "%d propagation steps, %d registered (lookme_set_propagation)",
                steps, h->prop_steps);
  if (n == 0 || n_keep == 0) return LOOKME_OK;
  LOOKME_TRY(check_lookup_ptrs(kept, scene, prim, w, hidden));
  Layout L;
  LOOKME_TRY(check_workspace(h, layers, n, &L));
  const lookme_desc_t& d = h->d;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(h->ws);
  Timed tm(h, LOOKME_GROUP_INJECT, st);
  LOOKME_TRY(hip_status(lookme::launch_gather_rows(d.dtype, 1, n, n_keep, kept, scene, prim, w,
                                                   h->values, d.num_scenes, d.prims_per_scene,
                                                   d.value_dim, d.top_k, ws + L.fus_r, st,
                                                   n_keep, 0),
                        "fusion gather launch"));
  LOOKME_TRY(hip_status(
      lookme::launch_propagate(d.dtype, h->prop_w, steps, n_keep, d.value_dim, ws + L.fus_r, st),
      "propagation launch"));
  return hip_status(lookme::launch_fusion(d.dtype, h->fus, layers, n, n_keep, kept, 0,
                                          d.value_dim, ws + L.fus_r, ws + L.fus_u, hidden, st),
                    "fusion launch");
}

lookme_status_t lookme_gate(lookme_t h, int32_t layers, int64_t n, const void* delta,
                            int64_t delta_rows, int32_t d_c, const int32_t* pos, const void* w_g,
                            int32_t* kept_out, int32_t* count_out, void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  LOOKME_TRY(check_crit_dim(h->d, d_c));
  LOOKME_TRY(check_ptr(count_out, "count_out"));
  if (n > 0) {
    if (delta_rows < 1)
      return fail(LOOKME_ERR_INVALID, "delta_rows must be positive (got %lld)",
                  (long long)delta_rows);
    if (pos == nullptr && delta_rows < n)
      return fail(LOOKME_ERR_INVALID, "delta_rows %lld < n %lld with no pos list",
                  (long long)delta_rows, (long long)n);
    if ((int64_t)layers * delta_rows > (int64_t)INT32_MAX)
      return fail(LOOKME_ERR_UNSUPPORTED, "layers * delta_rows exceeds 2^31 - 1 rows");
    LOOKME_TRY(check_ptr(delta, "delta"));
    LOOKME_TRY(check_ptr(w_g, "w_g"));
    LOOKME_TRY(check_ptr(kept_out, "kept_out"));
    if (pos != nullptr) LOOKME_TRY(check_ptr(pos, "pos"));
  }
  float* z = nullptr;
  if (n > 0) {
    Layout L;
    LOOKME_TRY(check_workspace(h, layers, n, &L));
    z = reinterpret_cast<float*>(static_cast<char*>(h->ws) + L.crit_key);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  Timed tm(h, LOOKME_GROUP_NORM, st);
  return hip_status(lookme::launch_gate(h->d.dtype, layers, n, delta, delta_rows, d_c, pos, w_g,
                                        z, kept_out, count_out, st),
                    "gate launch");
}

lookme_status_t lookme_inject_gated(lookme_t h, int32_t layers, int64_t n, const int32_t* kept,
                                    const int32_t* count, const int32_t* scene,
                                    const int32_t* prim, const float* w, void* hidden,
                                    int32_t d_h, void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  LOOKME_TRY(check_hidden_dim(h->d, d_h));
  if (n == 0) return LOOKME_OK;
  LOOKME_TRY(check_ptr(count, "count"));
  LOOKME_TRY(check_lookup_ptrs(kept, scene, prim, w, hidden));
  const lookme_desc_t& d = h->d;
  hipStream_t st = static_cast<hipStream_t>(stream);
  Timed tm(h, LOOKME_GROUP_INJECT, st);
  return hip_status(lookme::launch_inject_rows(d.dtype, layers, n, n, kept, scene, prim, w,
                                               h->values, d.num_scenes, d.prims_per_scene,
                                               d.value_dim, d.top_k, hidden, d_h, st, count),
                    "gated inject launch");
}

lookme_status_t lookme_inject_fused_gated(lookme_t h, int32_t layers, int64_t n,
                                          const int32_t* kept, const int32_t* count,
                                          const int32_t* scene, const int32_t* prim,
                                          const float* w, void* hidden, int32_t d_h,
                                          void* stream) {
  LOOKME_TRY(check_handle(h));
  LOOKME_TRY(check_layers_n(layers, n));
  LOOKME_TRY(check_fusion(h, layers, d_h));
  if (n == 0) return LOOKME_OK;
  LOOKME_TRY(check_ptr(count, "count"));
  LOOKME_TRY(check_lookup_ptrs(kept, scene, prim, w, hidden));
  Layout L;
  LOOKME_TRY(check_workspace(h, layers, n, &L));
  const lookme_desc_t& d = h->d;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(h->ws);
  Timed tm(h, LOOKME_GROUP_INJECT, st);
  LOOKME_TRY(hip_status(lookme::launch_gather_rows(d.dtype, layers, n, n, kept, scene, prim, w,
                                                   h->values, d.num_scenes, d.prims_per_scene,
                                                   d.value_dim, d.top_k, ws + L.fus_r, st, n, 0,
                                                   count),
                        "fusion gather launch"));
  return hip_status(lookme::launch_fusion(d.dtype, h->fus, layers, n, n, kept, n, d.value_dim,
                                          ws + L.fus_r, ws + L.fus_u, hidden, st, count),
                    "fusion launch");
}

lookme_status_t lookme_inject_propagated_gated(lookme_t h, int32_t steps, int64_t n,
                                               const int32_t* kept, const int32_t* count,
                                               const int32_t* scene, const int32_t* prim,
                                               const float* w, void* hidden, int32_t d_h,
                                               void* stream) {
  LOOKME_TRY(check_handle(h));
  if (steps < 0 || steps >= INT32_MAX)
    return fail(LOOKME_ERR_INVALID, "steps must be in [0, 2^31 - 2] (got %d)", steps);
  const int32_t layers = steps + 1;
  LOOKME_TRY(check_layers_n(layers, n));
  LOOKME_TRY(check_fusion(h, layers, d_h));
  if (steps > h->prop_steps)
    return fail(LOOKME_ERR_INVALID, "%d propagation steps, %d registered (lookme_set_propagation)",
                steps, h->prop_steps);
  if (n == 0) return LOOKME_OK;
  LOOKME_TRY(check_ptr(count, "count"));
  LOOKME_TRY(check_lookup_ptrs(kept, scene, prim, w, hidden));
  Layout L;
  LOOKME_TRY(check_workspace(h, layers, n, &L));
  const lookme_desc_t& d = h->d;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(h->ws);
  Timed tm(h, LOOKME_GROUP_INJECT, st);
  LOOKME_TRY(hip_status(lookme::launch_gather_rows(d.dtype, 1, n, n, kept, scene, prim, w,
                                                   h->values, d.num_scenes, d.prims_per_scene,
                                                   d.value_dim, d.top_k, ws + L.fus_r, st, n, 0,
                                                   count),
                        "fusion gather launch"));
  LOOKME_TRY(hip_status(lookme::launch_propagate(d.dtype, h->prop_w, steps, n, d.value_dim,
                                                 ws + L.fus_r, st, count),
                        "propagation launch"));
  return hip_status(lookme::launch_fusion(d.dtype, h->fus, layers, n, n, kept, 0, d.value_dim,
                                          ws + L.fus_r, ws + L.fus_u, hidden, st, count),
                    "fusion launch");
}

lookme_status_t lookme_index_errors(void* stream, uint64_t* count) {
  if (count == nullptr) return fail(LOOKME_ERR_INVALID, "count is NULL");
  return hip_status(lookme::take_index_errors(static_cast<hipStream_t>(stream), count),
                    "reading the index-error count");
}

lookme_status_t lookme_scene_keys(const lookme_desc_t* desc, const void* prim_keys,
                                  void* scene_keys, void* stream) {
  if (desc == nullptr) return fail(LOOKME_ERR_INVALID, "desc is NULL");
  const lookme_desc_t d = *desc;
  if (d.dtype != LOOKME_F32 && d.dtype != LOOKME_BF16)
    return fail(LOOKME_ERR_INVALID, "unknown dtype %d", d.dtype);
  if (d.num_scenes < 1 || d.prims_per_scene < 1 || d.key_dim < 1)
    return fail(LOOKME_ERR_INVALID, "num_scenes, prims_per_scene and key_dim must be positive");
  if (((int64_t)d.key_dim * elem_size(d.dtype)) % 16 != 0)
    return fail(LOOKME_ERR_UNSUPPORTED, "key_dim * elem_size must be a multiple of 16 bytes");
  if ((int64_t)d.num_scenes * d.prims_per_scene > (int64_t)INT32_MAX)
    return fail(LOOKME_ERR_UNSUPPORTED, "num_scenes * prims_per_scene exceeds 2^31 - 1 rows");
  LOOKME_TRY(check_ptr(prim_keys, "prim_keys"));
  LOOKME_TRY(check_ptr(scene_keys, "scene_keys"));
  return hip_status(lookme::launch_scene_keys(d.dtype, prim_keys, d.num_scenes,
                                              d.prims_per_scene, d.key_dim, scene_keys,
                                              static_cast<hipStream_t>(stream)),
                    "scene keys launch");
}

lookme_status_t lookme_inject_text(int32_t dtype, const void* table, int64_t vocab, int32_t d_t,
                                   int64_t n_text, const int32_t* pos, const int32_t* ids,
                                   const int32_t* kept, const int32_t* count, void* hidden,
                                   int64_t n, int32_t d_h, void* stream) {
  if (dtype != LOOKME_F32 && dtype != LOOKME_BF16)
    return fail(LOOKME_ERR_INVALID, "unknown dtype %d", dtype);
  const int es = elem_size(dtype);
  if (vocab < 1 || d_t < 1 || d_h < 1)
    return fail(LOOKME_ERR_INVALID, "vocab, d_t and d_h must be positive");
  if (d_t > d_h) return fail(LOOKME_ERR_INVALID, "d_t %d exceeds d_h %d", d_t, d_h);
  if (((int64_t)d_t * es) % 16 != 0 || ((int64_t)d_h * es) % 16 != 0)
    return fail(LOOKME_ERR_UNSUPPORTED, "d_t and d_h times elem_size must be multiples of 16");
  if (vocab > (int64_t)INT32_MAX) return fail(LOOKME_ERR_UNSUPPORTED, "vocab exceeds 2^31 - 1");
  if (n_text < 0 || n < 0) return fail(LOOKME_ERR_INVALID, "n_text and n must be >= 0");
  if (n_text > (int64_t)INT32_MAX / 2)
    return fail(LOOKME_ERR_UNSUPPORTED, "n_text exceeds 2^30");
  if (n_text == 0) return LOOKME_OK;
  if (n < 1) return fail(LOOKME_ERR_INVALID, "text entries given for n = 0 positions");
  LOOKME_TRY(check_ptr(table, "table"));
  LOOKME_TRY(check_ptr(pos, "pos"));
  LOOKME_TRY(check_ptr(ids, "ids"));
  LOOKME_TRY(check_ptr(hidden, "hidden"));
  if (kept != nullptr) LOOKME_TRY(check_ptr(kept, "kept"));
  if (count != nullptr) LOOKME_TRY(check_ptr(count, "count"));
  return hip_status(lookme::launch_text_inject(dtype, n_text, kept, count, pos, ids, table, vocab,
                                               d_t, hidden, n, d_h,
                                               static_cast<hipStream_t>(stream)),
                    "text inject launch");
}

lookme_status_t lookme_set_multiscale(lookme_t h, int32_t scales, int32_t d_h,
                                      const void* w_he_t) {
  LOOKME_TRY(check_handle(h));
  const lookme_desc_t& d = h->d;
  if (scales < 1 || scales > lookme::MS_MAX_SCALES)
    return fail(LOOKME_ERR_UNSUPPORTED, "scales must be in [1, %d] (got %d)",
                lookme::MS_MAX_SCALES, scales);
  if (d.num_scenes % scales != 0)
    return fail(LOOKME_ERR_INVALID, "%d scenes do not split evenly over %d scales",
                d.num_scenes, scales);
  LOOKME_TRY(check_hidden_dim(d, d_h));
  if (((int64_t)d_h * elem_size(d.dtype)) % 128 != 0)
    return fail(LOOKME_ERR_UNSUPPORTED, "d_h * elem_size must be a multiple of 128 bytes");
  LOOKME_TRY(check_ptr(w_he_t, "w_he_t"));
  h->ms_scales = scales;
  h->ms_dh = d_h;
  h->ms_w = w_he_t;
  return LOOKME_OK;
}

lookme_status_t lookme_inject_multiscale(lookme_t h, int64_t n, int64_t n_keep,
                                         const int32_t* kept, const int32_t* scene,
                                         const int32_t* prim, const float* w, void* hidden,
                                         int32_t d_h, void* stream) {
  LOOKME_TRY(check_handle(h));
  if (h->ms_scales < 1)
    return fail(LOOKME_ERR_INVALID, "no multi-scale router registered (lookme_set_multiscale)");
  LOOKME_TRY(check_layers_n(h->ms_scales, n));
  LOOKME_TRY(check_keep(n, n_keep));
  if (d_h != h->ms_dh)
    return fail(LOOKME_ERR_INVALID, "d_h %d, the router reads %d", d_h, h->ms_dh);
  if (n == 0 || n_keep == 0) return LOOKME_OK;
  LOOKME_TRY(check_lookup_ptrs(kept, scene, prim, w, hidden));
  Layout L;
  LOOKME_TRY(check_workspace(h, 1, n, &L));
  const lookme_desc_t& d = h->d;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(h->ws);
  Timed tm(h, LOOKME_GROUP_INJECT, st);
  return hip_status(lookme::launch_multiscale(d.dtype, h->ms_scales, n, n_keep, kept, scene,
                                              prim, w, h->values, d.num_scenes,
                                              d.prims_per_scene, d.value_dim, d.top_k, h->ms_w,
                                              d_h, hidden, ws + L.ms_r, ws + L.ms_q, st),
                    "multi-scale injection launch");
}

lookme_status_t lookme_inject_multiscale_gated(lookme_t h, int64_t n, const int32_t* kept,
                                               const int32_t* count, const int32_t* scene,
                                               const int32_t* prim, const float* w, void* hidden,
                                               int32_t d_h, void* stream) {
  LOOKME_TRY(check_handle(h));
  if (h->ms_scales < 1)
    return fail(LOOKME_ERR_INVALID, "no multi-scale router registered (lookme_set_multiscale)");
  LOOKME_TRY(check_layers_n(h->ms_scales, n));
  if (d_h != h->ms_dh)
    return fail(LOOKME_ERR_INVALID, "d_h %d, the router reads %d", d_h, h->ms_dh);
  if (n == 0) return LOOKME_OK;
  LOOKME_TRY(check_ptr(count, "count"));
  LOOKME_TRY(check_lookup_ptrs(kept, scene, prim, w, hidden));
  Layout L;
  LOOKME_TRY(check_workspace(h, 1, n, &L));
  const lookme_desc_t& d = h->d;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(h->ws);
  Timed tm(h, LOOKME_GROUP_INJECT, st);
  return hip_status(lookme::launch_multiscale(d.dtype, h->ms_scales, n, n, kept, scene, prim, w,
                                              h->values, d.num_scenes, d.prims_per_scene,
                                              d.value_dim, d.top_k, h->ms_w, d_h, hidden,
                                              ws + L.ms_r, ws + L.ms_q, st, count),
                    "multi-scale injection launch");
}

}  // extern "C"
