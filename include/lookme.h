/*
 * lookme.h -- C ABI of the LookME image-pathway hot path on AMD Instinct
 * MI355X (gfx950).
 *
 * Paper: "LookME: Lookup-Based Multimodal Embeddings for Layer Injection in
 * Vision-Language Models", arXiv 2607.16305.
 *
 * For every continuous multimodal token the library
 *   1. projects it into the table's key space      (Sec. 3.2, Level-1: v_e = v W_{v->e})
 *   2. routes it to one scene                        (Sec. 3.2, Eq. 5)
 *   3. picks the top-k primitives of that scene and  (Sec. 3.2, Eq. 6-7, dot-score form
 *      softmax-weights them                           against per-row primitive keys)
 *   4. selects the critical tokens                   (Sec. 3.3, Eq. 9-10: keep the n_keep
 *                                                     tokens of largest ||Delta_t||_2)
 *   5. adds the weighted table rows into their       (Eq. 2 and Eq. 10)
 *      hidden states,
 * for one or several layers that share the table (Sec. 3.3, inter-layer reuse).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  * Tensors are DEVICE pointers, row-major and contiguous, owned by the
 *    caller.  Every pointer must be 16-byte aligned.  Element type is the
 *    table dtype (LOOKME_F32 or LOOKME_BF16) unless stated (int32 indices,
 *    float32 weights and bias).
 *  * Calls are asynchronous on `stream` (a hipStream_t; NULL = default
 *    stream).  The library itself never allocates device memory: scratch
 *    space comes from the caller's workspace (lookme_set_workspace).
 *  * Every argument is validated before anything is launched; on any error
 *    nothing is written and the status says why (lookme_last_error() gives
 *    the message).  No C++ exception crosses this boundary.
 *  * n == 0 is a valid no-op.  A handle is not thread-safe (it owns one
 *    workspace); calls on one handle must be ordered on one stream.
 *  * Exact score ties resolve to the lowest index (scene, primitive, token).
 */
#ifndef LOOKME_H_
#define LOOKME_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lookme_s* lookme_t;           /* opaque; borrows the table */

typedef enum {
  LOOKME_OK = 0,
  LOOKME_ERR_INVALID = 1,       /* bad argument (null, size, alignment, range) */
  LOOKME_ERR_UNSUPPORTED = 2,   /* valid but outside what the library implements */
  LOOKME_ERR_WORKSPACE = 3,     /* no workspace set, or too small for the call */
  LOOKME_ERR_HIP = 4            /* a HIP runtime call or kernel launch failed */
} lookme_status_t;

typedef enum { LOOKME_F32 = 0, LOOKME_BF16 = 1 } lookme_dtype_t;
typedef enum { LOOKME_SCORE_DOT = 0, LOOKME_SCORE_COS = 1 } lookme_score_t;

/* Largest supported top-k (T~ in Eq. 6). */
#define LOOKME_KMAX 32
/* rows (layers * n) that lookme_inject_noalloc accepts */
#define LOOKME_NOALLOC_MAX_ROWS 131072

typedef struct {
  int32_t num_scenes;       /* N_s  (Sec. 3.2 "Two-level embedding table")            */
  int32_t prims_per_scene;  /* N_p                                                   */
  int32_t key_dim;          /* d_e: width of scene keys, primitive keys and queries;
                               key_dim * elem_size must be a multiple of 64 bytes
                               and at most 2048 bytes                               */
  int32_t value_dim;        /* d_v: width of a table row that is added into H;
                               value_dim * elem_size must be a multiple of 16 bytes  */
  int32_t top_k;            /* T~ (Eq. 6): 1 <= top_k <= min(N_p, LOOKME_KMAX)       */
  int32_t dtype;            /* lookme_dtype_t of keys, values, queries, hidden       */
  int32_t score;            /* lookme_score_t: DOT, the dot product of the configured
                               workloads, or COS, the cosine of Eq. 5 and Eq. 7
                               (q.k / (||q|| ||k||), 0 for a zero vector), used by
                               routing (plus the bias) and by the key-scored
                               Level-2, whose softmax then runs over the k cosines */
} lookme_desc_t;

/*
 * lookme_create -- describe an HBM-resident table (Sec. 3.2).
 *   scene_keys [N_s, d_e]        e_img of Eq. 4-5: one routing key per scene
 *   prim_keys  [N_s, N_p, d_e]   one key per table row, scored in Level-2
 *   values     [N_s * N_p, d_v]  table rows; row (s, p) is values[s*N_p + p]
 *   scene_bias [N_s] float32 or NULL (b of Eq. 5; NULL means 0)
 * The handle BORROWS the four pointers: they must stay valid and unmodified
 * until lookme_destroy.  Nothing is copied (a table may be tens of GiB).
 * No HIP call is made.
 */
lookme_status_t lookme_create(const lookme_desc_t* desc, const void* scene_keys,
                              const void* prim_keys, const void* values,
                              const float* scene_bias, lookme_t* out);

/* Bytes of device workspace needed by route/lookup/inject for `layers`
 * layers of `n_tokens` tokens each.  No HIP call is made. */
lookme_status_t lookme_workspace_size(lookme_t h, int32_t layers, int64_t n_tokens,
                                      size_t* bytes);

/* Attach caller-owned device workspace (256-byte aligned, at least 49408
 * bytes; lookme_workspace_size gives what a call needs).  The library
 * zero-fills a small counter region of it once here (hipMemset on the current
 * device); every call leaves those counters at zero again.  The workspace
 * must not be modified by the caller while the handle uses it. */
lookme_status_t lookme_set_workspace(lookme_t h, void* dev_ptr, size_t bytes);

/*
 * lookme_route -- query projection and Level-1 scene routing (Eq. 5).
 *   x         [n, d_in]            tokens v (vision-encoder outputs), shared by all layers
 *   w_proj    [layers, d_e, d_in]  W_{v->e} of each layer stored output-row-major
 *                                  (row j holds column j of the paper's d_in x d_e
 *                                  matrix), or NULL when the tokens already are
 *                                  the queries of every layer (then d_in must
 *                                  equal d_e; q_out may alias x for one layer)
 *   q_out     [layers, n, d_e]     q = round_to_dtype(x W), float32 accumulation
 *   scene_out [layers, n] int32    argmax_s <q, scene_keys[s]> + bias[s]
 * d_in * elem_size must be a multiple of 16 bytes.  Needs a workspace of at
 * least lookme_workspace_size(layers, n) (small batches pass partial arg
 * maxima between workgroups through it).
 */
lookme_status_t lookme_route(lookme_t h, int32_t layers, int64_t n, int32_t d_in,
                             const void* x, const void* w_proj, void* q_out,
                             int32_t* scene_out, void* stream);

/*
 * lookme_lookup -- Level-2 scene-primitive retrieval (Eq. 6-7, dot form).
 *   q        [layers, n, d_e]       queries (q_out of lookme_route)
 *   scene    [layers, n] int32      scenes in [0, N_s)
 *   prim_out [layers, n, k] int32   the k primitives p in [0, N_p) of largest
 *                                   <q, prim_keys[scene, p]>, score-descending
 *   w_out    [layers, n, k] float32 softmax of those k scores (temperature 1)
 * Needs a workspace of at least lookme_workspace_size(layers, n).  Launches
 * the bucketing, the Level-2 scoring and, for batches of at least 1024 rows
 * averaging at most 16 rows a scene, a small launch after it that merges the
 * parts of work units cut in two (the outputs are the same bits either way).
 */
lookme_status_t lookme_lookup(lookme_t h, int32_t layers, int64_t n, const void* q,
                              const int32_t* scene, int32_t* prim_out, float* w_out,
                              void* stream);

/*
 * lookme_lookup_select -- lookme_lookup and lookme_select of the same batch
 * in one call on one stream, for callers that would otherwise order a second
 * stream around the select (each cross-stream wait costs microseconds, which
 * at small batches is a tenth of the path).  For batches of at most 1024
 * rows (layers * n) the criticality norms of Eq. 9 are computed by extra
 * workgroups of the bucketing launch, and when n <= 4096 each layer's top
 * n_keep select (Eq. 10) runs as one extra workgroup of the Level-2 launch,
 * beside the scoring units; what does not fit (and any batch of a handle
 * with COS scores) runs as its own kernels after the bucketing.  The results
 * are the same bits as lookme_lookup followed by lookme_select:
 *   prim_out, w_out as for lookme_lookup; kept_out [layers, n_keep] int32
 *   ascending (unused when n_keep = 0); crit [layers, n, d_c].
 * Requires what both calls require; needs the workspace of
 * lookme_workspace_size(layers, n) and uses the part that lookme_select uses
 * (the two must not run concurrently on one handle).
 */
lookme_status_t lookme_lookup_select(lookme_t h, int32_t layers, int64_t n, const void* q,
                                     const int32_t* scene, int32_t* prim_out, float* w_out,
                                     int64_t n_keep, const void* crit, int32_t d_c,
                                     int32_t* kept_out, void* stream);

/*
 * Index checks of the row adds.  Every entry point that gathers table rows
 * for kept tokens (lookme_inject, lookme_inject_kept, lookme_inject_noalloc,
 * the gated, fused, propagated and multi-scale injections) checks each kept
 * entry's token id (in [0, n)), its scene (in [0, N_s), or in its scale's
 * partition) and its k primitives (in [0, N_p)) on the device.  An entry
 * with any of them out of range is not injected (its hidden row keeps its
 * bits; where the rows feed the fusion or the scale mix, its retrieved row is
 * zero) and is counted in the library's per-GPU index-error count instead.
 *
 * lookme_index_errors -- *count = the number of such entries since the last
 * call on the current GPU, and resets it.  Ordered on `stream` and
 * synchronises it (a debugging aid: the adds themselves never wait on it).
 */
lookme_status_t lookme_index_errors(void* stream, uint64_t* count);

/*
 * lookme_inject -- sparse injection (Eq. 9-10) and residual add (Eq. 2).
 *   crit     [layers, n, d_c]   Delta of each layer (the attention update);
 *                               criticality c_t = ||crit_t||_2
 *   scene, prim, w              outputs of route and lookup
 *   hidden   [layers, n, d_h]   H, updated IN PLACE: for the n_keep tokens of
 *                               largest c_t (ties: lowest t) and j < d_v,
 *                               H[t,j] <- round(H[t,j] + sum_i w[t,i] *
 *                               values[scene[t]*N_p + prim[t,i], j]);
 *                               every other element keeps its bits
 *   kept_out [layers, n_keep] int32, ascending kept token ids, or NULL
 * Requires 0 <= n_keep <= n, d_v <= d_h, d_c * elem_size and d_h * elem_size
 * multiples of 16 bytes.  Needs the workspace of lookme_workspace_size.
 */
lookme_status_t lookme_inject(lookme_t h, int32_t layers, int64_t n, int64_t n_keep,
                              const void* crit, int32_t d_c, const int32_t* scene,
                              const int32_t* prim, const float* w, void* hidden,
                              int32_t d_h, int32_t* kept_out, void* stream);

/*
 * lookme_inject_noalloc -- lookme_inject for callers that cannot allocate
 * device memory (code under stream capture, tight serving loops, harnesses
 * that forbid allocation): the same selection and row add, the same
 * arguments and the same results bit for bit, but no workspace is needed and
 * nothing is allocated.  Its scratch (the criticality keys and, when
 * kept_out is NULL, the kept lists) is a static device array of the library,
 * 1 MiB on every GPU it runs on, held until the process ends.
 * Requires layers * n <= LOOKME_NOALLOC_MAX_ROWS (else
 * LOOKME_ERR_UNSUPPORTED, nothing launched) and the conditions of
 * lookme_inject.  Every call on one GPU shares that GPU's scratch: calls that
 * overlap on one GPU (other streams, other threads) race and must be
 * ordered by the caller.  The profiling hooks do not time it.
 */
lookme_status_t lookme_inject_noalloc(lookme_t h, int32_t layers, int64_t n, int64_t n_keep,
                                      const void* crit, int32_t d_c, const int32_t* scene,
                                      const int32_t* prim, const float* w, void* hidden,
                                      int32_t d_h, int32_t* kept_out, void* stream);

/*
 * lookme_select -- the sparse injection set alone (Eq. 9): c_t = ||crit_t||_2
 * for every token, then per layer the n_keep tokens of largest c_t (ties:
 * lowest t) written to
 *   kept_out [layers, n_keep] int32, ascending token ids
 * -- the set that lookme_inject selects.  It reads no routing or lookup
 * result and its part of the workspace is disjoint from theirs, so it may run
 * on another stream, concurrently with lookme_route / lookme_lookup of the
 * same batch; lookme_inject_kept then adds the rows.  Made for that: its
 * norms run on one workgroup a CU (they leave most of every CU to the
 * kernels beside them, and take longer alone than lookme_inject's).  Requires
 * 0 <= n_keep <= n, d_c * elem_size a multiple of 16 bytes, kept_out non-NULL
 * when n_keep > 0 (n_keep = 0 does nothing).  Needs the workspace of
 * lookme_workspace_size.
 */
lookme_status_t lookme_select(lookme_t h, int32_t layers, int64_t n, int64_t n_keep,
                              const void* crit, int32_t d_c, int32_t* kept_out, void* stream);

/*
 * lookme_inject_kept -- the gather and residual add of lookme_inject (Eq. 10,
 * Eq. 2) for a kept set computed beforehand:
 *   kept [layers, n_keep] int32   token ids of each layer (kept_out of
 *                                 lookme_select); an id outside [0, n) is
 *                                 not injected and is counted (see
 *                                 lookme_index_errors), and an id listed
 *                                 twice in a layer races on its row of hidden
 * The other arguments as for lookme_inject; the result is the same when kept
 * is the set lookme_select writes.  Needs no workspace.
 */
lookme_status_t lookme_inject_kept(lookme_t h, int32_t layers, int64_t n, int64_t n_keep,
                                   const int32_t* kept, const int32_t* scene, const int32_t* prim,
                                   const float* w, void* hidden, int32_t d_h, void* stream);

/*
 * lookme_set_relevance -- registers the scene-shared relevance MLP that
 * Level-2 uses in the paper's own form (Sec. 3.2, Eq. 6).  The tensors are
 * borrowed like the table (they must stay alive and unmodified while used):
 *   hidden  width h of the hidden layer; h * elem_size a multiple of 128 bytes
 *   w1      [h, 2 * key_dim] dtype; columns [0, key_dim) act on the query,
 *           [key_dim, 2 key_dim) on the scene key e_img[j]
 *   b1      [h] float32, or NULL for zero
 *   w2      [prims_per_scene, h] dtype
 *   b2      [prims_per_scene] float32, or NULL for zero
 * Needs key_dim * elem_size a multiple of 128 bytes.  Replaces an earlier
 * registration.  From then on lookme_workspace_size includes the lookup's
 * logits, layers * n * prims_per_scene float32, and a per-scene table
 * T[s] = W1[:, key_dim:] scene_keys[s] + b1 (num_scenes * h float32) that
 * the first lookme_lookup_relevance after this call (or after
 * lookme_set_workspace) computes into the workspace and later calls reuse:
 * the first layer then multiplies only the query half per row.  The
 * workspace must be left alone between calls, and a change of the scene
 * keys, w1 or b1 in place needs this call again.
 */
lookme_status_t lookme_set_relevance(lookme_t h, int32_t hidden, const void* w1,
                                     const float* b1, const void* w2, const float* b2);

/*
 * lookme_lookup_relevance -- Level-2 in the paper's form (Eq. 6-7), with
 * the MLP of lookme_set_relevance:
 *   q, scene   as for lookme_lookup (q [layers, n, d_e], scene [layers, n])
 *   act_out    [layers, n, h] dtype: a = round(ReLU(W1 [q ; scene_keys[scene]]
 *              + b1)), float32 accumulation (the query half per row plus the
 *              per-scene table), one rounding to dtype
 *   prim_out   [layers, n, k] int32: the k primitives p of largest logit
 *              r_p = <W2[p], a> + b2[p] (ties: lowest p), logit-descending
 *   w_out      [layers, n, k] float32: softmax over the k of
 *              cos(q, prim_keys[scene, p]) + tanh(r_p) (cosine 0 for a zero
 *              vector)
 * Needs the workspace of lookme_workspace_size (queried after
 * lookme_set_relevance): the logits of every row go through it.
 */
lookme_status_t lookme_lookup_relevance(lookme_t h, int32_t layers, int64_t n, const void* q,
                                        const int32_t* scene, void* act_out, int32_t* prim_out,
                                        float* w_out, void* stream);

/*
 * lookme_set_fusion -- registers the SwiGLU fusion f of Eq. 10, one per
 * layer (borrowed, like the table):
 *   w_gate, w_up [layers, d_ff, value_dim] dtype
 *   w_down       [layers, d_h, d_ff] dtype
 *   f_l(R) = w_down[l] (silu(w_gate[l] R) * (w_up[l] R)), silu(x) = x / (1 + e^-x)
 * Needs d_ff * elem_size and value_dim * elem_size multiples of 128 bytes.
 * From then on lookme_workspace_size includes the fusion's buffers (R and
 * the inner activations of up to layers * n rows).
 */
lookme_status_t lookme_set_fusion(lookme_t h, int32_t layers, int32_t d_ff, int32_t d_h,
                                  const void* w_gate, const void* w_up, const void* w_down);

/*
 * lookme_inject_fused -- sparse injection through the fusion (Eq. 10, Eq. 2)
 * for a kept set (lookme_select): for every layer l and kept token t,
 *   R = round(sum_i w[t,i] values[scene[t]*N_p + prim[t,i], :])   (value_dim)
 *   U = round(silu(w_gate[l] R) * (w_up[l] R))                     (d_ff)
 *   hidden[l, t, :] <- round(hidden[l, t, :] + w_down[l] U)        (d_h)
 * float32 accumulation throughout; every other row keeps its bits.  A kept id
 * outside [0, n) is not injected and is counted (lookme_index_errors), and
 * an id listed twice in a layer races on its row.  d_h must be the fusion's.  Needs the workspace of
 * lookme_workspace_size (queried after lookme_set_fusion).
 */
lookme_status_t lookme_inject_fused(lookme_t h, int32_t layers, int64_t n, int64_t n_keep,
                                    const int32_t* kept, const int32_t* scene,
                                    const int32_t* prim, const float* w, void* hidden,
                                    int32_t d_h, void* stream);

/*
 * lookme_set_propagation -- registers the propagation projections of the
 * inter-layer sparse activation (Sec. 3.3, Eq. 11), one for each of `steps`
 * non-LookME layers after a LookME layer (borrowed, like the table):
 *   w_p_t [steps, value_dim, value_dim] dtype, w_p_t[j][o][i] = W_p^(j+1)[i, o]
 * (each matrix stored transposed, output-row-major, like the projection's W).
 * The propagated rows keep the retrieved width value_dim.  Needs value_dim *
 * elem_size a multiple of 128 bytes.
 */
lookme_status_t lookme_set_propagation(lookme_t h, int32_t steps, const void* w_p_t);

/*
 * lookme_inject_propagated -- sparse injection at a LookME layer and at the
 * `steps` non-LookME layers after it (Eq. 10-11): one lookup and one kept set
 * (the LookME layer's gate, reused by the layers after it), and for every
 * kept token t and j = 0..steps:
 *   R_0 = round(sum_i w[t,i] values[scene[t]*N_p + prim[t,i], :])
 *   R_j = round(R_{j-1} W_p^j + R_{j-1})                            (j >= 1)
 *   hidden[j, t, :] <- round(hidden[j, t, :] + f_j(R_j))
 * with f_j layer j of the registered fusion (lookme_set_fusion: at least
 * steps + 1 layers, d_h equal to the fusion's) and W_p^j projection j - 1 of
 * lookme_set_propagation (at least `steps` registered).  kept [n_keep],
 * scene [n], prim [n, top_k], w [n, top_k] are the LookME layer's (a
 * one-layer select and lookup); hidden [steps + 1, n, d_h] holds the
 * layers' hidden states, updated in place.  float32 accumulation, every other
 * row keeps its bits; steps = 0 is lookme_inject_fused on one layer.  Needs
 * the workspace of lookme_workspace_size(layers = steps + 1, n) queried after
 * lookme_set_fusion.
 */
lookme_status_t lookme_inject_propagated(lookme_t h, int32_t steps, int64_t n, int64_t n_keep,
                                         const int32_t* kept, const int32_t* scene,
                                         const int32_t* prim, const float* w, void* hidden,
                                         int32_t d_h, void* stream);

/*
 * lookme_set_multiscale -- registers the token-wise router of multi-scale
 * image retrieval (Sec. 3.2, Eq. 8) on the handle of the whole table:
 *   scales  M in [1, 8]; the num_scenes scenes split into M equal partitions,
 *           scale m owning scenes [m S/M, (m+1) S/M) (each scale is routed and
 *           looked up on a handle created over its partition's slices of
 *           scene_keys, prim_keys and values: its own ranker);
 *   w_he_t  [value_dim, d_h] dtype, W_{h->e} stored transposed (output-row-
 *           major), borrowed; it projects a hidden state to the width of the
 *           retrieved rows.
 * Needs d_h >= value_dim and d_h * elem_size a multiple of 128 bytes.  From
 * then on lookme_workspace_size includes the router's buffers.
 */
lookme_status_t lookme_set_multiscale(lookme_t h, int32_t scales, int32_t d_h,
                                      const void* w_he_t);

/*
 * lookme_inject_multiscale -- multi-scale injection of one layer (Eq. 8, then
 * Eq. 10 and Eq. 2): scene [M, n] (scale m's scene ids, local to its
 * partition), prim [M, n, top_k] and w [M, n, top_k] are the M scales'
 * lookups, kept [n_keep] the layer's kept set (lookme_select).  For every
 * kept token t:
 *   R^m = round(sum_i w[m,t,i] values[(m S/M + scene[m,t]) N_p + prim[m,t,i], :])
 *   q   = round(hidden[t, :] W_{h->e})                 (the states before the add)
 *   a   = softmax over m of (q . R^m) / sqrt(value_dim)
 *   hidden[t, :value_dim] <- round(hidden[t, :value_dim] + sum_m a_m R^m)
 * float32 accumulation; every other row keeps its bits.  hidden [n, d_h],
 * d_h equal to the registered one.  Needs the workspace of
 * lookme_workspace_size(1, n) queried after lookme_set_multiscale.
 */
lookme_status_t lookme_inject_multiscale(lookme_t h, int64_t n, int64_t n_keep,
                                         const int32_t* kept, const int32_t* scene,
                                         const int32_t* prim, const float* w, void* hidden,
                                         int32_t d_h, void* stream);

/*
 * lookme_inject_multiscale_gated -- lookme_inject_multiscale for the counted
 * list of lookme_gate (Eq. 8 with the learned gate of Eq. 9-10): kept [n]
 * int32 holds the layer's open token ids in its first count[0] entries (the
 * rest is not read), count [1] int32 is read on the device; scene, prim, w,
 * hidden and the workspace as for lookme_inject_multiscale, whose result it
 * gives bit for bit for the same set.  Launches for n entries; those past the
 * count do nothing.  count NULL or no router registered: INVALID.
 */
lookme_status_t lookme_inject_multiscale_gated(lookme_t h, int64_t n, const int32_t* kept,
                                               const int32_t* count, const int32_t* scene,
                                               const int32_t* prim, const float* w, void* hidden,
                                               int32_t d_h, void* stream);

/*
 * lookme_gate -- the learned SKA gate of the intra-layer sparse activation
 * (Sec. 3.3, Eq. 9) as it acts at inference: the Gumbel-Sigmoid is hard and
 * noise-free, so entry i of a layer opens exactly when
 *   z_i = Delta_{row(i)} . W_g > 0                (z_i = 0 stays closed)
 * with row(i) = pos[i] (pos non-NULL: the pathway's positions in a longer
 * sequence, e.g. the text positions) or i.  Per pathway and layer it gives
 * the variable set of positions whose retrieved rows Eq. 10 injects.
 *   delta     [layers, delta_rows, d_c] dtype, Delta = Attn(H_in) of each layer
 *   pos       [n] int32 row of each entry (clamped into [0, delta_rows)), or
 *             NULL (then delta_rows >= n and entry i reads row i)
 *   w_g       [layers, d_c] dtype, each layer's gate projection W_g
 *   kept_out  [layers, n] int32: the open entries i of layer l in ascending
 *             order, then -1 up to n
 *   count_out [layers] int32: the number of open entries of each layer
 * z is accumulated in float32 (fused multiply-adds over d_c) and compared
 * with 0 in that precision.  d_c * elem_size a multiple of 16 bytes.  n = 0
 * writes count_out = 0 and nothing else.  Needs the workspace of
 * lookme_workspace_size(layers, n); it uses the same part as lookme_select,
 * so a gate and a select on one handle must not run concurrently.
 */
lookme_status_t lookme_gate(lookme_t h, int32_t layers, int64_t n, const void* delta,
                            int64_t delta_rows, int32_t d_c, const int32_t* pos, const void* w_g,
                            int32_t* kept_out, int32_t* count_out, void* stream);

/*
 * lookme_lookup_gate -- lookme_lookup and lookme_gate (with pos = NULL,
 * delta_rows = n) of the same batch in one call on one stream, as
 * lookme_lookup_select is for the top-n_keep select: for batches of at most
 * 1024 rows the gate's logits are computed by extra workgroups of the
 * bucketing launch and, when n <= 4096, each layer's open rows are compacted
 * by one extra workgroup of the Level-2 launch; otherwise the gate's kernels
 * run after the bucketing.  The same bits as the two calls:
 *   delta [layers, n, d_c], w_g [layers, d_c]; kept_out [layers, n] (open
 *   token ids ascending, then -1), count_out [layers]; prim_out, w_out as
 *   for lookme_lookup.
 * Needs the workspace of lookme_workspace_size(layers, n); uses the part that
 * lookme_select and lookme_gate use.
 */
lookme_status_t lookme_lookup_gate(lookme_t h, int32_t layers, int64_t n, const void* q,
                                   const int32_t* scene, int32_t* prim_out, float* w_out,
                                   const void* delta, int32_t d_c, const void* w_g,
                                   int32_t* kept_out, int32_t* count_out, void* stream);

/*
 * lookme_inject_gated -- lookme_inject_kept for the counted lists of
 * lookme_gate (Eq. 10 with the learned gate, prefix add of Eq. 2):
 *   kept  [layers, n] int32, layer l's open token ids in its first count[l]
 *         entries (the rest is not read)
 *   count [layers] int32, read on the device
 * scene, prim, w and hidden as for lookme_inject_kept.  Launches layers * n
 * workgroups, those past a layer's count end at once.  Needs no workspace.
 */
lookme_status_t lookme_inject_gated(lookme_t h, int32_t layers, int64_t n, const int32_t* kept,
                                    const int32_t* count, const int32_t* scene,
                                    const int32_t* prim, const float* w, void* hidden,
                                    int32_t d_h, void* stream);

/*
 * lookme_inject_fused_gated -- lookme_inject_fused (Eq. 10 through the
 * SwiGLU fusion f) for the counted lists of lookme_gate: kept [layers, n]
 * and count [layers] as for lookme_inject_gated, S(R) = g . f(R[g]) on the
 * open rows only.  Needs the workspace of lookme_workspace_size(layers, n)
 * queried after lookme_set_fusion.
 */
lookme_status_t lookme_inject_fused_gated(lookme_t h, int32_t layers, int64_t n,
                                          const int32_t* kept, const int32_t* count,
                                          const int32_t* scene, const int32_t* prim,
                                          const float* w, void* hidden, int32_t d_h,
                                          void* stream);

/*
 * lookme_inject_propagated_gated -- lookme_inject_propagated (Eq. 11) with
 * the LookME layer's learned gate reused by the layers after it: kept [n]
 * int32 holds the open token ids in its first count[0] entries (a one-layer
 * lookme_gate), count [1] int32 is read on the device.  Everything else as
 * for lookme_inject_propagated; the workspace of
 * lookme_workspace_size(steps + 1, n) queried after lookme_set_fusion.
 */
lookme_status_t lookme_inject_propagated_gated(lookme_t h, int32_t steps, int64_t n,
                                               const int32_t* kept, const int32_t* count,
                                               const int32_t* scene, const int32_t* prim,
                                               const float* w, void* hidden, int32_t d_h,
                                               void* stream);

/*
 * lookme_scene_keys -- scene-centred keys (Sec. 3.2, Level-1, Eq. 4): a
 * scene's key is the mean of its primitive embeddings,
 *   scene_keys[s, :] = round( (sum over p of prim_keys[s, p, :]) / N_p ),
 * each element summed in float32 in increasing p, divided by N_p once and
 * rounded once to the dtype.  A preparation step for tables whose scene
 * keys are not given (the configured workloads give them): its output can be
 * passed to lookme_create as scene_keys.
 *   desc        num_scenes, prims_per_scene, key_dim and dtype are used (the
 *               rest is ignored); key_dim * elem_size a multiple of 16 bytes
 *   prim_keys   [N_s, N_p, d_e] of dtype, read once
 *   scene_keys  [N_s, d_e] of dtype, written (must not overlap prim_keys)
 * Needs no handle and no workspace.
 */
lookme_status_t lookme_scene_keys(const lookme_desc_t* desc, const void* prim_keys,
                                  void* scene_keys, void* stream);

/*
 * lookme_inject_text -- the text pathway of a LookME layer (Sec. 3.2, "Text
 * embedding index-based lookup", Eq. 1): a text position's token id indexes
 * the layer's text table, R_text = E_text[u], and the open entries of the
 * pathway's gate (Eq. 9-10) add it into their hidden rows:
 *   for the first count[0] entries j of kept (all n_text of them when count
 *   is NULL; kept NULL: j itself), with i = kept[j]:
 *     hidden[pos[i], :d_t] <- round(hidden[pos[i], :d_t] + table[ids[i], :])
 * float32 sum, one rounding; every other element keeps its bits.
 *   dtype  lookme_dtype_t of table and hidden (no handle: the text table is
 *          not the image table)
 *   table  [vocab, d_t], borrowed for the call
 *   pos    [n_text] int32 text positions in [0, n) (clamped), pairwise
 *          distinct (two entries on one position race)
 *   ids    [n_text] int32 token ids in [0, vocab) (clamped)
 *   kept   [n_text] int32 entries of pos/ids (lookme_gate with pos), or NULL
 *   count  [1] int32 on the device, or NULL
 *   hidden [n, d_h], updated in place
 * Requires d_t <= d_h and d_t * elem_size, d_h * elem_size multiples of 16
 * bytes.  n_text = 0 does nothing.  Needs no workspace.
 */
lookme_status_t lookme_inject_text(int32_t dtype, const void* table, int64_t vocab, int32_t d_t,
                                   int64_t n_text, const int32_t* pos, const int32_t* ids,
                                   const int32_t* kept, const int32_t* count, void* hidden,
                                   int64_t n, int32_t d_h, void* stream);

/*
 * Measurement support (not part of the method).  When enabled, each kernel
 * group that route/lookup/inject launches is bracketed by a pair of HIP timing
 * events recorded on the call's stream; the Level-2 scoring launch of the
 * bucketed lookups (lookme_lookup, lookme_lookup_select, lookme_lookup_gate)
 * instead records its own start and end in its pair (an extended launch), so
 * its time is the kernel's duration alone.  lookme_profile_read waits for the
 * recorded events, adds their durations to per-group totals and returns the
 * totals since the last reset.  Groups (lookme_group_t):
 *   PROJECT  query projection GEMM          ROUTE   Level-1 scoring + arg max
 *   BUCKET   scene bucketing (3 kernels)    SCORE   Level-2 scoring + top-k + softmax
 *   NORM     criticality norms              SELECT  top-n_keep select + compaction
 *   INJECT   row gather + residual add
 * Recorded events cost a few microseconds of launch overhead per group; leave
 * profiling off when measuring end-to-end throughput.
 */
typedef enum {
  LOOKME_GROUP_PROJECT = 0, LOOKME_GROUP_ROUTE = 1, LOOKME_GROUP_BUCKET = 2,
  LOOKME_GROUP_SCORE = 3, LOOKME_GROUP_NORM = 4, LOOKME_GROUP_SELECT = 5,
  LOOKME_GROUP_INJECT = 6, LOOKME_GROUP_COUNT = 7
} lookme_group_t;

lookme_status_t lookme_profile_enable(lookme_t h, int32_t enabled);
/* count: number of timed launches of `group`; total_ms: their summed time.
 * reset != 0 clears the totals after reading. */
lookme_status_t lookme_profile_read(lookme_t h, int32_t group, int64_t* count,
                                    double* total_ms, int32_t reset);

/* Release the handle (not the borrowed table or the workspace). NULL is OK. */
lookme_status_t lookme_destroy(lookme_t h);

/* Message of the last non-OK status returned on this thread ("" if none). */
const char* lookme_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LOOKME_H_ */
