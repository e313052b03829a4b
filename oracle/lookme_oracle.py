"""Plain fp64 CPU oracle for the LookME image-pathway hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
module: only the tests, the smoke check and the benchmark's CPU-baseline leg
use it.  It shares no code with the HIP library (no kernels, no headers, no
helpers); it receives the same input bytes and recomputes every result from
the paper's definitions, slowly and obviously.

Paper: "LookME: Lookup-Based Multimodal Embeddings for Layer Injection in
Vision-Language Models" (arXiv 2607.16305).

What is computed, step by step (each function cites its passage):

  project     Sec. 3.2 "Level-1: scene retrieval": v_e = v W_{v->e}
  scene_keys_from_primitives
              Eq. 4: a scene's key as the mean of its primitive embeddings
  route       Sec. 3.2 Level-1, Eq. 5: scene = argmax(score(v_e, e_img) + b)
  lookup      Sec. 3.2 Level-2, Eq. 6-7 in the configured form: top-k
              primitives of the chosen scene by dot score against per-row
              primitive keys, softmax weights over the k selected scores
  criticality Sec. 3.3 "Intra-Layer Sparse Activation", Eq. 9: the gate is
              driven by the size of Delta_i, the attention update
  select      Eq. 10: the pathway runs only at the gated positions; the
              configured gate keeps the n_keep positions of largest
              ||Delta_i||_2
  inject      Eq. 10 and Eq. 2: H_out = H + S(R_img) at the kept positions,
              S(R)[i] = sum_p w_p * E[scene_i, p, :]
  run         all of the above for L layers that share one table (Sec. 3.3,
              "Inter-Layer Sparse Activation": neighbouring layers retrieve
              similar primitives, so one table serves several layers)
  fusion      Eq. 10 with the SwiGLU fusion f: the kept tokens receive
              f(R) = W_down (silu(W_gate R) * (W_up R)) instead of R
  propagate   Eq. 11 (inter-layer sparse activation): a non-LookME layer k
              after LookME layer l carries R^(k) = R^(k-1) W_p^k + R^(k-1)
              and reuses layer l's gate; inject_propagated applies f^k to it
  multiscale  Sec. 3.2 "Multi-scale image retrieval", Eq. 8: M scales, each
              routed and looked up in its own scene partition of the table;
              a token-wise softmax router over the M retrieved rows, queried
              by the token's hidden state through W_{h->e}, mixes them
  relevance_* Level-2 in the paper's own form (Eq. 6-7): a scene-shared
              two-layer MLP over [v_e, e_img[j]] gives relevance logits r_j;
              the top-k primitives by r are weighted by the softmax of
              cos(v_e, e_{j,p}) + tanh(r_j[p])
  gate        Eq. 9 at inference: the hard, noise-free SKA gate keeps the
              positions with Delta_i W_g > 0 (a learned gate, variable count)
  text        Sec. 3.2 "Text embedding index-based lookup" (Eq. 1):
              R_text = E_text[u] at the text positions; inject_text adds it
  lookme_layer  Eq. 2: one LookME layer, L_dec(H_in) plus the text, image and
              cross-modal pathways' gated injections (the three retrievals of
              Eq. 3) in that order; the
              cross-modal pathway queries the two-level lookup with L_dec(H_in)
              itself at every position (Sec. 3.2, cross-modal embedding
              hierarchical two-level lookup)

Readings of the paper taken here (the paper is silent or differs from the
configured workloads; each is listed in the design notes of the repository):
  * Scores are dot products (the configured workloads); ``score="cos"``
    gives the cosine of Eq. 5 / Eq. 7 (both vectors normalised).
  * Level-2 candidates are scored against primitive keys K2[s, p, :], one key
    per table row; table rows V[s*P + p, :] are the values that are summed.
  * Softmax over the k selected scores, temperature 1, max subtracted.
  * Exact ties go to the lowest index (scene, primitive, token).
  * q is quantised once to the storage dtype (bf16 or fp32) with
    round-to-nearest-even from the exact product; later stages use that q.
  * The injected increment is added into the first d_v columns of H; the
    result is rounded once to the storage dtype.
  * Relevance MLP (Eq. 6): r = W2 act(W1 [v_e ; e_img[j]] + b1) + b2 with
    act = ReLU and a given hidden width; the hidden activations are rounded
    once to the storage dtype (the second layer runs on them as stored);
    e_img are the scene keys; the primitive rows whose cosine Eq. 7 takes are
    the primitive keys K2[j, p, :] (a zero vector has cosine 0).
  * Fusion f (Eq. 10): a SwiGLU FFN d_v -> d_ff -> d_h per layer, silu(x) =
    x / (1 + exp(-x)); R and the inner activations are rounded once to the
    storage dtype (each is the input of a product, as stored), H + f(R) once.

Inputs are numpy arrays.  bf16 tensors are passed as their raw uint16 bit
patterns (numpy has no bf16) together with ``dtype="bf16"``; fp32 tensors as
float32 arrays with ``dtype="f32"``.  All arithmetic is float64.
"""

from __future__ import annotations

import numpy as np

# ---------------------------------------------------------------------------
# Number formats (IEEE-754 binary32 and bfloat16: 1 sign, 8 exponent bits,
# 7 stored fraction bits).  These are written out here from the format
# definitions; the oracle does not use any GPU-side conversion routine.
# ---------------------------------------------------------------------------

_BF16_MANT_BITS = 8          # significand precision including the hidden bit
_BF16_EMIN = -126            # smallest normal exponent (same as binary32)
_BF16_EMAX = 127


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bfloat16 numbers given as uint16 bit patterns."""
    b = np.asarray(bits).astype(np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (ties to even), directly
    from the exact float64 value (no intermediate binary32 rounding).

    Returns float64 values that are exactly representable in bfloat16.
    Values beyond the largest finite bfloat16 after rounding become +-inf.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros_like(x)
    nz = (x != 0) & np.isfinite(x)
    ax = np.abs(x[nz])
    # exponent e with 2^e <= |x| < 2^(e+1)
    _, e2 = np.frexp(ax)            # ax = m * 2^e2, 0.5 <= m < 1
    e = e2 - 1
    e = np.maximum(e, _BF16_EMIN)   # subnormal range keeps the fixed quantum
    quantum_exp = e - (_BF16_MANT_BITS - 1)
    scaled = np.ldexp(ax, -quantum_exp)          # exact (power-of-two scale)
    r = np.ldexp(np.rint(scaled), quantum_exp)  # rint: half to even
    max_finite = np.ldexp(np.float64(2 ** _BF16_MANT_BITS - 1),
                          _BF16_EMAX - (_BF16_MANT_BITS - 1))
    r = np.where(r > max_finite, np.inf, r)
    out[nz] = np.sign(x[nz]) * r
    out[~np.isfinite(x)] = x[~np.isfinite(x)]
    return out


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Bit patterns of float64 values that are already bfloat16 values."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    return (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def round_to_dtype(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values once to the storage dtype; returns float64."""
    if dtype == "bf16":
        return round_to_bf16(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 value of a stored tensor (bf16 bits or float32)."""
    if dtype == "bf16":
        return bf16_bits_to_f64(a)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def from_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Storage representation of float64 values already in the dtype."""
    if dtype == "bf16":
        return f64_to_bf16_bits(x)
    return np.asarray(x, dtype=np.float64).astype(np.float32)


# ---------------------------------------------------------------------------
# The method
# ---------------------------------------------------------------------------

def project(x: np.ndarray, w_t: np.ndarray | None, dtype: str) -> np.ndarray:
    """Query projection v_e = v W_{v->e} (Sec. 3.2, Level-1 paragraph).

    x    : [n, d_in] float64 values of the stored tokens.
    w_t  : [d_e, d_in] float64 values of W stored output-row-major (the
           transpose of the paper's d_in x d_e matrix), or None when the
           tokens are already queries (d_in == d_e, no projection).
    Returns q: [n, d_e] float64 values rounded once to ``dtype``.
    """
    if w_t is None:
        return np.array(x, dtype=np.float64, copy=True)
    q_exact = x @ w_t.T           # (v W)[t, j] = sum_i v[t, i] W[i, j]
    return round_to_dtype(q_exact, dtype)


def scene_keys_from_primitives(prim_keys: np.ndarray) -> np.ndarray:
    """Scene-centred keys (Eq. 4): each scene's key is the mean of its
    primitive embeddings, e_img[j] = (1/N_p) sum_p E[j, p, :].

    prim_keys [S, P, d_e] float64 values -> [S, d_e] float64 (not rounded;
    a caller storing them rounds once to its dtype).
    """
    prim_keys = np.asarray(prim_keys, dtype=np.float64)
    return np.sum(prim_keys, axis=1) / prim_keys.shape[1]


def _unit_rows(a: np.ndarray) -> np.ndarray:
    n = np.sqrt(np.sum(a * a, axis=-1, keepdims=True))
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.where(n > 0, a / np.where(n > 0, n, 1.0), 0.0)


def scene_scores(q: np.ndarray, scene_keys: np.ndarray,
                 bias: np.ndarray | None = None, score: str = "dot") -> np.ndarray:
    """Level-1 scores (Eq. 5): score(v_e, e_img[s]) + b[s] for every scene.

    q [n, d_e], scene_keys [S, d_e], bias [S] or None.  Returns [n, S].
    """
    if score == "cos":
        s = _unit_rows(q) @ _unit_rows(scene_keys).T
    elif score == "dot":
        s = q @ scene_keys.T
    else:
        raise ValueError(score)
    if bias is not None:
        s = s + np.asarray(bias, dtype=np.float64)[None, :]
    return s


def route(q: np.ndarray, scene_keys: np.ndarray, bias: np.ndarray | None = None,
          score: str = "dot") -> np.ndarray:
    """Level-1 scene retrieval (Eq. 5): the arg max over scenes, lowest scene
    index on exact ties.  Returns scene [n] int32."""
    s = scene_scores(q, scene_keys, bias, score)
    if s.shape[1] == 0:
        raise ValueError("no scenes")
    return np.argmax(s, axis=1).astype(np.int32)   # first maximum = lowest s


def primitive_scores(q_t: np.ndarray, prim_keys_s: np.ndarray,
                     score: str = "dot") -> np.ndarray:
    """Level-2 scores of one token against every primitive key of its scene
    (Eq. 6-7, configured form).  q_t [d_e], prim_keys_s [P, d_e] -> [P]."""
    if score == "cos":
        return _unit_rows(prim_keys_s) @ _unit_rows(q_t[None, :])[0]
    return prim_keys_s @ q_t


def softmax_weights(top_scores: np.ndarray) -> np.ndarray:
    """phi in Eq. 7: softmax over the k selected scores (temperature 1),
    evaluated with the largest score subtracted."""
    z = top_scores - np.max(top_scores)
    e = np.exp(z)
    return e / np.sum(e)


def topk_order(scores: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest scores, ordered by (score descending,
    index ascending): a stable sort of the negated scores."""
    order = np.argsort(-scores, kind="stable")
    return order[:k]


def lookup(q: np.ndarray, scene: np.ndarray, prim_keys: np.ndarray, k: int,
           score: str = "dot"):
    """Level-2 scene-primitive retrieval (Eq. 6-7, configured form).

    q [n, d_e], scene [n], prim_keys [S, P, d_e] (float64 values).
    Returns (prim [n, k] int32 in [0, P), descending score; w [n, k] float64;
    top_scores [n, k] float64).
    """
    n = q.shape[0]
    P = prim_keys.shape[1]
    if not (1 <= k <= P):
        raise ValueError("k must be in [1, P]")
    prim = np.zeros((n, k), dtype=np.int32)
    w = np.zeros((n, k), dtype=np.float64)
    top = np.zeros((n, k), dtype=np.float64)
    for t in range(n):
        s2 = primitive_scores(q[t], prim_keys[scene[t]], score)
        idx = topk_order(s2, k)
        prim[t] = idx
        top[t] = s2[idx]
        w[t] = softmax_weights(s2[idx])
    return prim, w, top


def criticality(delta: np.ndarray) -> np.ndarray:
    """Size of the attention update that drives the SKA gate (Eq. 9):
    c_t = ||Delta_t||_2.  delta [n, d_c] -> [n]."""
    return np.sqrt(np.sum(delta * delta, axis=1))


def select(c: np.ndarray, n_keep: int) -> np.ndarray:
    """Sparse activation (Eq. 10) with the configured gate: keep the n_keep
    tokens of largest criticality, ties to the lowest token index; returned in
    ascending token order."""
    n = c.shape[0]
    if not (0 <= n_keep <= n):
        raise ValueError("n_keep must be in [0, n]")
    order = np.argsort(-c, kind="stable")
    return np.sort(order[:n_keep]).astype(np.int32)


def retrieved(values: np.ndarray, P: int, scene_t: int, prim_t: np.ndarray,
              w_t: np.ndarray) -> np.ndarray:
    """R_img for one token (Eq. 7): sum_i w_i * E[scene, prim_i, :], where
    table row (s, p) is stored at V[s*P + p, :]."""
    rows = values[scene_t * P + np.asarray(prim_t, dtype=np.int64)]
    return np.sum(np.asarray(w_t, dtype=np.float64)[:, None] * rows, axis=0)


def inject(hidden: np.ndarray, values: np.ndarray, P: int, scene: np.ndarray,
           prim: np.ndarray, w: np.ndarray, kept: np.ndarray, dtype: str) -> np.ndarray:
    """Residual injection (Eq. 2 and Eq. 10): for kept tokens,
    H[t, :d_v] <- round(H[t, :d_v] + R_img[t]); everything else unchanged.

    hidden [n, d_h] and values [S*P, d_v] are float64 values; returns the new
    hidden as float64 values of ``dtype``.
    """
    out = np.array(hidden, dtype=np.float64, copy=True)
    d_v = values.shape[1]
    for t in np.asarray(kept, dtype=np.int64):
        r = retrieved(values, P, int(scene[t]), prim[t], w[t])
        out[t, :d_v] = round_to_dtype(hidden[t, :d_v] + r, dtype)
    return out


def propagate(r: np.ndarray, w_p: np.ndarray, dtype: str) -> np.ndarray:
    """Eq. 11 chain: R^(0) = r, R^(j) = R^(j-1) W_p^j + R^(j-1) for j = 1..m,
    each stored (rounded once to dtype) before the next step.

    r [m_rows, d_v] (already rounded), w_p [m, d_v, d_v] in the paper's
    orientation (input index first).  Returns [m + 1, m_rows, d_v]."""
    out = [np.asarray(r, dtype=np.float64)]
    for j in range(w_p.shape[0]):
        prev = out[-1]
        out.append(round_to_dtype(prev @ w_p[j] + prev, dtype))
    return np.stack(out)


def inject_propagated(hidden: np.ndarray, values: np.ndarray, P: int, scene: np.ndarray,
                      prim: np.ndarray, w: np.ndarray, kept: np.ndarray, w_p: np.ndarray,
                      w_gate: np.ndarray, w_up: np.ndarray, w_down: np.ndarray,
                      dtype: str) -> np.ndarray:
    """Injection at a LookME layer and the m = w_p.shape[0] non-LookME layers
    after it (Eq. 10-11): the LookME layer's lookup (scene, prim, w) and gate
    (kept) serve all of them; layer j's kept rows receive f_j(R^(j)) with
    R^(j) from ``propagate``.

    hidden [m + 1, n, d_h]; w_gate, w_up [>= m + 1, d_ff, d_v]; w_down
    [>= m + 1, d_h, d_ff].  Returns float64 [m + 1, n, d_h]."""
    out = np.array(hidden, dtype=np.float64, copy=True)
    kept = np.asarray(kept, dtype=np.int64)
    if kept.size == 0:
        return out
    R0 = round_to_dtype(
        np.stack([retrieved(values, P, int(scene[t]), prim[t], w[t]) for t in kept]), dtype)
    Rs = propagate(R0, w_p, dtype)
    for j in range(Rs.shape[0]):
        F = fusion(Rs[j], w_gate[j], w_up[j], w_down[j], dtype)
        out[j, kept] = round_to_dtype(hidden[j, kept] + F, dtype)
    return out


def multiscale_mix(q: np.ndarray, r_scales: np.ndarray) -> np.ndarray:
    """Eq. 8's router for one token: alpha = softmax over the M scales of
    (q . R^m) / sqrt(d), d the width of q and of the rows; returns
    sum_m alpha_m R^m (float64, not rounded).  q [d], r_scales [M, d]."""
    logits = (r_scales @ q) / np.sqrt(q.shape[0])
    z = logits - np.max(logits)
    alpha = np.exp(z) / np.sum(np.exp(z))
    return alpha @ r_scales


def inject_multiscale(hidden: np.ndarray, values: np.ndarray, P: int, scenes_per_scale: int,
                      scene: np.ndarray, prim: np.ndarray, w: np.ndarray, kept: np.ndarray,
                      w_he: np.ndarray, dtype: str) -> np.ndarray:
    """Multi-scale injection (Eq. 8, then Eq. 10 and Eq. 2 in the prefix-add
    form): scale m's lookup (scene [M, n] local to its partition, whose
    scenes start at m * scenes_per_scale; prim, w [M, n, k]) gives the
    retrieved row R^m_t, stored (rounded); the router query is the token's
    hidden state projected, q_t = round(H[t] W_{h->e}); for kept tokens
    H[t, :d_v] <- round(H[t, :d_v] + multiscale_mix(q_t, [R^1_t .. R^M_t])).

    hidden [n, d_h] (the states before injection serve as the router's
    H_img), w_he [d_h, d_v] in the paper's orientation.  Returns float64."""
    out = np.array(hidden, dtype=np.float64, copy=True)
    kept = np.asarray(kept, dtype=np.int64)
    M = scene.shape[0]
    d_v = values.shape[1]
    for t in kept:
        R = np.stack([
            round_to_dtype(retrieved(values, P, m * scenes_per_scale + int(scene[m, t]),
                                     prim[m, t], w[m, t]), dtype) for m in range(M)])
        q = round_to_dtype(hidden[t] @ w_he, dtype)
        out[t, :d_v] = round_to_dtype(hidden[t, :d_v] + multiscale_mix(q, R), dtype)
    return out


def run_multiscale(x_scales, w_t_scales, scene_keys, prim_keys, values, delta, hidden, w_he, *,
                   k: int, n_keep: int, dtype: str):
    """One layer's image pathway over M scales (Sec. 3.2 multi-scale
    retrieval): scale m projects its own tokens x_scales[m] with its own W
    and is routed and looked up within scene partition m (the S scenes split
    evenly); the kept set comes from delta; the rows are mixed by the router
    and injected.  x_scales [M, n, d_in], w_t_scales [M, d_e, d_in],
    delta [n, d_c], hidden [n, d_h], w_he [d_h, d_v].  Returns a dict:
    q [M, n, d_e], scene [M, n] (local), prim, w [M, n, k], kept [n_keep],
    hidden [n, d_h]."""
    M = x_scales.shape[0]
    S, P = prim_keys.shape[0], prim_keys.shape[1]
    if S % M:
        raise ValueError("the scenes must split evenly over the scales")
    Sm = S // M
    qs, scs, prs, ws = [], [], [], []
    for m in range(M):
        q = project(x_scales[m], w_t_scales[m], dtype)
        sc = route(q, scene_keys[m * Sm:(m + 1) * Sm])
        pr, ww, _ = lookup(q, sc, prim_keys[m * Sm:(m + 1) * Sm], k)
        qs.append(q), scs.append(sc), prs.append(pr), ws.append(ww)
    scene, prim, w = np.stack(scs), np.stack(prs), np.stack(ws)
    kept = select(criticality(delta), n_keep)
    h = inject_multiscale(hidden, values, P, Sm, scene, prim, w, kept, w_he, dtype)
    return {"q": np.stack(qs), "scene": scene, "prim": prim, "w": w, "kept": kept, "hidden": h}


def run(x, w_t, scene_keys, prim_keys, values, bias, delta, hidden, *,
        k: int, n_keep: int, dtype: str, score: str = "dot", mlp=None, fusion=None,
        propagation=None, w_g=None):
    """Whole path for L layers sharing one table (Sec. 3.3 inter-layer reuse).

    x [n, d_in]; w_t [L, d_e, d_in] or None; delta [L, n, d_c];
    hidden [L, n, d_h]; all float64 values.  ``mlp`` = (w1, b1, w2, b2)
    selects Level-2 in the paper's form (relevance_hidden/relevance_lookup)
    instead of the key-scored one; ``fusion`` = (w_gate, w_up, w_down), each
    with a leading layer axis, injects through f (inject_fused) instead of
    the prefix add.  ``propagation`` = w_p [m, d_v, d_v] (with ``fusion`` of
    at least m + 1 layers): one LookME layer whose R is carried to the m
    layers after it (Eq. 11, inject_propagated); then hidden, w_t and delta
    hold [m + 1, ...], [1, ...] and [1, ...].  ``w_g`` [L, d_c]: the kept set
    of layer l is the learned gate's (Eq. 9, ``gate``) instead of the top
    n_keep by criticality (n_keep is then not used).  Returns a dict of per-layer
    results: q [L,n,d_e], scene [L,n], prim [L,n,k], w [L,n,k],
    kept [L,n_keep], hidden [L,n,d_h] (with ``propagation``: L = 1 and
    hidden [m + 1, n, d_h]).
    """
    L = hidden.shape[0] if propagation is None else 1
    P = prim_keys.shape[1]
    res = {k_: [] for k_ in ("q", "scene", "prim", "w", "kept", "hidden")}
    for l in range(L):
        q = project(x, None if w_t is None else w_t[l], dtype)
        sc = route(q, scene_keys, bias, score)
        if mlp is None:
            pr, ww, _ = lookup(q, sc, prim_keys, k, score)
        else:
            w1, b1, w2, b2 = mlp
            a = relevance_hidden(q, sc, scene_keys, w1, b1, dtype)
            pr, ww, _ = relevance_lookup(q, sc, a, w2, b2, prim_keys, k)
        if w_g is None:
            kept = select(criticality(delta[l]), n_keep)
        else:
            kept = gate(delta[l], w_g[l])
        if propagation is not None:
            h = inject_propagated(hidden, values, P, sc, pr, ww, kept, propagation, fusion[0],
                                  fusion[1], fusion[2], dtype)
        elif fusion is None:
            h = inject(hidden[l], values, P, sc, pr, ww, kept, dtype)
        else:
            h = inject_fused(hidden[l], values, P, sc, pr, ww, kept, fusion[0][l], fusion[1][l],
                             fusion[2][l], dtype)
        for name, v in zip(res, (q, sc, pr, ww, kept, h)):
            res[name].append(v)
    out = {name: (np.stack(v) if name != "kept" or w_g is None else v)
           for name, v in res.items()}     # gated kept lists differ in length
    if propagation is not None:
        out["hidden"] = out["hidden"][0]
    return out


# ---------------------------------------------------------------------------
# Level-2 in the paper's form: relevance MLP (Eq. 6) and cosine + tanh
# weights (Eq. 7)
# ---------------------------------------------------------------------------

def relevance_hidden(q: np.ndarray, scene: np.ndarray, scene_keys: np.ndarray,
                     w1: np.ndarray, b1: np.ndarray, dtype: str) -> np.ndarray:
    """First layer of the scene-shared relevance MLP (Sec. 3.2, Level-2,
    Eq. 6) on the concatenation [v_e, e_img[j]] of a token's query and its
    scene's key: a = ReLU(W1 [v_e ; e_img[j]] + b1), rounded once to dtype.

    q [n, d_e], scene [n], scene_keys [S, d_e], w1 [h, 2 d_e] (columns
    0..d_e-1 act on v_e, the rest on e_img[j]), b1 [h].  Returns [n, h].
    """
    inp = np.concatenate([q, scene_keys[np.asarray(scene, dtype=np.int64)]], axis=1)
    z = inp @ w1.T + np.asarray(b1, dtype=np.float64)[None, :]
    return round_to_dtype(np.maximum(z, 0.0), dtype)


def relevance_logits(a: np.ndarray, w2: np.ndarray, b2: np.ndarray) -> np.ndarray:
    """Second layer of the MLP (Eq. 6): r_j = W2 a + b2, one logit per
    primitive.  a [n, h], w2 [P, h], b2 [P] -> [n, P]."""
    return a @ w2.T + np.asarray(b2, dtype=np.float64)[None, :]


def cosine(u: np.ndarray, v: np.ndarray) -> float:
    """cos(u, v) = <u, v> / (|u| |v|); 0 when either vector is zero."""
    nu = np.sqrt(np.dot(u, u))
    nv = np.sqrt(np.dot(v, v))
    if nu == 0 or nv == 0:
        return 0.0
    return float(np.dot(u, v) / (nu * nv))


def relevance_lookup(q: np.ndarray, scene: np.ndarray, a: np.ndarray, w2: np.ndarray,
                     b2: np.ndarray, prim_keys: np.ndarray, k: int):
    """Level-2 retrieval in the paper's form (Eq. 6-7): the top-k primitives
    of the token's scene by relevance logit (ties to the lowest p), weighted
    by the softmax over those k of cos(v_e, e_{j,p}) + tanh(r_j[p]).

    q [n, d_e], scene [n], a [n, h] (relevance_hidden), w2 [P, h], b2 [P],
    prim_keys [S, P, d_e].  Returns (prim [n, k] int32, w [n, k] float64,
    r_top [n, k] float64: the logits of the chosen primitives).
    """
    n = q.shape[0]
    P = prim_keys.shape[1]
    if not (1 <= k <= P):
        raise ValueError("k must be in [1, P]")
    r = relevance_logits(a, w2, b2)
    prim = np.zeros((n, k), dtype=np.int32)
    w = np.zeros((n, k), dtype=np.float64)
    r_top = np.zeros((n, k), dtype=np.float64)
    for t in range(n):
        idx = topk_order(r[t], k)
        rows = prim_keys[int(scene[t])][idx]
        z = np.array([cosine(q[t], rows[i]) for i in range(k)]) + np.tanh(r[t, idx])
        prim[t] = idx
        r_top[t] = r[t, idx]
        w[t] = softmax_weights(z)
    return prim, w, r_top


# ---------------------------------------------------------------------------
# Sparse injection with the SwiGLU fusion (Eq. 10)
# ---------------------------------------------------------------------------

def silu(x: np.ndarray) -> np.ndarray:
    """x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


def fusion(r: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray, w_down: np.ndarray,
           dtype: str) -> np.ndarray:
    """f in Eq. 10, a SwiGLU-style FFN from the retrieved width to the
    backbone width: f(R) = W_down (silu(W_gate R) * (W_up R)).

    r [m, d_v] (already rounded to dtype), w_gate and w_up [d_ff, d_v],
    w_down [d_h, d_ff].  The inner activations are rounded once to dtype
    before W_down.  Returns [m, d_h] float64 (not rounded)."""
    u = round_to_dtype(silu(r @ w_gate.T) * (r @ w_up.T), dtype)
    return u @ w_down.T


def inject_fused(hidden: np.ndarray, values: np.ndarray, P: int, scene: np.ndarray,
                 prim: np.ndarray, w: np.ndarray, kept: np.ndarray, w_gate: np.ndarray,
                 w_up: np.ndarray, w_down: np.ndarray, dtype: str) -> np.ndarray:
    """Sparse injection through the fusion (Eq. 10 and Eq. 2): for kept
    tokens H[t, :] <- round(H[t, :] + f(round(R_img[t]))); every other row is
    unchanged.  hidden [n, d_h], values [S*P, d_v]; returns float64."""
    out = np.array(hidden, dtype=np.float64, copy=True)
    kept = np.asarray(kept, dtype=np.int64)
    if kept.size == 0:
        return out
    R = np.stack([retrieved(values, P, int(scene[t]), prim[t], w[t]) for t in kept])
    F = fusion(round_to_dtype(R, dtype), w_gate, w_up, w_down, dtype)
    out[kept] = round_to_dtype(hidden[kept] + F, dtype)
    return out


# ---------------------------------------------------------------------------
# Learned SKA gate (Eq. 9), the text pathway (Sec. 3.2, ID lookup) and one
# whole LookME layer with its three pathways (Eq. 2, retrievals of Eq. 3)
# ---------------------------------------------------------------------------

def gate_logits(delta: np.ndarray, w_g: np.ndarray) -> np.ndarray:
    """Argument of the SKA gate (Eq. 9): z_i = Delta_i W_g, with W_g a
    single column of width d_c.  delta [n, d_c], w_g [d_c] -> [n]."""
    return delta @ np.asarray(w_g, dtype=np.float64)


def gate(delta: np.ndarray, w_g: np.ndarray, pos: np.ndarray | None = None) -> np.ndarray:
    """The SKA gate as it acts at inference (Eq. 9-10): the Gumbel-Sigmoid is
    hard and noise-free, so g_i = 1 exactly when sigma(z_i) > 1/2, i.e. when
    z_i > 0 (z_i = 0 stays closed).  The gate reads the rows of delta at the
    pathway's positions ``pos`` (all rows when None) and returns the indices
    i (into ``pos``) of the open gates in ascending order: the positions
    R[g] of Eq. 10 takes."""
    rows = delta if pos is None else delta[np.asarray(pos, dtype=np.int64)]
    return np.flatnonzero(gate_logits(rows, w_g) > 0).astype(np.int32)


def text_rows(table: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """Text pathway retrieval (Eq. 1 and Sec. 3.2 "Text embedding index-based
    lookup"): R_text = E_text[u], one table row per text token id."""
    return table[np.asarray(ids, dtype=np.int64)]


def inject_text(hidden: np.ndarray, table: np.ndarray, pos: np.ndarray, ids: np.ndarray,
                kept: np.ndarray, dtype: str) -> np.ndarray:
    """Sparse injection of the text pathway (Eq. 10 with the prefix add):
    for every open gate i, H[pos[i], :d_t] <- round(H[pos[i], :d_t] +
    E_text[ids[i]]); every other element unchanged.  hidden [n, d_h], table
    [V, d_t]; returns float64 values of dtype."""
    out = np.array(hidden, dtype=np.float64, copy=True)
    d_t = table.shape[1]
    pos = np.asarray(pos, dtype=np.int64)
    for i in np.asarray(kept, dtype=np.int64):
        t = pos[i]
        out[t, :d_t] = round_to_dtype(hidden[t, :d_t] + text_rows(table, [ids[i]])[0], dtype)
    return out


def lookme_layer(h_dec: np.ndarray, delta: np.ndarray, *, dtype: str, text=None, image=None,
                 cross=None):
    """One LookME layer (Eq. 2): H_out = L_dec(H_in) + S(R_text) + S(R_img)
    + S(R_cross), the pathways' sparse injections fused into the backbone
    one after another in that order, each a residual add rounded once to
    dtype.  Every pathway reads the layer's inputs, not a partly injected
    state: the image and cross-modal queries and all three gates are taken
    before the first add.

    h_dec [n, d_h]  L_dec(H_in), the decoder layer's output (float64 values)
    delta [n, d_c]  Delta = Attn(H_in), shared by the three gates (Eq. 9)
    text  = (pos [n_t], ids [n_t], table [V, d_t], w_g [d_c]): the text
            positions and their token ids (Sec. 3.2, text pathway)
    image = (start, x [n_i, d_in], w_t [d_e, d_in], scene_keys, prim_keys,
            values, k, w_g): image positions start .. start + n_i - 1, whose
            encoder embeddings x are projected and looked up (Eq. 4-7)
    cross = (w_t [d_e, d_h], scene_keys, prim_keys, values, k, w_g): every
            position, queried by its own h_dec row (Sec. 3.2, cross-modal
            pathway), against the pathway's own table
    A pathway given as None is absent.  Returns a dict with "hidden" and the
    per-pathway results (gates, scenes, primitives, weights)."""
    out = np.array(h_dec, dtype=np.float64, copy=True)
    res = {}
    plans = []
    if text is not None:
        pos, ids, table, w_g = text
        kept = gate(delta, w_g, pos)
        res["text_kept"] = kept
        plans.append(("text", pos, ids, table, kept))
    if image is not None:
        start, x, w_t, sk, pk, vals, k, w_g = image
        n_i = x.shape[0]
        q = project(x, w_t, dtype)
        sc = route(q, sk)
        pr, ww, _ = lookup(q, sc, pk, k)
        kept = gate(delta[start:start + n_i], w_g)
        res.update(img_q=q, img_scene=sc, img_prim=pr, img_w=ww, img_kept=kept)
        plans.append(("image", start, n_i, vals, sk.shape[0], pk.shape[1], sc, pr, ww, kept))
    if cross is not None:
        w_t, sk, pk, vals, k, w_g = cross
        q = project(h_dec, w_t, dtype)
        sc = route(q, sk)
        pr, ww, _ = lookup(q, sc, pk, k)
        kept = gate(delta, w_g)
        res.update(cross_q=q, cross_scene=sc, cross_prim=pr, cross_w=ww, cross_kept=kept)
        plans.append(("cross", vals, pk.shape[1], sc, pr, ww, kept))
    for plan in plans:
        if plan[0] == "text":
            _, pos, ids, table, kept = plan
            out = inject_text(out, table, pos, ids, kept, dtype)
        elif plan[0] == "image":
            _, start, n_i, vals, _, P, sc, pr, ww, kept = plan
            out[start:start + n_i] = inject(out[start:start + n_i], vals, P, sc, pr, ww, kept,
                                            dtype)
        else:
            _, vals, P, sc, pr, ww, kept = plan
            out = inject(out, vals, P, sc, pr, ww, kept, dtype)
    res["hidden"] = out
    return res
