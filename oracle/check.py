"""Tie- and rounding-aware comparison of library outputs with the oracle.
TEST INFRASTRUCTURE ONLY (used by the tests, the smoke check and the
benchmark's CPU leg; never by the library).

Every comparison recomputes the oracle's view with ``lookme_oracle`` on the
inputs the library saw for that stage (stage-wise checking): the scene is
checked on the library's q, the primitives under the library's scene, the
injected rows with the library's (kept, scene, prim).  Index results must be
identical except where the oracle's own float64 scores of the competing
choices tie within

    |a - b| <= 1e-5 * max(|a|, |b|) + 1e-7 * ||q_t||_2

(the relative part is the stated acceptance rule; the small absolute floor is
the size of a float32 summation error for scores near zero).  Each such
exemption is counted; more than 1% of decisions of one kind exempted fails the
check, so a systematic error cannot hide inside the tolerance.
"""

from __future__ import annotations

import dataclasses

import numpy as np

from . import lookme_oracle as O

REL_TIE = 1e-5
ABS_TIE_PER_QNORM = 1e-7
MAX_EXEMPT_FRACTION = 0.01


@dataclasses.dataclass
class Report:
    decisions: dict = dataclasses.field(default_factory=dict)
    exemptions: dict = dataclasses.field(default_factory=dict)
    failures: list = dataclasses.field(default_factory=list)
    notes: dict = dataclasses.field(default_factory=dict)

    def count(self, kind: str, n: int = 1):
        self.decisions[kind] = self.decisions.get(kind, 0) + n

    def exempt(self, kind: str, n: int = 1):
        self.exemptions[kind] = self.exemptions.get(kind, 0) + n

    def fail(self, msg: str):
        if len(self.failures) < 50:
            self.failures.append(msg)

    def finish(self) -> "Report":
        for kind, n in self.decisions.items():
            e = self.exemptions.get(kind, 0)
            if n > 0 and e > max(1, MAX_EXEMPT_FRACTION * n):
                self.fail(f"{kind}: {e} tie exemptions out of {n} decisions (> 1%)")
        return self

    @property
    def ok(self) -> bool:
        return not self.failures

    def __str__(self):
        return (f"decisions={self.decisions} exemptions={self.exemptions} "
                f"notes={self.notes} failures={self.failures[:10]}")


def tie(a: float, b: float, qnorm: float = 0.0) -> bool:
    return abs(a - b) <= REL_TIE * max(abs(a), abs(b)) + ABS_TIE_PER_QNORM * qnorm


# ---------------------------------------------------------------------------
# Rounding distance in units in the last place
# ---------------------------------------------------------------------------

def _mono_bf16(bits: np.ndarray) -> np.ndarray:
    b = np.asarray(bits).astype(np.int64) & 0xFFFF
    mag = b & 0x7FFF
    return np.where(b >> 15 == 1, -mag, mag)


def _mono_f32(x: np.ndarray) -> np.ndarray:
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.int64)
    mag = b & 0x7FFFFFFF
    return np.where(b >> 31 == 1, -mag, mag)


def ulp_distance(a: np.ndarray, b: np.ndarray, dtype: str) -> np.ndarray:
    """Distance in representable steps between stored values (bf16 bit
    patterns or float32 arrays)."""
    if dtype == "bf16":
        return np.abs(_mono_bf16(a) - _mono_bf16(b))
    return np.abs(_mono_f32(a) - _mono_f32(b))


# ---------------------------------------------------------------------------
# Evaluation intervals for chains of float32 products with rounded stores
# ---------------------------------------------------------------------------
#
# The fused, propagated and multi-scale injections (Eq. 8, 10, 11) evaluate
# several products in float32 and round intermediate rows (R, U, q, R^(k)) to
# the storage dtype before the next product reads them.  The checks below
# follow the library's value through that chain as an interval (centre c,
# radius r) that provably contains it, starting from exact float64 values:
#
#  * a float32 sum of K products of values known within (c, r) errs from the
#    exact product of the centres by at most |W| r + (K + 2) u |W| (|c| + r),
#    u = 2^-24 (recursive summation, any order, plus the input radius);
#  * a store to the dtype maps [c - r, c + r] to [round(c - r), round(c + r)]
#    (rounding is monotone), which also covers a rounding decision that the
#    float32 error moved across a midpoint;
#  * silu is 1.1-Lipschitz (its largest slope is 1.0998), and its float32
#    evaluation x / (1 + expf(-x)) errs by at most 8 u relative;
#  * a softmax whose inputs move by at most D moves each output by a factor
#    within [e^-2D, e^2D].
#
# The library's stored value must lie in the final interval.  In float32 the
# interval is a few units of the summed magnitudes times K u; in bf16 it is
# one or two bf16 steps wide where an intermediate rounding was close to a
# midpoint, and a single value elsewhere.

U32 = 2.0 ** -24


def _iv_round(c: np.ndarray, r: np.ndarray, dtype: str):
    lo = O.round_to_dtype(c - r, dtype)
    hi = O.round_to_dtype(c + r, dtype)
    return (lo + hi) / 2, (hi - lo) / 2


def _iv_matvec(w: np.ndarray, c: np.ndarray, r: np.ndarray):
    """W (rows = outputs) times a vector known within (c, r), float32."""
    aw = np.abs(w)
    return w @ c, aw @ r + (w.shape[1] + 2) * U32 * (aw @ (np.abs(c) + r))


def _iv_gather(w_lib: np.ndarray, V: np.ndarray, dtype: str):
    """R = round(sum_i w_i V_i), the library's weights, k float32 FMAs."""
    wv = np.asarray(w_lib, dtype=np.float64)[:, None] * V
    e = np.sum(wv, axis=0)
    E = (len(w_lib) + 1) * U32 * np.sum(np.abs(wv), axis=0)
    return _iv_round(e, E, dtype)


def _iv_swiglu(cR, rR, w_gate, w_up, dtype: str):
    """U = round(silu(W_gate R) * (W_up R)) as an interval."""
    cg, rg = _iv_matvec(w_gate, cR, rR)
    cu, ru = _iv_matvec(w_up, cR, rR)
    cs = O.silu(cg)
    rs = 1.1 * rg + 8 * U32 * (np.abs(cs) + 1.1 * rg)
    cp = cs * cu
    rp = (np.abs(cs) * ru + np.abs(cu) * rs + rs * ru
          + 2 * U32 * (np.abs(cs) + rs) * (np.abs(cu) + ru))
    return _iv_round(cp, rp, dtype)


def _iv_add_store(h: np.ndarray, cf, rf, dtype: str):
    """round(H + F) for F within (cf, rf), one float32 add: (lo, hi)."""
    e = h + cf
    E = rf + U32 * (np.abs(h) + np.abs(cf) + rf)
    return O.round_to_dtype(e - E, dtype), O.round_to_dtype(e + E, dtype)


# ---------------------------------------------------------------------------
# Stage checks
# ---------------------------------------------------------------------------

def check_scene_keys(keys_lib, prim_keys, dtype: str, rep: Report):
    """Eq. 4 scene-centred keys: the library's [S, d_e] against the oracle's
    exact mean of each scene's primitive keys (prim_keys [S, P, d_e] in the
    stored form of ``dtype``).  A float32 sum of P terms in any order errs by
    at most (P - 1) 2^-24 sum|x| and the division by P adds one rounding, so
    the stored key must lie between the roundings of mean -/+ E with
    E = (P + 1) 2^-24 (sum|x| / P + |mean|)."""
    pk = O.to_f64(np.asarray(prim_keys), dtype)
    P = pk.shape[1]
    mean = O.scene_keys_from_primitives(pk)
    E = (P + 1) * U32 * (np.sum(np.abs(pk), axis=1) / P + np.abs(mean))
    lo, hi = O.round_to_dtype(mean - E, dtype), O.round_to_dtype(mean + E, dtype)
    got = O.to_f64(keys_lib, dtype)
    rep.count("scene_key", got.shape[0])
    bad = (got < lo) | (got > hi)
    if np.any(bad):
        s, c = np.argwhere(bad)[0]
        rep.fail(f"scene key [{s}, {c}]: {got[s, c]!r} outside [{lo[s, c]!r}, {hi[s, c]!r}] "
                 f"(mean {mean[s, c]!r}); {int(bad.sum())} elements")


def check_q(q_lib, q_orc, dtype: str, rep: Report, max_ulp: int = 1):
    """C1 (exact copies): every element within ``max_ulp`` of the oracle's."""
    d = ulp_distance(q_lib, q_orc, dtype)
    rep.count("q", d.size)
    bad = int(np.sum(d > max_ulp))
    if bad:
        i = np.unravel_index(int(np.argmax(d)), d.shape)
        rep.fail(f"q: {bad} elements beyond {max_ulp} ulp (worst {int(d[i])} at {i})")
    return d


def check_projection(q_lib, x: np.ndarray, w_t: np.ndarray, dtype: str, rep: Report):
    """C1 (projection): the library accumulates x . w in float32 and rounds
    once to ``dtype``.  A float32 sum of d_in exact products differs from the
    exact sum by at most d_in * 2^-24 * sum_i |x_i w_i| (the standard
    recursive-summation bound), so the library's value must lie between the
    roundings of (exact - E) and (exact + E).  Most elements land on the
    correctly rounded value; the count of those that do not is reported."""
    exact = x @ w_t.T
    E = x.shape[1] * 2.0 ** -24 * (np.abs(x) @ np.abs(w_t).T)
    lo = O.round_to_dtype(exact - E, dtype)
    hi = O.round_to_dtype(exact + E, dtype)
    got = O.to_f64(q_lib, dtype)
    rep.count("q", got.size)
    bad = (got < lo) | (got > hi)
    if np.any(bad):
        i = np.unravel_index(int(np.argmax(bad)), bad.shape)
        rep.fail(f"q: {int(bad.sum())} elements outside the float32 accumulation bound "
                 f"(first at {i}: got {got[i]!r}, exact {exact[i]!r}, bound {E[i]!r})")
    off = int(np.sum(got != O.round_to_dtype(exact, dtype)))
    rep.notes["q_not_correctly_rounded"] = rep.notes.get("q_not_correctly_rounded", 0) + off
    return off


def check_scene(q: np.ndarray, scene_keys: np.ndarray, bias, score: str,
                scene_lib: np.ndarray, rep: Report, tokens=None):
    """C2: the library's scene is the oracle's arg max, or ties with it."""
    tokens = np.arange(q.shape[0]) if tokens is None else np.asarray(tokens)
    s1 = O.scene_scores(q[tokens], scene_keys, bias, score)
    best = np.argmax(s1, axis=1)
    for r, t in enumerate(tokens):
        g = int(scene_lib[t])
        rep.count("scene")
        if g < 0 or g >= scene_keys.shape[0]:
            rep.fail(f"scene[{t}]={g} out of range")
            continue
        b = int(best[r])
        if g == b:
            continue
        qn = float(np.linalg.norm(q[t]))
        if tie(s1[r, g], s1[r, b], qn):
            rep.exempt("scene")
        else:
            rep.fail(f"scene[{t}]: library {g} score {s1[r, g]!r}, oracle {b} score {s1[r, b]!r}")


def _check_topk_set(t, s2: np.ndarray, qn: float, g: np.ndarray, k: int, rep: Report):
    """C3 for one row: the listed k indices ``g`` against the exact scores
    ``s2``: the set equals the top k except for swaps among scores tied with
    the k-th, listed score-descending (exact ties by ascending index).
    Returns the scores of the listed set, or None after a failure."""
    P = s2.shape[0]
    rep.count("prim")
    if np.any(g < 0) or np.any(g >= P) or len(set(g.tolist())) != k:
        rep.fail(f"prim[{t}]={g.tolist()} invalid (P={P})")
        return None
    ref = O.topk_order(s2, k)
    kth = s2[ref[-1]]
    gs = s2[g]
    exempt = False
    # every listed element must reach the k-th score (up to a tie)
    for p, v in zip(g, gs):
        if v < kth and not tie(v, kth, qn):
            rep.fail(f"prim[{t}]: p={p} score {v!r} below k-th {kth!r}")
            return None
        if v < kth:
            exempt = True
    # every element strictly above the k-th score must be listed
    gset = set(g.tolist())
    for p in ref:
        if int(p) not in gset:
            if not tie(s2[p], kth, qn):
                rep.fail(f"prim[{t}]: missing p={p} score {s2[p]!r} (k-th {kth!r})")
                return None
            exempt = True
    # order: descending score, exact ties ascending index
    for i in range(k - 1):
        a, b = gs[i], gs[i + 1]
        if a < b and not tie(a, b, qn):
            rep.fail(f"prim[{t}]: order {g.tolist()} not descending")
            break
        if a == b and g[i] > g[i + 1]:
            rep.fail(f"prim[{t}]: equal scores not in ascending p order")
            break
    if exempt:
        rep.exempt("prim")
    return gs


def check_prim(q: np.ndarray, scene: np.ndarray, scene_prim_keys, k: int, score: str,
               prim_lib: np.ndarray, w_lib: np.ndarray, rep: Report, tokens=None,
               w_tol: float = 1e-5):
    """C3 + C4: the library's k primitives under the library's scene.

    ``scene_prim_keys(s)`` returns the float64 [P, d_e] keys of scene s.
    The set must equal the oracle's top-k except for swaps among scores tied
    with the k-th; the listed order must be score-descending (exact ties by
    ascending p); the weights must equal the softmax of the oracle's scores of
    the library's set within ``w_tol``.  Returns the oracle weights of the
    library's set, [len(tokens), k].
    """
    tokens = np.arange(q.shape[0]) if tokens is None else np.asarray(tokens)
    w_orc = np.zeros((len(tokens), k))
    cache = {}
    for r, t in enumerate(tokens):
        s = int(scene[t])
        if s not in cache:
            if len(cache) > 64:
                cache.clear()
            cache[s] = scene_prim_keys(s)
        keys = cache[s]
        P = keys.shape[0]
        s2 = O.primitive_scores(q[t], keys, score)
        qn = float(np.linalg.norm(q[t]))
        g = np.asarray(prim_lib[t], dtype=np.int64)
        gs = _check_topk_set(t, s2, qn, g, k, rep)
        if gs is None:
            continue
        wo = O.softmax_weights(gs)
        w_orc[r] = wo
        rep.count("w", k)
        dw = np.max(np.abs(np.asarray(w_lib[t], dtype=np.float64) - wo))
        if not dw <= w_tol:
            rep.fail(f"w[{t}]: max |dw| = {dw:.3g} > {w_tol}")
    return w_orc


def check_relevance_hidden(act_lib, q: np.ndarray, scene: np.ndarray, scene_keys: np.ndarray,
                           w1: np.ndarray, b1: np.ndarray, dtype: str, rep: Report):
    """C1 for the relevance MLP's hidden layer (Eq. 6): the library sums the
    2 d_e products of [q, e_img[scene]] and W1 plus b1 in float32 and applies
    ReLU and one rounding; with E the recursive-summation bound, its value
    must lie between the roundings of ReLU(exact - E) and ReLU(exact + E)."""
    inp = np.concatenate([q, scene_keys[np.asarray(scene, dtype=np.int64)]], axis=1)
    b = np.asarray(b1, dtype=np.float64)[None, :]
    exact = inp @ w1.T + b
    E = (inp.shape[1] + 1) * 2.0 ** -24 * (np.abs(inp) @ np.abs(w1).T + np.abs(b))
    lo = O.round_to_dtype(np.maximum(exact - E, 0.0), dtype)
    hi = O.round_to_dtype(np.maximum(exact + E, 0.0), dtype)
    got = O.to_f64(act_lib, dtype)
    rep.count("act", got.size)
    bad = (got < lo) | (got > hi)
    if np.any(bad):
        i = np.unravel_index(int(np.argmax(bad)), bad.shape)
        rep.fail(f"act: {int(bad.sum())} elements outside the float32 accumulation bound "
                 f"(first at {i}: got {got[i]!r}, exact {exact[i]!r}, bound {E[i]!r})")
    off = int(np.sum(got != O.round_to_dtype(np.maximum(exact, 0.0), dtype)))
    rep.notes["act_not_correctly_rounded"] = rep.notes.get("act_not_correctly_rounded", 0) + off


def check_relevance_prim(act: np.ndarray, w2: np.ndarray, b2: np.ndarray, q: np.ndarray,
                         scene: np.ndarray, scene_prim_keys, k: int, prim_lib: np.ndarray,
                         w_lib: np.ndarray, rep: Report, w_tol: float = 1e-5):
    """C3 + C4 for Level-2 in the paper's form (Eq. 6-7), on the library's
    hidden activations: the k primitives must be the top k of the logits
    W2 a + b2 (ties as in C3), and the weights the softmax over that set of
    cos(q, e_{j,p}) + tanh(r_p) within ``w_tol``.  Rows are those of the
    arguments (already sampled).  Returns the oracle weights of the library's
    sets, [rows, k]."""
    r_all = O.relevance_logits(act, w2, b2)
    w_orc = np.zeros((act.shape[0], k))
    for t in range(act.shape[0]):
        rn = float(np.linalg.norm(act[t]) * np.max(np.linalg.norm(w2, axis=1)))
        g = np.asarray(prim_lib[t], dtype=np.int64)
        gs = _check_topk_set(t, r_all[t], rn, g, k, rep)
        if gs is None:
            continue
        keys = scene_prim_keys(int(scene[t]))
        z = np.array([O.cosine(q[t], keys[p]) for p in g]) + np.tanh(gs)
        wo = O.softmax_weights(z)
        w_orc[t] = wo
        rep.count("w", k)
        dw = np.max(np.abs(np.asarray(w_lib[t], dtype=np.float64) - wo))
        if not dw <= w_tol:
            rep.fail(f"w[{t}]: max |dw| = {dw:.3g} > {w_tol}")
    return w_orc


def _check_contract(rep: Report, t, layer, err, got, exp, dtype: str, contract_abs: float,
                    magnitude):
    """The stated acceptance rule for injected hidden states: bf16 within
    ``contract_abs`` max-abs, float32 within 1e-5 of the summed magnitudes
    of the terms (the relative rule)."""
    if dtype == "bf16":
        bad = err > contract_abs
    else:
        bad = err > 1e-5 * magnitude
    if np.any(bad):
        c = int(np.argmax(np.where(bad, err, -1.0)))
        where = f"{t}, {c}" if layer is None else f"{layer}, {t}, {c}"
        rep.fail(f"hidden[{where}]: library {got[c]!r}, expected {exp[c]!r} (contract)")


def _check_interval(rep: Report, t, layer, got, lo, hi, what: str):
    bad = (got < lo) | (got > hi)
    if np.any(bad):
        c = int(np.argmax(bad))
        where = f"{t}" if layer is None else f"{layer}, {t}"
        rep.fail(f"hidden[{where}]: {int(bad.sum())} elements outside the float32 evaluation "
                 f"interval (first column {c}: {got[c]!r} not in [{lo[c]!r}, {hi[c]!r}])")
    rep.notes[f"{what}_interval_checked"] = rep.notes.get(f"{what}_interval_checked", 0) + 1


def _iv_multiscale(h_row, H, w_he, cR, rR, dtype: str):
    """Eq. 8 mix as the library evaluates it: q = round(H W_{h->e}) (float32
    over d_h), logits (q . R^m) * fl(1/sqrt(d_v)) in float32, softmax with the
    largest logit subtracted, sum_m alpha_m R^m by float32 FMAs, one rounded
    add into H.  cR, rR [M, d_v].  Returns (lo, hi) of the stored columns."""
    M, d_v = cR.shape
    cq, rq = _iv_round(*_iv_matvec(w_he.T, h_row, np.zeros_like(h_row)), dtype)
    s = 1.0 / np.sqrt(d_v)
    cz = (cR @ cq) * s
    mag = (np.abs(cR) + rR) @ (np.abs(cq) + rq)
    rz = s * ((np.abs(cR) @ rq) + (rR @ np.abs(cq)) + (rR @ rq)
              + (d_v + 2) * U32 * mag) + 4 * U32 * s * mag
    D = float(np.max(rz))
    ca = O.softmax_weights(cz)
    ra = ca * (np.expm1(2 * D) + (M + 6 + float(np.max(cz) - np.min(cz))) * U32)
    cy = ca @ cR
    ry = (ra @ np.abs(cR) + ca @ rR + ra @ rR
          + (M + 1) * U32 * ((ca + ra) @ (np.abs(cR) + rR)))
    return _iv_add_store(H, cy, ry, dtype)


def check_fused_hidden(h_in: np.ndarray, h_out_lib, dtype: str, values_rows, P: int,
                       scene: np.ndarray, prim: np.ndarray, w_lib: np.ndarray, kept: np.ndarray,
                       w_gate: np.ndarray, w_up: np.ndarray, w_down: np.ndarray, rep: Report,
                       tokens, contract_abs: float = 2e-2):
    """C6 through the SwiGLU fusion (Eq. 10), on the library's kept set,
    primitives and weights: rows outside the kept set keep their bits; kept
    rows must equal round(H + f(round(R))) within the contract (bf16:
    ``contract_abs`` max-abs; float32: 1e-5 * (|H| + |W_down| |U|), the
    relative rule on the summed magnitudes) and lie inside the evaluation
    interval of the library's float32 chain (see the interval helpers above:
    R, U and H + f(R) each rounded once).  h_in and h_out_lib hold the rows
    of ``tokens``."""
    kept_set = set(np.asarray(kept).tolist())
    h_in_f = O.to_f64(h_in, dtype)
    h_lib_f = O.to_f64(h_out_lib, dtype)
    for r, t in enumerate(np.asarray(tokens)):
        rep.count("hidden_row")
        if int(t) not in kept_set:
            if not np.array_equal(np.asarray(h_in[r]).view(np.uint8),
                                  np.asarray(h_out_lib[r]).view(np.uint8)):
                rep.fail(f"hidden: untouched row {t} modified")
            continue
        rows = int(scene[t]) * P + np.asarray(prim[t], dtype=np.int64)
        V = values_rows(rows)
        R = O.round_to_dtype(np.sum(np.asarray(w_lib[t], dtype=np.float64)[:, None] * V, axis=0),
                             dtype)
        U = O.round_to_dtype(O.silu(w_gate @ R) * (w_up @ R), dtype)
        F = w_down @ U
        exp = O.round_to_dtype(h_in_f[r] + F, dtype)
        err = np.abs(h_lib_f[r] - exp)
        _check_contract(rep, t, None, err, h_lib_f[r], exp, dtype, contract_abs,
                        np.abs(h_in_f[r]) + np.abs(w_down) @ np.abs(U))
        cR, rR = _iv_gather(w_lib[t], V, dtype)
        cU, rU = _iv_swiglu(cR, rR, w_gate, w_up, dtype)
        lo, hi = _iv_add_store(h_in_f[r], *_iv_matvec(w_down, cU, rU), dtype)
        _check_interval(rep, t, None, h_lib_f[r], lo, hi, "fused")
        rep.notes["fused_max_abs"] = max(rep.notes.get("fused_max_abs", 0.0), float(err.max()))


def check_propagated_hidden(h_in: np.ndarray, h_out_lib, dtype: str, values_rows, P: int,
                            scene: np.ndarray, prim: np.ndarray, w_lib: np.ndarray,
                            kept: np.ndarray, w_p: np.ndarray, w_gate: np.ndarray,
                            w_up: np.ndarray, w_down: np.ndarray, rep: Report, tokens,
                            contract_abs: float = 2e-2):
    """The LookME layer and the propagated layers after it (Eq. 10-11) on the
    library's kept set, primitives and weights of the LookME layer: in every
    layer j rows outside the kept set keep their bits, and kept rows equal
    round(H_j + f_j(R_j)) with R_0 = round(R), R_j = round(R_{j-1} W_p^j +
    R_{j-1}), within the contract and the evaluation interval of
    check_fused_hidden (the interval carried through the chain of R_j).
    h_in and h_out_lib
    hold [steps + 1, len(tokens), d_h]; w_p [steps, d_v, d_v] indexed
    [input, output]."""
    kept_set = set(np.asarray(kept).tolist())
    steps = w_p.shape[0]
    h_in_f = O.to_f64(h_in, dtype)
    h_lib_f = O.to_f64(h_out_lib, dtype)
    for r, t in enumerate(np.asarray(tokens)):
        rep.count("hidden_row", steps + 1)
        if int(t) not in kept_set:
            if not np.array_equal(np.asarray(h_in[:, r]).view(np.uint8),
                                  np.asarray(h_out_lib[:, r]).view(np.uint8)):
                rep.fail(f"hidden: untouched row {t} modified")
            continue
        rows = int(scene[t]) * P + np.asarray(prim[t], dtype=np.int64)
        V = values_rows(rows)
        R = O.round_to_dtype(np.sum(np.asarray(w_lib[t], dtype=np.float64)[:, None] * V, axis=0),
                             dtype)
        cR, rR = _iv_gather(w_lib[t], V, dtype)
        for j in range(steps + 1):
            if j > 0:
                R = O.round_to_dtype(R @ w_p[j - 1] + R, dtype)
                # R W_p (float32 over d_v) plus R, one float32 add, one store
                cm, rm = _iv_matvec(w_p[j - 1].T, cR, rR)
                cR, rR = _iv_round(cm + cR, rm + rR + U32 * (np.abs(cm) + rm + np.abs(cR) + rR),
                                   dtype)
            U = O.round_to_dtype(O.silu(w_gate[j] @ R) * (w_up[j] @ R), dtype)
            F = w_down[j] @ U
            exp = O.round_to_dtype(h_in_f[j, r] + F, dtype)
            err = np.abs(h_lib_f[j, r] - exp)
            _check_contract(rep, t, j, err, h_lib_f[j, r], exp, dtype, contract_abs,
                            np.abs(h_in_f[j, r]) + np.abs(w_down[j]) @ np.abs(U))
            cU, rU = _iv_swiglu(cR, rR, w_gate[j], w_up[j], dtype)
            lo, hi = _iv_add_store(h_in_f[j, r], *_iv_matvec(w_down[j], cU, rU), dtype)
            _check_interval(rep, t, j, h_lib_f[j, r], lo, hi, "propagated")
            rep.notes["propagated_max_abs"] = max(rep.notes.get("propagated_max_abs", 0.0),
                                                  float(err.max()))


def check_multiscale_hidden(h_in: np.ndarray, h_out_lib, dtype: str, values_rows, P: int,
                            scenes_per_scale: int, scene: np.ndarray, prim: np.ndarray,
                            w_lib: np.ndarray, kept: np.ndarray, w_he: np.ndarray, rep: Report,
                            tokens, contract_abs: float = 2e-2):
    """Multi-scale injection (Eq. 8) on the library's kept set and per-scale
    primitives and weights: rows outside the kept set, and columns from d_v
    on, keep their bits; the first d_v columns of kept rows equal
    round(H + mix(round(H W_{h->e}), [round(R^m)])) within the contract (bf16:
    ``contract_abs`` max-abs; float32: 1e-5 * (|H| + sum_m |R^m|)) and lie
    inside the evaluation interval of the library's chain (q and each R^m
    rounded once, float32 logits, softmax and mix, one rounded add).  scene,
    prim, w_lib [M, n, ...]; w_he [d_h, d_v]; h_in, h_out_lib hold the rows
    of ``tokens``."""
    kept_set = set(np.asarray(kept).tolist())
    M = scene.shape[0]
    d_v = w_he.shape[1]
    h_in_f = O.to_f64(h_in, dtype)
    h_lib_f = O.to_f64(h_out_lib, dtype)
    for r, t in enumerate(np.asarray(tokens)):
        rep.count("hidden_row")
        if int(t) not in kept_set:
            if not np.array_equal(np.asarray(h_in[r]).view(np.uint8),
                                  np.asarray(h_out_lib[r]).view(np.uint8)):
                rep.fail(f"hidden: untouched row {t} modified")
            continue
        if not np.array_equal(np.asarray(h_in[r, d_v:]).view(np.uint8),
                              np.asarray(h_out_lib[r, d_v:]).view(np.uint8)):
            rep.fail(f"hidden: row {t} modified past column {d_v}")
        R, cRs, rRs = [], [], []
        for m in range(M):
            rows = (m * scenes_per_scale + int(scene[m, t])) * P + np.asarray(prim[m, t],
                                                                              dtype=np.int64)
            Vm = values_rows(rows)
            R.append(O.round_to_dtype(
                np.sum(np.asarray(w_lib[m, t], dtype=np.float64)[:, None] * Vm, axis=0), dtype))
            cm, rm = _iv_gather(w_lib[m, t], Vm, dtype)
            cRs.append(cm)
            rRs.append(rm)
        R = np.stack(R)
        q = O.round_to_dtype(h_in_f[r] @ w_he, dtype)
        H = h_in_f[r, :d_v]
        exp = O.round_to_dtype(H + O.multiscale_mix(q, R), dtype)
        err = np.abs(h_lib_f[r, :d_v] - exp)
        _check_contract(rep, t, None, err, h_lib_f[r, :d_v], exp, dtype, contract_abs,
                        np.abs(H) + np.sum(np.abs(R), axis=0))
        lo, hi = _iv_multiscale(h_in_f[r], H, w_he, np.stack(cRs), np.stack(rRs), dtype)
        _check_interval(rep, t, None, h_lib_f[r, :d_v], lo, hi, "multiscale")
        rep.notes["multiscale_max_abs"] = max(rep.notes.get("multiscale_max_abs", 0.0),
                                              float(err.max()))


def check_kept(c: np.ndarray, n_keep: int, kept_lib: np.ndarray, rep: Report):
    """C5: the kept set equals the oracle's except for swaps among
    criticalities tied with the n_keep-th; ascending, unique, in range."""
    n = c.shape[0]
    kept_lib = np.asarray(kept_lib, dtype=np.int64)
    rep.count("kept", max(1, n_keep))
    if kept_lib.shape[0] != n_keep:
        rep.fail(f"kept: {kept_lib.shape[0]} entries, expected {n_keep}")
        return
    if n_keep == 0:
        return
    if np.any(kept_lib < 0) or np.any(kept_lib >= n):
        rep.fail("kept: token index out of range")
        return
    if np.any(np.diff(kept_lib) <= 0):
        rep.fail("kept: not strictly ascending")
        return
    ref = O.select(c, n_keep)
    if np.array_equal(ref, kept_lib):
        return
    cut = np.sort(c)[::-1][n_keep - 1]
    swaps = 0
    for t in np.setdiff1d(kept_lib, ref):
        if not tie(c[t], cut):
            rep.fail(f"kept: token {t} (c={c[t]!r}) kept below the cut {cut!r}")
            return
        swaps += 1
    for t in np.setdiff1d(ref, kept_lib):
        if not tie(c[t], cut):
            rep.fail(f"kept: token {t} (c={c[t]!r}) above the cut {cut!r} missing")
            return
    rep.exempt("kept", swaps)


def check_hidden(h_in: np.ndarray, h_out_lib, dtype: str, values_rows, P: int,
                 scene: np.ndarray, prim: np.ndarray, w_orc_of, kept: np.ndarray,
                 rep: Report, tokens=None, contract_abs: float = 2e-2, w_lib_of=None):
    """C6: recompute the injection with the library's (kept, scene, prim).

    * Untouched elements (tokens not kept, columns >= d_v) must keep their bits.
    * Contract, against the oracle's weights: bf16 within ``contract_abs``
      max-abs; float32 within 1e-5 * (|H| + sum_i w_i |V_i|).
    * Evaluation bound (bf16), when the library's weights are given: with
      e = H + sum_i w_lib_i V_i in exact arithmetic, a float32 evaluation
      (k fused multiply-adds, one add of H) errs by at most
      E = (k + 1) * 2^-24 * (|H| + sum_i |w_lib_i V_i|), so the stored value
      must lie between the roundings of e - E and e + E.  (A flat one-ulp rule
      is wrong where H + R cancels towards zero.)

    h_in, h_out_lib : stored arrays [n, d_h] (bf16 bits or float32), or the
                      rows for ``tokens`` when given.
    values_rows(rows) -> float64 [len(rows), d_v]
    w_orc_of(t) -> float64 [k] oracle weights of the library's set for t.
    w_lib_of(t) -> float32 [k] library weights for t (optional).
    """
    n = h_in.shape[0]
    tokens = np.arange(n) if tokens is None else np.asarray(tokens)
    kept_set = set(np.asarray(kept).tolist())
    h_in_f = O.to_f64(h_in, dtype)
    h_lib_f = O.to_f64(h_out_lib, dtype)
    worst = 0.0
    for r, t in enumerate(tokens):
        rep.count("hidden_row")
        if int(t) not in kept_set:
            same = (np.array_equal(np.asarray(h_in[r]).view(np.uint8),
                                   np.asarray(h_out_lib[r]).view(np.uint8)))
            if not same:
                rep.fail(f"hidden: untouched row {t} modified")
            continue
        rows = int(scene[t]) * P + np.asarray(prim[t], dtype=np.int64)
        V = values_rows(rows)
        d_v = V.shape[1]
        w = w_orc_of(int(t))
        H = h_in_f[r, :d_v]
        exact = H + np.sum(w[:, None] * V, axis=0)
        got = h_lib_f[r, :d_v]
        if not np.array_equal(np.asarray(h_in[r, d_v:]).view(np.uint8),
                              np.asarray(h_out_lib[r, d_v:]).view(np.uint8)):
            rep.fail(f"hidden: row {t} columns >= d_v modified")
        if dtype == "bf16":
            err = float(np.max(np.abs(got - O.round_to_dtype(exact, dtype))))
            worst = max(worst, err)
            if err > contract_abs:
                rep.fail(f"hidden[{t}]: max-abs {err:.3g} > {contract_abs}")
            if w_lib_of is not None:
                wl = np.asarray(w_lib_of(int(t)), dtype=np.float64)
                e = H + np.sum(wl[:, None] * V, axis=0)
                E = (len(wl) + 1) * 2.0 ** -24 * (np.abs(H) + np.sum(np.abs(wl[:, None] * V),
                                                                     axis=0))
                lo = O.round_to_dtype(e - E, dtype)
                hi = O.round_to_dtype(e + E, dtype)
                bad = (got < lo) | (got > hi)
                if np.any(bad):
                    rep.fail(f"hidden[{t}]: {int(bad.sum())} elements outside the float32 "
                             f"evaluation bound")
                off = int(np.sum(got != O.round_to_dtype(e, dtype)))
                rep.notes["hidden_not_correctly_rounded"] = (
                    rep.notes.get("hidden_not_correctly_rounded", 0) + off)
        else:
            bound = 1e-5 * (np.abs(H) + np.sum(np.abs(w[:, None] * V), axis=0))
            err = np.abs(got - exact)
            worst = max(worst, float(np.max(err)))
            if np.any(err > bound + 1e-30):
                rep.fail(f"hidden[{t}]: float32 error beyond 1e-5 relative")
    return worst


def check_end_to_end(x_rows: np.ndarray, w_t, scene_keys: np.ndarray, bias, score: str,
                     prim_keys, values_rows, P: int, k: int, crit: np.ndarray, n_keep: int,
                     h_in_rows, h_lib_rows, dtype: str, q_lib_rows, scene_lib: np.ndarray,
                     prim_lib: np.ndarray, w_lib: np.ndarray, kept_lib: np.ndarray,
                     rep: Report, tokens, contract_abs: float = 2e-2):
    """End-to-end mode: the oracle runs the whole path on the original inputs
    (its own q, scene, primitives, weights, kept set and hidden rows) and the
    library's final results are compared with it, one layer, on the rows of
    ``tokens``.

    * q: within the float32 accumulation bound of check_projection (or
      bit-identical without a projection).
    * Decisions (scene, primitive set, kept set) must equal the oracle's, a
      difference being allowed only where the oracle's own scores tie (C2,
      C3, C5).  Where the library's q differs from the oracle's (an element
      that is not the correctly rounded value, which the bound allows), the
      token's decisions are judged on the library's q instead and counted
      in the notes.
    * Weights, where the sets agree: within 1e-5 of the oracle's, paired by
      primitive.
    * Hidden rows: rows kept by neither keep their bits; rows kept by both
      with identical decisions equal the oracle's final row within the
      contract (bf16: ``contract_abs`` max-abs and one bf16 step; float32:
      1e-5 of |H| + sum w |V|).  A row whose decisions differ by an exempted
      tie is counted as an exemption of kind "e2e_hidden" (the 1% rule
      applies).

    x_rows [rows, d_in] float64 (the tokens' inputs), w_t [d_e, d_in] or
    None; prim_keys indexable by scene (float64 [P, d_e]); crit [n] the
    criticalities of every token of the layer (the kept set is global);
    h_in_rows / h_lib_rows / q_lib_rows stored rows of ``tokens``;
    scene_lib, prim_lib, w_lib indexed by token; kept_lib the library's
    kept list of the layer.
    """
    toks = np.asarray(tokens, dtype=np.int64)
    q_o = O.project(x_rows, w_t, dtype)
    if w_t is not None:
        check_projection(q_lib_rows, x_rows, w_t, dtype, rep)
    else:
        check_q(q_lib_rows, O.from_f64(q_o, dtype), dtype, rep, max_ulp=0)
    q_lib = O.to_f64(q_lib_rows, dtype)
    kept_o = O.select(crit, n_keep)
    check_kept(crit, n_keep, kept_lib, rep)
    kept_o_set = set(kept_o.tolist())
    kept_l_set = set(np.asarray(kept_lib, dtype=np.int64).tolist())
    h_in_f = O.to_f64(h_in_rows, dtype)
    h_lib_f = O.to_f64(h_lib_rows, dtype)
    n_qdiff = 0
    for r, t in enumerate(toks):
        t = int(t)
        rep.count("e2e_hidden")
        same_q = np.array_equal(q_lib[r], q_o[r])
        qv = q_o[r] if same_q else q_lib[r]
        n_qdiff += 0 if same_q else 1
        qn = float(np.linalg.norm(qv))
        # Level-1
        s1 = O.scene_scores(qv[None], scene_keys, bias, score)[0]
        sc_o = int(np.argmax(s1))
        g = int(scene_lib[t])
        rep.count("scene")
        if not 0 <= g < scene_keys.shape[0]:
            rep.fail(f"e2e scene[{t}]={g} out of range")
            continue
        decisions_same = True
        if g != sc_o:
            if not tie(s1[g], s1[sc_o], qn):
                rep.fail(f"e2e scene[{t}]: library {g} ({s1[g]!r}), oracle {sc_o} "
                         f"({s1[sc_o]!r})")
                continue
            rep.exempt("scene")
            decisions_same = False
        # Level-2 under the library's scene (the oracle's, unless tie-exempted)
        s2 = O.primitive_scores(qv, prim_keys[g], score)
        pl = np.asarray(prim_lib[t], dtype=np.int64)
        gs = _check_topk_set(t, s2, qn, pl, k, rep)
        if gs is None:
            continue
        po = O.topk_order(s2, k)
        if set(pl.tolist()) != set(po.tolist()):
            decisions_same = False
        else:
            wo = dict(zip(po.tolist(), O.softmax_weights(s2[po]).tolist()))
            wl = np.asarray(w_lib[t], dtype=np.float64)
            rep.count("w", k)
            dw = max(abs(wl[i] - wo[int(p)]) for i, p in enumerate(pl))
            if not dw <= 1e-5:
                rep.fail(f"e2e w[{t}]: max |dw| = {dw:.3g}")
        # injection
        in_o, in_l = t in kept_o_set, t in kept_l_set
        if in_o != in_l:
            decisions_same = False      # a kept-set swap already judged by check_kept
        if not in_l and not in_o:
            if not np.array_equal(np.asarray(h_in_rows[r]).view(np.uint8),
                                  np.asarray(h_lib_rows[r]).view(np.uint8)):
                rep.fail(f"e2e hidden: untouched row {t} modified")
            continue
        if not decisions_same:
            rep.exempt("e2e_hidden")
            continue
        Vo = values_rows(g * P + po)
        wvec = O.softmax_weights(s2[po])
        d_v = Vo.shape[1]
        H = h_in_f[r, :d_v]
        exact = H + np.sum(wvec[:, None] * Vo, axis=0)
        want = O.round_to_dtype(exact, dtype)
        got = h_lib_f[r, :d_v]
        if not np.array_equal(np.asarray(h_in_rows[r, d_v:]).view(np.uint8),
                              np.asarray(h_lib_rows[r, d_v:]).view(np.uint8)):
            rep.fail(f"e2e hidden: row {t} columns >= d_v modified")
        if dtype == "bf16":
            err = float(np.max(np.abs(got - want)))
            steps = int(np.max(ulp_distance(O.from_f64(got, dtype), O.from_f64(want, dtype),
                                            dtype)))
            if err > contract_abs or steps > 1:
                rep.fail(f"e2e hidden[{t}]: max-abs {err:.3g}, {steps} bf16 steps from the "
                         f"oracle's row")
        else:
            bound = 1e-5 * (np.abs(H) + np.sum(np.abs(wvec[:, None] * Vo), axis=0))
            if np.any(np.abs(got - exact) > bound):
                rep.fail(f"e2e hidden[{t}]: float32 error beyond 1e-5 relative")
    rep.notes["e2e_q_not_oracle"] = rep.notes.get("e2e_q_not_oracle", 0) + n_qdiff


def check_gate(delta: np.ndarray, w_g: np.ndarray, kept_lib, rep: Report, pos=None):
    """The learned SKA gate (Eq. 9): the library's open set equals the
    oracle's {i : Delta_i . W_g > 0} except for gates whose logit lies within
    the tie band of zero, |z_i| <= 1e-5 * sum_j |Delta_ij W_g,j| (the relative
    rule applied to the size of the summed terms), each counted as an
    exemption; strictly ascending and in range.

    delta [rows, d_c] float64 (the rows the gate reads are delta[pos] when pos
    is given); kept_lib the library's open indices (its first count entries).
    """
    rows = delta if pos is None else delta[np.asarray(pos, dtype=np.int64)]
    n = rows.shape[0]
    kept_lib = np.asarray(kept_lib, dtype=np.int64)
    rep.count("gate", max(1, n))
    if kept_lib.size and (np.any(kept_lib < 0) or np.any(kept_lib >= n)):
        rep.fail("gate: index out of range")
        return
    if np.any(np.diff(kept_lib) <= 0):
        rep.fail("gate: not strictly ascending")
        return
    ref = O.gate(rows, w_g)
    if np.array_equal(ref, kept_lib):
        return
    z = O.gate_logits(rows, w_g)
    band = REL_TIE * (np.abs(rows) @ np.abs(np.asarray(w_g, dtype=np.float64)))
    diff = np.setxor1d(ref, kept_lib)
    for i in diff:
        if abs(z[i]) > band[i]:
            rep.fail(f"gate: row {i} (z={z[i]!r}) {'opened' if i in kept_lib else 'closed'} "
                     f"against the oracle")
            return
    rep.exempt("gate", int(diff.size))


def check_text_hidden(h_in: np.ndarray, h_out_lib, dtype: str, table: np.ndarray, pos, ids,
                      kept, rep: Report, contract_abs: float = 2e-2):
    """The text pathway's injection (Eq. 1, Eq. 10) recomputed with the
    library's open set: rows not at an open text position keep their bits,
    columns >= d_t keep their bits, and the sum H + E_text[u] (exact in
    float64) must come back correctly rounded: a float32 addition of two
    stored values rounds once, so bf16 results may differ from the direct
    rounding only where the float32 sum was itself inexact (counted in the
    notes, bounded by the contract) and float32 results must be bit-exact."""
    h_in_f = O.to_f64(h_in, dtype)
    h_lib_f = O.to_f64(h_out_lib, dtype)
    d_t = table.shape[1]
    touched = {int(pos[i]): int(ids[i]) for i in np.asarray(kept, dtype=np.int64)}
    for t in range(h_in.shape[0]):
        rep.count("text_row")
        if t not in touched:
            if not np.array_equal(np.asarray(h_in[t]).view(np.uint8),
                                  np.asarray(h_out_lib[t]).view(np.uint8)):
                rep.fail(f"text: untouched row {t} modified")
            continue
        if not np.array_equal(np.asarray(h_in[t, d_t:]).view(np.uint8),
                              np.asarray(h_out_lib[t, d_t:]).view(np.uint8)):
            rep.fail(f"text: row {t} columns >= d_t modified")
        exact = h_in_f[t, :d_t] + table[touched[t]]
        want = O.round_to_dtype(exact, dtype)
        got = h_lib_f[t, :d_t]
        if dtype == "f32":
            if not np.array_equal(got, want):
                rep.fail(f"text: row {t} differs from the correctly rounded float32 sum")
        else:
            err = float(np.max(np.abs(got - want)))
            if err > contract_abs:
                rep.fail(f"text: row {t} max-abs {err:.3g} > {contract_abs}")
            s32 = exact.astype(np.float32).astype(np.float64)
            ok = (got == want) | (got == O.round_to_dtype(s32, dtype))
            if not np.all(ok):
                rep.fail(f"text: row {t}: {int((~ok).sum())} elements neither the direct nor "
                         f"the float32-then-bf16 rounding")
            rep.notes["text_double_rounded"] = (rep.notes.get("text_double_rounded", 0)
                                                + int(np.sum(got != want)))
