"""Pins of the CPU oracle against facts that do not come from the oracle
itself: a hand-derived worked example, closed forms, library routines,
exact rational brute force and invariants (arXiv 2607.16305, Sec. 3.2-3.3).

Each test names the mistake it is there to catch.
"""

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import brute as B
from oracle import lookme_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bf16_values(rng, shape, scale=1.0):
    """Random float64 values that are exactly bfloat16 numbers."""
    return O.round_to_bf16(rng.standard_normal(shape) * scale)


def _unit(rng, shape):
    a = rng.standard_normal(shape)
    return a / np.linalg.norm(a, axis=-1, keepdims=True)


# --------------------------------------------------------------------------
# Number formats
# --------------------------------------------------------------------------

def test_round_bf16_matches_torch_on_float32_inputs():
    """Catches a wrong rounding rule: for values that are exact binary32
    numbers, direct rounding to bf16 must equal torch's fp32->bf16 (RNE)."""
    rng = np.random.default_rng(1)
    x = np.concatenate([
        rng.standard_normal(20000),
        rng.standard_normal(2000) * 1e-38,     # binary32 subnormal range
        rng.standard_normal(2000) * 1e30,
        np.array([0.0, -0.0, 1.0, -1.0]),
    ]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.round_to_bf16(x.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


def test_round_bf16_ties_to_even_and_no_double_rounding():
    """Catches round-half-up, truncation and rounding through binary32."""
    e = 2.0 ** -8
    assert O.round_to_bf16(np.array([1 + e]))[0] == 1.0               # tie -> even
    assert O.round_to_bf16(np.array([1 + 3 * e]))[0] == 1 + 2 ** -6    # tie -> even
    assert O.round_to_bf16(np.array([-(1 + 3 * e)]))[0] == -(1 + 2 ** -6)
    # just above the midpoint: binary32 would round to the midpoint first and
    # then tie to 1.0; the correct result is the upper neighbour.
    v = 1 + e + 2.0 ** -30
    assert np.float32(v) == np.float32(1 + e)
    assert O.round_to_bf16(np.array([v]))[0] == 1 + 2 ** -7


def test_round_bf16_matches_exact_rational_rounding():
    """Two independent roundings (float64 scaling vs exact Fractions)."""
    rng = np.random.default_rng(2)
    x = np.concatenate([rng.standard_normal(3000) * 10.0 ** rng.integers(-40, 38, 3000)])
    got = O.round_to_bf16(x)
    for a, g in zip(x, got):
        assert Fraction(float(g)) == B.round_bf16(Fraction(float(a)))


def test_round_f32_matches_exact_rational_rounding():
    rng = np.random.default_rng(3)
    x = rng.standard_normal(3000) * 10.0 ** rng.integers(-30, 30, 3000)
    got = O.round_to_dtype(x, "f32")
    for a, g in zip(x, got):
        assert Fraction(float(g)) == B.round_f32(Fraction(float(a)))


def test_bf16_bits_roundtrip():
    rng = np.random.default_rng(4)
    bits = rng.integers(0, 1 << 16, 5000).astype(np.uint16)
    vals = O.bf16_bits_to_f64(bits)
    fin = np.isfinite(vals)
    back = O.f64_to_bf16_bits(vals[fin])
    np.testing.assert_array_equal(back, bits[fin])
    # against torch's own reinterpretation of the same bits
    t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(vals[fin], t[fin])


# --------------------------------------------------------------------------
# Worked example (hand-derived, tests/golden)
# --------------------------------------------------------------------------

def _softmax_closed(scores):
    ex = [math.exp(s - max(scores)) for s in scores]
    return [e / sum(ex) for e in ex]


def test_worked_example():
    """Catches wrong tie-breaks (scene, primitive and token), a wrong table
    row index s*P + p, and a wrong weight formula."""
    with open(os.path.join(GOLDEN, "worked_example_s2_p3.json")) as f:
        g = json.load(f)
    q = np.array(g["queries"], dtype=np.float64)
    K1 = np.array(g["scene_keys"], dtype=np.float64)
    K2 = np.array(g["prim_keys"], dtype=np.float64)
    V = np.array(g["values"], dtype=np.float64)
    H = np.array(g["hidden"], dtype=np.float64)
    D = np.array(g["delta"], dtype=np.float64)
    k, n_keep = g["k"], g["n_keep"]
    exp = g["expected"]

    scene = O.route(q, K1)
    assert scene.tolist() == exp["scene"]
    prim, w, top = O.lookup(q, scene, K2, k)
    assert prim.tolist() == exp["prim"]
    np.testing.assert_array_equal(top, np.array(exp["top_scores"], dtype=np.float64))
    for t in range(4):
        np.testing.assert_allclose(w[t], _softmax_closed(exp["top_scores"][t]), rtol=1e-15)
    kept = O.select(O.criticality(D), n_keep)
    assert kept.tolist() == exp["kept"]
    out = O.inject(H, V, K2.shape[1], scene, prim, w, kept, "f32")
    for t in range(4):
        if t in exp["kept"]:
            ws = _softmax_closed(exp["top_scores"][t])
            r = [sum(ws[i] * V[exp["rows"][t][i]][j] for i in range(k)) for j in range(2)]
            np.testing.assert_array_equal(out[t], np.float32(r).astype(np.float64))
        else:
            np.testing.assert_array_equal(out[t], H[t])
    # t1 lives in scene 1: its rows are V[3*1 + 1] and V[3*1 + 0]
    np.testing.assert_allclose(out[1], [4 - w[1, 1], 40 - 10 * w[1, 1]], rtol=1e-6)


# --------------------------------------------------------------------------
# Projection
# --------------------------------------------------------------------------

def test_project_matches_exact_rational_brute_force():
    """Catches a transposed W (d_in != d_e), a missing rounding and a wrong
    rounding point."""
    rng = np.random.default_rng(10)
    n, d_in, d_e = 5, 7, 3
    x = _bf16_values(rng, (n, d_in))
    wt = _bf16_values(rng, (d_e, d_in), 0.3)
    q = O.project(x, wt, "bf16")
    ref = B.project(x.tolist(), wt.tolist(), B.round_bf16)
    assert q.shape == (n, d_e)
    for t in range(n):
        for j in range(d_e):
            assert Fraction(float(q[t, j])) == ref[t][j]


def test_project_one_hot_tokens_pick_columns():
    """Closed form: token e_i projects to column i of W (row i of W^T...)."""
    rng = np.random.default_rng(11)
    d_in, d_e = 6, 4
    wt = _bf16_values(rng, (d_e, d_in))
    x = np.eye(d_in)
    q = O.project(x, wt, "bf16")
    np.testing.assert_array_equal(q, wt.T)


def test_project_without_weights_is_identity():
    x = np.arange(12, dtype=np.float64).reshape(3, 4)
    np.testing.assert_array_equal(O.project(x, None, "f32"), x)


# --------------------------------------------------------------------------
# Level-1 routing (Eq. 5)
# --------------------------------------------------------------------------

def test_route_matches_brute_force():
    rng = np.random.default_rng(20)
    n, S, d = 40, 9, 8
    q = _bf16_values(rng, (n, d))
    K1 = O.round_to_bf16(_unit(rng, (S, d)))
    b = rng.standard_normal(S) * 0.1
    assert O.route(q, K1, b).tolist() == B.route(q.tolist(), K1.tolist(), b.tolist())
    assert O.route(q, K1).tolist() == B.route(q.tolist(), K1.tolist())


def test_route_exact_integer_ties_go_to_lowest_scene():
    """Catches highest-index or arbitrary tie-breaks."""
    K1 = np.array([[1, 0, 0], [0, 1, 0], [1, 0, 0], [0, 1, 0]], dtype=np.float64)
    q = np.array([[2, 2, 0], [0, 3, 1], [5, 1, 9]], dtype=np.float64)
    assert O.route(q, K1).tolist() == [0, 1, 0]


def test_route_bias_sign():
    """Catches a subtracted (rather than added) bias."""
    K1 = np.eye(2)
    q = np.array([[1.0, 2.0]])
    assert O.route(q, K1).tolist() == [1]
    assert O.route(q, K1, np.array([1.5, 0.0])).tolist() == [0]
    assert O.route(q, K1, np.array([0.0, -1.5])).tolist() == [0]


def test_route_planted_clusters_and_single_scene():
    rng = np.random.default_rng(21)
    S, d = 12, 32
    K1 = _unit(rng, (S, d))
    labels = rng.integers(0, S, 200)
    q = 5.0 * K1[labels] + 0.05 * rng.standard_normal((200, d))
    assert np.array_equal(O.route(q, K1), labels)
    assert O.route(q, K1[:1]).tolist() == [0] * 200


def test_route_cos_equals_dot_for_unit_keys_without_bias():
    """A positive per-token scale preserves the arg max."""
    rng = np.random.default_rng(22)
    K1 = _unit(rng, (30, 16))
    q = rng.standard_normal((50, 16)) * rng.uniform(0.1, 10, (50, 1))
    assert np.array_equal(O.route(q, K1, score="cos"), O.route(q, K1, score="dot"))


# --------------------------------------------------------------------------
# Cosine scoring (Eq. 5 and Eq. 7 in the paper's own cosine form)
# --------------------------------------------------------------------------

# integer patterns whose Euclidean norm is an integer (Pythagorean
# quadruples and quintuples): a vector made of one of them, scaled by an exact
# binary fraction, has a rational norm, so every cosine between two such
# vectors is an exact rational
_RATIONAL_NORM_PATTERNS = [(1, 2, 2), (2, 3, 6), (1, 4, 8), (4, 4, 7), (2, 6, 9), (6, 6, 7),
                           (3, 4, 12), (2, 10, 11), (1, 12, 12), (8, 9, 12), (1, 1, 1, 1),
                           (1, 1, 3, 5), (2, 4, 5, 6), (1, 2, 4, 10)]
_SCALES = (0.25, 0.5, 0.75, 1.0, 1.5, 2.0, 3.0, 5.0)


def _rational_norm_rows(rng, n, d, zero_rows=()):
    """n rows of width d, each one pattern with random signs at random
    positions times a random scale (exact in bf16); rows in ``zero_rows``
    are zero.  Norms are rational and deliberately uneven."""
    out = np.zeros((n, d))
    for i in range(n):
        if i in zero_rows:
            continue
        pat = _RATIONAL_NORM_PATTERNS[rng.integers(len(_RATIONAL_NORM_PATTERNS))]
        pos = rng.choice(d, len(pat), replace=False)
        out[i, pos] = np.array(pat) * rng.choice([-1.0, 1.0], len(pat))
        out[i] *= _SCALES[rng.integers(len(_SCALES))]
    assert np.array_equal(out, O.round_to_bf16(out))
    return out


def _exact_gap_ok(vals, i, j):
    """True when the exact rationals vals[i] and vals[j] differ by more than
    float64 can blur (no exact or near tie decided by rounding)."""
    return abs(vals[i] - vals[j]) > Fraction(1, 10 ** 9)


def _pin_cos_route():
    """Level-1 under the cosine with a scene bias (Eq. 5) against exact
    rationals, with queries and keys of uneven norms, a zero query and a zero
    key.  Every decision whose runner-up is not within 1e-9 must match."""
    rng = np.random.default_rng(120)
    n, S, d = 60, 9, 8
    q = _rational_norm_rows(rng, n, d, zero_rows=(7,))
    K1 = _rational_norm_rows(rng, S, d, zero_rows=(4,))
    b = rng.permutation(np.arange(-4, 5)) / 16.0        # distinct, exact
    got = O.route(q, K1, b, score="cos")
    want, rows = B.route_cos(q.tolist(), K1.tolist(), b.tolist())
    checked = 0
    for t in range(n):
        order = sorted(range(S), key=lambda s: (-rows[t][s], s))
        if _exact_gap_ok(rows[t], order[0], order[1]):
            assert got[t] == want[t], (t, got[t], want[t])
            checked += 1
    assert checked >= n - 3
    # the zero query scores every scene with its bias alone
    assert got[7] == int(np.argmax(b))
    # the scores themselves, including cos = 0 for the zero key
    s1 = O.scene_scores(q, K1, b, score="cos")
    for t in range(n):
        np.testing.assert_allclose(s1[t], [float(v) for v in rows[t]], rtol=0, atol=1e-15)
    assert np.all(s1[:, 4] == b[4])
    return q, K1, b


def _pin_cos_lookup():
    """Level-2 under the cosine (Eq. 7): the top-k of exact cosines within the
    scene and the softmax over the k selected cosines, evaluated in 40-digit
    decimal arithmetic."""
    rng = np.random.default_rng(121)
    n, S, P, d, k = 30, 3, 12, 8, 4
    q = _rational_norm_rows(rng, n, d, zero_rows=(5,))
    K2 = np.stack([_rational_norm_rows(rng, P, d, zero_rows=(3,)) for _ in range(S)])
    scene = rng.integers(0, S, n).astype(np.int32)
    prim, w, top = O.lookup(q, scene, K2, k, score="cos")
    bp, btop, alls = B.lookup_cos(q.tolist(), scene.tolist(), K2.tolist(), k)
    checked = 0
    for t in range(n):
        c = alls[t]
        order = sorted(range(P), key=lambda p: (-c[p], p))
        # no near tie at any listed position or at the cut
        if t != 5 and all(_exact_gap_ok(c, order[i], order[i + 1]) for i in range(k)):
            assert prim[t].tolist() == bp[t], (t, prim[t].tolist(), bp[t])
            np.testing.assert_allclose(top[t], [float(v) for v in btop[t]], rtol=0, atol=1e-15)
            np.testing.assert_allclose(w[t], B.softmax_decimal(btop[t]), rtol=1e-14, atol=0)
            checked += 1
    assert checked >= n // 2
    # the zero query: every cosine is 0, so the first k primitives, equal weights
    assert prim[5].tolist() == list(range(k))
    assert w[5].tolist() == [1.0 / k] * k
    return q, scene, K2


def _pin_cos_planted_angles():
    """Closed form: keys at planted cosines beta_p to q with arbitrary norms
    c_p give top-k = the k largest beta and weights = softmax(beta) under the
    cosine, whatever c_p and |q|; under the dot product the weights are
    softmax(c_p beta_p |q|) instead."""
    rng = np.random.default_rng(122)
    d, P, k = 48, 16, 5
    q = rng.standard_normal(d) * 3.7
    qh = q / np.linalg.norm(q)
    betas = rng.permutation(np.linspace(-0.9, 0.9, P))
    norms = rng.uniform(0.1, 10.0, P)
    keys = np.zeros((P, d))
    for p in range(P):
        u = rng.standard_normal(d)
        u -= (u @ qh) * qh
        u /= np.linalg.norm(u)
        keys[p] = norms[p] * (betas[p] * qh + math.sqrt(1 - betas[p] ** 2) * u)
    prim, w, top = O.lookup(q[None], np.array([0]), keys[None], k, score="cos")
    expect = np.argsort(-betas)[:k]
    assert prim[0].tolist() == expect.tolist()
    np.testing.assert_allclose(top[0], betas[expect], rtol=0, atol=1e-14)
    bt = betas[expect]
    np.testing.assert_allclose(w[0], np.exp(bt - bt.max()) / np.exp(bt - bt.max()).sum(),
                               rtol=1e-13)
    _, wd, _ = O.lookup(q[None], np.array([0]), keys[None], k, score="dot")
    assert np.max(np.abs(wd[0] - w[0])) > 1e-2
    # routing: planted cosines plus a bias that reverses the two best
    K1 = keys[expect[:2]]
    gap = float(betas[expect[0]] - betas[expect[1]])
    assert O.route(q[None], K1, np.array([0.0, 0.0]), score="cos").tolist() == [0]
    assert O.route(q[None], K1, np.array([0.0, 1.5 * gap]), score="cos").tolist() == [1]
    assert O.route(q[None], K1, np.array([0.0, 0.5 * gap]), score="cos").tolist() == [0]


def _pin_cos_scale_invariance():
    """Scaling a query or a key by a positive factor leaves the cosine scores,
    the decisions and the weights unchanged, while the dot-product scores
    change."""
    rng = np.random.default_rng(123)
    n, S, P, d, k = 20, 6, 10, 16, 3
    q = rng.standard_normal((n, d))
    K1 = rng.standard_normal((S, d))
    K2 = rng.standard_normal((S, P, d))
    b = rng.standard_normal(S) * 0.1
    fq = rng.uniform(0.2, 8.0, (n, 1))
    fk1 = rng.uniform(0.2, 8.0, (S, 1))
    fk2 = rng.uniform(0.2, 8.0, (S, P, 1))
    s_a = O.scene_scores(q, K1, b, score="cos")
    s_b = O.scene_scores(q * fq, K1 * fk1, b, score="cos")
    np.testing.assert_allclose(s_a, s_b, rtol=0, atol=1e-14)
    assert np.max(np.abs(O.scene_scores(q, K1, b) - O.scene_scores(q * fq, K1 * fk1, b))) > 1e-3
    scene = O.route(q, K1, b, score="cos")
    assert np.array_equal(scene, O.route(q * fq, K1 * fk1, b, score="cos"))
    pa, wa, _ = O.lookup(q, scene, K2, k, score="cos")
    pb, wb, _ = O.lookup(q * fq, scene, K2 * fk2, k, score="cos")
    assert np.array_equal(pa, pb)
    np.testing.assert_allclose(wa, wb, rtol=0, atol=1e-14)
    _, wd1, _ = O.lookup(q, scene, K2, k, score="dot")
    _, wd2, _ = O.lookup(q * fq, scene, K2 * fk2, k, score="dot")
    assert np.max(np.abs(wd1 - wd2)) > 1e-3


_COS_PINS = (_pin_cos_route, _pin_cos_lookup, _pin_cos_planted_angles, _pin_cos_scale_invariance)


def test_route_cos_with_bias_matches_exact_rational_brute_force():
    """Catches a query or key left unnormalised, the bias folded into the
    cosine, and a zero vector not scoring 0."""
    q, K1, b = _pin_cos_route()
    # the pin discriminates: with these uneven norms the dot product routes
    # differently for many tokens
    assert np.sum(O.route(q, K1, b, score="dot") != O.route(q, K1, b, score="cos")) >= 10


def test_lookup_cos_matches_exact_rational_brute_force():
    q, scene, K2 = _pin_cos_lookup()
    pd, _, _ = O.lookup(q, scene, K2, 4, score="dot")
    pc, _, _ = O.lookup(q, scene, K2, 4, score="cos")
    assert np.sum(np.any(pd != pc, axis=1)) >= 5


def test_cos_planted_angles_closed_form():
    _pin_cos_planted_angles()


def test_cos_scale_invariance_and_dot_sensitivity():
    _pin_cos_scale_invariance()


def _mut_scene_scores_q_raw(q, scene_keys, bias=None, score="dot"):
    if score != "cos":
        return _REAL_SCENE_SCORES(q, scene_keys, bias, score)
    s = q @ O._unit_rows(scene_keys).T
    return s if bias is None else s + bias[None, :]


def _mut_scene_scores_k_raw(q, scene_keys, bias=None, score="dot"):
    if score != "cos":
        return _REAL_SCENE_SCORES(q, scene_keys, bias, score)
    s = O._unit_rows(q) @ scene_keys.T
    return s if bias is None else s + bias[None, :]


def _mut_scene_scores_bias_inside(q, scene_keys, bias=None, score="dot"):
    if score != "cos":
        return _REAL_SCENE_SCORES(q, scene_keys, bias, score)
    num = q @ scene_keys.T + (0.0 if bias is None else bias[None, :])
    nq = np.linalg.norm(q, axis=1)[:, None]
    nk = np.linalg.norm(scene_keys, axis=1)[None, :]
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.where((nq > 0) & (nk > 0), num / (nq * nk), 0.0)


def _mut_prim_scores_q_raw(q_t, prim_keys_s, score="dot"):
    if score != "cos":
        return _REAL_PRIM_SCORES(q_t, prim_keys_s, score)
    return O._unit_rows(prim_keys_s) @ q_t


def _mut_prim_scores_k_raw(q_t, prim_keys_s, score="dot"):
    if score != "cos":
        return _REAL_PRIM_SCORES(q_t, prim_keys_s, score)
    return prim_keys_s @ O._unit_rows(q_t[None, :])[0]


_REAL_SCENE_SCORES = O.scene_scores
_REAL_PRIM_SCORES = O.primitive_scores


@pytest.mark.parametrize("target,mutant", [
    ("scene_scores", _mut_scene_scores_q_raw),
    ("scene_scores", _mut_scene_scores_k_raw),
    ("scene_scores", _mut_scene_scores_bias_inside),
    ("primitive_scores", _mut_prim_scores_q_raw),
    ("primitive_scores", _mut_prim_scores_k_raw),
])
def test_cos_pins_kill_planted_mistakes(monkeypatch, target, mutant):
    """Each planted mistake in the oracle's cosine branch (query not
    normalised, keys not normalised, bias inside the cosine) makes at least
    one of the cosine pins fail."""
    monkeypatch.setattr(O, target, mutant)
    failed = 0
    for pin in _COS_PINS:
        try:
            pin()
        except AssertionError:
            failed += 1
    assert failed >= 1, f"no cosine pin catches the planted mistake {mutant.__name__}"


def test_scene_keys_are_primitive_means_eq4():
    """Eq. 4: e_img[j] = (1/N_p) sum_p E[j, p, :], against exact rationals
    (S != P != d catches a mean over the wrong axis), a scene of identical
    primitives (its key is that primitive) and invariance under relabelling
    the primitives of a scene."""
    rng = np.random.default_rng(124)
    S, P, d = 3, 7, 5
    E = _bf16_values(rng, (S, P, d))
    got = O.scene_keys_from_primitives(E)
    want = B.scene_means(E.reshape(S * P, d).tolist(), P)
    assert got.shape == (S, d)
    for j in range(S):
        np.testing.assert_allclose(got[j], [float(v) for v in want[j]], rtol=1e-15, atol=0)
    E2 = E.copy()
    E2[1] = E[1, 4]
    np.testing.assert_array_equal(O.scene_keys_from_primitives(E2)[1], E[1, 4])
    perm = rng.permutation(P)
    np.testing.assert_allclose(O.scene_keys_from_primitives(E[:, perm]), got, rtol=1e-15)


# --------------------------------------------------------------------------
# Level-2 lookup (Eq. 6-7, configured form)
# --------------------------------------------------------------------------

def test_lookup_equals_exhaustive_search_within_scene():
    """spec brute force: the two-level result equals an exhaustive top-k
    over the rows [s*P, (s+1)*P) of the chosen scene in the flat table.
    Catches a wrong scene offset and a transposed key operand (S != P != d)."""
    rng = np.random.default_rng(30)
    n, S, P, d, k = 25, 5, 11, 6, 4
    q = _bf16_values(rng, (n, d))
    K2 = O.round_to_bf16(_unit(rng, (S, P, d)))
    scene = rng.integers(0, S, n).astype(np.int32)
    prim, w, top = O.lookup(q, scene, K2, k)
    bp, btop = B.lookup_flat_sim(q.tolist(), scene.tolist(), K2.reshape(S * P, d).tolist(), P, k)
    assert prim.tolist() == bp
    for t in range(n):
        assert [Fraction(float(v)) for v in top[t]] == btop[t]
        np.testing.assert_allclose(w[t], B.softmax(btop[t]), rtol=1e-14)


def test_lookup_planted_ranking():
    """Keys at known angles to q: the top-k and the weights are known."""
    rng = np.random.default_rng(31)
    d, P, k = 64, 20, 5
    q = rng.standard_normal(d)
    qh = q / np.linalg.norm(q)
    betas = rng.permutation(np.linspace(-0.9, 0.95, P))
    keys = np.zeros((P, d))
    for p in range(P):
        u = rng.standard_normal(d)
        u -= (u @ qh) * qh
        u /= np.linalg.norm(u)
        keys[p] = betas[p] * qh + math.sqrt(1 - betas[p] ** 2) * u
    prim, w, top = O.lookup(q[None], np.array([0]), keys[None], k)
    expect = np.argsort(-betas)[:k]
    assert prim[0].tolist() == expect.tolist()
    s = betas[expect] * np.linalg.norm(q)
    np.testing.assert_allclose(top[0], s, rtol=1e-12)
    np.testing.assert_allclose(w[0], np.exp(s - s.max()) / np.exp(s - s.max()).sum(), rtol=1e-12)


def test_lookup_k_equals_p_and_integer_ties():
    """k = P lists every primitive; exact ties list the lower p first."""
    K2 = np.array([[[1, 0], [0, 1], [1, 0], [2, 0], [0, 1]]], dtype=np.float64)
    q = np.array([[1.0, 1.0]])
    prim, w, top = O.lookup(q, np.array([0]), K2, 5)
    # scores 1, 1, 1, 2, 1 -> 3 first, then 0, 1, 2, 4 in index order
    assert prim[0].tolist() == [3, 0, 1, 2, 4]
    prim, _, _ = O.lookup(q, np.array([0]), K2, 2)
    assert prim[0].tolist() == [3, 0]


def test_lookup_many_exact_ties_against_brute_force():
    """Integer keys with few distinct scores over P = 300: an unstable sort
    (e.g. an introsort on long arrays) would list tied primitives out of
    index order."""
    rng = np.random.default_rng(32)
    P, d, k = 300, 4, 40
    K2 = rng.integers(-1, 2, (1, P, d)).astype(np.float64)
    q = rng.integers(-2, 3, (3, d)).astype(np.float64)
    prim, _, top = O.lookup(q, np.zeros(3, dtype=np.int32), K2, k)
    bp, btop = B.lookup_flat_sim(q.tolist(), [0, 0, 0], K2[0].tolist(), P, k)
    assert prim.tolist() == bp


def test_softmax_closed_forms():
    """k = 1 gives exactly 1; equal scores give exactly 1/k; ln3 vs 0 gives
    3/4 and 1/4; huge scores do not overflow (max subtracted)."""
    assert O.softmax_weights(np.array([7.25])).tolist() == [1.0]
    assert O.softmax_weights(np.array([2.0] * 4)).tolist() == [0.25] * 4
    np.testing.assert_allclose(O.softmax_weights(np.array([math.log(3), 0.0])), [0.75, 0.25],
                               rtol=1e-15)
    w = O.softmax_weights(np.array([1000.0, 999.0]))
    np.testing.assert_allclose(w, [1 / (1 + math.exp(-1)), math.exp(-1) / (1 + math.exp(-1))])
    assert abs(O.softmax_weights(np.random.default_rng(0).standard_normal(16)).sum() - 1) < 1e-15


# --------------------------------------------------------------------------
# Criticality select (Eq. 9-10, configured gate)
# --------------------------------------------------------------------------

def test_select_matches_brute_force_and_is_ascending():
    rng = np.random.default_rng(40)
    D = rng.standard_normal((60, 9)) * rng.lognormal(size=(60, 1))
    c = O.criticality(D)
    nsq = [sum(Fraction(float(v)) ** 2 for v in row) for row in D]
    for n_keep in (0, 1, 7, 30, 60):
        assert O.select(c, n_keep).tolist() == B.select(nsq, n_keep)


def test_select_planted_and_ties():
    """Planted norms gamma_t e_1; equal norms keep the lowest indices.
    Catches keeping the smallest instead of the largest."""
    gam = np.array([3.0, 9.0, 1.0, 7.0, 5.0])
    D = np.zeros((5, 4))
    D[:, 0] = gam
    assert O.select(O.criticality(D), 2).tolist() == [1, 3]
    assert O.select(O.criticality(-D), 3).tolist() == [1, 3, 4]
    E = np.ones((6, 3))
    assert O.select(O.criticality(E), 4).tolist() == [0, 1, 2, 3]
    # long arrays with few distinct norms: ties must still keep low indices
    rng = np.random.default_rng(41)
    F = rng.integers(0, 3, (500, 2)).astype(np.float64)
    nsq = [int(a * a + b * b) for a, b in F]
    for n_keep in (37, 250, 499):
        assert O.select(O.criticality(F), n_keep).tolist() == B.select(nsq, n_keep)
    assert O.select(O.criticality(E), 6).tolist() == list(range(6))
    assert O.select(O.criticality(E), 0).tolist() == []


# --------------------------------------------------------------------------
# Injection (Eq. 2, Eq. 10)
# --------------------------------------------------------------------------

def test_inject_matches_exact_rational_brute_force_bf16():
    """Catches a double rounding, a missing H term and a wrong row index."""
    rng = np.random.default_rng(50)
    n, S, P, d_v, d_h, k = 6, 3, 4, 5, 7, 3
    H = _bf16_values(rng, (n, d_h))
    V = _bf16_values(rng, (S * P, d_v), 0.5)
    scene = rng.integers(0, S, n)
    prim = np.array([rng.permutation(P)[:k] for _ in range(n)])
    w = np.array([O.softmax_weights(rng.standard_normal(k)) for _ in range(n)])
    kept = np.array([0, 2, 3, 5])
    out = O.inject(H, V, P, scene, prim, w, kept, "bf16")
    ref = B.inject(H.tolist(), V.tolist(), P, scene.tolist(), prim.tolist(), w.tolist(),
                   kept.tolist(), B.round_bf16)
    for t in range(n):
        for j in range(d_h):
            assert Fraction(float(out[t, j])) == ref[t][j], (t, j)


def test_inject_k1_float32_is_one_correctly_rounded_add():
    """k = 1 in float32: out = fl(H + V_row) bit for bit."""
    rng = np.random.default_rng(51)
    n, S, P, d = 8, 2, 3, 16
    H32 = rng.standard_normal((n, d)).astype(np.float32)
    V32 = (rng.standard_normal((S * P, d)) * 1e-3).astype(np.float32)
    scene = rng.integers(0, S, n)
    prim = rng.integers(0, P, (n, 1))
    w = np.ones((n, 1))
    kept = np.arange(n)
    out = O.inject(H32.astype(np.float64), V32.astype(np.float64), P, scene, prim, w, kept, "f32")
    ref = H32 + V32[scene * P + prim[:, 0]]
    np.testing.assert_array_equal(out.astype(np.float32), ref)


def test_inject_zero_hidden_gives_retrieved_rows_and_leaves_rest():
    """Rows that encode their own index reveal which rows were gathered;
    untouched rows and columns >= d_v keep their bits."""
    S, P, d_v, d_h = 3, 4, 2, 3
    V = np.array([[r, -r] for r in range(S * P)], dtype=np.float64)
    H = np.zeros((4, d_h))
    H[:, 2] = 9.0
    scene = np.array([2, 0, 1, 1])
    prim = np.array([[3], [1], [0], [2]])
    w = np.ones((4, 1))
    out = O.inject(H, V, P, scene, prim, w, np.array([0, 2]), "f32")
    assert out[0].tolist() == [11.0, -11.0, 9.0]      # row 2*4 + 3
    assert out[2].tolist() == [4.0, -4.0, 9.0]        # row 1*4 + 0
    assert out[1].tolist() == [0.0, 0.0, 9.0]
    assert out[3].tolist() == [0.0, 0.0, 9.0]


def test_retrieved_is_in_convex_hull_of_rows():
    rng = np.random.default_rng(52)
    V = rng.standard_normal((12, 5))
    w = O.softmax_weights(rng.standard_normal(4))
    r = O.retrieved(V, 4, 2, np.array([0, 3, 1, 2]), w)
    rows = V[8:12][[0, 3, 1, 2]]
    assert np.all(r <= rows.max(axis=0) + 1e-15) and np.all(r >= rows.min(axis=0) - 1e-15)


# --------------------------------------------------------------------------
# Whole path
# --------------------------------------------------------------------------

def _tiny_inputs(seed, L=2, n=24, d_in=12, d_e=8, S=4, P=6, d_v=5, d_h=7, k=3):
    rng = np.random.default_rng(seed)
    return dict(
        x=_bf16_values(rng, (n, d_in)),
        w_t=_bf16_values(rng, (L, d_e, d_in), 0.3),
        scene_keys=O.round_to_bf16(_unit(rng, (S, d_e))),
        prim_keys=O.round_to_bf16(_unit(rng, (S, P, d_e))),
        values=_bf16_values(rng, (S * P, d_v), 0.02),
        bias=None,
        delta=_bf16_values(rng, (L, n, d_h)),
        hidden=_bf16_values(rng, (L, n, d_h)),
    ), k


def test_run_layers_equal_independent_single_layer_runs():
    """Table reuse across layers must not change any layer's result."""
    inp, k = _tiny_inputs(60)
    full = O.run(**inp, k=k, n_keep=7, dtype="bf16")
    for l in range(2):
        one = dict(inp)
        one["w_t"] = inp["w_t"][l:l + 1]
        one["delta"] = inp["delta"][l:l + 1]
        one["hidden"] = inp["hidden"][l:l + 1]
        r = O.run(**one, k=k, n_keep=7, dtype="bf16")
        for name in full:
            np.testing.assert_array_equal(full[name][l], r[name][0])


def test_run_token_permutation_equivariance():
    inp, k = _tiny_inputs(61, L=1)
    perm = np.random.default_rng(5).permutation(inp["x"].shape[0])
    a = O.run(**inp, k=k, n_keep=24, dtype="bf16")    # keep all: no cut ties
    pinp = dict(inp)
    pinp["x"] = inp["x"][perm]
    pinp["delta"] = inp["delta"][:, perm]
    pinp["hidden"] = inp["hidden"][:, perm]
    b = O.run(**pinp, k=k, n_keep=24, dtype="bf16")
    for name in ("q", "scene", "prim", "w", "hidden"):
        np.testing.assert_array_equal(a[name][0][perm], b[name][0])


def test_run_matches_brute_force_end_to_end():
    """Every stage of the whole path against the rational brute force."""
    inp, k = _tiny_inputs(62, L=1, n=10)
    n_keep = 4
    res = O.run(**inp, k=k, n_keep=n_keep, dtype="bf16")
    q = B.project(inp["x"].tolist(), inp["w_t"][0].tolist(), B.round_bf16)
    assert [[Fraction(float(v)) for v in row] for row in res["q"][0]] == q
    scenes = B.route(q, inp["scene_keys"].tolist())
    assert res["scene"][0].tolist() == scenes
    S, P, d_e = inp["prim_keys"].shape
    prim, top = B.lookup_flat_sim(q, scenes, inp["prim_keys"].reshape(S * P, d_e).tolist(), P, k)
    assert res["prim"][0].tolist() == prim
    nsq = [sum(Fraction(float(v)) ** 2 for v in row) for row in inp["delta"][0]]
    kept = B.select(nsq, n_keep)
    assert res["kept"][0].tolist() == kept
    w = [B.softmax(tp) for tp in top]
    np.testing.assert_allclose(res["w"][0], w, rtol=1e-13)
    hid = B.inject(inp["hidden"][0].tolist(), inp["values"].tolist(), P, scenes, prim,
                   res["w"][0].tolist(), kept, B.round_bf16)
    for t in range(10):
        assert [Fraction(float(v)) for v in res["hidden"][0][t]] == hid[t]


def test_oracle_rejects_bad_sizes():
    with pytest.raises(ValueError):
        O.select(np.ones(3), 4)
    with pytest.raises(ValueError):
        O.lookup(np.ones((1, 2)), np.array([0]), np.ones((1, 3, 2)), 4)


# --------------------------------------------------------------------------
# Level-2 in the paper's form: relevance MLP (Eq. 6), cos + tanh weights
# (Eq. 7)
# --------------------------------------------------------------------------

def _relevance_tiny(seed, n=6, d_e=4, S=3, P=7, h=5, dtype="bf16"):
    rng = np.random.default_rng(seed)
    rnd = _bf16_values if dtype == "bf16" else (lambda r, sh, sc=1.0: r.standard_normal(sh) * sc)
    q = rnd(rng, (n, d_e))
    keys = rnd(rng, (S, d_e))
    w1 = rnd(rng, (h, 2 * d_e), 0.5)
    b1 = rng.standard_normal(h) * 0.25
    w2 = rnd(rng, (P, h), 0.5)
    b2 = rng.standard_normal(P) * 0.25
    K2 = rnd(rng, (S, P, d_e))
    scene = rng.integers(0, S, n)
    return q, scene, keys, w1, b1, w2, b2, K2


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_relevance_matches_exact_rational_brute_force(dtype):
    """Catches swapped halves of W1 (query vs scene key), a transposed W2, a
    missing bias, the activation applied after the rounding or not at all,
    and a top-k over the wrong axis."""
    q, scene, keys, w1, b1, w2, b2, K2 = _relevance_tiny(40, dtype=dtype)
    k = 3
    a = O.relevance_hidden(q, scene, keys, w1, b1, dtype)
    prim, w, r_top = O.relevance_lookup(q, scene, a, w2, b2, K2, k)
    mant = 8 if dtype == "bf16" else 24
    P = K2.shape[1]
    ba, bp, bw = B.relevance(q.tolist(), scene.tolist(), keys.tolist(), w1.tolist(), b1.tolist(),
                             w2.tolist(), b2.tolist(), K2.reshape(-1, K2.shape[2]).tolist(), P, k,
                             mant)
    for t in range(q.shape[0]):
        assert [Fraction(float(v)) for v in a[t]] == ba[t]
    assert prim.tolist() == bp
    np.testing.assert_allclose(w, np.array(bw), rtol=1e-12, atol=1e-15)


def test_relevance_constant_hidden_gives_planted_ranking():
    """W1 = 0 and b1 > 0 make the hidden layer a constant; with one hidden
    unit of value 1 the logits are the rows of W2 plus b2, so the top k is
    known by construction (and independent of the token and its scene)."""
    d_e, S, P, k = 4, 2, 9, 4
    planted = np.array([0.5, -1.0, 2.0, 0.25, 2.0, -3.0, 1.5, 0.75, 1.0])   # two equal maxima
    w1 = np.zeros((1, 2 * d_e))
    b1 = np.array([1.0])
    w2 = planted[:, None] - 0.125
    b2 = np.full(P, 0.125)
    rng = np.random.default_rng(41)
    q = rng.standard_normal((3, d_e))
    keys = rng.standard_normal((S, d_e))
    K2 = rng.standard_normal((S, P, d_e))
    a = O.relevance_hidden(q, np.array([0, 1, 1]), keys, w1, b1, "f32")
    assert np.all(a == 1.0)
    prim, _, r_top = O.relevance_lookup(q, np.array([0, 1, 1]), a, w2, b2, K2, k)
    for t in range(3):
        assert prim[t].tolist() == [2, 4, 6, 8]      # 2.0 (p=2 before p=4), 1.5, 1.0
        assert r_top[t].tolist() == [2.0, 2.0, 1.5, 1.0]


def test_relevance_relu_zeroes_negative_preactivations():
    """Pre-activations all below zero leave a = 0, so the logits are b2:
    catches a missing or sign-flipped activation."""
    d_e, P, h = 3, 6, 4
    q = np.array([[1.0, 2.0, 0.5]])
    keys = np.array([[0.25, 0.5, 1.0]])
    w1 = np.full((h, 2 * d_e), 1.0)
    b1 = np.full(h, -100.0)
    b2 = np.array([0.3, -0.2, 0.9, 0.1, 0.9, -1.0])
    w2 = np.ones((P, h))
    a = O.relevance_hidden(q, np.array([0]), keys, w1, b1, "f32")
    assert np.all(a == 0.0)
    prim, _, r_top = O.relevance_lookup(q, np.array([0]), a, w2, b2, np.ones((1, P, d_e)), 3)
    assert prim[0].tolist() == [2, 4, 0]
    assert r_top[0].tolist() == [0.9, 0.9, 0.3]


def test_relevance_weights_closed_forms():
    """Eq. 7 in closed form: rows parallel to v_e have cosine 1 and rows
    opposite to it -1, so the weights are a softmax of 1 + tanh(r) or
    -1 + tanh(r); k = 1 gives exactly 1."""
    d_e, P = 4, 3
    q = np.array([[1.0, -2.0, 0.5, 3.0]])
    K2 = np.stack([2.0 * q[0], 0.5 * q[0], -3.0 * q[0]])[None]        # cos = 1, 1, -1
    r = np.array([0.0, math.atanh(0.5), math.atanh(-0.25)])
    # one hidden unit equal to 1 carries the logits
    w1 = np.zeros((1, 2 * d_e))
    b1 = np.array([1.0])
    a = O.relevance_hidden(q, np.array([0]), np.zeros((1, d_e)), w1, b1, "f32")
    prim, w, _ = O.relevance_lookup(q, np.array([0]), a, r[:, None], np.zeros(P), K2, 3)
    assert prim[0].tolist() == [1, 0, 2]
    z = np.array([1 + 0.5, 1 + 0.0, -1 - 0.25])
    np.testing.assert_allclose(w[0], np.exp(z) / np.exp(z).sum(), rtol=1e-14)
    _, w1k, _ = O.relevance_lookup(q, np.array([0]), a, r[:, None], np.zeros(P), K2, 1)
    assert w1k[0].tolist() == [1.0]


def test_relevance_invariants():
    """Relabelling the hidden units (rows of W1 and b1, columns of W2 alike)
    leaves the logits unchanged; scaling primitive rows by positive factors
    leaves the cosines, hence the weights, unchanged.  Catches W1/W2 index
    mix-ups and a dot product used in place of the cosine."""
    q, scene, keys, w1, b1, w2, b2, K2 = _relevance_tiny(42, n=8, d_e=6, S=2, P=11, h=7,
                                                         dtype="f32")
    k = 4
    a = O.relevance_hidden(q, scene, keys, w1, b1, "f32")
    prim, w, r_top = O.relevance_lookup(q, scene, a, w2, b2, K2, k)
    perm = np.random.default_rng(43).permutation(w1.shape[0])
    a2 = O.relevance_hidden(q, scene, keys, w1[perm], b1[perm], "f32")
    prim2, w2_, r2 = O.relevance_lookup(q, scene, a2, w2[:, perm], b2, K2, k)
    assert prim2.tolist() == prim.tolist()
    np.testing.assert_allclose(r2, r_top, rtol=1e-12)
    scale = np.random.default_rng(44).uniform(0.1, 10.0, K2.shape[:2])[..., None]
    prim3, w3, _ = O.relevance_lookup(q, scene, a, w2, b2, K2 * scale, k)
    assert prim3.tolist() == prim.tolist()
    np.testing.assert_allclose(w3, w, rtol=1e-12)


# --------------------------------------------------------------------------
# Sparse injection through the SwiGLU fusion (Eq. 10)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_fusion_matches_brute_force(dtype):
    """Catches a swapped gate/up pair, silu applied to the wrong factor, a
    transposed W_down and a missing rounding of the inner activations."""
    rng = np.random.default_rng(50)
    m, d_v, d_ff, d_h = 4, 5, 6, 3
    rnd = _bf16_values if dtype == "bf16" else (lambda r, sh, sc=1.0: r.standard_normal(sh) * sc)
    R = rnd(rng, (m, d_v))
    wg, wu, wd = rnd(rng, (d_ff, d_v), 0.7), rnd(rng, (d_ff, d_v), 0.7), rnd(rng, (d_h, d_ff), 0.7)
    F = O.fusion(R, wg, wu, wd, dtype)
    ref = B.fusion_rows(R.tolist(), wg.tolist(), wu.tolist(), wd.tolist(),
                        8 if dtype == "bf16" else 24)
    np.testing.assert_allclose(F, np.array([[float(v) for v in row] for row in ref]),
                               rtol=1e-12, atol=1e-14)


def test_fusion_closed_form():
    """One inner unit: u = silu(a) * b, f = (2u, -u), with silu(a) =
    a / (1 + e^-a) computed by hand."""
    a, b = 1.5, -0.75
    R = np.array([[a, b]])
    F = O.fusion(R, np.array([[1.0, 0.0]]), np.array([[0.0, 1.0]]), np.array([[2.0], [-1.0]]),
                 "f32")
    u = float(np.float32(a / (1 + math.exp(-a)) * b))
    np.testing.assert_allclose(F[0], [2 * u, -u], rtol=1e-15)
    assert O.silu(np.array([0.0]))[0] == 0.0


def test_inject_fused_touches_only_kept_rows_and_zero_up_is_identity():
    """Rows outside the kept set keep their bits; W_up = 0 gives f = 0, so
    the kept rows keep theirs too; a nonzero f changes exactly the kept
    rows."""
    rng = np.random.default_rng(51)
    n, S, P, d_v, d_ff, d_h, k = 9, 2, 5, 4, 3, 6, 2
    H = _bf16_values(rng, (n, d_h))
    V = _bf16_values(rng, (S * P, d_v))
    scene = rng.integers(0, S, n)
    prim = np.stack([rng.permutation(P)[:k] for _ in range(n)])
    w = np.full((n, k), 0.5)
    kept = np.array([1, 4, 7])
    wg = _bf16_values(rng, (d_ff, d_v))
    wd = _bf16_values(rng, (d_h, d_ff))
    out0 = O.inject_fused(H, V, P, scene, prim, w, kept, wg, np.zeros((d_ff, d_v)), wd, "bf16")
    assert np.array_equal(out0, H)
    wu = _bf16_values(rng, (d_ff, d_v))
    out = O.inject_fused(H, V, P, scene, prim, w, kept, wg, wu, wd, "bf16")
    others = np.setdiff1d(np.arange(n), kept)
    assert np.array_equal(out[others], H[others])
    assert not np.array_equal(out[kept], H[kept])


def test_fusion_inner_unit_relabelling_invariance():
    """Permuting the inner units (rows of W_gate and W_up, columns of W_down
    alike) leaves f unchanged: catches gate/up rows and down columns indexed
    differently."""
    rng = np.random.default_rng(52)
    R = rng.standard_normal((3, 7))
    wg, wu, wd = rng.standard_normal((5, 7)), rng.standard_normal((5, 7)), rng.standard_normal((4, 5))
    perm = rng.permutation(5)
    np.testing.assert_allclose(O.fusion(R, wg[perm], wu[perm], wd[:, perm], "f32"),
                               O.fusion(R, wg, wu, wd, "f32"), rtol=1e-12)


# --------------------------------------------------------------------------
# Inter-layer propagation (Eq. 11)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_propagate_matches_brute_force(dtype):
    """Three steps against exact rational loops with one rounding per step:
    catches a transposed W_p, a missing residual, a missing or doubled
    rounding between steps and steps applied out of order."""
    rng = np.random.default_rng(53)
    m, d_v, steps = 3, 6, 3
    rnd = _bf16_values if dtype == "bf16" else (lambda r, sh, sc=1.0: r.standard_normal(sh) * sc)
    R = O.round_to_dtype(rnd(rng, (m, d_v)), dtype)
    wp = rnd(rng, (steps, d_v, d_v), 0.6)
    chain = O.propagate(R, wp, dtype)
    ref = B.propagate_rows(R.tolist(), [w.tolist() for w in wp], 8 if dtype == "bf16" else 24)
    assert chain.shape == (steps + 1, m, d_v)
    for j in range(steps + 1):
        np.testing.assert_array_equal(chain[j], np.array([[float(v) for v in row]
                                                          for row in ref[j]]))


def test_propagate_orientation_and_order():
    """W_p^1 moves input 0 into output 1 and W_p^2 input 1 into output 2 (a
    matrix indexed [input, output], applied as R W_p): R_1[1] = R_0[1] + R_0[0]
    and R_2[2] = R_0[2] + R_0[1] + R_0[0], every other column unchanged; the
    transposed or reversed chain gives other sums."""
    R = np.array([[1.0, 2.0, 4.0, 8.0], [-3.0, 5.0, 0.5, 1.0]])
    wp = np.zeros((2, 4, 4))
    wp[0, 0, 1] = 1.0
    wp[1, 1, 2] = 1.0
    chain = O.propagate(R, wp, "f32")
    r1 = R.copy()
    r1[:, 1] = R[:, 1] + R[:, 0]
    r2 = r1.copy()
    r2[:, 2] = R[:, 2] + R[:, 1] + R[:, 0]
    np.testing.assert_array_equal(chain[0], R)
    np.testing.assert_array_equal(chain[1], r1)
    np.testing.assert_array_equal(chain[2], r2)


def _prop_case(rng, n=10, S=2, P=5, d_v=4, d_ff=3, d_h=6, k=2, steps=2):
    H = _bf16_values(rng, (steps + 1, n, d_h))
    V = _bf16_values(rng, (S * P, d_v))
    scene = rng.integers(0, S, n)
    prim = np.stack([rng.permutation(P)[:k] for _ in range(n)])
    w = np.full((n, k), 0.5)
    kept = np.array([0, 3, 8])
    wg = _bf16_values(rng, (steps + 1, d_ff, d_v))
    wu = _bf16_values(rng, (steps + 1, d_ff, d_v))
    wd = _bf16_values(rng, (steps + 1, d_h, d_ff))
    return H, V, P, scene, prim, w, kept, wg, wu, wd


def test_propagate_minus_identity_cancels():
    """W_p = -I gives R_1 = R_0 - R_0 = 0 exactly and f(0) = 0, so the
    propagated layer keeps its bits while the LookME layer's kept rows move;
    rows outside the kept set keep theirs in every layer (the gate of the
    LookME layer is reused, Eq. 11)."""
    rng = np.random.default_rng(54)
    H, V, P, scene, prim, w, kept, wg, wu, wd = _prop_case(rng, steps=1)
    wp = -np.eye(V.shape[1])[None]
    assert np.array_equal(O.propagate(np.ones((2, V.shape[1])), wp, "bf16")[1], np.zeros((2, 4)))
    out = O.inject_propagated(H, V, P, scene, prim, w, kept, wp, wg, wu, wd, "bf16")
    assert np.array_equal(out[1], H[1])
    assert not np.array_equal(out[0, kept], H[0, kept])
    others = np.setdiff1d(np.arange(H.shape[1]), kept)
    assert np.array_equal(out[:, others], H[:, others])


def test_inject_propagated_special_cases_reduce_to_inject_fused():
    """No steps: the LookME layer alone, i.e. inject_fused on one layer.
    W_p = 0 at every step: R_j = R_0, so layer j is inject_fused with f_j
    on the LookME layer's lookup and kept set."""
    rng = np.random.default_rng(55)
    H, V, P, scene, prim, w, kept, wg, wu, wd = _prop_case(rng, steps=2)
    d_v = V.shape[1]
    out0 = O.inject_propagated(H[:1], V, P, scene, prim, w, kept, np.zeros((0, d_v, d_v)),
                               wg, wu, wd, "bf16")
    np.testing.assert_array_equal(
        out0[0], O.inject_fused(H[0], V, P, scene, prim, w, kept, wg[0], wu[0], wd[0], "bf16"))
    out = O.inject_propagated(H, V, P, scene, prim, w, kept, np.zeros((2, d_v, d_v)),
                              wg, wu, wd, "bf16")
    for j in range(3):
        np.testing.assert_array_equal(
            out[j], O.inject_fused(H[j], V, P, scene, prim, w, kept, wg[j], wu[j], wd[j], "bf16"))


# --------------------------------------------------------------------------
# Multi-scale retrieval with the token-wise router (Eq. 8)
# --------------------------------------------------------------------------

def _ms_case(rng, n=8, M=2, Sm=3, P=5, d_v=4, d_h=6, k=2):
    H = _bf16_values(rng, (n, d_h))
    V = _bf16_values(rng, (M * Sm * P, d_v))
    scene = rng.integers(0, Sm, (M, n))
    prim = np.stack([np.stack([rng.permutation(P)[:k] for _ in range(n)]) for _ in range(M)])
    w = rng.dirichlet(np.ones(k), (M, n))
    kept = np.array([1, 2, 6])
    return H, V, P, Sm, scene, prim, w, kept


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_multiscale_injection_matches_brute_force(dtype):
    """inject_multiscale against exact rational loops for the router query,
    logits, softmax over scales and mix (k = 1 with weight 1, so R^m is a
    table row exactly; a square W_{h->e}, so a transposed one differs):
    catches a transposed W_{h->e}, a missing 1/sqrt(d), a softmax over the
    wrong axis, an unrounded query and a scale reading another partition."""
    rng = np.random.default_rng(56)
    n, M, Sm, P, d = 4, 3, 2, 3, 4
    rnd = _bf16_values if dtype == "bf16" else (lambda r, sh, sc=1.0: r.standard_normal(sh) * sc)
    H = O.round_to_dtype(rnd(rng, (n, d), 1.5), dtype)
    W = O.round_to_dtype(rnd(rng, (d, d), 1.5), dtype)
    V = O.round_to_dtype(rnd(rng, (M * Sm * P, d), 2.0), dtype)
    scene = rng.integers(0, Sm, (M, n))
    prim = rng.integers(0, P, (M, n, 1))
    w = np.ones((M, n, 1))
    kept = np.arange(n)
    got = O.inject_multiscale(H, V, P, Sm, scene, prim, w, kept, W, dtype)
    R = [[V[(m * Sm + scene[m, t]) * P + prim[m, t, 0]].tolist() for m in range(M)]
         for t in range(n)]
    mix = B.multiscale_rows(H.tolist(), W.tolist(), R, 8 if dtype == "bf16" else 24)
    exp = O.round_to_dtype(H + np.array([[float(v) for v in row] for row in mix]), dtype)
    np.testing.assert_array_equal(got, exp)


def test_multiscale_one_scale_adds_the_rounded_row():
    """M = 1: the router weight is 1, so a kept row gets round(H + round(R))."""
    rng = np.random.default_rng(57)
    H, V, P, Sm, scene, prim, w, kept = _ms_case(rng, M=1)
    out = O.inject_multiscale(H, V, P, Sm, scene, prim, w, kept,
                              _bf16_values(rng, (H.shape[1], V.shape[1])), "bf16")
    for t in kept:
        R = O.round_to_dtype(O.retrieved(V, P, int(scene[0, t]), prim[0, t], w[0, t]), "bf16")
        np.testing.assert_array_equal(out[t, :4], O.round_to_dtype(H[t, :4] + R, "bf16"))
    others = np.setdiff1d(np.arange(H.shape[0]), kept)
    np.testing.assert_array_equal(out[others], H[others])


def test_multiscale_zero_router_takes_the_mean_and_scales_use_their_partitions():
    """W_{h->e} = 0: equal logits, weights 1/M, the mean of the scales' rows;
    scale m reads rows of its own partition (scenes from m * Sm)."""
    rng = np.random.default_rng(58)
    H, V, P, Sm, scene, prim, w, kept = _ms_case(rng, M=3)
    out = O.inject_multiscale(H, V, P, Sm, scene, prim, w, kept, np.zeros((H.shape[1], 4)), "bf16")
    for t in kept:
        R = [O.round_to_dtype(O.retrieved(V, P, m * Sm + int(scene[m, t]), prim[m, t], w[m, t]),
                              "bf16") for m in range(3)]
        np.testing.assert_allclose(out[t, :4], O.round_to_dtype(H[t, :4] + sum(R) / 3, "bf16"),
                                   rtol=0, atol=0)


def test_multiscale_planted_scale_wins_and_scale_order_does_not_matter():
    """A router query aligned with scale 1's row by a margin of 1000 in the
    logit puts all weight there (exp(-1000) = 0): round(H + R^1).  Reordering
    the scales (their table partitions and lookups alike) changes nothing."""
    rng = np.random.default_rng(59)
    H, V, P, Sm, scene, prim, w, kept = _ms_case(rng, n=4, M=2, d_v=4, d_h=4, k=1)
    kept = np.array([2])
    prim[:, 2, 0] = 0
    scene[:, 2] = 0
    w[:, 2, 0] = 1.0
    V[0 * Sm * P] = [1.0, 0.0, 0.0, 0.0]          # scale 0's row for token 2
    V[1 * Sm * P] = [0.0, 1.0, 0.0, 0.0]          # scale 1's row
    H[2] = [0.0, 1.0, 0.0, 0.0]
    W = np.eye(4) * 2000.0                        # q = (0, 2000, 0, 0): logits 0 and 1000
    out = O.inject_multiscale(H, V, P, Sm, scene, prim, w, kept, W, "f32")
    np.testing.assert_array_equal(out[2], [0.0, 2.0, 0.0, 0.0])
    # scales swapped: partition blocks exchanged, lookups exchanged
    V2 = np.concatenate([V[Sm * P:], V[:Sm * P]])
    out2 = O.inject_multiscale(H, V2, P, Sm, scene[::-1], prim[::-1], w[::-1], kept, W, "f32")
    np.testing.assert_array_equal(out2, out)
    H3, V3, P3, Sm3, sc3, pr3, w3, kept3 = _ms_case(np.random.default_rng(60), M=3)
    W3 = _bf16_values(np.random.default_rng(61), (H3.shape[1], 4))
    perm = [2, 0, 1]
    V3p = np.concatenate([V3[m * Sm3 * P3:(m + 1) * Sm3 * P3] for m in perm])
    np.testing.assert_array_equal(
        O.inject_multiscale(H3, V3p, P3, Sm3, sc3[perm], pr3[perm], w3[perm], kept3, W3, "bf16"),
        O.inject_multiscale(H3, V3, P3, Sm3, sc3, pr3, w3, kept3, W3, "bf16"))


def test_run_multiscale_routes_each_scale_within_its_partition():
    """One scale reproduces the single-scale path's q, scene, prim and w; a
    key planted in partition 0 that beats every other key moves scale 0's
    routing onto it and leaves scale 1's untouched."""
    rng = np.random.default_rng(62)
    n, d_in, d_e, S, P, d_v, d_h, k = 12, 8, 8, 4, 6, 4, 6, 2
    x = rng.standard_normal((2, n, d_in))
    wt = rng.standard_normal((2, d_e, d_in))
    K1 = rng.standard_normal((S, d_e))
    K2 = rng.standard_normal((S, P, d_e))
    V = rng.standard_normal((S * P, d_v))
    D = rng.standard_normal((n, 5))
    H = rng.standard_normal((n, d_h))
    Whe = rng.standard_normal((d_h, d_v))
    one = O.run_multiscale(x[:1], wt[:1], K1, K2, V, D, H, Whe, k=k, n_keep=4, dtype="f32")
    ref = O.run(x[0], wt[:1], K1, K2, V, None, D[None], H[None], k=k, n_keep=4, dtype="f32")
    for key in ("q", "scene", "prim", "w"):
        np.testing.assert_array_equal(one[key][0], ref[key][0])
    two = O.run_multiscale(x, wt, K1, K2, V, D, H, Whe, k=k, n_keep=4, dtype="f32")
    assert np.all(two["scene"] < S // 2)
    K1p = K1.copy()
    K1p[1] = 1e6 * np.sign(two["q"][0].sum(axis=0))   # partition 0's second key
    planted = O.run_multiscale(x, wt, K1p, K2, V, D, H, Whe, k=k, n_keep=4, dtype="f32")
    assert np.mean(planted["scene"][0] == 1) > 0.5
    np.testing.assert_array_equal(planted["scene"][1], two["scene"][1])


# --------------------------------------------------------------------------
# Learned SKA gate (Eq. 9), text pathway (Eq. 1), one LookME layer (Eq. 2)
# --------------------------------------------------------------------------

def test_gate_matches_exact_rational_brute_force_with_exact_zeros():
    """Catches a wrong threshold (>= instead of >), a transposed operand or a
    dropped row: small-integer Delta and W_g make many logits exactly 0,
    which must stay closed, and every other sign is exact."""
    rng = np.random.default_rng(70)
    delta = rng.integers(-2, 3, size=(60, 6)).astype(np.float64)
    w_g = rng.integers(-2, 3, size=6).astype(np.float64)
    z = [B.dot(r, w_g.tolist()) for r in delta.tolist()]
    assert sum(1 for v in z if v == 0) >= 3      # the case is exercised
    assert O.gate(delta, w_g).tolist() == B.gate(delta.tolist(), w_g.tolist())
    pos = rng.permutation(60)[:25]
    assert O.gate(delta, w_g, pos).tolist() == B.gate(delta.tolist(), w_g.tolist(),
                                                      pos.tolist())


def test_gate_planted_signs_and_degenerate_weights():
    """Planted: Delta_i = gamma_i e_3 and W_g = e_3 open exactly where
    gamma_i > 0; W_g = 0 closes every gate; a positive scale of W_g changes
    nothing and a negated W_g opens exactly the complement (no zero logits in
    Gaussian data)."""
    rng = np.random.default_rng(71)
    gamma = rng.standard_normal(40)
    delta = np.zeros((40, 5))
    delta[:, 3] = gamma
    e3 = np.eye(5)[3]
    assert O.gate(delta, e3).tolist() == np.flatnonzero(gamma > 0).tolist()
    assert O.gate(delta, np.zeros(5)).size == 0
    d2 = _bf16_values(rng, (300, 16))
    w = _bf16_values(rng, 16)
    a = O.gate(d2, w)
    np.testing.assert_array_equal(a, O.gate(d2, 2.0 ** 7 * w))
    b = O.gate(d2, -w)
    assert np.intersect1d(a, b).size == 0
    np.testing.assert_array_equal(np.union1d(a, b), np.arange(300))
    # opens about half the gates on zero-mean data, in ascending order
    assert 100 < a.size < 200 and np.all(np.diff(a) > 0)


def test_inject_text_matches_brute_force_and_float32_addition():
    """Catches a wrong row (id vs position), a write outside the open gates or
    a second rounding: exact rational brute force in bf16, and in float32 the
    result must equal numpy's own float32 addition (one correctly rounded
    add) bit for bit."""
    rng = np.random.default_rng(72)
    V, d_t, d_h, n = 11, 5, 7, 9
    table = _bf16_values(rng, (V, d_t), 0.5)
    hidden = _bf16_values(rng, (n, d_h))
    pos = np.array([8, 0, 3, 5, 6])
    ids = np.array([4, 4, 10, 0, 7])
    kept = np.array([0, 1, 3])
    got = O.inject_text(hidden, table, pos, ids, kept, "bf16")
    ref = B.inject_text(hidden.tolist(), table.tolist(), pos.tolist(), ids.tolist(),
                        kept.tolist(), B.round_bf16)
    for t in range(n):
        assert [Fraction(float(v)) for v in got[t]] == ref[t]
    # untouched: positions 3 (gate closed), 6 (closed), 1, 2, 4, 7 (not text)
    for t in (1, 2, 3, 4, 6, 7):
        np.testing.assert_array_equal(got[t], hidden[t])
    h32 = rng.standard_normal((n, d_h)).astype(np.float32)
    t32 = rng.standard_normal((V, d_t)).astype(np.float32)
    g32 = O.inject_text(h32.astype(np.float64), t32.astype(np.float64), pos, ids, kept, "f32")
    want = h32.copy()
    for i in kept:
        want[pos[i], :d_t] = h32[pos[i], :d_t] + t32[ids[i]]
    np.testing.assert_array_equal(g32.astype(np.float32), want)
    zero = O.inject_text(np.zeros((n, d_h)), table, pos, ids, np.arange(5), "bf16")
    np.testing.assert_array_equal(zero[8, :d_t], table[4])
    np.testing.assert_array_equal(zero[0, :d_t], table[4])


def _layer_inputs(seed, n=20, d_h=16, d_c=12, start=6, n_i=9):
    rng = np.random.default_rng(seed)
    d_in, d_e, S, P, d_v, k, V, d_t = 10, 8, 4, 6, 12, 3, 13, 10
    h_dec = _bf16_values(rng, (n, d_h))
    delta = _bf16_values(rng, (n, d_c))
    text_pos = np.array([0, 1, 2, 3, 17, 19])
    text = (text_pos, rng.integers(0, V, size=text_pos.size), _bf16_values(rng, (V, d_t), 0.5),
            _bf16_values(rng, d_c))
    image = (start, _bf16_values(rng, (n_i, d_in)), _bf16_values(rng, (d_e, d_in), 0.3),
             O.round_to_bf16(_unit(rng, (S, d_e))), O.round_to_bf16(_unit(rng, (S, P, d_e))),
             _bf16_values(rng, (S * P, d_v), 0.5), k, _bf16_values(rng, d_c))
    cross = (_bf16_values(rng, (d_e, d_h), 0.3), O.round_to_bf16(_unit(rng, (S, d_e))),
             O.round_to_bf16(_unit(rng, (S, P, d_e))), _bf16_values(rng, (S * P, d_v), 0.5),
             k, _bf16_values(rng, d_c))
    return h_dec, delta, text, image, cross


def test_lookme_layer_closed_gates_and_single_pathways():
    """W_g = 0 for every pathway leaves L_dec(H_in) bit-identical; with one
    pathway present the layer reduces to that pathway's own injection (text:
    inject_text at the gated positions; image: route/lookup/inject on the
    image block; cross: the same on every position, queried by h_dec)."""
    h_dec, delta, text, image, cross = _layer_inputs(73)
    zt = text[:3] + (np.zeros_like(text[3]),)
    zi = image[:7] + (np.zeros_like(image[7]),)
    zc = cross[:5] + (np.zeros_like(cross[5]),)
    r = O.lookme_layer(h_dec, delta, dtype="bf16", text=zt, image=zi, cross=zc)
    np.testing.assert_array_equal(r["hidden"], h_dec)
    rt = O.lookme_layer(h_dec, delta, dtype="bf16", text=text)
    kept_t = B.gate(delta.tolist(), text[3].tolist(), text[0].tolist())
    assert kept_t and rt["text_kept"].tolist() == kept_t
    ref = B.inject_text(h_dec.tolist(), text[2].tolist(), text[0].tolist(), text[1].tolist(),
                        kept_t, B.round_bf16)
    np.testing.assert_array_equal(rt["hidden"], np.array([[float(v) for v in r_] for r_ in ref]))
    start, x, w_t, sk, pk, vals, k, w_g = image
    ri = O.lookme_layer(h_dec, delta, dtype="bf16", image=image)
    q = B.project(x.tolist(), w_t.tolist(), B.round_bf16)
    sc = B.route(q, sk.tolist())
    S, P, d_e = pk.shape
    prim, top = B.lookup_flat_sim(q, sc, pk.reshape(S * P, d_e).tolist(), P, k)
    assert ri["img_scene"].tolist() == sc and ri["img_prim"].tolist() == prim
    kept_i = B.gate(delta[start:start + x.shape[0]].tolist(), w_g.tolist())
    assert kept_i and ri["img_kept"].tolist() == kept_i
    blk = B.inject(h_dec[start:start + x.shape[0]].tolist(), vals.tolist(), P, sc, prim,
                   ri["img_w"].tolist(), kept_i, B.round_bf16)
    want = h_dec.copy()
    want[start:start + x.shape[0]] = np.array([[float(v) for v in r_] for r_ in blk])
    np.testing.assert_array_equal(ri["hidden"], want)
    rc = O.lookme_layer(h_dec, delta, dtype="bf16", cross=cross)
    qc = B.project(h_dec.tolist(), cross[0].tolist(), B.round_bf16)
    assert rc["cross_scene"].tolist() == B.route(qc, cross[1].tolist())
    kept_c = B.gate(delta.tolist(), cross[5].tolist())
    assert kept_c and rc["cross_kept"].tolist() == kept_c


def test_lookme_layer_pathways_read_the_layer_inputs_and_add_in_order():
    """The cross-modal query is L_dec(H_in), not a partly injected state: the
    full layer's cross-modal lookup equals the cross-only layer's even with
    loud text and image rows.  The adds run text, image, cross, each rounded:
    the full result equals chaining the three single-pathway layers, each on
    the previous result, with the cross-modal lookup kept from h_dec."""
    h_dec, delta, text, image, cross = _layer_inputs(74)
    full = O.lookme_layer(h_dec, delta, dtype="bf16", text=text, image=image, cross=cross)
    rc = O.lookme_layer(h_dec, delta, dtype="bf16", cross=cross)
    for name in ("cross_q", "cross_scene", "cross_prim", "cross_w", "cross_kept"):
        np.testing.assert_array_equal(full[name], rc[name])
    a = O.lookme_layer(h_dec, delta, dtype="bf16", text=text)["hidden"]
    b = O.lookme_layer(a, delta, dtype="bf16", image=image)["hidden"]
    c = O.inject(b, cross[3], cross[2].shape[1], rc["cross_scene"], rc["cross_prim"],
                 rc["cross_w"], rc["cross_kept"], "bf16")
    np.testing.assert_array_equal(full["hidden"], c)
    # the text and image positions overlap the cross-modal ones: a changed
    # order would round differently somewhere
    assert np.intersect1d(text[0][full["text_kept"]], full["cross_kept"]).size > 0


def test_run_with_learned_gate_composes_gate_and_inject():
    """run(w_g=...) keeps exactly the gate's positions of each layer and
    injects them as inject does; a gate that opens where the criticality
    select keeps gives the same result as the select."""
    inp, k = _tiny_inputs(75, L=2)
    rng = np.random.default_rng(75)
    w_g = _bf16_values(rng, (2, inp["delta"].shape[2]))
    r = O.run(**inp, k=k, n_keep=0, dtype="bf16", w_g=w_g)
    P = inp["prim_keys"].shape[1]
    for l in range(2):
        kept = B.gate(inp["delta"][l].tolist(), w_g[l].tolist())
        assert r["kept"][l].tolist() == kept
        want = O.inject(inp["hidden"][l], inp["values"], P, r["scene"][l], r["prim"][l],
                        r["w"][l], np.array(kept), "bf16")
        np.testing.assert_array_equal(r["hidden"][l], want)
    # planted: Delta_t = c_t e_0 with W_g = e_0 opens the positive c_t, which
    # (all |c| distinct) are the top n_keep by norm when the rest are tiny
    one = dict(inp)
    n, d_c = inp["delta"].shape[1], inp["delta"].shape[2]
    c = np.concatenate([np.arange(1, 9) * 1.0, -np.arange(1, n - 7) * 2.0 ** -12])
    d = np.zeros((1, n, d_c))
    d[0, :, 0] = c
    one.update(delta=d, hidden=inp["hidden"][:1], w_t=inp["w_t"][:1])
    a = O.run(**one, k=k, n_keep=8, dtype="bf16")
    b = O.run(**one, k=k, n_keep=0, dtype="bf16", w_g=np.eye(d_c)[:1])
    np.testing.assert_array_equal(a["kept"][0], b["kept"][0])
    np.testing.assert_array_equal(a["hidden"], b["hidden"])
