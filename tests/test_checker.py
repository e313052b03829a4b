"""The checker must accept the oracle's own results, accept genuine ties, and
reject planted mistakes (all on the CPU, no library involved)."""

import numpy as np
import pytest

from oracle import check as C
from oracle import lookme_oracle as O


def _setup(seed=0, n=40, S=6, P=30, d=16, k=4, d_v=8, d_h=10):
    rng = np.random.default_rng(seed)
    q = O.round_to_bf16(rng.standard_normal((n, d)))
    K1 = O.round_to_bf16(rng.standard_normal((S, d)) / np.sqrt(d))
    K2 = O.round_to_bf16(rng.standard_normal((S, P, d)) / np.sqrt(d))
    V = O.round_to_bf16(rng.standard_normal((S * P, d_v)) * 0.02)
    H = O.round_to_bf16(rng.standard_normal((n, d_h)))
    D = rng.standard_normal((n, d_h)) * rng.lognormal(size=(n, 1))
    return q, K1, K2, V, H, D, k


def test_checker_accepts_oracle_results():
    q, K1, K2, V, H, D, k = _setup()
    rep = C.Report()
    scene = O.route(q, K1)
    C.check_scene(q, K1, None, "dot", scene, rep)
    prim, w, _ = O.lookup(q, scene, K2, k)
    w_orc = C.check_prim(q, scene, lambda s: K2[s], k, "dot", prim, w.astype(np.float32), rep)
    c = O.criticality(D)
    kept = O.select(c, 13)
    C.check_kept(c, 13, kept, rep)
    out = O.inject(H, V, K2.shape[1], scene, prim, w, kept, "bf16")
    C.check_hidden(O.from_f64(H, "bf16"), O.from_f64(out, "bf16"), "bf16", lambda r: V[r],
                   K2.shape[1], scene, prim, lambda t: w_orc[t], kept, rep)
    assert rep.finish().ok, str(rep)
    assert not rep.exemptions


def test_checker_rejects_planted_mistakes():
    q, K1, K2, V, H, D, k = _setup(1)
    scene = O.route(q, K1)
    # a wrong scene
    bad = scene.copy()
    bad[3] = (bad[3] + 1) % K1.shape[0]
    rep = C.Report()
    C.check_scene(q, K1, None, "dot", bad, rep)
    assert not rep.ok
    # a primitive set missing its best element
    prim, w, _ = O.lookup(q, scene, K2, k)
    bp = prim.copy()
    bp[5, 0] = [p for p in range(K2.shape[1]) if p not in prim[5]][0]
    rep = C.Report()
    C.check_prim(q, scene, lambda s: K2[s], k, "dot", bp, w, rep)
    assert not rep.ok
    # ascending instead of descending order
    rep = C.Report()
    C.check_prim(q, scene, lambda s: K2[s], k, "dot", prim[:, ::-1], w[:, ::-1], rep)
    assert not rep.ok
    # weights off by 1e-4
    rep = C.Report()
    C.check_prim(q, scene, lambda s: K2[s], k, "dot", prim, w + 1e-4, rep)
    assert not rep.ok
    # kept set with the smallest instead of the largest
    c = O.criticality(D)
    rep = C.Report()
    C.check_kept(c, 5, np.sort(np.argsort(c)[:5]), rep)
    assert not rep.ok
    rep = C.Report()
    C.check_kept(c, 5, O.select(c, 5)[::-1], rep)
    assert not rep.ok
    # an untouched row modified, and a touched row off by one bf16 step x2
    kept = O.select(c, 10)
    out = O.inject(H, V, K2.shape[1], scene, prim, w, kept, "bf16")
    bits = O.from_f64(out, "bf16")
    untouched = [t for t in range(q.shape[0]) if t not in kept][0]
    b2 = bits.copy()
    b2[untouched, 0] ^= 1
    rep = C.Report()
    C.check_hidden(O.from_f64(H, "bf16"), b2, "bf16", lambda r: V[r], K2.shape[1], scene, prim,
                   lambda t: w[t], kept, rep)
    assert not rep.ok
    b3 = bits.copy()
    b3[kept[0], 1] = (b3[kept[0], 1].astype(np.int32) + 2).astype(np.uint16)
    rep = C.Report()
    C.check_hidden(O.from_f64(H, "bf16"), b3, "bf16", lambda r: V[r], K2.shape[1], scene, prim,
                   lambda t: w[t], kept, rep, w_lib_of=lambda t: w[t].astype(np.float32))
    assert not rep.ok
    # the untouched result with the library weights passes the evaluation bound
    rep = C.Report()
    C.check_hidden(O.from_f64(H, "bf16"), bits, "bf16", lambda r: V[r], K2.shape[1], scene, prim,
                   lambda t: w[t], kept, rep, w_lib_of=lambda t: w[t])
    assert rep.ok, str(rep)


def test_checker_exempts_true_ties_only():
    # two scenes whose scores for the token differ by 1e-7 relative
    q = np.array([[1.0, 0.0]])
    K1 = np.array([[1.0, 0.0], [1.0 - 1e-7, 0.0]])
    rep = C.Report()
    C.check_scene(q, K1, None, "dot", np.array([1]), rep)
    assert rep.ok and rep.exemptions == {"scene": 1}
    K1b = np.array([[1.0, 0.0], [0.999, 0.0]])
    rep = C.Report()
    C.check_scene(q, K1b, None, "dot", np.array([1]), rep)
    assert not rep.ok


def test_checker_fails_when_exemptions_exceed_one_percent():
    rep = C.Report()
    rep.count("prim", 1000)
    rep.exempt("prim", 11)
    assert not rep.finish().ok
    rep = C.Report()
    rep.count("prim", 1000)
    rep.exempt("prim", 9)
    assert rep.finish().ok


def test_ulp_distance():
    a = O.from_f64(np.array([1.0, -1.0, 0.0]), "bf16")
    b = O.from_f64(np.array([1 + 2 ** -7, -1.0 - 2 ** -6, -0.0]), "bf16")
    assert C.ulp_distance(a, b, "bf16").tolist() == [1, 2, 0]


def test_projection_bound_accepts_float32_accumulation_and_rejects_errors():
    """A float32 left-to-right accumulation (what any float32 kernel may do)
    lies inside the bound even under heavy cancellation; a value one bf16
    step beyond the bound's rounding is rejected."""
    rng = np.random.default_rng(7)
    n, d_in, d_e = 50, 768, 40
    x = O.round_to_bf16(rng.standard_normal((n, d_in)))
    w = O.round_to_bf16(rng.standard_normal((d_e, d_in)) / np.sqrt(d_in))
    acc = np.zeros((n, d_e), dtype=np.float32)
    for i in range(d_in):
        acc = (acc + (x[:, i:i + 1] * w[:, i][None, :]).astype(np.float32)).astype(np.float32)
    lib = O.from_f64(O.round_to_bf16(acc.astype(np.float64)), "bf16")
    rep = C.Report()
    C.check_projection(lib, x, w, "bf16", rep)
    assert rep.ok, str(rep)
    exact = x @ w.T
    E = d_in * 2.0 ** -24 * (np.abs(x) @ np.abs(w).T)
    bad = O.round_to_bf16(exact + E)
    bad_bits = O.from_f64(bad, "bf16").astype(np.int32)
    bad_bits[3, 5] += 1 if bad[3, 5] >= 0 else -1       # one step beyond the upper rounding
    rep = C.Report()
    C.check_projection(bad_bits.astype(np.uint16), x, w, "bf16", rep)
    assert not rep.ok


def test_relevance_checks_accept_the_oracle_and_reject_planted_errors():
    """The relevance-mode checks pass the oracle's own answer and fail a
    swapped primitive, a wrong weight and an activation off by a lot."""
    rng = np.random.default_rng(7)
    n, d_e, S, P, h, k = 5, 8, 3, 20, 6, 4
    q = rng.standard_normal((n, d_e))
    keys = rng.standard_normal((S, d_e))
    w1 = rng.standard_normal((h, 2 * d_e)) * 0.3
    b1 = rng.standard_normal(h) * 0.1
    w2 = rng.standard_normal((P, h))
    b2 = rng.standard_normal(P) * 0.1
    K2 = rng.standard_normal((S, P, d_e))
    scene = rng.integers(0, S, n)
    a = O.relevance_hidden(q, scene, keys, w1, b1, "f32")
    prim, w, _ = O.relevance_lookup(q, scene, a, w2, b2, K2, k)
    rep = C.Report()
    C.check_relevance_hidden(a.astype(np.float32), q, scene, keys, w1, b1, "f32", rep)
    C.check_relevance_prim(a, w2, b2, q, scene, lambda s: K2[s], k, prim, w, rep)
    assert rep.finish().ok, str(rep)
    bad = prim.copy()
    r = O.relevance_logits(a, w2, b2)
    bad[0, -1] = int(np.argsort(r[0])[0])          # the worst primitive instead
    rep = C.Report()
    C.check_relevance_prim(a, w2, b2, q, scene, lambda s: K2[s], k, bad, w, rep)
    assert not rep.ok
    w_bad = w.copy()
    w_bad[1, 0] += 1e-3
    rep = C.Report()
    C.check_relevance_prim(a, w2, b2, q, scene, lambda s: K2[s], k, prim, w_bad, rep)
    assert not rep.ok
    a_bad = a.astype(np.float32).copy()
    a_bad[2, 1] += 0.5
    rep = C.Report()
    C.check_relevance_hidden(a_bad, q, scene, keys, w1, b1, "f32", rep)
    assert not rep.ok


def test_propagated_check_accepts_the_oracle_and_rejects_planted_errors():
    """check_propagated_hidden on bf16 data: the oracle's own result passes;
    a result built with W_p transposed, or with an untouched row changed,
    fails."""
    rng = np.random.default_rng(9)
    n, S, P, d_v, d_ff, d_h, k, steps = 12, 3, 6, 16, 8, 10, 2, 2
    bf = lambda a: O.round_to_dtype(a, "bf16")
    H = bf(rng.standard_normal((steps + 1, n, d_h)))
    V = bf(rng.standard_normal((S * P, d_v)))
    scene = rng.integers(0, S, n)
    prim = np.stack([rng.permutation(P)[:k] for _ in range(n)])
    w = np.full((n, k), 0.5)
    kept = np.array([1, 5, 6, 11])
    wp = bf(rng.standard_normal((steps, d_v, d_v)) * 0.5)
    wg = bf(rng.standard_normal((steps + 1, d_ff, d_v)))
    wu = bf(rng.standard_normal((steps + 1, d_ff, d_v)))
    wd = bf(rng.standard_normal((steps + 1, d_h, d_ff)))
    bits = O.f64_to_bf16_bits
    toks = np.arange(n)

    def check(out):
        rep = C.Report()
        C.check_propagated_hidden(bits(H), bits(out), "bf16", lambda rows: V[rows], P, scene,
                                  prim, w, kept, wp, wg, wu, wd, rep, toks)
        return rep.finish()

    good = O.inject_propagated(H, V, P, scene, prim, w, kept, wp, wg, wu, wd, "bf16")
    assert check(good).ok
    transposed = O.inject_propagated(H, V, P, scene, prim, w, kept, wp.transpose(0, 2, 1), wg,
                                     wu, wd, "bf16")
    assert not check(transposed).ok
    touched = good.copy()
    touched[2, 0, 3] = bf(touched[2, 0, 3] + 1.0)
    assert not check(touched).ok


def test_multiscale_check_accepts_the_oracle_and_rejects_planted_errors():
    """check_multiscale_hidden on bf16 data: the oracle's result passes; one
    computed without the partition offset of each scale, or with a column
    past d_v changed, fails."""
    rng = np.random.default_rng(10)
    n, M, Sm, P, d_v, d_h, k = 10, 2, 3, 5, 16, 24, 2
    bf = lambda a: O.round_to_dtype(a, "bf16")
    H = bf(rng.standard_normal((n, d_h)))
    V = bf(rng.standard_normal((M * Sm * P, d_v)) * 2)
    scene = rng.integers(0, Sm, (M, n))
    prim = np.stack([np.stack([rng.permutation(P)[:k] for _ in range(n)]) for _ in range(M)])
    w = rng.dirichlet(np.ones(k), (M, n))
    kept = np.array([0, 3, 4, 9])
    W = bf(rng.standard_normal((d_h, d_v)) / np.sqrt(d_h))
    bits = O.f64_to_bf16_bits

    def check(out):
        rep = C.Report()
        C.check_multiscale_hidden(bits(H), bits(out), "bf16", lambda rows: V[rows], P, Sm, scene,
                                  prim, w, kept, W, rep, np.arange(n))
        return rep.finish()

    good = O.inject_multiscale(H, V, P, Sm, scene, prim, w, kept, W, "bf16")
    assert check(good).ok
    assert not check(O.inject_multiscale(H, V, P, 0, scene, prim, w, kept, W, "bf16")).ok
    bad = good.copy()
    bad[3, d_v + 2] = bf(bad[3, d_v + 2] + 1.0)
    assert not check(bad).ok


def _fused_case(rng, dtype, n=16, S=3, P=6, d_v=24, d_ff=40, d_h=32, k=3):
    rd = lambda a: O.round_to_dtype(a, dtype)
    H = rd(rng.standard_normal((n, d_h)))
    V = rd(rng.standard_normal((S * P, d_v)))
    scene = rng.integers(0, S, n)
    prim = np.stack([rng.permutation(P)[:k] for _ in range(n)])
    w = rng.dirichlet(np.ones(k), n).astype(np.float32).astype(np.float64)
    kept = np.array([0, 2, 3, 7, 8, 15])
    wg = rd(rng.standard_normal((d_ff, d_v)) / np.sqrt(d_v))
    wu = rd(rng.standard_normal((d_ff, d_v)) / np.sqrt(d_v))
    wd = rd(rng.standard_normal((d_h, d_ff)) / np.sqrt(d_ff))
    return H, V, P, scene, prim, w, kept, wg, wu, wd


def _fused_float32_evaluation(H, V, P, scene, prim, w, kept, wg, wu, wd, dtype):
    """The fused injection evaluated the way a float32 kernel would (float32
    sums in another order than the oracle's), each stored row rounded."""
    f32 = np.float32
    rd = lambda a: O.round_to_dtype(np.asarray(a, dtype=np.float64), dtype)
    out = H.copy()
    for t in kept:
        rows = scene[t] * P + prim[t]
        acc = np.zeros(V.shape[1], dtype=f32)
        for i in range(len(rows)):
            acc = acc + f32(w[t, i]) * V[rows[i]].astype(f32)
        R = rd(acc)
        g = (wg.astype(f32) @ R.astype(f32)).astype(f32)
        u = (wu.astype(f32) @ R.astype(f32)).astype(f32)
        U = rd((g / (f32(1) + np.exp(-g))) * u)
        F = (wd.astype(f32)[:, ::-1] @ U.astype(f32)[::-1]).astype(f32)
        d_v = V.shape[1]
        out[t] = H[t]
        out[t] = rd(H[t].astype(f32) + F)
    return out


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_fused_check_interval_accepts_float32_evaluation_and_rejects_small_errors(dtype):
    """check_fused_hidden accepts a float32 evaluation of the chain in another
    summation order; in bf16 its evaluation interval rejects one bf16 step
    (far below the 2e-2 contract) where the interval is a single value; in
    float32 the 1e-5 relative rule rejects 3e-5 of the summed magnitudes.
    (In float32 the worst-case interval of the two chained products is wider
    than the relative rule; there the rule is the binding one.)"""
    rng = np.random.default_rng(11)
    H, V, P, scene, prim, w, kept, wg, wu, wd = _fused_case(rng, dtype)
    enc = (lambda a: O.f64_to_bf16_bits(a)) if dtype == "bf16" else (lambda a: a.astype(np.float32))
    n = H.shape[0]

    def check(out):
        rep = C.Report()
        C.check_fused_hidden(enc(H), enc(out), dtype, lambda rows: V[rows], P, scene, prim,
                             w.astype(np.float32), kept, wg, wu, wd, rep, np.arange(n))
        return rep.finish()

    got = _fused_float32_evaluation(H, V, P, scene, prim, w, kept, wg, wu, wd, dtype)
    rep = check(got)
    assert rep.ok, rep
    assert rep.notes["fused_interval_checked"] == len(kept)
    bad = got.copy()
    t, c = int(kept[2]), 5
    if dtype == "bf16":
        # step one bf16 value up
        bits = O.f64_to_bf16_bits(bad[t, c:c + 1]).astype(np.int64)
        step = 1 if bad[t, c] >= 0 else -1
        bad[t, c] = O.bf16_bits_to_f64(np.array([bits[0] + step], dtype=np.uint16))[0]
        assert abs(bad[t, c] - got[t, c]) < 2e-2
    else:
        # 3e-5 of the summed magnitudes: inside the earlier 1e-4 rule,
        # outside the 1e-5 relative contract
        R = O.round_to_dtype(w[t] @ V[scene[t] * P + prim[t]], dtype)
        U = O.round_to_dtype(O.silu(wg @ R) * (wu @ R), dtype)
        mag = abs(H[t, c]) + np.abs(wd[c]) @ np.abs(U)
        bad[t, c] = np.float32(bad[t, c] + 3e-5 * mag)
    rep = check(bad)
    assert not rep.ok
    assert any(("interval" if dtype == "bf16" else "contract") in f for f in rep.failures)


def test_gate_checker_accepts_oracle_exempts_near_zero_and_rejects_flips():
    rng = np.random.default_rng(30)
    D = O.round_to_bf16(rng.standard_normal((200, 24)))
    wg = O.round_to_bf16(rng.standard_normal(24))
    kept = O.gate(D, wg)
    rep = C.Report()
    C.check_gate(D, wg, kept, rep)
    assert rep.finish().ok and not rep.exemptions
    # a logit planted at a few ulps above zero may go either way
    D2 = D.copy()
    D2[7] = 0.0
    D2[7, 0], D2[7, 1] = 1.0, -(1.0 - 2.0 ** -20)
    wg2 = wg.copy()
    wg2[0], wg2[1] = 1.0, 1.0
    ref = O.gate(D2, wg2)
    assert 7 in ref
    rep = C.Report()
    C.check_gate(D2, wg2, np.setdiff1d(ref, [7]), rep)
    assert rep.finish().ok and rep.exemptions == {"gate": 1}
    # a clear sign flip, a duplicate and an unsorted list are rejected
    bad = np.union1d(kept, [int(np.argmin(O.gate_logits(D, wg)))])
    for wrong in (bad, np.concatenate([kept[:3], kept[2:]]), kept[::-1]):
        rep = C.Report()
        C.check_gate(D, wg, wrong, rep)
        assert not rep.finish().ok
    pos = rng.permutation(200)[:50]
    rep = C.Report()
    C.check_gate(D, wg, O.gate(D, wg, pos), rep, pos=pos)
    assert rep.finish().ok


def test_text_checker_accepts_oracle_and_rejects_wrong_rows():
    rng = np.random.default_rng(31)
    table = O.round_to_bf16(rng.standard_normal((17, 6)) * 0.5)
    H = O.round_to_bf16(rng.standard_normal((12, 9)))
    pos, ids, kept = np.array([11, 2, 5, 0]), np.array([3, 16, 3, 8]), np.array([0, 1, 3])
    out = O.inject_text(H, table, pos, ids, kept, "bf16")
    hb, ob = O.from_f64(H, "bf16"), O.from_f64(out, "bf16")
    rep = C.Report()
    C.check_text_hidden(hb, ob, "bf16", table, pos, ids, kept, rep)
    assert rep.finish().ok, str(rep)
    wrong = O.from_f64(O.inject_text(H, table, pos, ids[::-1], kept, "bf16"), "bf16")
    rep = C.Report()
    C.check_text_hidden(hb, wrong, "bf16", table, pos, ids, kept, rep)
    assert not rep.finish().ok
    extra = O.from_f64(O.inject_text(H, table, pos, ids, np.arange(4), "bf16"), "bf16")
    rep = C.Report()
    C.check_text_hidden(hb, extra, "bf16", table, pos, ids, kept, rep)
    assert not rep.finish().ok


def _e2e_case(dtype, seed=12, n=40, d_in=24, d_e=16, S=5, P=9, d_v=12, d_h=14, k=3, n_keep=13):
    rng = np.random.default_rng(seed)
    rd = lambda a: O.round_to_dtype(a, dtype)
    x = rd(rng.standard_normal((n, d_in)))
    wt = rd(rng.standard_normal((d_e, d_in)) / np.sqrt(d_in))
    K1 = rd(rng.standard_normal((S, d_e)) / np.sqrt(d_e))
    K2 = rd(rng.standard_normal((S, P, d_e)) / np.sqrt(d_e))
    V = rd(rng.standard_normal((S * P, d_v)))
    D = rd(rng.standard_normal((1, n, 8)) * rng.lognormal(0, 1, (1, n, 1)))
    H = rd(rng.standard_normal((1, n, d_h)))
    res = O.run(x, wt[None], K1, K2, V, None, D, H, k=k, n_keep=n_keep, dtype=dtype)
    return dict(x=x, wt=wt, K1=K1, K2=K2, V=V, D=D, H=H, k=k, n_keep=n_keep, P=P, res=res)


def _e2e_check(c, dtype, q=None, scene=None, prim=None, w=None, kept=None, hidden=None):
    res = c["res"]
    enc = (lambda a: O.f64_to_bf16_bits(a)) if dtype == "bf16" else (lambda a: a.astype(np.float32))
    rep = C.Report()
    n = c["x"].shape[0]
    C.check_end_to_end(c["x"], c["wt"], c["K1"], None, "dot", c["K2"], lambda rows: c["V"][rows],
                       c["P"], c["k"], O.criticality(c["D"][0]), c["n_keep"], enc(c["H"][0]),
                       enc(res["hidden"][0] if hidden is None else hidden), dtype,
                       enc(res["q"][0] if q is None else q),
                       res["scene"][0] if scene is None else scene,
                       res["prim"][0] if prim is None else prim,
                       (res["w"][0] if w is None else w).astype(np.float32),
                       res["kept"][0] if kept is None else kept, rep, np.arange(n))
    return rep.finish()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_end_to_end_check_accepts_the_oracle_and_rejects_planted_errors(dtype):
    """check_end_to_end: the oracle's own whole-path results pass; a wrong
    scene, a wrong primitive, a dropped kept token, a hidden row two bf16
    steps (or 1e-4 relative) off and a q two steps off each fail."""
    c = _e2e_case(dtype)
    res = c["res"]
    rep = _e2e_check(c, dtype)
    assert rep.ok, rep
    t = int(res["kept"][0][3])
    sc = res["scene"][0].copy()
    sc[t] = (sc[t] + 1) % c["K1"].shape[0]
    assert not _e2e_check(c, dtype, scene=sc).ok
    pr = res["prim"][0].copy()
    pr[t, 0] = [p for p in range(c["P"]) if p not in pr[t]][0]
    assert not _e2e_check(c, dtype, prim=pr).ok
    kp = res["kept"][0].copy()
    kp[3] = [i for i in range(40) if i not in kp][0]
    assert not _e2e_check(c, dtype, kept=np.sort(kp)).ok
    h = res["hidden"][0].copy()
    if dtype == "bf16":
        bits = O.f64_to_bf16_bits(h[t, :1]).astype(np.int64)
        h[t, 0] = O.bf16_bits_to_f64(np.array([bits[0] + 2], dtype=np.uint16))[0]
    else:
        h[t, 0] = np.float32(h[t, 0] * (1 + 1e-4) + 1e-4)
    assert not _e2e_check(c, dtype, hidden=h).ok
    q = res["q"][0].copy()
    if dtype == "bf16":
        bits = O.f64_to_bf16_bits(q[t, :1]).astype(np.int64)
        q[t, 0] = O.bf16_bits_to_f64(np.array([bits[0] + 2], dtype=np.uint16))[0]
    else:
        q[t, 0] = np.float32(q[t, 0] * (1 + 1e-3))
    assert not _e2e_check(c, dtype, q=q).ok


def test_scene_key_check_accepts_float32_means_and_rejects_errors():
    """check_scene_keys: a float32 running sum divided by P (either storage
    dtype) passes; a key off by one bf16 ulp where the bound is tight, or a
    sum that skips a primitive, fails."""
    rng = np.random.default_rng(7)
    S, P, d = 6, 300, 16
    pk32 = rng.standard_normal((S, P, d)).astype(np.float32)
    acc = np.zeros((S, d), dtype=np.float32)
    for p in range(P):                                  # the library's order, float32
        acc = (acc + pk32[:, p, :]).astype(np.float32)
    lib32 = (acc / np.float32(P)).astype(np.float32)
    rep = C.Report()
    C.check_scene_keys(lib32, pk32, "f32", rep)
    assert rep.ok, rep
    # the same means stored as bf16 (keys of bf16 values, rounded once more)
    pkb = O.round_to_dtype(pk32.astype(np.float64), "bf16").astype(np.float32)
    accb = np.zeros((S, d), dtype=np.float32)
    for p in range(P):
        accb = (accb + pkb[:, p, :]).astype(np.float32)
    libb = O.f64_to_bf16_bits(O.round_to_dtype((accb / np.float32(P)).astype(np.float64),
                                               "bf16"))
    rep = C.Report()
    C.check_scene_keys(libb, O.f64_to_bf16_bits(pkb.astype(np.float64)), "bf16", rep)
    assert rep.ok, rep
    # planted mistakes: one primitive left out, and the sum not divided
    bad = ((acc - pk32[:, 0, :]) / np.float32(P)).astype(np.float32)
    rep = C.Report()
    C.check_scene_keys(bad, pk32, "f32", rep)
    assert not rep.ok
    rep = C.Report()
    C.check_scene_keys(acc, pk32, "f32", rep)
    assert not rep.ok
    # integer keys with P a power of two: the mean is exact in float32 and passes
    ik = rng.integers(-2, 3, size=(3, 256, 8)).astype(np.float32)
    exact = (ik.sum(axis=1) / 256).astype(np.float32)
    rep = C.Report()
    C.check_scene_keys(exact, ik, "f32", rep)
    assert rep.ok, rep
