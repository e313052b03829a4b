"""Pure-Python brute force for tiny inputs.  TEST INFRASTRUCTURE ONLY.

An independent second route to the same definitions as ``lookme_oracle``:
plain loops over Python numbers, repeated maximum extraction instead of
sorting, exact rational arithmetic (``fractions.Fraction``) for sums, and an
exact rational round-to-nearest-even to bfloat16 / binary32.  It pins the
oracle; it is far too slow for anything but a few dozen tokens.

Paper: arXiv 2607.16305, Sec. 3.2 (Eq. 4-7) and Sec. 3.3 (Eq. 9-10).
The cosine scores of Eq. 5 and Eq. 7 are exact rationals here for vectors
built to have rational norms; softmax weights over them are evaluated in
40-digit decimal arithmetic.
"""

from __future__ import annotations

import math
from fractions import Fraction


def round_fraction(v: Fraction, mant_bits: int, emin: int = -126) -> Fraction:
    """Exact round-to-nearest-even of a rational to a binary format with
    ``mant_bits`` significand bits (hidden bit included) and minimum normal
    exponent ``emin``.  Overflow is not handled (inputs here are small)."""
    if v == 0:
        return Fraction(0)
    sign = -1 if v < 0 else 1
    a = abs(v)
    # find e with 2^e <= a < 2^(e+1)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, emin)
    quantum = Fraction(2) ** (e - (mant_bits - 1))
    m = a / quantum
    fl = m.numerator // m.denominator
    rem = m - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return sign * fl * quantum


def round_bf16(v: Fraction) -> Fraction:
    return round_fraction(v, 8)


def round_f32(v: Fraction) -> Fraction:
    return round_fraction(v, 24)


def dot(a, b) -> Fraction:
    s = Fraction(0)
    for x, y in zip(a, b):
        s += Fraction(x) * Fraction(y)
    return s


def matvec_rows(x_rows, w_rows):
    """[(x . w_j) for each output row j] for every token row."""
    return [[dot(xr, wr) for wr in w_rows] for xr in x_rows]


def argmax_lowest(vals) -> int:
    best = 0
    for i in range(1, len(vals)):
        if vals[i] > vals[best]:
            best = i
    return best


def topk_by_extraction(vals, k):
    """k largest by repeated extraction of the maximum (lowest index wins an
    exact tie), in extraction order."""
    taken = []
    used = [False] * len(vals)
    for _ in range(k):
        best = -1
        for i, v in enumerate(vals):
            if used[i]:
                continue
            if best < 0 or v > vals[best]:
                best = i
        used[best] = True
        taken.append(best)
    return taken


def project(x_rows, w_t_rows, rounder):
    """q = round(x W) with W given output-row-major (w_t_rows[j] = column j)."""
    return [[rounder(v) for v in row] for row in matvec_rows(x_rows, w_t_rows)]


def route(q_rows, scene_keys, bias=None):
    out = []
    for q in q_rows:
        s = [dot(q, key) + (Fraction(bias[j]) if bias is not None else 0)
             for j, key in enumerate(scene_keys)]
        out.append(argmax_lowest(s))
    return out


def rational_sqrt(v: Fraction) -> Fraction:
    """Exact square root of a non-negative rational whose numerator and
    denominator are perfect squares; raises ValueError otherwise (the
    cosine routines below are only used on vectors built to have rational
    norms)."""
    v = Fraction(v)
    if v < 0:
        raise ValueError("negative")
    rn, rd = math.isqrt(v.numerator), math.isqrt(v.denominator)
    if rn * rn != v.numerator or rd * rd != v.denominator:
        raise ValueError(f"{v} is not the square of a rational")
    return Fraction(rn, rd)


def cosine_exact(a, b) -> Fraction:
    """cos(a, b) = <a, b> / (|a| |b|) as an exact rational (Eq. 5 and Eq. 7
    in their cosine form); 0 when either vector is zero.  Needs |a|^2 |b|^2
    to be the square of a rational."""
    na, nb = dot(a, a), dot(b, b)
    if na == 0 or nb == 0:
        return Fraction(0)
    return dot(a, b) / rational_sqrt(na * nb)


def route_cos(q_rows, scene_keys, bias=None):
    """Level-1 under the cosine of Eq. 5: arg max over s of
    cos(q, e_img[s]) + b[s], exact rationals, lowest s on exact ties.
    Returns (scenes, exact score rows)."""
    out, rows = [], []
    for q in q_rows:
        s = [cosine_exact(q, key) + (Fraction(bias[j]) if bias is not None else 0)
             for j, key in enumerate(scene_keys)]
        out.append(argmax_lowest(s))
        rows.append(s)
    return out, rows


def lookup_cos(q_rows, scenes, prim_keys, k):
    """Level-2 under the cosine of Eq. 7: the k largest exact cosines of the
    chosen scene's primitive keys (prim_keys[s][p]) by repeated extraction
    (lowest p on exact ties).  Returns (prim, exact top cosines, all exact
    cosines per row)."""
    prim, top, alls = [], [], []
    for q, s in zip(q_rows, scenes):
        c = [cosine_exact(q, key) for key in prim_keys[s]]
        idx = topk_by_extraction(c, k)
        prim.append(idx)
        top.append([c[i] for i in idx])
        alls.append(c)
    return prim, top, alls


def softmax_decimal(vals, digits: int = 40):
    """Softmax of exact rationals evaluated in ``digits``-digit decimal
    arithmetic (correctly rounded exp of the decimal module), returned as
    floats: an evaluation independent of float64 and of NumPy."""
    import decimal
    ctx = decimal.Context(prec=digits)
    dv = [ctx.divide(decimal.Decimal(v.numerator), decimal.Decimal(v.denominator))
          for v in map(Fraction, vals)]
    e = [ctx.exp(x) for x in dv]
    tot = sum(e, decimal.Decimal(0))
    return [float(ctx.divide(x, tot)) for x in e]


def scene_means(prim_key_rows, P):
    """Eq. 4 by plain loops: e_img[j] = (1/N_p) sum_p E[j, p, :] for the
    flat primitive rows of every scene, exact rationals."""
    S = len(prim_key_rows) // P
    d = len(prim_key_rows[0])
    out = []
    for j in range(S):
        row = []
        for c in range(d):
            acc = Fraction(0)
            for p in range(P):
                acc += Fraction(prim_key_rows[j * P + p][c])
            row.append(acc / P)
        out.append(row)
    return out


def lookup_flat_sim(q_rows, scenes, flat_keys, P, k):
    """Two-level result via a one-level similarity search restricted to the
    chosen scene's rows [s*P, (s+1)*P) of the flat key table (the 1-L(sim)
    baseline of the paper restricted to one scene).  Returns (prim, scores)
    with prim relative to the scene."""
    prim, top = [], []
    for q, s in zip(q_rows, scenes):
        scores = [dot(q, flat_keys[s * P + p]) for p in range(P)]
        idx = topk_by_extraction(scores, k)
        prim.append(idx)
        top.append([scores[i] for i in idx])
    return prim, top


def softmax(vals):
    m = max(vals)
    e = [math.exp(float(v - m)) for v in vals]
    s = math.fsum(e)
    return [x / s for x in e]


def select(norm_sq, n_keep):
    """Top n_keep by criticality via repeated extraction (ties lowest index),
    reported ascending.  Comparing squared norms orders exactly like norms."""
    return sorted(topk_by_extraction(norm_sq, n_keep))


def inject(hidden_rows, value_rows, P, scenes, prim, w, kept, rounder):
    """Exact rational sum of the weighted rows plus H, rounded once."""
    out = [list(map(Fraction, r)) for r in hidden_rows]
    d_v = len(value_rows[0])
    for t in kept:
        for j in range(d_v):
            acc = Fraction(hidden_rows[t][j])
            for i, p in enumerate(prim[t]):
                acc += Fraction(w[t][i]) * Fraction(value_rows[scenes[t] * P + p][j])
            out[t][j] = rounder(acc)
    return out


def relevance(q_rows, scene, scene_key_rows, w1_rows, b1, w2_rows, b2, prim_key_rows, P, k,
              mant_bits):
    """Level-2 in the paper's form (Eq. 6-7) by plain loops: exact rational
    MLP layers (ReLU, one rounding of the hidden activations), repeated
    maximum extraction for the top k (lowest p among equal logits), then
    cos + tanh and a softmax in floating point.  Returns (a, prim, w)."""
    a_rows, prims, ws = [], [], []
    for t, qt in enumerate(q_rows):
        inp = list(qt) + list(scene_key_rows[scene[t]])
        a = []
        for j, wr in enumerate(w1_rows):
            z = dot(inp, wr) + Fraction(b1[j])
            a.append(round_fraction(z, mant_bits) if z > 0 else Fraction(0))
        a_rows.append(a)
        r = [dot(a, w2_rows[p]) + Fraction(b2[p]) for p in range(P)]
        left = list(range(P))
        chosen = []
        for _ in range(k):
            best = left[0]
            for p in left[1:]:
                if r[p] > r[best]:
                    best = p
            chosen.append(best)
            left.remove(best)
        z = []
        for p in chosen:
            e = prim_key_rows[scene[t] * P + p]
            num = float(dot(qt, e))
            nq = math.sqrt(float(dot(qt, qt)))
            ne = math.sqrt(float(dot(e, e)))
            c = 0.0 if nq == 0 or ne == 0 else num / (nq * ne)
            z.append(c + math.tanh(float(r[p])))
        m = max(z)
        ex = [math.exp(v - m) for v in z]
        tot = sum(ex)
        prims.append(chosen)
        ws.append([v / tot for v in ex])
    return a_rows, prims, ws


def fusion_rows(r_rows, w_gate_rows, w_up_rows, w_down_rows, mant_bits):
    """f of Eq. 10 by plain loops: exact rational products, silu in floating
    point, one rounding of the inner activations (as a rational), then the
    exact down product.  Returns rationals [m][d_h]."""
    out = []
    for r in r_rows:
        u = []
        for gw, uw in zip(w_gate_rows, w_up_rows):
            g = float(dot(r, gw))
            val = Fraction(g / (1.0 + math.exp(-g))) * dot(r, uw)
            u.append(round_fraction(val, mant_bits))
        out.append([dot(u, dw) for dw in w_down_rows])
    return out


def propagate_rows(r_rows, w_p_mats, mant_bits):
    """Eq. 11 by plain loops: R_j[o] = sum_i R_{j-1}[i] W_p^j[i][o] +
    R_{j-1}[o], exact, then one rounding (as a rational) per element.
    w_p_mats[j] is a list of d_v rows indexed [i][o].  Returns the list of
    the m + 1 row lists (R_0 first)."""
    chain = [[list(r) for r in r_rows]]
    for wp in w_p_mats:
        nxt = []
        for r in chain[-1]:
            row = []
            for o in range(len(r)):
                acc = Fraction(r[o])
                for i in range(len(r)):
                    acc += Fraction(r[i]) * Fraction(wp[i][o])
                row.append(round_fraction(acc, mant_bits))
            nxt.append(row)
        chain.append(nxt)
    return chain


def multiscale_rows(h_rows, w_he_rows, r_scale_rows, mant_bits):
    """Eq. 8 by plain loops for each token: q = round(h W_{h->e}) exactly
    rounded, logits (q . R^m) / sqrt(d) as exact rationals evaluated in
    floating point, alpha by repeated max subtraction, then sum_m alpha_m R^m
    as rationals.  h_rows [t][d_h], w_he_rows [d_h][d_v] (input index first),
    r_scale_rows [t][M][d_v].  Returns rationals [t][d_v]."""
    out = []
    for h, rs in zip(h_rows, r_scale_rows):
        d_v = len(rs[0])
        q = []
        for o in range(d_v):
            acc = Fraction(0)
            for i in range(len(h)):
                acc += Fraction(h[i]) * Fraction(w_he_rows[i][o])
            q.append(round_fraction(acc, mant_bits))
        logits = [float(dot(q, r)) / math.sqrt(d_v) for r in rs]
        top = max(logits)
        e = [math.exp(v - top) for v in logits]
        tot = sum(e)
        alpha = [Fraction(v / tot) for v in e]
        out.append([sum((a * Fraction(r[c]) for a, r in zip(alpha, rs)), Fraction(0))
                    for c in range(d_v)])
    return out


def gate(delta_rows, w_g, pos=None):
    """Hard SKA gate (Eq. 9) by exact rational dot products: the indices i
    (into pos, or rows when pos is None) with Delta_{pos[i]} . W_g > 0."""
    rows = list(range(len(delta_rows))) if pos is None else list(pos)
    out = []
    for i, r in enumerate(rows):
        if dot(delta_rows[r], w_g) > 0:
            out.append(i)
    return out


def inject_text(hidden_rows, table_rows, pos, ids, kept, rounder):
    """Text pathway (Eq. 1): H[pos[i]] <- round(H[pos[i]] + E[ids[i]]) for
    the open gates i, in exact rational arithmetic."""
    out = [list(map(Fraction, r)) for r in hidden_rows]
    d_t = len(table_rows[0])
    for i in kept:
        t = pos[i]
        for j in range(d_t):
            out[t][j] = rounder(Fraction(hidden_rows[t][j]) + Fraction(table_rows[ids[i]][j]))
    return out
