"""GPU parity of the learned SKA gate (Eq. 9), the injections for its counted
lists (prefix add, SwiGLU fusion, propagation), the text pathway (Eq. 1) and
one whole LookME layer (Eq. 2), through the C ABI, against the CPU oracle on
the same seeded inputs.
"""

import numpy as np
import pytest
import torch

from oracle import check as C
from synth import (WORKLOADS, Workload, make_fusion, make_gate, make_inputs, make_layer,
                   make_propagation, make_text)

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _announce(msg):
    print(f"[gpu-gate] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    from paper_2607_16305_amd import lookme as lk
    lk.load()          # fails loudly if the library was not built
    yield
    torch.cuda.synchronize()


def _small_table(dtype):
    from paper_2607_16305_amd import lookme as lk
    wl = Workload("gate_table", dtype, 16, 1, 64, 64, 2, 8, 16, 16, 2, 50)
    inp = make_inputs(wl, seed=2, device=DEV)
    return lk.Table(inp["scene_keys"], inp["prim_keys"], inp["values"], 2), inp


def _gate_and_check(table, delta, w_g, layers, pos=None, expect_exempt=True):
    from tests.harness import f64, to_np
    rows = delta.shape[-2]
    n = rows if pos is None else pos.numel()
    kept = torch.full((layers, max(n, 1)), -7, dtype=torch.int32, device=DEV)
    count = torch.full((layers,), -7, dtype=torch.int32, device=DEV)
    table.gate(delta, w_g, kept, count, pos=pos, layers=layers)
    torch.cuda.synchronize()
    rep = C.Report()
    cnt = to_np(count)
    kk = to_np(kept)
    p = None if pos is None else to_np(pos).astype(np.int64)
    for l in range(layers):
        c = int(cnt[l])
        assert 0 <= c <= n
        assert np.all(kk[l, c:n] == -1)
        C.check_gate(f64(delta[l]), f64(w_g[l]), kk[l, :c], rep, pos=p)
    rep.finish()
    assert rep.ok, str(rep)
    if not expect_exempt:
        assert not rep.exemptions, rep.exemptions
    return kept, count, rep


GATE = {
    # (dtype, layers, rows, d_c, pos entries or None)
    "bf16_image": ("bf16", 1, 1024, 2048, None),
    "f32_l3_ragged": ("f32", 3, 777, 96, None),
    "bf16_two_rounds": ("bf16", 2, 40000, 256, None),    # 32768 rows a compaction round
    "bf16_pos": ("bf16", 2, 1200, 512, 500),
    "f32_one_row": ("f32", 1, 1, 16, None),
    "bf16_zipf_width": ("bf16", 1, 32768, 4096, None),
}


@pytest.mark.parametrize("case", list(GATE))
def test_gate(case):
    """Open set {i : Delta_i W_g > 0} in ascending order, -1 past the count,
    the count itself; exemptions only within the tie band of zero."""
    dtype, layers, rows, d_c, npos = GATE[case]
    _announce(f"gate {case}")
    table, _ = _small_table(dtype)
    wl = Workload("g", dtype, rows, layers, 64, 64, 2, 8, 16, 16, 2, 50, d_c=d_c)
    g = torch.Generator(device="cpu").manual_seed(41)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    a = torch.exp(torch.randn((layers, rows, 1), generator=g))
    delta = (a * torch.randn((layers, rows, d_c), generator=g) / d_c ** 0.5).to(tdt).to(DEV)
    w_g = make_gate(wl, 41, device=DEV, layers=layers)
    pos = None
    if npos:
        pos = torch.randint(0, rows, (npos,), generator=g, dtype=torch.int32).to(DEV)
    kept, count, _ = _gate_and_check(table, delta, w_g, layers, pos)
    frac = count.float().mean().item() / (rows if pos is None else npos)
    assert 0.3 < frac < 0.7 or rows < 10


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_gate_integer_logits_exact(dtype):
    """Small-integer Delta and W_g: every logit is an exact integer in fp32,
    many exactly 0 (closed): the open set must match with no exemption."""
    _announce(f"gate integers {dtype}")
    table, _ = _small_table(dtype)
    g = torch.Generator(device="cpu").manual_seed(43)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    delta = torch.randint(-2, 3, (2, 3001, 64), generator=g).to(tdt).to(DEV)
    w_g = torch.randint(-1, 2, (2, 64), generator=g).to(tdt).to(DEV)
    _, count, _ = _gate_and_check(table, delta, w_g, 2, expect_exempt=False)
    z = (delta.double() @ w_g.double()[:, :, None])[..., 0]
    assert torch.equal(count.long().cpu(), (z > 0).sum(dim=1).cpu())
    assert (z == 0).sum().item() > 50


def test_gate_edges():
    """W_g = 0 closes every gate (count 0, list all -1); a W_g aligned with a
    positive Delta opens all; n = 0 writes count 0."""
    from paper_2607_16305_amd import lookme as lk
    _announce("gate edges")
    table, _ = _small_table("bf16")
    delta = torch.rand((1, 300, 64), device=DEV).add_(0.1).to(torch.bfloat16)
    kept = torch.full((1, 300), 5, dtype=torch.int32, device=DEV)
    count = torch.full((1,), 9, dtype=torch.int32, device=DEV)
    table.gate(delta, torch.zeros((1, 64), dtype=torch.bfloat16, device=DEV), kept, count)
    torch.cuda.synchronize()
    assert count.item() == 0 and torch.all(kept == -1)
    table.gate(delta, torch.ones((1, 64), dtype=torch.bfloat16, device=DEV), kept, count)
    torch.cuda.synchronize()
    assert count.item() == 300
    assert torch.equal(kept[0].cpu(), torch.arange(300, dtype=torch.int32))
    e = torch.empty(0, device=DEV)
    lk.lookme_gate(table.handle, 1, 0, e, 0, 64, None, e, e, count)
    torch.cuda.synchronize()
    assert count.item() == 0


GATED = {
    # name: (workload, mode, d_ff, sample)
    "plain_bf16_l2": (Workload("gp", "bf16", 300, 2, 768, 512, 20, 200, 392, 520, 8, 33,
                               usage="uniform"), "plain", 0, None),
    "plain_f32_l3": (Workload("gp32", "f32", 77, 3, 96, 256, 5, 37, 36, 40, 3, 40), "plain", 0,
                     None),
    "plain_image": (WORKLOADS[1], "plain", 0, 150),
    "fused_bf16_l2": (Workload("gf", "bf16", 700, 2, 256, 128, 20, 60, 128, 160, 8, 25,
                               usage="uniform", value_std=1.0), "fused", 256, None),
    "fused_image": (WORKLOADS[1].scaled(value_std=1.0), "fused", 2048, 60),
    "propagated_bf16": (Workload("gpr", "bf16", 300, 3, 256, 128, 20, 60, 128, 80, 8, 30,
                                 usage="uniform", value_std=1.0), "propagated", 192, None),
}


@pytest.mark.parametrize("name", list(GATED))
def test_gated_injection(name):
    """Route, lookup, the learned gate and the injection for its counted
    lists, against the oracle on the library's lookup; the counted fused
    path gives the same bits as lookme_inject_fused given the same set as a
    plain list."""
    from tests.harness import GatedRun, check_gated_run
    wl, mode, d_ff, sample = GATED[name]
    _announce(f"gated {name}: {wl} {mode}")
    inp = make_inputs(wl, seed=8, device=DEV)
    w_g = make_gate(wl, 8, device=DEV)
    fus = make_fusion(wl, 8, d_ff, device=DEV) if d_ff else None
    w_p_t = make_propagation(wl, 8, wl.layers - 1, device=DEV) if mode == "propagated" else None
    r = GatedRun(inp, w_g, mode, fus, w_p_t).run()
    toks = None
    if sample:
        k0 = r.kept[0].cpu().numpy()[:40]
        toks = np.unique(np.concatenate(
            [np.random.default_rng(8).choice(wl.n_tokens, sample, replace=False), k0]))
    rep = check_gated_run(r, tokens=toks)
    assert rep.ok, str(rep)
    if mode == "fused":
        from paper_2607_16305_amd import lookme as lk
        counts = r.count.cpu().tolist()
        for l in range(wl.layers):
            c = counts[l]
            ref = lk.Table(inp["scene_keys"], inp["prim_keys"], inp["values"], wl.top_k)
            ref.set_fusion(fus["w_gate"][l:l + 1], fus["w_up"][l:l + 1],
                           fus["w_down"][l:l + 1])      # layer l's fusion as a one-layer one
            hid = inp["hidden"][l:l + 1].clone()
            if c:
                ref.inject_fused(r.kept[l, :c].contiguous(), r.scene[l], r.prim[l], r.w[l], hid,
                                 c, layers=1)
            torch.cuda.synchronize()
            assert torch.equal(hid[0], r.hidden[l]), f"layer {l}"


SMALL_MS = {
    "ms_bf16": (Workload("ms_bf16", "bf16", 300, 1, 256, 128, 20, 60, 128, 192, 8, 30,
                         value_std=1.0), 2),
    "ms_f32_three": (Workload("ms_f32", "f32", 77, 1, 96, 64, 15, 37, 64, 96, 3, 20,
                              value_std=1.0), 3),
}


@pytest.mark.parametrize("name", list(SMALL_MS))
def test_gated_multiscale_injection(name):
    """The learned gate with the multi-scale router (Eq. 8-10): the gate's
    counted list into lookme_inject_multiscale_gated gives the oracle's mix of
    the scales' rows on the open tokens (and the gate the oracle's set), and
    the same bits as lookme_inject_multiscale given that set as a plain list."""
    from paper_2607_16305_amd import lookme as lk
    from synth import make_multiscale
    from tests.harness import MultiScaleRun, f64, to_np
    wl, scales = SMALL_MS[name]
    _announce(f"gated multi-scale {name}: {wl}")
    inp = make_inputs(wl, seed=12, device=DEV)
    ms = make_multiscale(wl, 12, scales, device=DEV)
    r = MultiScaleRun(inp, ms).run()
    w_g = make_gate(wl, 12, device=DEV, layers=1)
    n = r.n
    kept = torch.full((n,), -7, dtype=torch.int32, device=DEV)
    count = torch.full((4,), -7, dtype=torch.int32, device=DEV)
    r.table.gate(inp["delta"][0], w_g, kept, count[:1])
    hid = r.h_in.clone()
    r.table.inject_multiscale_gated(kept, count[:1], r.scene, r.prim, r.w, hid)
    torch.cuda.synchronize()
    c = int(count[0])
    assert 0 < c < n
    kept_np = kept.cpu().numpy()
    rep = C.Report()
    C.check_gate(f64(inp["delta"][0]), f64(w_g[0]), kept_np[:c], rep)
    dt = "bf16" if inp["x"].dtype == torch.bfloat16 else "f32"
    values = inp["values"]

    def values_rows(rows):
        idx = torch.as_tensor(np.asarray(rows), device=values.device, dtype=torch.long)
        return f64(values[idx])

    toks = np.arange(n)
    C.check_multiscale_hidden(to_np(r.h_in), to_np(hid), dt, values_rows, r.P, r.S // r.M,
                              to_np(r.scene), to_np(r.prim), to_np(r.w), kept_np[:c],
                              f64(ms["w_he_t"]).T, rep, toks)
    rep = rep.finish()
    assert rep.ok, str(rep)
    plain = r.h_in.clone()
    r.table.inject_multiscale(kept[:c].contiguous(), r.scene, r.prim, r.w, plain, c)
    torch.cuda.synchronize()
    assert torch.equal(plain, hid)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_text_injection(dtype):
    """The text pathway: the gate over the text positions, then
    lookme_inject_text for its counted list; every open entry adds its
    token's row once (float32 exactly, bf16 one rounding), nothing else
    moves; with no list every entry is injected."""
    from paper_2607_16305_amd import lookme as lk
    from tests.harness import f64, to_np
    _announce(f"text {dtype}")
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    n, d_h, d_c, vocab, d_t = 900, 256, 128, 5003, 192
    g = torch.Generator(device="cpu").manual_seed(51)
    pos = torch.randperm(n, generator=g)[:333].to(torch.int32)
    tx = make_text(51, vocab, d_t, pos, dtype, DEV, value_std=0.5)
    hidden = torch.randn((n, d_h), generator=g).to(tdt).to(DEV)
    delta = torch.randn((1, n, d_c), generator=g).to(tdt).to(DEV)
    w_g = torch.randn((1, d_c), generator=g).to(tdt).to(DEV)
    table, _ = _small_table(dtype)
    kept, count, _ = _gate_and_check(table, delta, w_g, 1, pos=tx["pos"])
    h0 = hidden.clone()
    lk.inject_text(tx["table"], tx["pos"], tx["ids"], hidden, kept[0], count)
    torch.cuda.synchronize()
    rep = C.Report()
    c = count.item()
    C.check_text_hidden(to_np(h0), to_np(hidden), dtype, f64(tx["table"]), to_np(tx["pos"]),
                        to_np(tx["ids"]), to_np(kept[0])[:c], rep)
    assert rep.finish().ok, str(rep)
    h1 = h0.clone()
    lk.inject_text(tx["table"], tx["pos"], tx["ids"], h1)
    torch.cuda.synchronize()
    rep = C.Report()
    C.check_text_hidden(to_np(h0), to_np(h1), dtype, f64(tx["table"]), to_np(tx["pos"]),
                        to_np(tx["ids"]), np.arange(333), rep)
    assert rep.finish().ok, str(rep)


LAYER = {
    # name: (image workload, text before, text after, vocab, d_t, cross S, P, k, sample)
    "bf16_small": (Workload("lay", "bf16", 200, 1, 256, 128, 12, 40, 128, 192, 4, 20,
                            value_std=0.5), 30, 50, 997, 64, 9, 32, 5, None),
    "f32_small": (Workload("lay32", "f32", 90, 1, 64, 64, 5, 24, 32, 48, 3, 20,
                           value_std=0.5), 7, 11, 101, 16, 4, 16, 3, None),
    "bf16_image": (WORKLOADS[1], 64, 192, 151936, 2048, 512, 256, 8, 200),
}


@pytest.mark.parametrize("name", list(LAYER))
def test_lookme_layer(name):
    """One LookME layer (Eq. 2): text, image and cross-modal pathways with
    their own gates, all reading the layer's inputs, added in order; against
    the oracle's recomputation from the library's decisions."""
    from tests.harness import LayerRun, check_layer_run
    wl, tb, ta, vocab, d_t, cs, cp, ck, sample = LAYER[name]
    _announce(f"layer {name}")
    lay = make_layer(wl, 9, tb, ta, vocab, d_t, cs, cp, ck, device=DEV)
    r = LayerRun(lay).run()
    toks = None
    if sample:
        toks = np.random.default_rng(9).choice(lay["n_seq"], sample, replace=False)
    rep = check_layer_run(r, tokens=toks)
    assert rep.ok, str(rep)
    opened = rep.notes["layer_open"]
    assert all(o > 0 for o in opened), opened


@pytest.mark.parametrize("name", ["gp_bf16_l2", "gp_f32_l3", "one_token", "image", "many"])
def test_lookup_gate_one_launch(name):
    """lookme_lookup_gate (the gate's logits in the bucketing launch and its
    compaction in the Level-2 launch for batches of at most 1024 rows, its own
    kernels after the bucketing otherwise): the same bits as lookme_lookup +
    lookme_gate, the gate against the oracle, and again on a second call."""
    from tests.harness import f64, to_np
    cases = {
        "gp_bf16_l2": Workload("gp", "bf16", 300, 2, 768, 512, 20, 200, 392, 520, 8, 33,
                               usage="uniform"),
        "gp_f32_l3": Workload("gp32", "f32", 77, 3, 96, 256, 5, 37, 36, 40, 3, 40),
        "one_token": Workload("one", "bf16", 1, 1, 64, 64, 9, 24, 16, 16, 4, 100),
        "image": WORKLOADS[1],
        "many": Workload("many", "bf16", 40000, 1, 64, 64, 8, 16, 16, 16, 2, 10),
    }
    wl = cases[name]
    _announce(f"lookup_gate {name}")
    from paper_2607_16305_amd import lookme as lk
    inp = make_inputs(wl, seed=21, device=DEV)
    w_g = make_gate(wl, 21, device=DEV)
    L, n, k = wl.layers, wl.n_tokens, wl.top_k
    t = lk.Table(inp["scene_keys"], inp["prim_keys"], inp["values"], k)
    q = torch.empty((L, n, wl.d_e), dtype=inp["x"].dtype, device=DEV)
    scene = torch.empty((L, n), dtype=torch.int32, device=DEV)
    t.route(inp["x"], inp["wt"], q, scene, layers=L)
    outs = []
    for mode in ("two_calls", "one", "one_again"):
        prim = torch.full((L, n, k), -7, dtype=torch.int32, device=DEV)
        w = torch.full((L, n, k), -7.0, dtype=torch.float32, device=DEV)
        kept = torch.full((L, n), -7, dtype=torch.int32, device=DEV)
        count = torch.full((L,), -7, dtype=torch.int32, device=DEV)
        if mode == "two_calls":
            t.lookup(q, scene, prim, w, layers=L)
            t.gate(inp["delta"], w_g, kept, count, layers=L)
        else:
            t.lookup_gate(q, scene, prim, w, inp["delta"], w_g, kept, count, layers=L)
        torch.cuda.synchronize()
        outs.append((prim, w, kept, count))
    for o in outs[1:]:
        for a, b, key in zip(outs[0], o, ("prim", "w", "kept", "count")):
            assert torch.equal(a, b), key
    rep = C.Report()
    cnt, kk = to_np(outs[1][3]), to_np(outs[1][2])
    for l in range(L):
        c = int(cnt[l])
        assert np.all(kk[l, c:] == -1)
        C.check_gate(f64(inp["delta"][l]), f64(w_g[l]), kk[l, :c], rep)
    assert rep.finish().ok, str(rep)
