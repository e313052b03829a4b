"""GPU parity: the library (through its C ABI) against the CPU oracle on the
same seeded inputs, stage by stage (q, scene, primitives, weights, kept set,
injected hidden states), with the tie rules of oracle/check.py.

Sizes: small shapes that span several 16-row tiles, several 16-key blocks
per wave and ragged tails, checked on every token; the benchmark workloads
at full size, checked on sampled tokens (and the full kept set).
"""

import numpy as np
import pytest
import torch

from oracle import lookme_oracle as O
from synth import (WORKLOADS, Workload, make_fusion, make_inputs, make_integer_inputs,
                   make_multiscale, make_propagation, make_relevance)

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _announce(msg):
    print(f"[gpu-parity] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    from paper_2607_16305_amd import lookme as lk
    lk.load()          # fails loudly if the library was not built
    yield
    torch.cuda.synchronize()


def _run_check(inp, tokens=None, **kw):
    from tests.harness import Run, check_run
    r = Run(inp, **kw).run()
    rep = check_run(r, tokens=tokens)
    assert rep.ok, str(rep)
    return r, rep


SMALL = {
    "bf16_ragged_l2": Workload("bf16_ragged_l2", "bf16", 300, 2, 768, 512, 20, 200, 392, 520,
                               8, 33, usage="uniform"),
    "f32_proj_l3": Workload("f32_proj_l3", "f32", 77, 3, 96, 256, 5, 37, 36, 40, 3, 40,
                            usage="iid"),
    "bf16_narrow_keys": Workload("bf16_narrow_keys", "bf16", 130, 1, 160, 96, 7, 50, 64, 64,
                                 5, 50, usage="iid"),
    "bf16_wide_keys": Workload("bf16_wide_keys", "bf16", 90, 1, 256, 1024, 6, 70, 128, 128, 8,
                               30, usage="iid"),
    "bf16_zipf_tiles": Workload("bf16_zipf_tiles", "bf16", 2000, 1, 512, 512, 50, 64, 256, 256,
                                16, 20, usage="zipf"),
    "f32_k1": Workload("f32_k1", "f32", 64, 1, 64, 64, 3, 16, 64, 64, 1, 100, usage="iid",
                       project=False, value_std=1.0),
    "bf16_k_eq_p": Workload("bf16_k_eq_p", "bf16", 40, 1, 128, 128, 2, 16, 64, 64, 16, 50),
    "bf16_k32": Workload("bf16_k32", "bf16", 40, 1, 128, 128, 2, 40, 64, 64, 32, 50),
    "bf16_one_scene": Workload("bf16_one_scene", "bf16", 33, 1, 128, 256, 1, 19, 32, 32, 4, 50),
    # buckets of about 150 rows: shared units (64 rows, the last ragged) with
    # the widest lists, and fp32 with k = 16
    "bf16_k32_shared": Workload("bf16_k32_shared", "bf16", 300, 1, 128, 128, 2, 70, 32, 32, 32,
                                30, usage="uniform"),
    "f32_k16_shared": Workload("f32_k16_shared", "f32", 450, 1, 64, 128, 3, 90, 16, 16, 16, 30,
                               usage="uniform"),
    "bf16_one_prim": Workload("bf16_one_prim", "bf16", 21, 1, 64, 64, 9, 1, 16, 16, 1, 50),
    "bf16_one_token": Workload("bf16_one_token", "bf16", 1, 1, 64, 64, 9, 24, 16, 16, 4, 100),
    # projections large enough for the direct-to-LDS kernel (>= 256 tiles of
    # 128 x 128), with ragged row and K edges
    "bf16_dtl_proj_l4": Workload("bf16_dtl_proj_l4", "bf16", 1999, 4, 320, 512, 12, 40, 64, 64,
                                 4, 20, usage="uniform"),
    "f32_dtl_proj_l4": Workload("f32_dtl_proj_l4", "f32", 2100, 4, 96, 512, 5, 24, 32, 32, 3,
                                30, usage="iid"),
    # more tokens per layer than the select kernel caches in LDS
    "bf16_many_tokens": Workload("bf16_many_tokens", "bf16", 40000, 1, 64, 64, 8, 16, 16, 16, 2,
                                 10, usage="iid"),
    # the largest scene count the bucketing holds (one LDS histogram entry a
    # scene), with a ragged key width
    "bf16_max_scenes": Workload("bf16_max_scenes", "bf16", 3000, 1, 96, 96, 16384, 4, 32, 48,
                                2, 20, usage="uniform"),
    # same size, K not in whole 128-byte steps: the register-staged kernel
    "f32_ragged_k_proj_l4": Workload("f32_ragged_k_proj_l4", "f32", 2100, 4, 48, 512, 5, 24, 32,
                                     32, 3, 30, usage="iid"),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_small_workloads_every_token(name):
    """Stage-wise and end-to-end checks on every token."""
    from tests.harness import check_end_to_end_run
    wl = SMALL[name]
    _announce(f"{name}: {wl}")
    inp = make_inputs(wl, seed=3, device=DEV)
    r, rep = _run_check(inp)
    e2e = check_end_to_end_run(r)
    assert e2e.ok, str(e2e)
    if wl.usage != "iid" and wl.project:
        # planted clusters: layer-0 routing recovers the cluster label
        lab = inp["labels"].cpu().numpy()
        got = r.scene[0].cpu().numpy()
        assert np.mean(got == lab) > 0.99


# Batches whose last round of Level-2 units is cut in two parts (more than two
# rounds of single-bucket streaming units, P >= 512): masked bf16 keys with
# k = 16, fp32 with k = 32 (the widest partial list) and a ragged last key
# block (P = 520) over two layers, the cosine scores, and Zipf buckets (shared
# units in groups with streaming ones ahead of the parts); and one batch the
# host allows to cut but whose buckets are too few (no parts, the merge
# launch finds nothing).
CUT = {
    "bf16_cut_k16": (Workload("bf16_cut_k16", "bf16", 2048, 1, 64, 64, 2048, 512, 16, 16, 16,
                              20, usage="uniform"), "dot", True),
    "f32_cut_k32_p520": (Workload("f32_cut_k32_p520", "f32", 1500, 2, 64, 64, 3000, 520, 16, 16,
                                  32, 20, usage="uniform"), "dot", True),
    "bf16_cut_cos": (Workload("bf16_cut_cos", "bf16", 2048, 1, 64, 64, 2048, 512, 16, 16, 8, 20,
                              usage="uniform"), "cos", True),
    "bf16_cut_zipf": (Workload("bf16_cut_zipf", "bf16", 8000, 1, 64, 64, 2048, 512, 16, 16, 16,
                               20, usage="zipf"), "dot", True),
    "bf16_cut_declined": (Workload("bf16_cut_declined", "bf16", 1100, 1, 64, 64, 100, 512, 16,
                                   16, 8, 20, usage="uniform"), "dot", False),
    # the narrowest lists (k = 2, eight merge lanes a row) on 512-byte keys
    "f32_cut_k2_ks8": (Workload("f32_cut_k2_ks8", "f32", 2600, 1, 64, 128, 1300, 512, 16, 16, 2,
                                20, usage="uniform"), "dot", True),
}


@pytest.mark.parametrize("name", list(CUT))
def test_cut_last_round_every_token(name):
    """The Level-2 launch whose last 512 streaming units run as two parts
    each (partial top-k lists merged after the launch) against the oracle on
    every token; the work list's counters show the parts were made and
    taken."""
    wl, score, cut = CUT[name]
    _announce(f"{name}: {wl} score={score}")
    r, _ = _run_check(make_inputs(wl, seed=5, device=DEV), score=score)
    torch.cuda.synchronize()
    entries, first_part, taken = r.table.ws[:12].view(torch.int32).cpu().tolist()
    assert entries - first_part == (2 * 512 if cut else 0), (entries, first_part)
    assert taken >= (2 * 512 if cut else 0)
    # the merge's row names (after the routing counters at the start of the
    # workspace) are back at zero, and a second lookup gives the same bits
    named = r.table.ws[256 + 4096 * 4:256 + 4096 * 4 + 512 * 16 * 4].view(torch.int32)
    assert int(named.abs().sum()) == 0
    prim2, w2 = torch.full_like(r.prim, -7), torch.full_like(r.w, -7.0)
    r.table.lookup(r.q, r.scene, prim2, w2, layers=r.L)
    torch.cuda.synchronize()
    assert torch.equal(prim2, r.prim) and torch.equal(w2, r.w)


def test_tiny_f32_workload_every_token():
    from tests.harness import check_end_to_end_run
    wl = WORKLOADS[0]
    _announce(f"config 0: {wl}")
    r, _ = _run_check(make_inputs(wl, seed=0, device=DEV))
    e2e = check_end_to_end_run(r)
    assert e2e.ok, str(e2e)
    assert e2e.decisions["e2e_hidden"] == wl.n_tokens


@pytest.mark.parametrize("dtype,n,S", [("bf16", 211, 7), ("f32", 211, 7), ("bf16", 4500, 300),
                                       ("f32", 4400, 600)])
def test_integer_scores_tie_break_exactly(dtype, n, S):
    """Exact integer scores: every tie (scene, primitive, kept token) must go
    to the lowest index, with no tolerance and no exemption."""
    _announce(f"integer ties {dtype}")
    # n >= 4096: routing on the matrix-core tile kernel, whose last key tile
    # is ragged (moved back to end at the last scene)
    inp = make_integer_inputs(n=n, S=S, P=45, d_e=128, d_v=32, d_h=48, k=6, n_keep=70,
                              seed=5, dtype=dtype, device=DEV, layers=2)
    _, rep = _run_check(inp)
    assert not rep.exemptions, rep.exemptions


SPLIT_ROUTE = {
    # 16-row tiles, keys in 5 ranges of 64, 64, 64, 64 and 44 (13 / 25 tiles)
    "stream_l1_bias": (Workload("bf16_split_route", "bf16", 200, 1, 256, 256, 300, 16, 32, 32,
                                4, 25, usage="uniform"), True),
    "stream_l2": (Workload("bf16_split_route", "bf16", 200, 2, 256, 256, 300, 16, 32, 32, 4,
                           25, usage="uniform"), False),
    # matrix-core kernel: 33 blocks of 128 rows (the last ragged) x 3 key
    # tiles of 256, 256 and 188 keys, one tile per workgroup
    "tiles_bias": (Workload("bf16_tile_route", "bf16", 4100, 1, 256, 256, 700, 16, 32, 32, 4,
                            20, usage="uniform"), True),
    # fp32, 2 key tiles (256 + 44) over 2 workgroups
    "tiles_f32": (Workload("f32_tile_route", "f32", 4200, 1, 128, 128, 300, 16, 32, 32, 4, 20,
                           usage="iid"), False),
    # 313 row blocks, 4 key tiles (the last of 232 keys, read from key 744 on)
    # in 2 ranges of 2 tiles: a workgroup crosses into the ragged tile
    "tiles_multi_bias": (Workload("bf16_tile_route_multi", "bf16", 40000, 1, 128, 128, 1000, 4,
                                  16, 16, 2, 10, usage="uniform"), True),
}


@pytest.mark.parametrize("case", list(SPLIT_ROUTE))
def test_routing_with_split_keys(case):
    """Routing splits the scene keys of a row tile over several workgroups;
    the scene is the arg max over all of them, bias included, and repeated
    calls reuse the arrival counters."""
    wl, with_bias = SPLIT_ROUTE[case]
    _announce(f"split routing: {wl}, bias={with_bias}")
    inp = make_inputs(wl, seed=12, device=DEV)
    if with_bias:
        g = torch.Generator(device="cpu").manual_seed(77)
        inp["bias"] = (torch.randn(wl.scenes, generator=g) * 0.5).to(DEV)
    r1, _ = _run_check(inp)
    r2, _ = _run_check(inp, table=r1.table)   # same workspace: counters were reset
    assert torch.equal(r1.scene, r2.scene)


def test_f32_k1_inject_is_one_rounded_add():
    wl = SMALL["f32_k1"]
    inp = make_inputs(wl, seed=9, device=DEV)
    from tests.harness import Run
    r = Run(inp).run()
    torch.cuda.synchronize()
    assert torch.all(r.w == 1.0)
    s = r.scene[0].long()
    p = r.prim[0, :, 0].long()
    rows = inp["values"][s * wl.prims + p]
    ref = r.h_in[0].clone()
    ref[:, : wl.d_v] = r.h_in[0][:, : wl.d_v] + rows
    assert torch.equal(r.hidden[0], ref)


def test_edge_counts():
    from tests.harness import Run
    wl = SMALL["bf16_ragged_l2"].scaled(layers=1)
    inp = make_inputs(wl, seed=4, device=DEV)
    # n_keep = 0 leaves H untouched; n_keep = n touches every row
    r = Run(inp, n_keep=0).run()
    torch.cuda.synchronize()
    assert torch.equal(r.hidden, r.h_in)
    _run_check(inp, n_keep=wl.n_tokens)
    # n = 0 is a no-op
    from paper_2607_16305_amd import lookme as lk
    t = lk.Table(inp["scene_keys"], inp["prim_keys"], inp["values"], wl.top_k)
    e = torch.empty(0, device=DEV)
    t.reserve(1, 0)
    lk.lookme_route(t.handle, 1, 0, wl.d_e, e, None, e, e)
    lk.lookme_lookup(t.handle, 1, 0, e, e, e, e)
    lk.lookme_inject(t.handle, 1, 0, 0, e, wl.d_h, e, e, e, e, wl.d_h)
    torch.cuda.synchronize()


def test_deterministic_reruns():
    from tests.harness import Run
    wl = SMALL["bf16_zipf_tiles"]
    inp = make_inputs(wl, seed=11, device=DEV)
    a = Run(inp).run()
    b = Run(inp, table=a.table).run()
    torch.cuda.synchronize()
    for name in ("q", "scene", "prim", "w", "kept", "hidden"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name


@pytest.mark.parametrize("name", ["bf16_ragged_l2", "f32_proj_l3", "bf16_many_tokens",
                                  "bf16_one_token"])
def test_select_on_second_stream_then_inject_kept(name):
    """lookme_select on its own stream, concurrent with route and lookup, then
    lookme_inject_kept: the oracle's results, and the same bits as
    lookme_inject on one stream."""
    from tests.harness import Run, check_run
    wl = SMALL[name]
    inp = make_inputs(wl, seed=31, device=DEV)
    ref = Run(inp).run()
    r = Run(inp, table=ref.table).run_split()
    rep = check_run(r)
    assert rep.ok, str(rep)
    for key in ("q", "scene", "prim", "w", "kept", "hidden"):
        assert torch.equal(getattr(ref, key), getattr(r, key)), key


@pytest.mark.parametrize("name", ["bf16_ragged_l2", "f32_proj_l3", "bf16_one_token",
                                  "bf16_k32_shared", "bf16_many_tokens", "image",
                                  "max_scenes_small"])
def test_lookup_select_one_launch(name):
    """lookme_lookup_select (the select riding in the bucketing launch for
    batches of at most 1024 rows, after it otherwise): the oracle's results,
    the same bits as lookme_lookup + lookme_select, and again on a second
    call (the arrival counters were left at zero)."""
    from tests.harness import Run, check_run, run_fused_select
    wl = (WORKLOADS[1] if name == "image" else
          SMALL["bf16_max_scenes"].scaled(n_tokens=1000) if name == "max_scenes_small" else
          SMALL[name])
    _announce(f"lookup_select {name}")
    inp = make_inputs(wl, seed=32, device=DEV)
    ref = Run(inp).run()
    for rep_i in range(2):
        r = run_fused_select(Run(inp, table=ref.table))
        toks = np.arange(0, wl.n_tokens, 7) if wl.n_tokens > 2000 else None
        rep = check_run(r, tokens=toks)
        assert rep.ok, str(rep)
        for key in ("q", "scene", "prim", "w", "kept", "hidden"):
            assert torch.equal(getattr(ref, key), getattr(r, key)), (rep_i, key)


def test_profiling_hooks_time_every_group_and_change_nothing():
    """With the measurement hooks on, every group of a pass is timed once per
    launch (the Level-2 launch through its own start/end stamps, the others
    through events recorded around them), the durations are positive and
    below a second, a reset clears them, and the outputs carry the same bits
    as with the hooks off."""
    from paper_2607_16305_amd import lookme as lk
    from tests.harness import Run, run_fused_select
    _announce("profiling hooks")
    inp = make_inputs(SMALL["bf16_ragged_l2"], seed=41, device=DEV)
    ref = run_fused_select(Run(inp))
    torch.cuda.synchronize()
    h = ref.table.handle
    lk.lookme_profile_enable(h, True)
    try:
        for g in range(len(lk.GROUPS)):
            lk.lookme_profile_read(h, g, reset=True)
        passes = 3
        for _ in range(passes):
            r = run_fused_select(Run(inp, table=ref.table))
        torch.cuda.synchronize()
        for key in ("q", "scene", "prim", "w", "kept", "hidden"):
            assert torch.equal(getattr(ref, key), getattr(r, key)), key
        for name in ("project", "route", "bucket", "score", "inject"):
            count, ms = lk.lookme_profile_read(h, lk.GROUPS.index(name))
            assert count == passes, (name, count)
            assert 0.0 < ms < 1000.0 * passes, (name, ms)
        g = lk.GROUPS.index("score")
        count, _ = lk.lookme_profile_read(h, g, reset=True)
        assert count == passes
        assert lk.lookme_profile_read(h, g) == (0, 0.0)
    finally:
        lk.lookme_profile_enable(h, False)
    r = run_fused_select(Run(inp, table=ref.table))
    torch.cuda.synchronize()
    assert lk.lookme_profile_read(h, lk.GROUPS.index("score"))[0] == 0
    assert torch.equal(ref.prim, r.prim) and torch.equal(ref.hidden, r.hidden)


def test_lookup_select_integer_ties_and_edges():
    """Exact integer criticalities (many equal norms at the cut): the fused
    select keeps the lowest tokens like the stand-alone one; n_keep = n and
    n_keep = 0."""
    from tests.harness import Run, run_fused_select
    _announce("lookup_select ties")
    inp = make_integer_inputs(n=211, S=7, P=45, d_e=128, d_v=32, d_h=48, k=6, n_keep=70,
                              seed=5, dtype="bf16", device=DEV, layers=2)
    for n_keep in (70, 211, 1):
        ref = Run(inp, n_keep=n_keep).run()
        r = run_fused_select(Run(inp, n_keep=n_keep, table=ref.table))
        torch.cuda.synchronize()
        for key in ("prim", "w", "kept", "hidden"):
            assert torch.equal(getattr(ref, key), getattr(r, key)), (n_keep, key)
    r = run_fused_select(Run(inp, n_keep=0))
    torch.cuda.synchronize()
    assert torch.equal(r.hidden, r.h_in)


def _cos_inputs(wl, seed):
    """The workload's inputs with keys of uneven norms (each key row scaled by
    a factor in [0.25, 4), one key of each table zero), one zero query row
    and a scene bias: the cosine then ranks differently from the dot
    product."""
    inp = make_inputs(wl, seed=seed, device=DEV)
    g = torch.Generator(device="cpu").manual_seed(seed)
    S, P, d_e = inp["prim_keys"].shape
    f1 = torch.exp2(torch.rand((S, 1), generator=g) * 4 - 2).to(DEV)
    f2 = torch.exp2(torch.rand((S, P, 1), generator=g) * 4 - 2).to(DEV)
    k1 = (inp["scene_keys"].float() * f1).to(inp["scene_keys"].dtype)
    k2 = (inp["prim_keys"].float() * f2).to(inp["prim_keys"].dtype)
    k1[S // 2] = 0
    k2[0, P // 2] = 0
    inp["scene_keys"], inp["prim_keys"] = k1.contiguous(), k2.contiguous()
    inp["x"] = inp["x"].clone()
    inp["x"][1] = 0
    inp["bias"] = (torch.randn(S, generator=g) * 0.05).to(DEV)
    return inp


@pytest.mark.parametrize("name", ["bf16_ragged_l2", "f32_proj_l3", "bf16_k32_shared",
                                  "bf16_zipf_tiles", "bf16_many_tokens", "f32_k16_shared"])
def test_cosine_scores(name):
    """COS handles (the cosine of Eq. 5 and Eq. 7): routing with the bias and
    Level-2 against the oracle's cosines, in the streaming and shared units;
    the one-stream select falls back to its own kernels and stays the same
    bits."""
    from tests.harness import Run, check_run, run_fused_select
    wl = SMALL[name]
    _announce(f"cosine {name}")
    inp = _cos_inputs(wl, 41)
    toks = np.arange(0, wl.n_tokens, 5) if wl.n_tokens > 5000 else None
    r = Run(inp, score="cos").run()
    rep = check_run(r, tokens=toks)
    assert rep.ok, str(rep)
    d = Run(inp, score="dot").run()
    torch.cuda.synchronize()
    assert not torch.equal(r.w, d.w)          # the cosine form was taken
    f = run_fused_select(Run(inp, table=r.table, score="cos"))
    torch.cuda.synchronize()
    for key in ("scene", "prim", "w", "kept", "hidden"):
        assert torch.equal(getattr(r, key), getattr(f, key)), key


def test_layers_batched_equal_sequential():
    from tests.harness import Run
    wl = SMALL["bf16_ragged_l2"].scaled(layers=3)
    inp = make_inputs(wl, seed=12, device=DEV)
    full = Run(inp).run()
    for l in range(3):
        one = dict(inp)
        one["wt"] = inp["wt"][l:l + 1]
        one["delta"] = inp["delta"][l:l + 1]
        one["hidden"] = inp["hidden"][l:l + 1]
        r = Run(one, table=full.table).run()
        torch.cuda.synchronize()
        for name in ("q", "scene", "prim", "w", "kept", "hidden"):
            assert torch.equal(getattr(full, name)[l], getattr(r, name)[0]), (l, name)


# Level-2 in the paper's form (Eq. 6-7): (workload, hidden width, sampled
# tokens or None for all).  Ragged rows and primitive counts (200, 37, 300)
# leave partial 64 x 64 tiles in both layers; the image and multi-scale
# cases have the benchmarks' shapes.  Hidden rows of 512 or 1024 bytes take
# the fused second layer + top-k (bf16 batches of >= 4096 rows with k <= 16:
# the 32 x 32 tile form, else 16 x 16): the "fused" and "rel32" cases cover
# both widths in both dtypes and both forms, ragged last blocks of W2 rows
# (P 37, 300, 1000; at P 300 the last 32-key block's second image lies
# wholly past P), W2 split into ranges merged afterwards (P 300 over 2,
# P 1000 over 4 with a short last range, the image shape over 8), units with
# rows for one wave only (130 rows, 4200 rows) and one range of 4096 rows
# (Zipf).
RELEVANCE = {
    "bf16_rel_fused_h256": (Workload("bf16_rel_fused_h256", "bf16", 130, 1, 128, 64, 7, 300, 32,
                                     32, 32, 30, usage="uniform"), 256, None),
    "bf16_rel_fused_h256_k8": (Workload("bf16_rel_fused_h256_k8", "bf16", 130, 1, 128, 64, 7, 300,
                                        32, 32, 8, 30, usage="uniform"), 256, None),
    "f32_rel_fused_h128": (Workload("f32_rel_fused_h128", "f32", 77, 1, 96, 64, 5, 37, 40, 40,
                                    3, 40, usage="iid"), 128, None),
    "f32_rel_fused_h256": (Workload("f32_rel_fused_h256", "f32", 200, 1, 96, 64, 6, 1000, 40, 40,
                                    8, 40, usage="uniform"), 256, None),
    "bf16_rel_zipf": (WORKLOADS[4], 512, 40),
    # 1032 tiles of 128 x 128 in the first layer, a ragged last row block and
    # K of two 64-byte stages (fewer than the ring holds)
    "bf16_rel_big_ragged": (Workload("bf16_rel_big_ragged", "bf16", 33001, 1, 128, 64, 9, 300,
                                     32, 32, 8, 30, usage="uniform"), 512, 48),
    # batches of >= 4096 rows take the 32 x 32 form: 512-byte hidden rows with
    # ragged P (300: the last 32-key block's second image wholly past P; two
    # ranges) and a ragged last unit (4200 rows), 1024-byte rows with P 1000
    # and k 16, and k 4
    "bf16_rel32_h256_p300": (Workload("bf16_rel32_h256_p300", "bf16", 4200, 1, 128, 64, 7, 300,
                                      32, 32, 8, 30, usage="uniform"), 256, 48),
    "bf16_rel32_h512_p1000_k16": (Workload("bf16_rel32_h512_p1000_k16", "bf16", 4100, 1, 128, 64,
                                           5, 1000, 32, 32, 16, 30, usage="uniform"), 512, 48),
    "bf16_rel32_k4": (Workload("bf16_rel32_k4", "bf16", 4096, 1, 128, 64, 3, 200, 32, 32, 4, 30,
                               usage="iid"), 256, 48),
    # query rows of 512 and 1024 bytes with k < 32 take the weights on the
    # matrix cores: both widths, both dtypes, k < 16 (one tile with the
    # query), k = 16 (the query broadcast) and k = 20 (two tiles); k = 32
    # the vector form
    "bf16_rel_wmma_k32": (Workload("bf16_rel_wmma_k32", "bf16", 90, 1, 256, 256, 5, 300, 32, 32,
                                   32, 30, usage="uniform"), 128, None),
    "f32_rel_wmma_d128": (Workload("f32_rel_wmma_d128", "f32", 70, 1, 128, 128, 4, 100, 32, 32, 8,
                                   30, usage="uniform"), 64, None),
    "f32_rel_wmma_k16": (Workload("f32_rel_wmma_k16", "f32", 50, 1, 128, 128, 3, 90, 32, 32, 16,
                                  30, usage="iid"), 64, None),
    "f32_rel_wmma_k20": (Workload("f32_rel_wmma_k20", "f32", 60, 1, 256, 256, 3, 150, 32, 32, 20,
                                  30, usage="iid"), 96, None),
    "bf16_rel_l2": (Workload("bf16_rel_l2", "bf16", 300, 2, 256, 128, 20, 200, 64, 64, 8, 30,
                             usage="uniform"), 192, None),
    "f32_rel": (Workload("f32_rel", "f32", 77, 1, 96, 64, 5, 37, 40, 40, 3, 40, usage="iid"),
                96, None),
    "bf16_rel_k32": (Workload("bf16_rel_k32", "bf16", 130, 1, 128, 64, 7, 300, 32, 32, 32, 30,
                              usage="uniform"), 64, None),
    "bf16_rel_image": (WORKLOADS[1], 512, 80),
    # enough rows for the logits on the 256 x 256 projection tiles
    "bf16_rel_multiscale": (WORKLOADS[2], 512, 80),
}


@pytest.mark.parametrize("name", list(RELEVANCE))
def test_relevance_lookup(name):
    """Routing, the relevance MLP, top-k by logit, cos + tanh weights and the
    injection, stage by stage against the oracle."""
    from tests.harness import RelevanceRun, check_relevance_run
    wl, hidden, sample = RELEVANCE[name]
    _announce(f"relevance {name}: {wl} hidden {hidden}")
    inp = make_inputs(wl, seed=5, device=DEV)
    mlp = make_relevance(wl, 5, hidden, device=DEV)
    r = RelevanceRun(inp, mlp).run()
    toks = None
    if sample:
        # random rows plus the first and the last ones (the ragged edge)
        toks = np.unique(np.concatenate([
            np.random.default_rng(5).choice(wl.n_tokens, sample, replace=False),
            [0, wl.n_tokens - 2, wl.n_tokens - 1]]))
    rep = check_relevance_run(r, tokens=toks)
    assert rep.ok, str(rep)
    assert min(rep.decisions.get(kind, 0) for kind in ("act", "prim", "w", "hidden_row")) > 0
    r2 = RelevanceRun(inp, mlp, table=r.table).run()
    torch.cuda.synchronize()
    for key in ("act", "prim", "w"):
        assert torch.equal(getattr(r, key), getattr(r2, key)), key


def test_relevance_table_follows_registration():
    """The per-scene half of the first layer is computed once per
    registration and workspace: re-registering another MLP, or the first
    one again, gives what a fresh handle gives, bit for bit."""
    from tests.harness import RelevanceRun
    wl = Workload("bf16_rel_tab", "bf16", 200, 1, 128, 128, 9, 64, 32, 32, 8, 30, usage="uniform")
    _announce(f"relevance table refresh: {wl}")
    inp = make_inputs(wl, seed=11, device=DEV)
    mlp_a = make_relevance(wl, 11, 256, device=DEV)
    mlp_b = make_relevance(wl, 12, 256, device=DEV)
    ra = RelevanceRun(inp, mlp_a).run()
    act_a = ra.act.clone()
    rb = RelevanceRun(inp, mlp_b, table=ra.table).run()       # re-registers B on A's handle
    fresh_b = RelevanceRun(inp, mlp_b).run()
    ra2 = RelevanceRun(inp, mlp_a, table=ra.table).run()      # and A again
    torch.cuda.synchronize()
    assert not torch.equal(act_a, rb.act)
    for key in ("act", "prim", "w"):
        assert torch.equal(getattr(rb, key), getattr(fresh_b, key)), key
    assert torch.equal(ra2.act, act_a)


# Sparse injection through the SwiGLU fusion (Eq. 10): (workload, d_ff,
# sampled tokens or None).  Rows of unit scale (value_std 1) so that f is of
# the order of H; ragged kept counts and widths (d_h 80, d_ff 192, n_keep
# 90 and 11) leave partial tiles in both products.
FUSION = {
    "bf16_fus_l2": (Workload("bf16_fus_l2", "bf16", 300, 2, 256, 128, 20, 60, 128, 80, 8, 30,
                             usage="uniform", value_std=1.0), 192, None),
    "f32_fus": (Workload("f32_fus", "f32", 77, 1, 96, 64, 5, 37, 64, 48, 3, 15, usage="iid",
                         value_std=1.0), 96, None),
    "bf16_fus_image": (WORKLOADS[1].scaled(value_std=1.0), 2048, 80),
    # a gate/up grid of 1024 workgroups: the product's two-stage ring
    "bf16_fus_wide": (Workload("bf16_fus_wide", "bf16", 4000, 2, 256, 128, 20, 60, 256, 320, 8,
                               25, usage="uniform", value_std=1.0), 1024, 60),
}


@pytest.mark.parametrize("name", list(FUSION))
def test_fused_injection(name):
    """lookme_select then lookme_inject_fused against the oracle's
    round(H + f(round(R))) on the library's primitives; other rows keep
    their bits; two passes from the same inputs agree bit for bit."""
    from tests.harness import FusedRun, check_fused_run
    wl, d_ff, sample = FUSION[name]
    _announce(f"fusion {name}: {wl} d_ff {d_ff}")
    inp = make_inputs(wl, seed=6, device=DEV)
    fus = make_fusion(wl, 6, d_ff, device=DEV)
    r = FusedRun(inp, fus).run()
    toks = None
    if sample:
        kept0 = r.kept[0].cpu().numpy()[:40]
        toks = np.unique(np.concatenate(
            [np.random.default_rng(6).choice(wl.n_tokens, sample, replace=False), kept0]))
    rep = check_fused_run(r, tokens=toks)
    assert rep.ok, str(rep)
    assert rep.decisions.get("hidden_row", 0) > 0
    r2 = FusedRun(inp, fus, table=r.table).run()
    torch.cuda.synchronize()
    assert torch.equal(r.hidden, r2.hidden)


# layers = the LookME layer + the propagated ones
PROPAGATION = {
    "bf16_prop_small": (Workload("bf16_prop_small", "bf16", 300, 3, 256, 128, 20, 60, 128, 80,
                                 8, 30, usage="uniform", value_std=1.0), 192, None),
    "f32_prop": (Workload("f32_prop", "f32", 77, 2, 96, 64, 5, 37, 64, 48, 3, 15, usage="iid",
                          value_std=1.0), 96, None),
    "bf16_prop_image": (WORKLOADS[1].scaled(layers=4, value_std=1.0), 2048, 80),
}


def _sample_with_kept(r, wl, sample, seed):
    if not sample:
        return None
    kept0 = r.kept[0].cpu().numpy()[:40]
    return np.unique(np.concatenate(
        [np.random.default_rng(seed).choice(wl.n_tokens, sample, replace=False), kept0]))


@pytest.mark.parametrize("name", list(PROPAGATION))
def test_propagated_injection(name):
    """One lookup and kept set at the LookME layer, R carried through the
    propagation of Eq. 11 to the layers after it, each injected through its
    own fusion: against the oracle's chain on the library's primitives and
    weights; two passes agree bit for bit."""
    from tests.harness import PropagatedRun, check_propagated_run
    wl, d_ff, sample = PROPAGATION[name]
    _announce(f"propagation {name}: {wl} d_ff {d_ff}")
    inp = make_inputs(wl, seed=7, device=DEV)
    fus = make_fusion(wl, 7, d_ff, device=DEV)
    w_p_t = make_propagation(wl, 7, wl.layers - 1, device=DEV)
    r = PropagatedRun(inp, fus, w_p_t).run()
    rep = check_propagated_run(r, tokens=_sample_with_kept(r, wl, sample, 7))
    assert rep.ok, str(rep)
    assert rep.decisions.get("hidden_row", 0) > 0
    r2 = PropagatedRun(inp, fus, w_p_t, table=r.table).run()
    torch.cuda.synchronize()
    assert torch.equal(r.hidden, r2.hidden)


def test_propagated_special_cases_match_fused_injection():
    """No steps: the same bits as lookme_inject_fused on one layer.  W_p = 0:
    every R_j is R_0 exactly, so layer j gets the bits of lookme_inject_fused
    over three layers that all carry the LookME layer's lookup and kept set."""
    from tests.harness import FusedRun, PropagatedRun
    wl = Workload("bf16_prop_eq", "bf16", 300, 3, 256, 128, 20, 60, 128, 80, 8, 30,
                  usage="uniform", value_std=1.0)
    _announce(f"propagation special cases: {wl}")
    inp = make_inputs(wl, seed=8, device=DEV)
    fus = make_fusion(wl, 8, 192, device=DEV)
    zeros = torch.zeros((2, wl.d_v, wl.d_v), dtype=torch.bfloat16, device=DEV)
    r = PropagatedRun(inp, fus, zeros).run()
    n_keep = r.n_keep
    rep3 = lambda t: t[:1].expand(3, *t.shape[1:]).contiguous()
    hidden = inp["hidden"].clone()
    r.table.inject_fused(rep3(r.kept), rep3(r.scene), rep3(r.prim), rep3(r.w), hidden, n_keep,
                         layers=3)
    torch.cuda.synchronize()
    assert torch.equal(r.hidden, hidden)
    assert not torch.equal(r.hidden[2], inp["hidden"][2])

    one = {k: (v[:1].contiguous() if k in ("wt", "delta", "hidden") else v)
           for k, v in inp.items()}
    fus1 = {k: (v[:1].contiguous() if torch.is_tensor(v) else v) for k, v in fus.items()}
    p0 = PropagatedRun(one, fus1, zeros).run()
    f0 = FusedRun(one, fus1).run()
    torch.cuda.synchronize()
    assert p0.steps == 0
    assert torch.equal(p0.hidden, f0.hidden)


# (workload, scales, sampled tokens or None for all)
MULTISCALE = {
    "bf16_ms_small": (Workload("bf16_ms_small", "bf16", 300, 1, 256, 128, 20, 60, 128, 192, 8,
                               30, usage="iid", value_std=1.0), 2, None),
    "f32_ms_three": (Workload("f32_ms_three", "f32", 77, 1, 96, 64, 15, 37, 64, 96, 3, 20,
                              usage="iid", value_std=1.0), 3, None),
    "bf16_ms_image": (WORKLOADS[1].scaled(value_std=1.0), 2, 80),
    # the multi-scale batch's shape: 23040 tokens a scale, 1024 scenes split
    # over two scales, rows of width 1536 into hidden 2048
    "bf16_ms_batch": (WORKLOADS[2].scaled(value_std=1.0), 2, 80),
}


@pytest.mark.parametrize("name", list(MULTISCALE))
def test_multiscale_injection(name):
    """Per-scale projection, routing within the scale's scene partition and
    lookup, the kept set, and the router's mix of the scales' rows (Eq. 8)
    against the oracle; two passes agree bit for bit."""
    from tests.harness import MultiScaleRun, check_multiscale_run
    wl, scales, sample = MULTISCALE[name]
    _announce(f"multi-scale {name}: {wl} scales {scales}")
    inp = make_inputs(wl, seed=9, device=DEV)
    ms = make_multiscale(wl, 9, scales, device=DEV)
    r = MultiScaleRun(inp, ms).run()
    toks = None
    if sample:
        kept0 = r.kept.cpu().numpy()[:40]
        toks = np.unique(np.concatenate(
            [np.random.default_rng(9).choice(wl.n_tokens, sample, replace=False), kept0]))
    rep = check_multiscale_run(r, tokens=toks)
    assert rep.ok, str(rep)
    assert min(rep.decisions.get(kind, 0) for kind in ("scene", "prim", "hidden_row")) > 0
    r2 = MultiScaleRun(inp, ms, table=r.table).run()
    torch.cuda.synchronize()
    assert torch.equal(r.hidden, r2.hidden)
    assert int(r.scene.max()) < wl.scenes // scales


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_benchmark_workloads_sampled(cfg):
    """Full-size workloads in the benchmark's launch configuration; sampled
    tokens are checked stage-wise, the kept set in full."""
    from tests.harness import Run, check_end_to_end_run, check_run
    wl = WORKLOADS[cfg]
    _announce(f"config {cfg}: {wl}")
    inp = make_inputs(wl, seed=cfg, device=DEV)
    r = Run(inp).run()
    rng = np.random.default_rng(cfg)
    kept0 = r.kept[0].cpu().numpy()[: min(48, wl.n_keep)]
    toks = np.unique(np.concatenate([rng.choice(wl.n_tokens, 80, replace=False), kept0]))
    rep = check_run(r, tokens=toks)
    assert rep.ok, str(rep)
    # end-to-end mode: the oracle's own decisions from the original inputs
    e2e = check_end_to_end_run(r, tokens=toks)
    assert e2e.ok, str(e2e)
    if wl.usage != "iid":
        lab = inp["labels"].cpu().numpy()
        assert np.mean(r.scene[0].cpu().numpy() == lab) > 0.99
    del inp, r
    torch.cuda.empty_cache()


@pytest.mark.parametrize("case", ["bf16_ragged", "f32_small", "bf16_zipf_prims"])
def test_scene_keys_eq4(case):
    """lookme_scene_keys (Eq. 4) against the oracle's exact means within the
    float32 summation bound (oracle/check.py:check_scene_keys), on the
    primitive keys of seeded workloads: ragged sizes, fp32, and 4096
    primitives a scene as in the Zipf workload."""
    from oracle import check as C
    from paper_2607_16305_amd import lookme as lk
    from tests.harness import to_np
    wl = {"bf16_ragged": SMALL["bf16_ragged_l2"], "f32_small": SMALL["f32_proj_l3"],
          "bf16_zipf_prims": Workload("bf16_zipf_prims", "bf16", 16, 1, 512, 512, 48, 4096,
                                      64, 64, 16, 20)}[case]
    _announce(f"scene keys {case}: S={wl.scenes} P={wl.prims} d_e={wl.d_e} {wl.dtype}")
    inp = make_inputs(wl, seed=3, device=DEV)
    pk = inp["prim_keys"]
    keys = lk.scene_keys(pk)
    torch.cuda.synchronize()
    rep = C.Report()
    C.check_scene_keys(to_np(keys.cpu()), to_np(pk.cpu()), wl.dtype, rep)
    assert rep.ok, str(rep)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_scene_keys_exact_on_integer_keys(dtype):
    """Integer keys in [-2, 2] with P a power of two: every float32 partial
    sum is exact and so is the division, so the library's keys must be the
    correctly rounded means bit for bit."""
    from paper_2607_16305_amd import lookme as lk
    from tests.harness import to_np
    _announce(f"scene keys exact {dtype}")
    g = torch.Generator(device="cpu").manual_seed(11)
    S, P, d = 5, 1024, 96 if dtype == "bf16" else 48
    ik = torch.randint(-2, 3, (S, P, d), generator=g).to(torch.float32)
    pk = ik.to(torch.bfloat16 if dtype == "bf16" else torch.float32).to(DEV)
    keys = lk.scene_keys(pk)
    torch.cuda.synchronize()
    exact = O.round_to_dtype(ik.double().numpy().sum(axis=1) / P, dtype)
    got = O.to_f64(to_np(keys.cpu()), dtype)
    assert np.array_equal(got, exact)


def test_out_of_range_indices_are_counted_not_injected():
    """Kept entries with a token id, scene or primitive out of range are left
    out (their hidden rows keep their bits), every other kept row gets the
    same bits as with a clean list, and lookme_index_errors reports the bad
    entries once (then zero)."""
    from paper_2607_16305_amd import lookme as lk
    from tests.harness import Run
    wl = SMALL["bf16_ragged_l2"]
    _announce("index errors bf16_ragged_l2")
    inp = make_inputs(wl, seed=5, device=DEV)
    ref = Run(inp).run()
    torch.cuda.synchronize()
    assert lk.lookme_index_errors() == 0   # nothing counted by a clean pass
    L, n = ref.L, ref.n
    kept = ref.kept.clone()
    scene = ref.scene.clone()
    prim = ref.prim.clone()
    bad_tokens = []
    kept[0, 0] = -1                          # token id below the range
    kept[1, 1] = n                           # and above it
    t2 = int(kept[0, 2])
    scene[0, t2] = wl.scenes                 # scene out of range
    t3 = int(kept[1, 3])
    prim[1, t3, wl.top_k - 1] = wl.prims     # one primitive out of range
    bad_tokens = [(0, t2), (1, t3)]
    hidden = inp["hidden"].clone()
    ref.table.inject_kept(kept, scene, prim, ref.w, hidden, ref.n_keep, layers=L)
    assert lk.lookme_index_errors() == 4
    assert lk.lookme_index_errors() == 0
    # the bad entries' rows (where they exist) keep their bits
    for l, t in bad_tokens:
        assert torch.equal(hidden[l, t], inp["hidden"][l, t])
    # every other kept row as injected by the clean pass; the rest untouched
    skip = {(0, int(ref.kept[0, 0])), (1, int(ref.kept[1, 1]))} | set(bad_tokens)
    for l in range(L):
        for t in ref.kept[l].tolist():
            if (l, t) in skip:
                assert torch.equal(hidden[l, t], inp["hidden"][l, t])
            else:
                assert torch.equal(hidden[l, t], ref.hidden[l, t]), (l, t)
