"""GPU test of lookme_inject_noalloc, the variant of lookme_inject that
allocates nothing (its scratch is a static device array of the library):
through the C ABI, on the same inputs, its results must be the bits of
lookme_inject's, for two calls in a row, the second on a smaller batch, with
and without a kept output."""

import pytest
import torch

from synth import Workload, make_inputs

pytestmark = pytest.mark.gpu


def _announce(msg):
    print(f"[gpu-noalloc] {msg}", flush=True)


def _lookup(inp, table, wl):
    L, n = wl.layers, wl.n_tokens
    dev = inp["x"].device
    q = torch.empty((L, n, wl.d_e), dtype=inp["x"].dtype, device=dev)
    scene = torch.empty((L, n), dtype=torch.int32, device=dev)
    prim = torch.empty((L, n, wl.top_k), dtype=torch.int32, device=dev)
    w = torch.empty((L, n, wl.top_k), dtype=torch.float32, device=dev)
    table.route(inp["x"], inp["wt"], q, scene, layers=L)
    table.lookup(q, scene, prim, w, layers=L)
    return scene, prim, w


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_inject_noalloc_matches_inject_on_two_calls(dtype):
    from paper_2607_16305_amd import lookme as lk
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    lk.load()
    big = Workload(f"noalloc_{dtype}_big", dtype, 3000, 2, 256, 256, 24, 64, 384, 512, 8, 20,
                   usage="uniform")
    small = Workload(f"noalloc_{dtype}_small", dtype, 700, 1, 256, 256, 24, 64, 384, 512, 8, 35,
                     usage="uniform")
    for wl in (big, small):
        _announce(f"{wl}")
        inp = make_inputs(wl, seed=11, device="cuda")
        table = lk.Table(inp["scene_keys"], inp["prim_keys"], inp["values"], wl.top_k)
        table.reserve(wl.layers, wl.n_tokens)
        scene, prim, w = _lookup(inp, table, wl)
        L, n, nk = wl.layers, wl.n_tokens, wl.n_keep
        ref_h = inp["hidden"].clone()
        ref_kept = torch.full((L, nk), -7, dtype=torch.int32, device="cuda")
        lk.lookme_inject(table.handle, L, n, nk, inp["delta"], wl.crit_dim, scene, prim, w,
                         ref_h, wl.d_h, ref_kept)
        got_h = inp["hidden"].clone()
        got_kept = torch.full((L, nk), -7, dtype=torch.int32, device="cuda")
        lk.lookme_inject_noalloc(table.handle, L, n, nk, inp["delta"], wl.crit_dim, scene, prim,
                                 w, got_h, wl.d_h, got_kept)
        # and with the kept lists in the library's scratch
        got_h2 = inp["hidden"].clone()
        lk.lookme_inject_noalloc(table.handle, L, n, nk, inp["delta"], wl.crit_dim, scene, prim,
                                 w, got_h2, wl.d_h, None)
        torch.cuda.synchronize()
        assert torch.equal(got_kept, ref_kept)
        assert torch.equal(got_h, ref_h)
        assert torch.equal(got_h2, ref_h)
        assert not torch.equal(ref_h, inp["hidden"])
        # the kept set is the oracle's (ties within the relative rule exempt)
        from oracle import check as C
        from oracle import lookme_oracle as O
        from tests.harness import f64
        rep = C.Report()
        for l in range(L):
            C.check_kept(O.criticality(f64(inp["delta"][l])), nk, ref_kept[l].cpu().numpy(), rep)
        assert rep.finish().ok, str(rep)
        del table
