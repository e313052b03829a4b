"""Test-side driver: runs the library through its C ABI on one workload and
checks every stage against the oracle (stage-wise, see oracle/check.py).

Used by the GPU tests, the smoke check and the benchmark's parity sample.
"""

from __future__ import annotations

import numpy as np
import torch

from oracle import check as C
from oracle import lookme_oracle as O
from paper_2607_16305_amd import lookme as lk


def to_np(t: torch.Tensor) -> np.ndarray:
    """Stored representation: bf16 -> uint16 bits, fp32 -> float32, ints as is."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def dtype_name(t: torch.Tensor) -> str:
    return "bf16" if t.dtype == torch.bfloat16 else "f32"


def f64(t: torch.Tensor) -> np.ndarray:
    return O.to_f64(to_np(t), dtype_name(t))


class Run:
    """Outputs of one pass of the path (device tensors) plus the inputs."""

    def __init__(self, inp: dict, n_keep: int | None = None, k: int | None = None,
                 table: lk.Table | None = None, with_kept=True, stream=None, score: str = "dot"):
        self.inp = inp
        self.score = score
        x, wt = inp["x"], inp["wt"]
        self.dev = x.device
        self.L = inp["hidden"].shape[0]
        self.n = x.shape[0]
        self.k = k if k is not None else inp["k"]
        self.n_keep = n_keep if n_keep is not None else inp["n_keep"]
        S, P, d_e = inp["prim_keys"].shape
        self.S, self.P, self.d_e = S, P, d_e
        self.table = table or lk.Table(
            inp["scene_keys"], inp["prim_keys"], inp["values"], self.k, inp.get("bias"),
            score=lk.LOOKME_SCORE_COS if score == "cos" else lk.LOOKME_SCORE_DOT)
        self.table.reserve(self.L, self.n)
        L, n = self.L, self.n
        dt = x.dtype
        self.q = torch.empty((L, n, d_e), dtype=dt, device=self.dev)
        self.scene = torch.full((L, n), -7, dtype=torch.int32, device=self.dev)
        self.prim = torch.full((L, n, self.k), -7, dtype=torch.int32, device=self.dev)
        self.w = torch.full((L, n, self.k), -7.0, dtype=torch.float32, device=self.dev)
        self.kept = (torch.full((L, max(self.n_keep, 1)), -7, dtype=torch.int32,
                                device=self.dev) if with_kept else None)
        self.h_in = inp["hidden"].clone()
        self.hidden = inp["hidden"].clone()
        self.stream = stream

    def run(self):
        inp, L = self.inp, self.L
        self.table.route(inp["x"], inp["wt"], self.q, self.scene, layers=L, stream=self.stream)
        self.table.lookup(self.q, self.scene, self.prim, self.w, layers=L, stream=self.stream)
        self.table.inject(inp["delta"], self.scene, self.prim, self.w, self.hidden, self.n_keep,
                          kept_out=self.kept, layers=L, stream=self.stream)
        return self

    def run_split(self):
        """The same pass with the kept set selected on a second stream while
        routing and lookup run, then the rows added for that set."""
        inp, L = self.inp, self.L
        main = torch.cuda.current_stream()
        side = torch.cuda.Stream()
        self.table.reserve(L, self.n)
        side.wait_stream(main)
        with torch.cuda.stream(side):
            self.table.select(inp["delta"], self.kept, self.n_keep, layers=L, stream=side)
        self.table.route(inp["x"], inp["wt"], self.q, self.scene, layers=L, stream=main)
        self.table.lookup(self.q, self.scene, self.prim, self.w, layers=L, stream=main)
        main.wait_stream(side)
        self.table.inject_kept(self.kept, self.scene, self.prim, self.w, self.hidden, self.n_keep,
                               layers=L, stream=main)
        return self


def run_fused_select(r: Run) -> Run:
    """The pass of ``r`` with lookme_lookup_select (the select carried by the
    lookup's bucketing launch, one stream), then lookme_inject_kept."""
    inp, L = r.inp, r.L
    r.table.route(inp["x"], inp["wt"], r.q, r.scene, layers=L, stream=r.stream)
    r.table.lookup_select(r.q, r.scene, r.prim, r.w, inp["delta"], r.kept, r.n_keep, layers=L,
                          stream=r.stream)
    r.table.inject_kept(r.kept, r.scene, r.prim, r.w, r.hidden, r.n_keep, layers=L,
                        stream=r.stream)
    return r


class RelevanceRun(Run):
    """A pass with Level-2 in the paper's form (Eq. 6-7): routing, the
    relevance lookup (hidden activations, primitives, weights), then the kept
    set and the injection as in the configured path."""

    def __init__(self, inp: dict, mlp: dict, **kw):
        super().__init__(inp, **kw)
        self.mlp = mlp
        self.act = torch.full((self.L, self.n, mlp["hidden"]), 7, dtype=inp["x"].dtype,
                              device=self.dev)
        self.table.set_relevance(mlp["w1"], mlp["b1"], mlp["w2"], mlp["b2"])

    def run(self):
        inp, L = self.inp, self.L
        self.table.route(inp["x"], inp["wt"], self.q, self.scene, layers=L, stream=self.stream)
        self.table.lookup_relevance(self.q, self.scene, self.act, self.prim, self.w, layers=L,
                                    stream=self.stream)
        self.table.inject(inp["delta"], self.scene, self.prim, self.w, self.hidden, self.n_keep,
                          kept_out=self.kept, layers=L, stream=self.stream)
        return self


class FusedRun(Run):
    """A pass whose injection goes through the SwiGLU fusion of Eq. 10:
    route, lookup, the kept set (lookme_select), then lookme_inject_fused."""

    def __init__(self, inp: dict, fus: dict, **kw):
        super().__init__(inp, **kw)
        self.fus = fus
        self.table.set_fusion(fus["w_gate"], fus["w_up"], fus["w_down"])

    def run(self):
        inp, L = self.inp, self.L
        self.table.route(inp["x"], inp["wt"], self.q, self.scene, layers=L, stream=self.stream)
        self.table.lookup(self.q, self.scene, self.prim, self.w, layers=L, stream=self.stream)
        self.table.select(inp["delta"], self.kept, self.n_keep, layers=L, stream=self.stream)
        self.table.inject_fused(self.kept, self.scene, self.prim, self.w, self.hidden,
                                self.n_keep, layers=L, stream=self.stream)
        return self


class PropagatedRun(Run):
    """A LookME layer followed by ``steps`` non-LookME layers (Eq. 11): the
    first layer's route, lookup and kept set, then lookme_inject_propagated
    into the hidden states of all steps + 1 layers (the workload's layer
    count)."""

    def __init__(self, inp: dict, fus: dict, w_p_t: torch.Tensor, **kw):
        super().__init__(inp, **kw)
        self.fus, self.w_p_t = fus, w_p_t
        self.steps = self.L - 1
        self.table.set_fusion(fus["w_gate"], fus["w_up"], fus["w_down"])
        if self.steps > 0:
            self.table.set_propagation(w_p_t)

    def run(self):
        inp, st = self.inp, self.stream
        self.table.route(inp["x"], inp["wt"][:1], self.q[:1], self.scene[:1], layers=1, stream=st)
        self.table.lookup(self.q[:1], self.scene[:1], self.prim[:1], self.w[:1], layers=1,
                          stream=st)
        self.table.select(inp["delta"][:1], self.kept[:1], self.n_keep, layers=1, stream=st)
        self.table.inject_propagated(self.kept[0], self.scene[0], self.prim[0], self.w[0],
                                     self.hidden, self.n_keep, self.steps, stream=st)
        return self


def check_propagated_run(r: PropagatedRun, tokens=None) -> C.Report:
    """The LookME layer's kept set in full and every layer's injected rows on
    the sampled tokens."""
    torch.cuda.synchronize()
    inp, fus = r.inp, r.fus
    dt = dtype_name(inp["x"])
    rep = C.Report()
    toks = np.arange(r.n) if tokens is None else np.asarray(tokens)
    tsel = torch.as_tensor(toks, device=r.dev)
    values = inp["values"]

    def values_rows(rows):
        idx = torch.as_tensor(np.asarray(rows), device=values.device, dtype=torch.long)
        return f64(values[idx])

    c = O.criticality(f64(inp["delta"][0]))
    kept = to_np(r.kept[0])[: r.n_keep]
    C.check_kept(c, r.n_keep, kept, rep)
    w_p = f64(r.w_p_t[: r.steps]).transpose(0, 2, 1) if r.steps else np.zeros((0, 1, 1))
    C.check_propagated_hidden(to_np(r.h_in[:, tsel]), to_np(r.hidden[:, tsel]), dt, values_rows,
                              r.P, to_np(r.scene[0]), to_np(r.prim[0]), to_np(r.w[0]), kept, w_p,
                              f64(fus["w_gate"]), f64(fus["w_up"]), f64(fus["w_down"]), rep, toks)
    return rep.finish()


class MultiScaleRun:
    """Multi-scale image pathway of one layer (Sec. 3.2, Eq. 8): scale m's
    tokens are projected, routed and looked up on a table over its scene
    partition (Table.scale_view), the kept set comes from the layer's
    criticality, and lookme_inject_multiscale mixes the scales' rows into the
    hidden states."""

    def __init__(self, inp: dict, ms: dict, table: lk.Table | None = None, stream=None):
        self.inp, self.ms = inp, ms
        x = ms["x"]
        self.M, self.n = ms["scales"], x.shape[1]
        self.k, self.n_keep = inp["k"], inp["n_keep"]
        S, P, d_e = inp["prim_keys"].shape
        self.S, self.P, self.d_e = S, P, d_e
        self.dev = x.device
        self.stream = stream
        self.table = table or lk.Table(inp["scene_keys"], inp["prim_keys"], inp["values"], self.k)
        self.table.set_multiscale(self.M, ms["w_he_t"])
        self.table.reserve(1, self.n)
        self.scales = [self.table.scale_view(m, self.M) for m in range(self.M)]
        M, n, k = self.M, self.n, self.k
        # one buffer per scale (16-byte aligned whatever n is), stacked into
        # the [M, n, ...] tensors that the injection reads
        self.qs = [torch.empty((n, d_e), dtype=x.dtype, device=self.dev) for _ in range(M)]
        self.scenes = [torch.full((n,), -7, dtype=torch.int32, device=self.dev) for _ in range(M)]
        self.prims = [torch.full((n, k), -7, dtype=torch.int32, device=self.dev)
                      for _ in range(M)]
        self.ws = [torch.full((n, k), -7.0, dtype=torch.float32, device=self.dev)
                   for _ in range(M)]
        self.kept = torch.full((max(self.n_keep, 1),), -7, dtype=torch.int32, device=self.dev)
        self.h_in = self.inp["hidden"][0].clone()
        self.hidden = self.inp["hidden"][0].clone()

    def run(self):
        ms, st = self.ms, self.stream
        for m, t in enumerate(self.scales):
            t.route(ms["x"][m], ms["wt"][m:m + 1], self.qs[m], self.scenes[m], layers=1,
                    stream=st)
            t.lookup(self.qs[m], self.scenes[m], self.prims[m], self.ws[m], layers=1, stream=st)
        self.q, self.scene = torch.stack(self.qs), torch.stack(self.scenes)
        self.prim, self.w = torch.stack(self.prims), torch.stack(self.ws)
        self.table.select(self.inp["delta"][:1], self.kept, self.n_keep, layers=1, stream=st)
        self.table.inject_multiscale(self.kept, self.scene, self.prim, self.w, self.hidden,
                                     self.n_keep, stream=st)
        return self


def check_multiscale_run(r: MultiScaleRun, tokens=None) -> C.Report:
    """Every scale's projection, routing (within its partition) and lookup on
    the sampled tokens, the kept set in full, and the mixed injection."""
    torch.cuda.synchronize()
    inp, ms = r.inp, r.ms
    dt = dtype_name(inp["x"])
    rep = C.Report()
    toks = np.arange(r.n) if tokens is None else np.asarray(tokens)
    tsel = torch.as_tensor(toks, device=r.dev)
    Sm = r.S // r.M
    K1 = f64(inp["scene_keys"])
    prim_keys, values = inp["prim_keys"], inp["values"]

    def values_rows(rows):
        idx = torch.as_tensor(np.asarray(rows), device=values.device, dtype=torch.long)
        return f64(values[idx])

    w_lib = to_np(r.w)
    for m in range(r.M):
        q_bits = to_np(r.q[m])[toks]
        C.check_projection(q_bits, f64(ms["x"][m][tsel]), f64(ms["wt"][m]), dt, rep)
        q_lib = O.to_f64(q_bits, dt)
        scene = to_np(r.scene[m]).astype(np.int64)
        C.check_scene(q_lib, K1[m * Sm:(m + 1) * Sm], None, "dot", scene[toks], rep)
        C.check_prim(q_lib, scene[toks], lambda s, m=m: f64(prim_keys[m * Sm + s]), r.k, "dot",
                     to_np(r.prim[m])[toks], w_lib[m][toks], rep)
    c = O.criticality(f64(inp["delta"][0]))
    kept = to_np(r.kept)[: r.n_keep]
    C.check_kept(c, r.n_keep, kept, rep)
    C.check_multiscale_hidden(to_np(r.h_in[tsel]), to_np(r.hidden[tsel]), dt, values_rows, r.P, Sm,
                              to_np(r.scene), to_np(r.prim), w_lib, kept,
                              f64(ms["w_he_t"]).T, rep, toks)
    return rep.finish()


def check_fused_run(r: FusedRun, tokens=None) -> C.Report:
    """The kept set in full and the fused injection on the sampled tokens
    (routing and lookup are checked by check_run and are the same here)."""
    torch.cuda.synchronize()
    inp, fus = r.inp, r.fus
    dt = dtype_name(inp["x"])
    rep = C.Report()
    toks = np.arange(r.n) if tokens is None else np.asarray(tokens)
    tsel = torch.as_tensor(toks, device=r.dev)
    values = inp["values"]

    def values_rows(rows):
        idx = torch.as_tensor(np.asarray(rows), device=values.device, dtype=torch.long)
        return f64(values[idx])

    for l in range(r.L):
        c = O.criticality(f64(inp["delta"][l]))
        kept = to_np(r.kept[l])[: r.n_keep]
        C.check_kept(c, r.n_keep, kept, rep)
        C.check_fused_hidden(to_np(r.h_in[l][tsel]), to_np(r.hidden[l][tsel]), dt, values_rows,
                             r.P, to_np(r.scene[l]), to_np(r.prim[l]), to_np(r.w[l]), kept,
                             f64(fus["w_gate"][l]), f64(fus["w_up"][l]), f64(fus["w_down"][l]),
                             rep, toks)
    return rep.finish()


def check_relevance_run(r: RelevanceRun, tokens=None) -> C.Report:
    """Stage-wise check of a relevance pass on the sampled tokens: q and the
    scene as in check_run, the hidden activations (C1 bound), the primitives
    and weights on the library's activations (C3/C4), the injected rows."""
    torch.cuda.synchronize()
    inp, mlp = r.inp, r.mlp
    dt = dtype_name(inp["x"])
    rep = C.Report()
    toks = np.arange(r.n) if tokens is None else np.asarray(tokens)
    tsel = torch.as_tensor(toks, device=r.dev)
    K1 = f64(inp["scene_keys"])
    w1, w2 = f64(mlp["w1"]), f64(mlp["w2"])
    b1 = mlp["b1"].cpu().numpy().astype(np.float64)
    b2 = mlp["b2"].cpu().numpy().astype(np.float64)
    prim_keys = inp["prim_keys"]
    values = inp["values"]
    x64 = f64(inp["x"][tsel])

    def values_rows(rows):
        idx = torch.as_tensor(np.asarray(rows), device=values.device, dtype=torch.long)
        return f64(values[idx])

    for l in range(r.L):
        q_bits = to_np(r.q[l])[toks]
        if inp["wt"] is not None:
            C.check_projection(q_bits, x64, f64(inp["wt"][l]), dt, rep)
        q_lib = O.to_f64(q_bits, dt)
        scene = to_np(r.scene[l]).astype(np.int64)
        C.check_scene(q_lib, K1, None, "dot", scene[toks], rep)
        act_bits = to_np(r.act[l])[toks]
        C.check_relevance_hidden(act_bits, q_lib, scene[toks], K1, w1, b1, dt, rep)
        prim = to_np(r.prim[l])
        w = to_np(r.w[l])
        w_orc = C.check_relevance_prim(O.to_f64(act_bits, dt), w2, b2, q_lib, scene[toks],
                                       lambda s: f64(prim_keys[s]), r.k, prim[toks], w[toks],
                                       rep)
        w_of = {int(t): w_orc[i] for i, t in enumerate(toks)}
        c = O.criticality(f64(inp["delta"][l]))
        kept = to_np(r.kept[l])[: r.n_keep]
        C.check_kept(c, r.n_keep, kept, rep)
        C.check_hidden(to_np(r.h_in[l][tsel]), to_np(r.hidden[l][tsel]), dt, values_rows, r.P,
                       scene, prim, lambda t: w_of[t], kept, rep, tokens=toks,
                       w_lib_of=lambda t: w[t])
    return rep.finish()


def check_run(r: Run, tokens=None, layers=None) -> C.Report:
    """Stage-wise comparison of a finished run against the oracle.

    ``tokens``: None for every token, else an array of token indices that are
    checked for route/lookup/inject (the kept set is always checked in full,
    since it is a global selection)."""
    torch.cuda.synchronize()
    inp = r.inp
    dt = dtype_name(inp["x"])
    rep = C.Report()
    L = r.L
    layers = range(L) if layers is None else layers
    toks = np.arange(r.n) if tokens is None else np.asarray(tokens)
    K1 = f64(inp["scene_keys"])
    bias = None if inp.get("bias") is None else inp["bias"].detach().cpu().numpy().astype(np.float64)
    prim_keys = inp["prim_keys"]
    values = inp["values"]
    x64 = f64(inp["x"][torch.as_tensor(toks, device=inp["x"].device)])

    def scene_keys_of(s):
        return f64(prim_keys[s])

    def values_rows(rows):
        idx = torch.as_tensor(np.asarray(rows), device=values.device, dtype=torch.long)
        return f64(values[idx])

    for l in layers:
        # C1: projection of the sampled tokens
        q_lib_bits = to_np(r.q[l])[toks]
        if inp["wt"] is not None:
            C.check_projection(q_lib_bits, x64, f64(inp["wt"][l]), dt, rep)
        else:
            C.check_q(q_lib_bits, O.from_f64(x64, dt), dt, rep, max_ulp=0)
        q_lib = O.to_f64(q_lib_bits, dt)
        # C2: scene on the library's q
        scene = to_np(r.scene[l]).astype(np.int64)
        C.check_scene(q_lib, K1, bias, r.score, scene[toks], rep)
        # C3/C4: primitives under the library's scene
        prim = to_np(r.prim[l])
        w = to_np(r.w[l])
        w_orc = C.check_prim(q_lib, scene[toks], scene_keys_of, r.k, r.score, prim[toks],
                             w[toks], rep)
        w_of = {int(t): w_orc[i] for i, t in enumerate(toks)}
        # C5: kept set (global)
        c = O.criticality(f64(inp["delta"][l]))
        kept_lib = to_np(r.kept[l])[: r.n_keep] if r.kept is not None else None
        if kept_lib is not None:
            C.check_kept(c, r.n_keep, kept_lib, rep)
        kept = kept_lib if kept_lib is not None else O.select(c, r.n_keep)
        # C6: hidden rows of the sampled tokens
        tsel = torch.as_tensor(toks, device=r.h_in.device)
        C.check_hidden(to_np(r.h_in[l][tsel]), to_np(r.hidden[l][tsel]), dt, values_rows, r.P,
                       scene, prim, lambda t: w_of[t], kept, rep, tokens=toks,
                       w_lib_of=lambda t: w[t])
    return rep.finish()


def check_end_to_end_run(r: Run, tokens=None, layers=None) -> C.Report:
    """End-to-end comparison of a finished run: the oracle computes every
    stage from the original inputs (oracle/check.py: check_end_to_end) and
    the library's final hidden rows, decisions and weights are compared with
    its own, ties counted."""
    torch.cuda.synchronize()
    inp = r.inp
    dt = dtype_name(inp["x"])
    rep = C.Report()
    layers = range(r.L) if layers is None else layers
    toks = np.arange(r.n) if tokens is None else np.asarray(tokens)
    tsel = torch.as_tensor(toks, device=r.dev)
    K1 = f64(inp["scene_keys"])
    bias = None if inp.get("bias") is None else inp["bias"].detach().cpu().numpy().astype(np.float64)
    prim_keys, values = inp["prim_keys"], inp["values"]
    x64 = f64(inp["x"][tsel])

    class Keys:
        def __getitem__(self, s):
            return f64(prim_keys[int(s)])

    def values_rows(rows):
        idx = torch.as_tensor(np.asarray(rows), device=values.device, dtype=torch.long)
        return f64(values[idx])

    for l in layers:
        wt = None if inp["wt"] is None else f64(inp["wt"][l])
        C.check_end_to_end(x64, wt, K1, bias, r.score, Keys(), values_rows, r.P, r.k,
                           O.criticality(f64(inp["delta"][l])), r.n_keep,
                           to_np(r.h_in[l][tsel]), to_np(r.hidden[l][tsel]), dt,
                           to_np(r.q[l])[toks], to_np(r.scene[l]).astype(np.int64),
                           to_np(r.prim[l]), to_np(r.w[l]), to_np(r.kept[l])[: r.n_keep], rep,
                           toks)
    return rep.finish()


class GatedRun(Run):
    """A pass with the learned SKA gate (Eq. 9-10): route and lookup, the
    gate of every layer (lookme_gate: a counted, ascending kept list), then
    the injection for those lists -- the prefix add (mode "plain",
    lookme_inject_gated), the SwiGLU fusion ("fused") or the fusion with the
    gate reused by ``steps`` propagated layers ("propagated", Eq. 11)."""

    def __init__(self, inp: dict, w_g: torch.Tensor, mode: str = "plain", fus=None,
                 w_p_t=None, **kw):
        super().__init__(inp, with_kept=False, **kw)
        self.w_g, self.mode, self.fus, self.w_p_t = w_g, mode, fus, w_p_t
        self.steps = self.L - 1 if mode == "propagated" else 0
        if mode in ("fused", "propagated"):
            self.table.set_fusion(fus["w_gate"], fus["w_up"], fus["w_down"])
        if self.steps > 0:
            self.table.set_propagation(w_p_t)
        gl = 1 if mode == "propagated" else self.L
        self.glayers = gl
        self.kept = torch.full((gl, self.n), -7, dtype=torch.int32, device=self.dev)
        self.count = torch.full((gl,), -7, dtype=torch.int32, device=self.dev)

    def run(self):
        inp, st, gl = self.inp, self.stream, self.glayers
        wt = None if inp["wt"] is None else inp["wt"][:gl]
        self.table.route(inp["x"], wt, self.q[:gl], self.scene[:gl], layers=gl, stream=st)
        self.table.lookup(self.q[:gl], self.scene[:gl], self.prim[:gl], self.w[:gl], layers=gl,
                          stream=st)
        self.table.gate(inp["delta"][:gl], self.w_g[:gl], self.kept, self.count, layers=gl,
                        stream=st)
        if self.mode == "plain":
            self.table.inject_gated(self.kept, self.count, self.scene, self.prim, self.w,
                                    self.hidden, layers=gl, stream=st)
        elif self.mode == "fused":
            self.table.inject_fused_gated(self.kept, self.count, self.scene, self.prim, self.w,
                                          self.hidden, layers=gl, stream=st)
        else:
            self.table.inject_propagated_gated(self.kept[0], self.count, self.scene[0],
                                               self.prim[0], self.w[0], self.hidden, self.steps,
                                               stream=st)
        return self


def check_gated_run(r: GatedRun, tokens=None) -> C.Report:
    """Every layer's gate in full (open set, ascending, -1 tail, count) and
    the injected rows of the sampled tokens against the oracle, on the
    library's lookup (routing and lookup themselves are checked by check_run
    on the same kernels)."""
    torch.cuda.synchronize()
    inp = r.inp
    dt = dtype_name(inp["x"])
    rep = C.Report()
    toks = np.arange(r.n) if tokens is None else np.asarray(tokens)
    tsel = torch.as_tensor(toks, device=r.dev)
    values = inp["values"]

    def values_rows(rows):
        idx = torch.as_tensor(np.asarray(rows), device=values.device, dtype=torch.long)
        return f64(values[idx])

    counts = to_np(r.count)
    kept_all = to_np(r.kept)
    kepts = []
    for l in range(r.glayers):
        c = int(counts[l])
        if not 0 <= c <= r.n:
            rep.fail(f"gate: count {c} of layer {l} outside [0, {r.n}]")
            return rep.finish()
        if np.any(kept_all[l, c:] != -1):
            rep.fail(f"gate: layer {l} list not -1 past its count")
        C.check_gate(f64(inp["delta"][l]), f64(r.w_g[l]), kept_all[l, :c], rep)
        kepts.append(kept_all[l, :c])
    if r.mode == "plain":
        prim_keys = inp["prim_keys"]
        for l in range(r.L):
            prim, w = to_np(r.prim[l]), to_np(r.w[l])
            scene = to_np(r.scene[l]).astype(np.int64)
            q_lib = O.to_f64(to_np(r.q[l])[toks], dt)
            w_orc = C.check_prim(q_lib, scene[toks], lambda s: f64(prim_keys[s]), r.k, "dot",
                                 prim[toks], w[toks], rep)
            w_of = {int(t): w_orc[i] for i, t in enumerate(toks)}
            C.check_hidden(to_np(r.h_in[l][tsel]), to_np(r.hidden[l][tsel]), dt, values_rows,
                           r.P, scene, prim, lambda t: w_of[t], kepts[l], rep, tokens=toks,
                           w_lib_of=lambda t, w=w: w[t])
    elif r.mode == "fused":
        fus = r.fus
        for l in range(r.L):
            C.check_fused_hidden(to_np(r.h_in[l][tsel]), to_np(r.hidden[l][tsel]), dt,
                                 values_rows, r.P, to_np(r.scene[l]), to_np(r.prim[l]),
                                 to_np(r.w[l]), kepts[l], f64(fus["w_gate"][l]),
                                 f64(fus["w_up"][l]), f64(fus["w_down"][l]), rep, toks)
    else:
        fus = r.fus
        w_p = f64(r.w_p_t[: r.steps]).transpose(0, 2, 1) if r.steps else np.zeros((0, 1, 1))
        C.check_propagated_hidden(to_np(r.h_in[:, tsel]), to_np(r.hidden[:, tsel]), dt,
                                  values_rows, r.P, to_np(r.scene[0]), to_np(r.prim[0]),
                                  to_np(r.w[0]), kepts[0], w_p, f64(fus["w_gate"]),
                                  f64(fus["w_up"]), f64(fus["w_down"]), rep, toks)
    return rep.finish()


class LayerRun:
    """One LookME layer (Eq. 2) over a sequence of text and image positions:
    the cross-modal pathway routes and looks up every position's L_dec(H_in)
    row against its own table, the image pathway the image block's encoder
    embeddings, each pathway's gate reads Delta at its positions, and then the
    text, image and cross-modal injections are added in that order -- every
    step a library call (lookme_route / lookup / gate / inject_text /
    inject_gated)."""

    def __init__(self, lay: dict, stream=None):
        self.lay = lay
        img, cr, tx = lay["image"], lay["cross"], lay["text"]
        self.dev = lay["h_dec"].device
        dt = lay["h_dec"].dtype
        self.stream = stream
        self.start, self.n_seq = lay["start"], lay["n_seq"]
        self.n_img = img["x"].shape[0]
        self.k, self.kc = img["k"], cr["k"]
        d_e = img["prim_keys"].shape[2]
        self.img_table = lk.Table(img["scene_keys"], img["prim_keys"], img["values"], self.k)
        self.cross_table = lk.Table(cr["scene_keys"], cr["prim_keys"], cr["values"], self.kc)
        self.img_table.reserve(1, max(self.n_img, tx["pos"].numel()))
        self.cross_table.reserve(1, self.n_seq)
        ni, ns, nt = self.n_img, self.n_seq, tx["pos"].numel()
        mk = lambda shape, dtype, fill: torch.full(shape, fill, dtype=dtype, device=self.dev)
        self.q_img, self.q_c = mk((ni, d_e), dt, 0), mk((ns, d_e), dt, 0)
        self.scene_img, self.scene_c = mk((ni,), torch.int32, -7), mk((ns,), torch.int32, -7)
        self.prim_img = mk((ni, self.k), torch.int32, -7)
        self.prim_c = mk((ns, self.kc), torch.int32, -7)
        self.w_img = mk((ni, self.k), torch.float32, -7.0)
        self.w_c = mk((ns, self.kc), torch.float32, -7.0)
        self.kept_t, self.kept_i, self.kept_c = (mk((nt,), torch.int32, -7),
                                                 mk((ni,), torch.int32, -7),
                                                 mk((ns,), torch.int32, -7))
        # one 16-byte row per pathway's count (text, image, cross)
        self.count = mk((3, 4), torch.int32, -7)
        self.hidden = lay["h_dec"].clone()

    def run(self):
        lay, st = self.lay, self.stream
        img, cr, tx = lay["image"], lay["cross"], lay["text"]
        s0, s1 = self.start, self.start + self.n_img
        # every pathway reads the layer's inputs before the first add
        self.cross_table.route(lay["h_dec"], cr["wt"], self.q_c, self.scene_c, stream=st)
        self.cross_table.lookup(self.q_c, self.scene_c, self.prim_c, self.w_c, stream=st)
        self.img_table.route(img["x"], img["wt"][:1], self.q_img, self.scene_img, stream=st)
        self.img_table.lookup(self.q_img, self.scene_img, self.prim_img, self.w_img, stream=st)
        c_t, c_i, c_c = self.count[0, :1], self.count[1, :1], self.count[2, :1]
        self.img_table.gate(lay["delta"], lay["w_g"][0:1], self.kept_t, c_t, pos=tx["pos"],
                            stream=st)
        self.img_table.gate(lay["delta"][s0:s1], lay["w_g"][1:2], self.kept_i, c_i, stream=st)
        self.cross_table.gate(lay["delta"], lay["w_g"][2:3], self.kept_c, c_c, stream=st)
        lk.inject_text(tx["table"], tx["pos"], tx["ids"], self.hidden, self.kept_t, c_t,
                       stream=st)
        self.img_table.inject_gated(self.kept_i, c_i, self.scene_img, self.prim_img, self.w_img,
                                    self.hidden[s0:s1], stream=st)
        self.cross_table.inject_gated(self.kept_c, c_c, self.scene_c, self.prim_c, self.w_c,
                                      self.hidden, stream=st)
        return self


def check_layer_run(r: LayerRun, tokens=None) -> C.Report:
    """Stage-wise check of one LookME layer: both pathways' projections,
    scenes and primitives on the sampled positions (C1-C4), the three gates
    in full, and the layer output recomputed in float64 from the library's
    decisions and weights with one rounding per add (text, image, cross):
    untouched rows bit-identical; touched elements within two bf16 ulps, at
    most 0.5% of them off the recomputed value (float32: within 1e-5 of the
    summed magnitudes)."""
    torch.cuda.synchronize()
    lay = r.lay
    img, cr, tx = lay["image"], lay["cross"], lay["text"]
    dt = dtype_name(lay["h_dec"])
    rep = C.Report()
    ni, ns = r.n_img, r.n_seq
    s0 = r.start
    h_dec = f64(lay["h_dec"])
    delta = f64(lay["delta"])
    w_g = f64(lay["w_g"])
    counts = to_np(r.count)[:, 0]
    pos, ids = to_np(tx["pos"]).astype(np.int64), to_np(tx["ids"]).astype(np.int64)
    kept_t = to_np(r.kept_t)[: counts[0]]
    kept_i = to_np(r.kept_i)[: counts[1]]
    kept_c = to_np(r.kept_c)[: counts[2]]
    C.check_gate(delta, w_g[0], kept_t, rep, pos=pos)
    C.check_gate(delta[s0:s0 + ni], w_g[1], kept_i, rep)
    C.check_gate(delta, w_g[2], kept_c, rep)
    # the two lookups on sampled positions
    ti = np.arange(ni) if tokens is None else np.asarray(tokens)[np.asarray(tokens) < ni]
    tc = np.arange(ns) if tokens is None else np.asarray(tokens)
    for name, x, wt, sk, pk, q, sc, pr, w, tk, k in (
            ("image", img["x"], img["wt"][0], img["scene_keys"], img["prim_keys"], r.q_img,
             r.scene_img, r.prim_img, r.w_img, ti, r.k),
            ("cross", lay["h_dec"], cr["wt"][0], cr["scene_keys"], cr["prim_keys"], r.q_c,
             r.scene_c, r.prim_c, r.w_c, tc, r.kc)):
        tsel = torch.as_tensor(tk, device=r.dev)
        q_bits = to_np(q)[tk]
        C.check_projection(q_bits, f64(x[tsel]), f64(wt), dt, rep)
        q_lib = O.to_f64(q_bits, dt)
        scene = to_np(sc).astype(np.int64)
        C.check_scene(q_lib, f64(sk), None, "dot", scene[tk], rep)
        C.check_prim(q_lib, scene[tk], lambda s, pk=pk: f64(pk[s]), k, "dot", to_np(pr)[tk],
                     to_np(w)[tk], rep)
    # the layer output from the library's decisions, one rounding per add
    want = h_dec.copy()
    mag = np.abs(h_dec)
    touched = np.zeros(ns, dtype=bool)
    table = tx["table"]
    d_t = table.shape[1]
    for i in kept_t:
        t = pos[i]
        row = f64(table[int(ids[i])])
        want[t, :d_t] = O.round_to_dtype(want[t, :d_t] + row, dt)
        mag[t, :d_t] += np.abs(row)
        touched[t] = True
    for pathway, kept, sc, pr, w, vals, P, off in (
            ("image", kept_i, r.scene_img, r.prim_img, r.w_img, img["values"],
             img["prim_keys"].shape[1], s0),
            ("cross", kept_c, r.scene_c, r.prim_c, r.w_c, cr["values"], cr["prim_keys"].shape[1],
             0)):
        scene, prim, w = to_np(sc).astype(np.int64), to_np(pr).astype(np.int64), to_np(w)
        d_v = vals.shape[1]
        for t in kept:
            rows = torch.as_tensor(scene[t] * P + prim[t], device=vals.device, dtype=torch.long)
            V = f64(vals[rows])
            ww = w[t].astype(np.float64)
            tt = off + int(t)
            want[tt, :d_v] = O.round_to_dtype(want[tt, :d_v] + np.sum(ww[:, None] * V, axis=0),
                                              dt)
            mag[tt, :d_v] += np.sum(np.abs(ww[:, None] * V), axis=0)
            touched[tt] = True
    got_bits = to_np(r.hidden)
    in_bits = to_np(lay["h_dec"])
    got = O.to_f64(got_bits, dt)
    rows = np.arange(ns) if tokens is None else np.union1d(np.asarray(tokens),
                                                           np.flatnonzero(touched)[:4096])
    off_count, n_el = 0, 0
    for t in rows:
        rep.count("layer_row")
        if not touched[t]:
            if not np.array_equal(got_bits[t].view(np.uint8), in_bits[t].view(np.uint8)):
                rep.fail(f"layer: untouched position {t} modified")
            continue
        d = np.abs(got[t] - want[t])
        if dt == "bf16":
            ulp = np.ldexp(1.0, np.frexp(np.maximum(np.abs(want[t]), 2.0 ** -126))[1] - 8)
            bad = d > 2 * ulp
        else:
            bad = d > 1e-5 * mag[t] + 1e-30
        if np.any(bad):
            rep.fail(f"layer: position {t}: {int(bad.sum())} elements beyond the bound")
        off_count += int(np.sum(d > 0))
        n_el += d.size
    rep.notes["layer_elements_off"] = off_count
    if dt == "bf16" and n_el and off_count > 0.005 * n_el:
        rep.fail(f"layer: {off_count} of {n_el} touched elements off the recomputed value")
    rep.notes["layer_open"] = [int(c) for c in counts]
    return rep.finish()
