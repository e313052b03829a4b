#!/usr/bin/env python3
"""Throughput of the LookME hot path on one MI355X.

One step = one pass of the hot path over one batch of synthetic tokens
(projection, Level-1 routing, bucketing, Level-2 top-k scoring with softmax,
criticality select, row gather and residual add), with every input resident
in HBM before the timed region starts: lookme_select runs on a second stream
while lookme_route runs on the first (the kept set depends on neither routing
nor lookup), then lookme_inject_kept adds the rows.  The metric is tokens
looked up and injected per second, counting tokens x layers.

The default workload is the largest one that fits one GPU: 32768 tokens
(32 images of 1024) against 4096 scenes x 4096 primitives with Zipf(1.1)
scene popularity (a 32 GiB value table and 16 GiB of primitive keys, bf16).
Smaller workloads (--workload 1..3) reuse a table in several copies so that
consecutive steps cannot find the previous step's keys in the 256 MiB
Infinity Cache.

Printed: one JSON line with the throughput, the roofline of the dominant
kernel (Level-2 scoring: its key stream is HBM-bound) measured with HIP
events inside the library on the launch stream, and the CPU oracle's
throughput on a bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--workload 0..4] [--no-cpu-baseline]
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}     # dense, MI355X
METRIC = "multimodal tokens looked up+injected/sec at 1 MI355X; % HBM BW / % MFMA peak"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--reps", type=int, default=5,
                    help="K-step blocks timed in all (the first gives value; all give the "
                         "median and spread)")
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", type=int, default=4,
                    help="index into synth.WORKLOADS (default: the 32 GiB Zipf table, the "
                         "largest single-GPU workload)")
    ap.add_argument("--copies", type=int, default=0, help="table copies (0: automatic)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-tokens", type=int, default=0, help="oracle sample size (0: auto)")
    ap.add_argument("--relevance", type=int, default=0, metavar="HIDDEN",
                    help="Level-2 in the paper's form (relevance MLP of this hidden width, "
                         "seeded weights) instead of the key-scored Level-2")
    ap.add_argument("--fusion", type=int, default=0, metavar="D_FF",
                    help="inject through the SwiGLU fusion of Eq. 10 (inner width D_FF, seeded "
                         "weights) instead of the prefix add of the retrieved rows")
    ap.add_argument("--netprop", type=int, default=0, metavar="M",
                    help="with --fusion on a one-layer workload: the LookME layer's R is carried "
                         "to M more layers by the propagation of Eq. 11 (seeded W_p), each "
                         "injected through its own fusion")
    ap.add_argument("--scales", type=int, default=0, metavar="M",
                    help="multi-scale image retrieval (Eq. 8) on a one-layer workload: M scales "
                         "(seeded tokens and rankers) each routed and looked up in its own scene "
                         "partition, mixed by the token-wise router and injected")
    ap.add_argument("--gate", action="store_true",
                    help="the kept set of each layer from the learned SKA gate of Eq. 9 "
                         "(seeded W_g; open where Delta W_g > 0, a variable count) instead of "
                         "the top n_keep by criticality")
    ap.add_argument("--layer", action="store_true",
                    help="time one whole LookME layer (Eq. 2) on a sequence of 64 + 192 text "
                         "positions around the workload's image block: text, image and "
                         "cross-modal pathways, each with its learned gate")
    ap.add_argument("--two-streams", action="store_true",
                    help="select the kept set on a second stream even where the lookup's "
                         "bucketing launch can carry it (batches of at most 1024 rows)")
    ap.add_argument("--select-on-main", action="store_true",
                    help="run the select on the launch stream instead of on a second stream "
                         "beside projection and routing (times its kernels without the overlap: "
                         "the plain path through lookme_inject after the lookup, the others "
                         "through lookme_select before routing)")
    ap.add_argument("--pmc-calibrate", action="store_true",
                    help="first run a plain 256 MiB read+write kernel (counter calibration)")
    ap.add_argument("--traffic-from", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "BENCH_JSON"),
                    help="summarise two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of this "
                         "script into profiles/, with the algorithmic bytes of a bench line "
                         "of the same workload, and exit (no GPU needed)")
    return ap.parse_args()


# --------------------------------------------------------------------------
# HBM traffic of the dominant kernel from PMC counters
# --------------------------------------------------------------------------

CALIB_BYTES = 256 << 20
SCORE_KERNEL = "score_kernel"
KERNEL_SOURCES = ("paper_2607_16305_amd/csrc/score.hip", "paper_2607_16305_amd/csrc/topk.h",
                  "paper_2607_16305_amd/csrc/common.h", "paper_2607_16305_amd/csrc/kernels.h",
                  "paper_2607_16305_amd/csrc/crit.h", "paper_2607_16305_amd/csrc/dtl.h",
                  "paper_2607_16305_amd/csrc/route_merge.h")


def kernel_source_sha() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_path(workload_name: str) -> str:
    return os.path.join(ROOT, "profiles", f"traffic_score_kernel_{workload_name}.json")


def calibration_copy():
    """A plain elementwise kernel of known traffic: reads and writes 256 MiB."""
    import torch
    src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()


def _counter_rows(d: str):
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    rows = []
    for f in files:
        with open(f) as fh:
            rows += list(csv.DictReader(fh))
    return rows


def _per_dispatch(rows, counter, match):
    vals = {}
    for r in rows:
        if r.get("Counter_Name") != counter or match not in r.get("Kernel_Name", ""):
            continue
        key = r.get("Dispatch_Id") or r.get("Correlation_Id")
        vals[key] = vals.get(key, 0.0) + float(r["Counter_Value"])
    return list(vals.values())


def summarise_traffic(fetch_dir: str, write_dir: str, wl, wl_index: int, algorithmic: int):
    """Scale FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the scoring kernel by
    what the same counters read for the 256 MiB calibration kernel."""
    fr, wr = _counter_rows(fetch_dir), _counter_rows(write_dir)
    cal_f = _per_dispatch(fr, "FETCH_SIZE", "neg_kernel") or _per_dispatch(fr, "FETCH_SIZE", "elementwise")
    cal_w = _per_dispatch(wr, "WRITE_SIZE", "neg_kernel") or _per_dispatch(wr, "WRITE_SIZE", "elementwise")
    sc_f = _per_dispatch(fr, "FETCH_SIZE", SCORE_KERNEL)
    sc_w = _per_dispatch(wr, "WRITE_SIZE", SCORE_KERNEL)
    # the routing launch of the scoring kernel is the smaller one; keep the
    # Level-2 launches (every other dispatch, the larger reading)
    sc_f = sorted(sc_f)[len(sc_f) // 2:]
    sc_w = sorted(sc_w)[len(sc_w) // 2:]
    mean = lambda v: sum(v) / len(v)
    f_read = max(cal_f) * 1024 / CALIB_BYTES
    f_write = max(cal_w) * 1024 / CALIB_BYTES
    fetch_b = mean(sc_f) * 1024 / f_read
    write_b = mean(sc_w) * 1024 / f_write
    out = {
        "kernel": SCORE_KERNEL + " (Level-2 launch)", "workload": wl.name,
        "kernel_source_sha": kernel_source_sha(),
        "fetch_kib_per_launch_raw": mean(sc_f), "write_kib_per_launch_raw": mean(sc_w),
        "calibration": {"bytes_read": CALIB_BYTES, "bytes_written": CALIB_BYTES,
                        "fetch_kib": max(cal_f), "write_kib": max(cal_w),
                        "read_factor": f_read, "write_factor": f_write},
        "traffic_bytes_per_launch": fetch_b + write_b,
        "algorithmic_bytes_per_launch": algorithmic,
        "traffic_over_algorithmic": (fetch_b + write_b) / algorithmic,
        "commands": [
            "rocprofv3 --pmc FETCH_SIZE --output-format csv -d <FETCH_DIR> -o run -- "
            f"python3 bench.py --workload {wl_index} --steps 20 --warmup 2 --reps 1 --no-cpu-baseline "
            "--pmc-calibrate",
            "rocprofv3 --pmc WRITE_SIZE --output-format csv -d <WRITE_DIR> -o run -- "
            f"python3 bench.py --workload {wl_index} --steps 20 --warmup 2 --reps 1 --no-cpu-baseline "
            "--pmc-calibrate",
            f"python3 bench.py --workload {wl_index} --traffic-from <FETCH_DIR> <WRITE_DIR> "
            "<BENCH_JSON>"],
    }
    with open(traffic_path(wl.name), "w") as fh:
        json.dump(out, fh, indent=1)
    return out


def stored_traffic(wl):
    """Measured traffic per launch, if taken on the current kernel source."""
    try:
        with open(traffic_path(wl.name)) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha") != kernel_source_sha():
        return None
    return t.get("traffic_bytes_per_launch")


class Bench:
    def __init__(self, wl, seed, copies, relevance=0, fusion=0, netprop=0, scales=0,
                 gate=False, two_streams=False, select_on_main=False):
        import torch
        from paper_2607_16305_amd import lookme as lk
        from synth import make_inputs
        self.torch, self.lk, self.wl = torch, lk, wl
        self.inp = make_inputs(wl, seed=seed, device="cuda")
        inp = self.inp
        table_bytes = sum(inp[k].numel() * inp[k].element_size()
                          for k in ("scene_keys", "prim_keys", "values"))
        if copies <= 0:
            copies = max(1, min(4, (24 << 30) // max(table_bytes, 1)))
        self.copies = copies
        self.tables = []
        for c in range(copies):
            if c == 0:
                sk, pk, v = inp["scene_keys"], inp["prim_keys"], inp["values"]
            else:
                sk, pk, v = (inp["scene_keys"].clone(), inp["prim_keys"].clone(),
                             inp["values"].clone())
            t = lk.Table(sk, pk, v, wl.top_k)
            t.reserve(wl.layers, wl.n_tokens)
            self.tables.append(t)
        L, n, k = wl.layers, wl.n_tokens, wl.top_k
        dt = inp["x"].dtype
        dev = inp["x"].device
        self.q = torch.empty((L, n, wl.d_e), dtype=dt, device=dev)
        self.scene = torch.empty((L, n), dtype=torch.int32, device=dev)
        self.prim = torch.empty((L, n, k), dtype=torch.int32, device=dev)
        self.w = torch.empty((L, n, k), dtype=torch.float32, device=dev)
        self.kept = torch.empty((L, max(wl.n_keep, 1)), dtype=torch.int32, device=dev)
        self.hidden = inp["hidden"].clone()
        self.mlp = None
        if relevance:
            from synth import make_relevance
            self.mlp = make_relevance(wl, seed, relevance, device="cuda")
            m = self.mlp
            for t in self.tables:
                t.set_relevance(m["w1"], m["b1"], m["w2"], m["b2"])
                t.reserve(L, n)          # the relevance logits need a larger workspace
            self.act = torch.empty((L, n, relevance), dtype=dt, device=dev)
        self.fus = None
        self.netprop = netprop
        if fusion:
            from synth import make_fusion, make_propagation
            self.fus = make_fusion(wl, seed, fusion, device="cuda", layers=L + netprop)
            f = self.fus
            if netprop:
                # the propagated layers' hidden states (synthetic: copies of
                # the LookME layer's)
                self.w_p_t = make_propagation(wl, seed, netprop, device="cuda")
                self.hidden = inp["hidden"][:1].repeat(1 + netprop, 1, 1)
            for t in self.tables:
                t.set_fusion(f["w_gate"], f["w_up"], f["w_down"])
                if netprop:
                    t.set_propagation(self.w_p_t)
                t.reserve(L + netprop, n)   # the fusion's buffers enlarge the workspace
        self.scales = scales
        self.gate = gate
        if gate:
            from synth import make_gate
            gl = 1 if netprop else L
            self.w_g = make_gate(wl, seed, device="cuda", layers=gl)
            self.kept = torch.empty((gl, n), dtype=torch.int32, device=dev)
            self.count = torch.zeros((gl,), dtype=torch.int32, device=dev)
        self.handles = [t.handle for t in self.tables]
        self.select_on_main = select_on_main
        # small batches: the select rides in the lookup's bucketing launch on
        # the one stream (lookme_lookup_select); a second stream's waits would
        # cost more than the select itself
        self.one_stream = (not two_streams and L * n <= 1024 and not relevance and not scales
                           and not netprop)
        if scales:
            from synth import make_multiscale
            self.ms = make_multiscale(wl, seed, scales, device="cuda")
            # stacked per-scale outputs (row m of each is 16-byte aligned: n % 4 == 0)
            self.q = torch.empty((scales, n, wl.d_e), dtype=dt, device=dev)
            self.scene = torch.empty((scales, n), dtype=torch.int32, device=dev)
            self.prim = torch.empty((scales, n, k), dtype=torch.int32, device=dev)
            self.w = torch.empty((scales, n, k), dtype=torch.float32, device=dev)
            self.scale_tables = []
            for t in self.tables:
                t.set_multiscale(scales, self.ms["w_he_t"])
                t.reserve(1, n)
                views = [t.scale_view(m, scales) for m in range(scales)]
                for v in views:
                    v.reserve(1, n)
                self.scale_tables.append(views)
                self.handles += [v.handle for v in views]
        # the kept set is selected on a second stream (default priority, as
        # the first) while routing and lookup run; two reusable events order
        # the streams within a step
        self.main = torch.cuda.current_stream()
        self.side = torch.cuda.Stream()
        self.stream = self.main.cuda_stream
        self.side_handle = self.side.cuda_stream
        self.ev_start = torch.cuda.Event()
        self.ev_kept = torch.cuda.Event()
        torch.cuda.synchronize()

    def step(self, i):
        lk, wl, inp = self.lk, self.wl, self.inp
        h = self.tables[i % self.copies].handle
        L, n = wl.layers, wl.n_tokens
        if self.one_stream and self.gate:
            lk.lookme_route(h, L, n, wl.d_in, inp["x"], inp["wt"], self.q, self.scene,
                            self.stream)
            lk.lookme_lookup_gate(h, L, n, self.q, self.scene, self.prim, self.w, inp["delta"],
                                  wl.crit_dim, self.w_g, self.kept, self.count, self.stream)
            if self.fus is None:
                lk.lookme_inject_gated(h, L, n, self.kept, self.count, self.scene, self.prim,
                                       self.w, self.hidden, wl.d_h, self.stream)
            else:
                lk.lookme_inject_fused_gated(h, L, n, self.kept, self.count, self.scene,
                                             self.prim, self.w, self.hidden, wl.d_h, self.stream)
            return
        if self.one_stream:
            lk.lookme_route(h, L, n, wl.d_in, inp["x"], inp["wt"], self.q, self.scene,
                            self.stream)
            lk.lookme_lookup_select(h, L, n, self.q, self.scene, self.prim, self.w, wl.n_keep,
                                    inp["delta"], wl.crit_dim, self.kept, self.stream)
            if self.fus is None:
                lk.lookme_inject_kept(h, L, n, wl.n_keep, self.kept, self.scene, self.prim,
                                      self.w, self.hidden, wl.d_h, self.stream)
            else:
                lk.lookme_inject_fused(h, L, n, wl.n_keep, self.kept, self.scene, self.prim,
                                       self.w, self.hidden, wl.d_h, self.stream)
            return
        # the select starts after the previous step's inject (which reads the
        # kept buffer it overwrites) and runs beside the projection and
        # routing; measured faster than beside the Level-2 lookup, whose
        # workgroups it would slow
        plain = not self.gate and self.fus is None and not self.scales
        if self.select_on_main and not self.gate and not plain:
            lk.lookme_select(h, L, n, wl.n_keep, inp["delta"], wl.crit_dim, self.kept,
                             self.stream)
        self.ev_start.record(self.main)
        self.side.wait_event(self.ev_start)
        if self.gate:
            gl = self.w_g.shape[0]
            lk.lookme_gate(h, gl, n, inp["delta"], n, wl.crit_dim, None, self.w_g, self.kept,
                           self.count, self.side_handle)
        elif not self.select_on_main:
            lk.lookme_select(h, L, n, wl.n_keep, inp["delta"], wl.crit_dim, self.kept,
                             self.side_handle)
        self.ev_kept.record(self.side)
        if self.scales:
            ms = self.ms
            for m, v in enumerate(self.scale_tables[i % self.copies]):
                lk.lookme_route(v.handle, 1, n, wl.d_in, ms["x"][m], ms["wt"][m], self.q[m],
                                self.scene[m], self.stream)
                lk.lookme_lookup(v.handle, 1, n, self.q[m], self.scene[m], self.prim[m],
                                 self.w[m], self.stream)
            self.main.wait_event(self.ev_kept)
            lk.lookme_inject_multiscale(h, n, wl.n_keep, self.kept, self.scene, self.prim, self.w,
                                        self.hidden[0], wl.d_h, self.stream)
            return
        lk.lookme_route(h, L, n, wl.d_in, inp["x"], inp["wt"], self.q, self.scene, self.stream)
        if self.mlp is None:
            lk.lookme_lookup(h, L, n, self.q, self.scene, self.prim, self.w, self.stream)
        else:
            lk.lookme_lookup_relevance(h, L, n, self.q, self.scene, self.act, self.prim, self.w,
                                       self.stream)
        self.main.wait_event(self.ev_kept)
        if self.gate:
            if self.fus is None:
                lk.lookme_inject_gated(h, L, n, self.kept, self.count, self.scene, self.prim,
                                       self.w, self.hidden, wl.d_h, self.stream)
            elif self.netprop:
                lk.lookme_inject_propagated_gated(h, self.netprop, n, self.kept[0], self.count,
                                                  self.scene[0], self.prim[0], self.w[0],
                                                  self.hidden, wl.d_h, self.stream)
            else:
                lk.lookme_inject_fused_gated(h, L, n, self.kept, self.count, self.scene,
                                             self.prim, self.w, self.hidden, wl.d_h, self.stream)
        elif plain and self.select_on_main:
            # norms, select and the adds in one call on the launch stream, each
            # kernel alone on the chip (the norms in their full-grid form)
            lk.lookme_inject(h, L, n, wl.n_keep, inp["delta"], wl.crit_dim, self.scene,
                             self.prim, self.w, self.hidden, wl.d_h, self.kept, self.stream)
        elif self.fus is None:
            lk.lookme_inject_kept(h, L, n, wl.n_keep, self.kept, self.scene, self.prim, self.w,
                                  self.hidden, wl.d_h, self.stream)
        elif self.netprop:
            lk.lookme_inject_propagated(h, self.netprop, n, wl.n_keep, self.kept[0], self.scene[0],
                                        self.prim[0], self.w[0], self.hidden, wl.d_h,
                                        self.stream)
        else:
            lk.lookme_inject_fused(h, L, n, wl.n_keep, self.kept, self.scene, self.prim, self.w,
                                   self.hidden, wl.d_h, self.stream)

    def timed(self, steps):
        torch = self.torch
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            self.step(i)
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    def profiled(self, steps):
        """Per-kernel-group times from the library's HIP events (launch stream)."""
        lk = self.lk
        for h in self.handles:
            lk.lookme_profile_read(h, 0, reset=True)
            lk.lookme_profile_enable(h, True)
        self.timed(steps)
        out = {}
        for g, name in enumerate(lk.GROUPS):
            cnt, ms = 0, 0.0
            for h in self.handles:
                c, m = lk.lookme_profile_read(h, g)
                cnt += c
                ms += m
            if cnt:
                out[name] = ms / cnt
        for h in self.handles:
            lk.lookme_profile_enable(h, False)
            lk.lookme_profile_read(h, 0, reset=True)
        return out   # average milliseconds per launch

    def algorithmic_bytes(self):
        """Bytes each kernel group must move per launch."""
        torch, wl = self.torch, self.wl
        es = self.inp["x"].element_size()
        L, n, k = wl.layers, wl.n_tokens, wl.top_k
        rows = L * n
        nonempty = int(torch.unique(self.scene).numel())
        scenes = wl.scenes
        if self.scales:
            # a launch of each group serves one scale: its rows and partition;
            # the used scenes averaged over the scales
            nonempty = sum(int(torch.unique(self.scene[m]).numel())
                           for m in range(self.scales)) / self.scales
            scenes = wl.scenes // self.scales
        keep = L * wl.n_keep
        if self.gate:
            # the open rows (the gate's count varies with the inputs, not the step)
            keep = int(self.count.sum().item())
        b = {}
        b["project"] = (n * wl.d_in + L * wl.d_e * wl.d_in + rows * wl.d_e) * es
        b["route"] = (rows * wl.d_e + scenes * wl.d_e) * es + rows * 4
        b["score"] = int(nonempty * wl.prims * wl.d_e * es   # key stream of each used scene
                      + rows * wl.d_e * es                    # queries
                      + rows * 4                              # bucketed row ids
                      + rows * k * 8)                         # prim + weights written
        b["norm"] = rows * wl.crit_dim * es + rows * 4
        if self.gate:
            gl = self.w_g.shape[0]
            b["norm"] = gl * n * wl.crit_dim * es + gl * wl.crit_dim * es + gl * n * 4
        # the injection reads each distinct value row of the kept tokens'
        # picks once (the caches serve its repeats), H read and written, the
        # picks and weights read
        fetched = keep * k
        self.inject_rows = {"fetched": fetched, "distinct": fetched}
        if not (self.gate or self.scales or self.fus is not None):
            kept = self.kept[:, :wl.n_keep].long()
            sc = torch.gather(self.scene.long(), 1, kept)
            pr = torch.gather(self.prim.long(), 1, kept.unsqueeze(-1).expand(-1, -1, k))
            self.inject_rows["distinct"] = int(torch.unique(sc.unsqueeze(-1) * wl.prims + pr).numel())
        b["inject"] = (self.inject_rows["distinct"] * wl.d_v * es
                       + keep * (2 * wl.d_v * es + k * 8 + 8))
        flops = {"project": 2 * n * wl.d_in * L * wl.d_e, "route": 2 * rows * wl.d_e * scenes,
                 "score": 2 * rows * wl.d_e * wl.prims}
        if self.scales:
            # the router's query product; the gather and mix move
            # n_keep (M k d_v + 2 M d_v + 2 d_v) elements besides
            flops["inject"] = 2 * keep * wl.d_h * wl.d_v
            b["inject"] = None
        if self.fus is not None:
            d_ff = self.fus["d_ff"]
            m = self.netprop
            flops["inject"] = 2 * keep * ((1 + m) * (2 * wl.d_v * d_ff + d_ff * wl.d_h)
                                          + m * wl.d_v * wl.d_v)
            b["inject"] = None
        if self.mlp is not None:
            hid = self.mlp["hidden"]
            # the two MLP layers per row: the query half of the first (its
            # scene half is a per-scene table, computed once per registered
            # MLP, not per step) and the second; the cosines are 2 k d_e per
            # row, negligible
            flops["score"] = 2 * rows * wl.d_e * hid + 2 * rows * hid * wl.prims
            b["score"] = None
        return b, flops, nonempty


class LayerBench:
    """One whole LookME layer (Eq. 2) per step on a sequence of TEXT_BEFORE
    text positions, the workload's image block and TEXT_AFTER text
    positions: the cross-modal pathway routes and looks up every position's
    L_dec(H_in) row in its own table (the paper's N_s = 512 scenes of
    N_p = 256 primitives, top-8), the image pathway the image block's
    embeddings in the workload's table, each with its learned gate carried
    by the lookup's launches (lookme_lookup_gate); the text gate runs on its
    own; then the text, image and cross-modal injections are added in that
    order.  One stream."""

    TEXT_BEFORE, TEXT_AFTER, VOCAB = 64, 192, 151936
    CROSS_SCENES, CROSS_PRIMS, CROSS_K = 512, 256, 8

    def __init__(self, wl, seed):
        import torch
        from paper_2607_16305_amd import lookme as lk
        from synth import make_layer
        self.torch, self.lk, self.wl = torch, lk, wl
        self.lay = lay = make_layer(wl, seed, self.TEXT_BEFORE, self.TEXT_AFTER, self.VOCAB,
                                    wl.d_h, self.CROSS_SCENES, self.CROSS_PRIMS, self.CROSS_K,
                                    device="cuda")
        img, cr = lay["image"], lay["cross"]
        self.n_seq, self.start, self.n_img = lay["n_seq"], lay["start"], wl.n_tokens
        self.n_text = lay["text"]["pos"].numel()
        self.img = lk.Table(img["scene_keys"], img["prim_keys"], img["values"], wl.top_k)
        self.cross = lk.Table(cr["scene_keys"], cr["prim_keys"], cr["values"], self.CROSS_K)
        self.img.reserve(1, max(self.n_img, self.n_text))
        self.cross.reserve(1, self.n_seq)
        dev, dt = lay["h_dec"].device, lay["h_dec"].dtype
        e = lambda shape, dtype: torch.empty(shape, dtype=dtype, device=dev)
        ni, ns = self.n_img, self.n_seq
        self.q_i, self.q_c = e((ni, wl.d_e), dt), e((ns, wl.d_e), dt)
        self.sc_i, self.sc_c = e((ni,), torch.int32), e((ns,), torch.int32)
        self.pr_i, self.pr_c = e((ni, wl.top_k), torch.int32), e((ns, self.CROSS_K), torch.int32)
        self.w_i, self.w_c = e((ni, wl.top_k), torch.float32), e((ns, self.CROSS_K), torch.float32)
        self.k_t, self.k_i, self.k_c = (e((self.n_text,), torch.int32), e((ni,), torch.int32),
                                        e((ns,), torch.int32))
        self.count = torch.zeros((3, 4), dtype=torch.int32, device=dev)   # a 16-byte row each
        self.hidden = lay["h_dec"].clone()
        self.main = torch.cuda.current_stream()
        self.handles = [self.img.handle, self.cross.handle]
        torch.cuda.synchronize()

    def step(self, i):
        lk, wl, lay = self.lk, self.wl, self.lay
        img, cr, tx = lay["image"], lay["cross"], lay["text"]
        st = self.main.cuda_stream
        hi, hc = self.img.handle, self.cross.handle
        s0, s1 = self.start, self.start + self.n_img
        ct, ci, cc = self.count[0, :1], self.count[1, :1], self.count[2, :1]
        d_c = lay["delta"].shape[1]
        # one stream: the image and cross-modal gates ride in their lookups'
        # launches, the text gate is its own pair of launches
        lk.lookme_route(hc, 1, self.n_seq, wl.d_h, lay["h_dec"], cr["wt"], self.q_c, self.sc_c, st)
        lk.lookme_lookup_gate(hc, 1, self.n_seq, self.q_c, self.sc_c, self.pr_c, self.w_c,
                              lay["delta"], d_c, lay["w_g"][2], self.k_c, cc, st)
        lk.lookme_route(hi, 1, self.n_img, wl.d_in, img["x"], img["wt"], self.q_i, self.sc_i, st)
        lk.lookme_lookup_gate(hi, 1, self.n_img, self.q_i, self.sc_i, self.pr_i, self.w_i,
                              lay["delta"][s0:s1], d_c, lay["w_g"][1], self.k_i, ci, st)
        lk.lookme_gate(hi, 1, self.n_text, lay["delta"], self.n_seq, d_c, tx["pos"],
                       lay["w_g"][0], self.k_t, ct, st)
        lk.lookme_inject_text(lk.DTYPE_CODE[tx["table"].dtype], tx["table"], tx["vocab"],
                              tx["d_t"], self.n_text, tx["pos"], tx["ids"], self.k_t, ct,
                              self.hidden, self.n_seq, wl.d_h, st)
        lk.lookme_inject_gated(hi, 1, self.n_img, self.k_i, ci, self.sc_i, self.pr_i, self.w_i,
                               self.hidden[s0:s1], wl.d_h, st)
        lk.lookme_inject_gated(hc, 1, self.n_seq, self.k_c, cc, self.sc_c, self.pr_c, self.w_c,
                               self.hidden, wl.d_h, st)

    timed = Bench.timed

    def profiled(self, steps):
        """Per-kernel-group times of each pathway's handle (HIP events on the
        launch streams), milliseconds per launch."""
        lk = self.lk
        for h in self.handles:
            lk.lookme_profile_read(h, 0, reset=True)
            lk.lookme_profile_enable(h, True)
        self.timed(steps)
        out = {}
        for h, name in zip(self.handles, ("image", "cross")):
            for g, grp in enumerate(lk.GROUPS):
                c, ms = lk.lookme_profile_read(h, g)
                if c:
                    out[f"{name}.{grp}"] = ms / c
            lk.lookme_profile_enable(h, False)
            lk.lookme_profile_read(h, 0, reset=True)
        return out


def run_layer(args, wl):
    b = LayerBench(wl, args.workload)
    for i in range(args.warmup):
        b.step(i)
    el = b.timed(args.steps)
    ms_step = el * 1000.0 / args.steps
    prof = b.profiled(args.steps)
    es = b.lay["h_dec"].element_size()
    nonempty = int(b.torch.unique(b.sc_i).numel())
    score_bytes = int(nonempty * wl.prims * wl.d_e * es + wl.n_tokens * wl.d_e * es
                      + wl.n_tokens * 4 + wl.n_tokens * wl.top_k * 8)
    score_ms = prof.get("image.score")
    achieved = score_bytes / (score_ms * 1e-3) / 1e9 if score_ms else None
    counts = b.count[:, 0].tolist()
    line = {
        "metric": METRIC, "value": round(b.n_seq / (el / args.steps), 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": f"layer_{wl.name}_text{b.n_text}", "positions": b.n_seq,
                   "image_positions": b.n_img, "text_positions": b.n_text,
                   "text_vocab": b.VOCAB, "cross_table": [b.CROSS_SCENES, b.CROSS_PRIMS,
                                                          b.CROSS_K],
                   "open_gates": {"text": counts[0], "image": counts[1], "cross": counts[2]},
                   "d_h": wl.d_h, "d_e": wl.d_e},
        "roofline": {"bound": "hbm", "kernel": "score_kernel of the image pathway",
                     "achieved": round(achieved, 1) if achieved else None,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4) if achieved else None,
                     "traffic": None, "algorithmic_bytes_per_launch": score_bytes},
        "cpu_baseline": None,
        "kernels": {k: {"avg_us": round(v * 1000.0, 3)} for k, v in prof.items()},
    }
    print(json.dumps(line), flush=True)


class DeviceRows:
    """A device tensor read by the oracle one leading index (or an index
    array) at a time: each access copies only those rows to the host as
    stored bits (bf16 bits or float32) and caches them, so the CPU leg never
    holds the whole table (48 GiB on the largest workload).  ``f64`` turns
    each access into the oracle's float64 values, as a host-resident table
    would be read."""

    def __init__(self, t, dtype: str, f64: bool = True):
        self.t, self.dt, self.f64 = t, dtype, f64
        self.shape = tuple(t.shape)
        self.cache = {}

    def raw(self, i):
        from tests.harness import to_np
        key = i if isinstance(i, int) else None
        if key is not None and key in self.cache:
            return self.cache[key]
        import numpy as np
        import torch
        if isinstance(i, int):
            a = to_np(self.t[i])
        else:
            idx = torch.as_tensor(np.asarray(i, dtype=np.int64), device=self.t.device)
            a = to_np(self.t[idx])
        if key is not None:
            self.cache[key] = a
        return a

    def __getitem__(self, i):
        from oracle import lookme_oracle as O
        if isinstance(i, slice):            # a scale's partition (multi-scale): still lazy
            return DeviceRows(self.t[i], self.dt, self.f64)
        import numpy as np
        if isinstance(i, (np.integer,)):
            i = int(i)
        a = self.raw(i)
        return O.to_f64(a, self.dt) if self.f64 else a


def host_cores() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def cpu_baseline(b: "Bench", m: int, min_seconds: float = 10.0):
    """The oracle, unchanged, on the first m tokens of the same workload
    (single thread); returns tokens/s and details.  The table stays on the
    device: before the clock starts, the oracle's own projection and routing
    of the sample (untimed) name the scenes it will read, and only those
    scenes' primitive keys are copied to the host as stored bits; the value
    rows it gathers are copied when it reads them (inside the timed region,
    a few MB)."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    from oracle import lookme_oracle as O
    from tests.harness import to_np

    wl, inp = b.wl, b.inp
    dt = wl.dtype
    n_keep = (wl.keep_pct * m + 50) // 100
    x = to_np(inp["x"][:m])
    wt = None if inp["wt"] is None else to_np(inp["wt"])
    K1 = to_np(inp["scene_keys"])
    K2 = DeviceRows(inp["prim_keys"], dt)
    V = DeviceRows(inp["values"], dt)
    D = to_np(inp["delta"][:, :m])
    H = to_np(b.hidden[:, :m] if b.netprop else inp["hidden"][:, :m])
    cores = host_cores()

    mlp = None
    if b.mlp is not None:
        f = lambda t: t.detach().cpu().numpy().astype(np.float64)
        mlp = (O.to_f64(to_np(b.mlp["w1"]), dt), f(b.mlp["b1"]), O.to_f64(to_np(b.mlp["w2"]), dt),
               f(b.mlp["b2"]))

    fusion = None
    if b.fus is not None:
        fusion = tuple(O.to_f64(to_np(b.fus[key]), dt) for key in ("w_gate", "w_up", "w_down"))
    w_p = None
    if b.netprop:
        w_p = O.to_f64(to_np(b.w_p_t), dt).transpose(0, 2, 1)
    w_g = O.to_f64(to_np(b.w_g), dt) if b.gate else None

    # the sample is repeated until about min_seconds of CPU work have been
    # timed (the same inputs each time), so that the rate is not a single
    # short measurement
    reps, el = 0, 0.0
    if b.scales:
        ms = b.ms
        xs = O.to_f64(to_np(ms["x"][:, :m]), dt)
        wts = O.to_f64(to_np(ms["wt"]), dt)
        w_he = O.to_f64(to_np(ms["w_he_t"]), dt).T
        with threadpool_limits(limits=1):
            while reps == 0 or el < min_seconds:
                t0 = time.perf_counter()
                res = O.run_multiscale(xs, wts, O.to_f64(K1, dt), K2, V,
                                       O.to_f64(D[0], dt), O.to_f64(H[0], dt), w_he, k=wl.top_k,
                                       n_keep=n_keep, dtype=dt)
                el += time.perf_counter() - t0
                reps += 1
                assert res["hidden"].shape == (m, wl.d_h)
        return {"value": reps * m / el, "unit": "tokens/s", "cores": 1, "host_cores": cores,
                "kind": "oracle",
                "sample": f"first {m} of {wl.n_tokens} image positions x {b.scales} scales, "
                          f"whole path (per-scale projection, routing and lookup, select, "
                          f"router mix and injection, n_keep={n_keep}), float64 NumPy, "
                          f"1 thread, {reps} repetitions, {el:.1f} s"}
    # the scenes the oracle will read (its own projection and routing of the
    # sample, untimed): their keys are copied to the host before the clock
    # starts, as stored bits
    x64 = O.to_f64(x, dt)
    K1_64 = O.to_f64(K1, dt)
    with threadpool_limits(limits=1):
        for l in range(wl.layers if b.netprop == 0 else 1):
            q = O.project(x64, None if wt is None else O.to_f64(wt[l], dt), dt)
            for s in np.unique(O.route(q, K1_64)):
                K2.raw(int(s))
        while reps == 0 or el < min_seconds:
            t0 = time.perf_counter()
            res = O.run(x64, None if wt is None else O.to_f64(wt, dt),
                        K1_64, K2, V, None, O.to_f64(D, dt),
                        O.to_f64(H, dt), k=wl.top_k, n_keep=n_keep, dtype=dt, mlp=mlp,
                        fusion=fusion, propagation=w_p, w_g=w_g)
            el += time.perf_counter() - t0
            reps += 1
            assert res["hidden"].shape == (wl.layers + b.netprop, m, wl.d_h)
    return {"value": reps * wl.layers * m / el, "unit": "tokens/s", "cores": 1,
            "host_cores": cores, "kind": "oracle",
            "sample": f"first {m} of {wl.n_tokens} tokens x {wl.layers} layer(s), whole path "
                      f"(projection..injection, "
                      f"{'learned gate' if w_g is not None else f'n_keep={n_keep}'}"
                      f"{', relevance Level-2' if mlp is not None else ''}"
                      f"{', SwiGLU fusion' if fusion is not None else ''}"
                      f"{f', propagated to {b.netprop} more layers' if b.netprop else ''}), "
                      f"float64 NumPy, 1 thread (BLAS pinned) of {cores} host cores, "
                      f"{len(K2.cache)} scenes' keys on the host, {reps} repetitions, "
                      f"{el:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    from synth import WORKLOADS
    wl = WORKLOADS[args.workload]
    if args.traffic_from:
        with open(args.traffic_from[2]) as fh:
            line = json.load(fh)
        if line["config"]["workload"] != wl.name:
            raise SystemExit("the bench line is for another workload")
        out = summarise_traffic(args.traffic_from[0], args.traffic_from[1], wl, args.workload,
                                line["roofline"]["algorithmic_bytes_per_launch"])
        print(json.dumps(out))
        return
    import torch
    torch.cuda.set_device(0)
    if args.pmc_calibrate:
        calibration_copy()
    if args.netprop and (not args.fusion or wl.layers != 1):
        raise SystemExit("--netprop needs --fusion and a one-layer workload")
    if args.scales and (wl.layers != 1 or args.relevance or args.fusion or wl.n_tokens % 4
                        or wl.scenes % args.scales):
        raise SystemExit("--scales needs a one-layer workload (tokens a multiple of 4, scenes "
                         "divisible by the scales) without --relevance or --fusion")
    if args.layer:
        if args.relevance or args.fusion or args.scales or args.gate or wl.layers != 1:
            raise SystemExit("--layer runs the layer's own pathways on a one-layer workload")
        run_layer(args, wl)
        return
    if args.gate and args.scales:
        raise SystemExit("--gate is not combined with --scales")
    b = Bench(wl, args.workload, args.copies, args.relevance, args.fusion, args.netprop,
              args.scales, args.gate, args.two_streams, args.select_on_main)

    for i in range(args.warmup):
        b.step(i)
    el = b.timed(args.steps)
    ms_step = el * 1000.0 / args.steps
    value = wl.layers * wl.n_tokens / (el / args.steps)
    # the same K-step block repeated, for the spread of the figure
    rep_ms = sorted([el * 1000.0 / args.steps] +
                    [b.timed(args.steps) * 1000.0 / args.steps for _ in range(args.reps - 1)])

    prof = b.profiled(args.steps)
    bytes_, flops, nonempty = b.algorithmic_bytes()
    kern = {}
    for name, ms in prof.items():
        e = {"avg_us": round(ms * 1000.0, 3)}
        if bytes_.get(name):
            gbs = bytes_[name] / (ms * 1e-3) / 1e9
            e["gbps"] = round(gbs, 1)
            e["hbm_frac"] = round(gbs / HBM_PEAK_GBS, 4)
        if name in flops:
            e["tflops"] = round(flops[name] / (ms * 1e-3) / 1e12, 2)
        if name == "inject" and bytes_.get(name):
            e["value_rows"] = b.inject_rows
        kern[name] = e
    score_ms = prof.get("score")
    if b.mlp is None:
        achieved = bytes_["score"] / (score_ms * 1e-3) / 1e9 if score_ms else None
        roofline = {"bound": "hbm", "kernel": "score_kernel (Level-2 scoring + top-k + softmax; "
                    "with split_merge_kernel where the last round is cut)",
                    "achieved": round(achieved, 1) if achieved else None, "peak": HBM_PEAK_GBS,
                    "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4) if achieved else None,
                    # counters were taken on the single-scale launch
                    "traffic": None if args.scales else stored_traffic(wl),
                    "algorithmic_bytes_per_launch": bytes_["score"], "nonempty_scenes": nonempty}
    else:
        # the relevance lookup is a pair of dense products: judged on the
        # matrix cores, whole launch group (both MLP layers and the weights)
        peak = MFMA_PEAK_TFLOPS[wl.dtype]
        achieved = flops["score"] / (score_ms * 1e-3) / 1e12 if score_ms else None
        roofline = {"bound": "mfma",
                    "kernel": "relevance lookup (MLP layers, top-k, cos + tanh weights)",
                    "achieved": round(achieved, 2) if achieved else None, "peak": peak,
                    "unit": "TFLOP/s", "frac": round(achieved / peak, 4) if achieved else None,
                    "traffic": None, "algorithmic_flops_per_launch": flops["score"]}

    cpu = None
    if not args.no_cpu_baseline:
        # a sample of about 10-30 s of oracle work: each token converts and
        # scores its scene's P x d_e keys in float64
        m = args.cpu_tokens or min(wl.n_tokens, max(64, (1024 * 1024) // wl.prims))
        cpu = cpu_baseline(b, m)

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "tokens": wl.n_tokens, "layers": wl.layers,
                   "d_in": wl.d_in, "d_e": wl.d_e, "scenes": wl.scenes, "prims": wl.prims,
                   "d_v": wl.d_v, "d_h": wl.d_h, "top_k": wl.top_k, "n_keep": wl.n_keep,
                   "usage": wl.usage, "table_copies": b.copies,
                   "level2": (f"relevance MLP, hidden {args.relevance}" if args.relevance
                              else "primitive keys"),
                   "injection": (f"SwiGLU fusion, d_ff {args.fusion}" if args.fusion
                                 else "prefix add of the retrieved rows"),
                   "propagated_layers": args.netprop, "scales": args.scales,
                   "select": (("gate logits in the bucketing launch, compaction in the Level-2 "
                               "launch (one stream)" if args.gate else
                               "norms in the bucketing launch, top-n_keep in the Level-2 launch "
                               "(one stream)") if b.one_stream
                              else ("launch stream, in lookme_inject after the lookup"
                                    if not (args.fusion or args.scales) else
                                    "launch stream, before routing") if b.select_on_main
                              else "second stream beside projection and routing"),
                   "kept_set": ("learned gate, " + "+".join(str(c) for c in b.count.tolist())
                                + " open" if args.gate else f"top {wl.n_keep} by criticality")},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "timing": {"blocks": len(rep_ms), "steps_per_block": args.steps,
                   "ms_per_step_median": round(rep_ms[len(rep_ms) // 2], 5),
                   "ms_per_step_min": round(rep_ms[0], 5), "ms_per_step_max": round(rep_ms[-1], 5)},
        "kernels": kern,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
