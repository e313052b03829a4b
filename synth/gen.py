"""Seeded, chunked generation of synthetic LookME workloads.

The paper's own inputs (vision-encoder tokens of Qwen2.5-VL on its fifteen
evaluation benchmarks, and its trained tables) are not available; these
synthetic tensors stand in for them with the shapes of the paper's
configuration (Sec. 4.1: d_e = 512, top-8 primitives, LookME at several LLM
layers) scaled to the sizes of the benchmark workloads.  No benchmark item is
reproduced.

Recipe (all normal draws are std, not variance):
  tokens x          iid N(0, 1), or clustered: x_t = c_{label_t} + N(0, 0.3^2)
                    with centroids c_s ~ N(0, I) and labels uniform or Zipf
  projection W_l    N(0, 1/d_in), stored as W_l^T  [d_e, d_in]
  scene keys K1     unit-norm Gaussian rows, or for clustered tokens
                    normalize(c_s W_0) so that layer-0 routing recovers labels
  primitive keys K2 unit-norm Gaussian rows  [S, P, d_e]
  table values V    N(0, value_std)          [S*P, d_v]
  criticality Delta Delta_t = a_t z_t, a_t ~ LogNormal(0, 1), z_t ~ N(0, I/d_c)
  hidden H          iid N(0, 1)              [L, N, d_h]

Seeds: sub-seed = 1000 * seed + tensor id (x=1, K1=2, K2=3, V=4, labels=5,
centroids=6, zipf permutation=7, W_l=10+l, Delta_l=20+l, H_l=30+l); large
tensors are drawn in chunks of 2^26 elements, chunk c seeded from
(sub-seed, c), so the bytes depend only on (workload, seed, device type).
Tensors are drawn in float32 and rounded to the storage dtype (bf16 by
round-to-nearest-even in torch); keys are normalised in float32 first.
"""

from __future__ import annotations

import dataclasses
import math

import torch

CHUNK = 1 << 26

TID_X, TID_K1, TID_K2, TID_V, TID_LABELS, TID_CENT, TID_PERM = 1, 2, 3, 4, 5, 6, 7
TID_W, TID_DELTA, TID_H = 10, 20, 30
TID_MLP_W1, TID_MLP_B1, TID_MLP_W2, TID_MLP_B2 = 40, 41, 42, 43
TID_FUS_GATE, TID_FUS_UP, TID_FUS_DOWN = 50, 60, 70
TID_PROP = 80
TID_MS_X, TID_MS_W, TID_MS_HE = 90, 100, 110
TID_GATE, TID_TEXT_TAB, TID_TEXT_IDS, TID_TEXT_POS = 120, 130, 131, 132
TID_CROSS_W, TID_CROSS_K1, TID_CROSS_K2, TID_CROSS_V, TID_HDEC, TID_SEQ_DELTA = (
    140, 141, 142, 143, 144, 145)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    dtype: str            # "bf16" | "f32"
    n_tokens: int
    layers: int
    d_in: int
    d_e: int
    scenes: int
    prims: int
    d_v: int
    d_h: int
    top_k: int
    keep_pct: int         # percent of tokens kept per layer
    usage: str = "iid"    # "iid" | "uniform" | "zipf"
    zipf_s: float = 1.1
    project: bool = True  # False: tokens are used directly as queries
    value_std: float = 0.02
    noise_std: float = 0.3
    d_c: int = 0          # criticality width; 0 means d_h

    @property
    def crit_dim(self) -> int:
        return self.d_c or self.d_h

    @property
    def n_keep(self) -> int:
        return n_keep_for(self.keep_pct, self.n_tokens)

    def scaled(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def n_keep_for(pct: int, n: int) -> int:
    """Kept-token count: pct percent of n rounded half up, in integers."""
    return (pct * n + 50) // 100


# The five benchmark workloads (sizes as stated for the benchmark suite).
WORKLOADS = {
    0: Workload("tiny_f32_n256_s16_p64", "f32", 256, 1, 256, 256, 16, 64, 256, 256,
                4, 25, usage="iid", project=False),
    1: Workload("image_n1024_s256_p1024_dv2048", "bf16", 1024, 1, 2048, 512, 256, 1024,
                2048, 2048, 8, 20, usage="iid"),
    2: Workload("multiscale_n23040_s1024_p1024_dv1536", "bf16", 23040, 1, 2048, 512, 1024,
                1024, 1536, 2048, 8, 15, usage="uniform"),
    3: Workload("reuse4_n23040_s1024_p1024_dv2048", "bf16", 23040, 4, 2048, 512, 1024, 1024,
                2048, 2048, 8, 10, usage="uniform"),
    4: Workload("zipf_n32768_s4096_p4096_dv1024", "bf16", 32768, 1, 4096, 512, 4096, 4096,
                1024, 4096, 16, 20, usage="zipf"),
}

TORCH_DTYPE = {"bf16": torch.bfloat16, "f32": torch.float32}


def _gen(seed: int, chunk: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1_000_003 + chunk * 7919 + 12345) & 0x7FFF_FFFF_FFFF)
    return g


def _randn_rows(rows: int, cols: int, sub_seed: int, device, std: float,
                dtype, normalize: bool = False) -> torch.Tensor:
    """[rows, cols] N(0, std) drawn in row-aligned chunks, optionally with
    every row scaled to unit L2 norm, then rounded to ``dtype``."""
    out = torch.empty((rows, cols), dtype=dtype, device=device)
    rows_per = max(1, CHUNK // max(cols, 1))
    for c, r0 in enumerate(range(0, rows, rows_per)):
        r1 = min(rows, r0 + rows_per)
        t = torch.randn((r1 - r0, cols), generator=_gen(sub_seed, c, device),
                        device=device, dtype=torch.float32)
        if normalize:
            t = t / t.norm(dim=1, keepdim=True).clamp_min(1e-30)
        else:
            t.mul_(std)
        out[r0:r1] = t.to(dtype)
    return out


def _labels(wl: Workload, base: int, device) -> torch.Tensor:
    n, S = wl.n_tokens, wl.scenes
    g = _gen(base + TID_LABELS, 0, device)
    if wl.usage == "uniform":
        return torch.randint(0, S, (n,), generator=g, device=device, dtype=torch.int64)
    if wl.usage == "zipf":
        ranks = torch.arange(1, S + 1, device=device, dtype=torch.float64)
        p = ranks.pow(-wl.zipf_s)
        p = (p / p.sum()).to(torch.float32)
        r = torch.multinomial(p, n, replacement=True, generator=g)
        perm = torch.randperm(S, generator=_gen(base + TID_PERM, 0, device), device=device)
        return perm[r]
    raise ValueError(wl.usage)


def make_inputs(wl: Workload, seed: int, device="cpu") -> dict:
    """Draw every input of one workload.

    Returns a dict of torch tensors on ``device``:
      x [N, d_in]; wt [L, d_e, d_in] (None when tokens are queries);
      scene_keys [S, d_e]; prim_keys [S, P, d_e]; values [S*P, d_v];
      bias None; delta [L, N, d_c]; hidden [L, N, d_h]; labels [N] or None;
    plus the workload and the integer parameters k and n_keep.
    """
    dev = torch.device(device)
    dt = TORCH_DTYPE[wl.dtype]
    base = 1000 * seed
    N, L = wl.n_tokens, wl.layers
    if not wl.project and wl.d_in != wl.d_e:
        raise ValueError("unprojected workloads need d_in == d_e")

    labels = None
    centroids = None
    if wl.usage == "iid":
        x = _randn_rows(N, wl.d_in, base + TID_X, dev, 1.0, dt)
    else:
        labels = _labels(wl, base, dev)
        centroids = _randn_rows(wl.scenes, wl.d_in, base + TID_CENT, dev, 1.0, torch.float32)
        noise = _randn_rows(N, wl.d_in, base + TID_X, dev, wl.noise_std, torch.float32)
        x = (centroids[labels] + noise).to(dt)
        del noise

    wt = None
    if wl.project:
        wt = torch.empty((L, wl.d_e, wl.d_in), dtype=dt, device=dev)
        for l in range(L):
            wt[l] = _randn_rows(wl.d_e, wl.d_in, base + TID_W + l, dev,
                                1.0 / math.sqrt(wl.d_in), dt)

    if centroids is not None and wt is not None:
        k1 = centroids @ wt[0].to(torch.float32).T
        k1 = k1 / k1.norm(dim=1, keepdim=True).clamp_min(1e-30)
        scene_keys = k1.to(dt)
    else:
        scene_keys = _randn_rows(wl.scenes, wl.d_e, base + TID_K1, dev, 1.0, dt,
                                 normalize=True)
    prim_keys = _randn_rows(wl.scenes * wl.prims, wl.d_e, base + TID_K2, dev, 1.0, dt,
                            normalize=True).view(wl.scenes, wl.prims, wl.d_e)
    values = _randn_rows(wl.scenes * wl.prims, wl.d_v, base + TID_V, dev, wl.value_std, dt)

    delta = torch.empty((L, N, wl.crit_dim), dtype=dt, device=dev)
    hidden = torch.empty((L, N, wl.d_h), dtype=dt, device=dev)
    for l in range(L):
        g = _gen(base + TID_DELTA + l, 0, dev)
        a = torch.exp(torch.randn((N, 1), generator=g, device=dev, dtype=torch.float32))
        z = _randn_rows(N, wl.crit_dim, base + TID_DELTA + l + 500, dev,
                        1.0 / math.sqrt(wl.crit_dim), torch.float32)
        delta[l] = (a * z).to(dt)
        del z
        hidden[l] = _randn_rows(N, wl.d_h, base + TID_H + l, dev, 1.0, dt)

    return dict(workload=wl, x=x, wt=wt, scene_keys=scene_keys, prim_keys=prim_keys,
                values=values, bias=None, delta=delta, hidden=hidden, labels=labels,
                k=wl.top_k, n_keep=wl.n_keep)


def make_integer_inputs(n: int, S: int, P: int, d_e: int, d_v: int, d_h: int, k: int,
                        n_keep: int, seed: int, dtype: str = "bf16", device="cpu",
                        layers: int = 1) -> dict:
    """Inputs whose scores are small exact integers (entries in {-2..2}), so
    that many scores tie exactly; queries are used directly (no projection).
    Exact in fp32 and bf16 arithmetic for d_e <= 256: every tie-break is
    decided by index alone."""
    dev = torch.device(device)
    dt = TORCH_DTYPE[dtype]
    g = _gen(1000 * seed + 90, 0, dev)
    ri = lambda shape, lo, hi: torch.randint(lo, hi + 1, shape, generator=g, device=dev,
                                             dtype=torch.int64).to(dt)
    x = ri((n, d_e), -2, 2)
    scene_keys = ri((S, d_e), -1, 1)
    prim_keys = ri((S, P, d_e), -1, 1)
    values = ri((S * P, d_v), -3, 3)
    delta = ri((layers, n, d_h), -1, 1)       # few distinct norms: ties at the cut
    hidden = ri((layers, n, d_h), -4, 4)
    return dict(workload=None, x=x, wt=None, scene_keys=scene_keys, prim_keys=prim_keys,
                values=values, bias=None, delta=delta, hidden=hidden, labels=None, k=k,
                n_keep=n_keep)


def make_relevance(wl: Workload, seed: int, hidden: int, device="cpu") -> dict:
    """Seeded weights of a scene-shared relevance MLP (the paper trains them;
    none are available here): W1 [hidden, 2 d_e] ~ N(0, 1/(2 d_e)) and
    W2 [P, hidden] ~ N(0, 2/hidden), so that activations and logits stay of
    order one, in the workload's dtype; biases b1 [hidden], b2 [P] ~ N(0, 0.1)
    in float32."""
    dev = torch.device(device)
    dt = TORCH_DTYPE[wl.dtype]
    base = 1000 * seed
    w1 = _randn_rows(hidden, 2 * wl.d_e, base + TID_MLP_W1, dev,
                     1.0 / math.sqrt(2 * wl.d_e), dt)
    b1 = _randn_rows(1, hidden, base + TID_MLP_B1, dev, 0.1, torch.float32)[0]
    w2 = _randn_rows(wl.prims, hidden, base + TID_MLP_W2, dev, math.sqrt(2.0 / hidden), dt)
    b2 = _randn_rows(1, wl.prims, base + TID_MLP_B2, dev, 0.1, torch.float32)[0]
    return dict(w1=w1, b1=b1.contiguous(), w2=w2, b2=b2.contiguous(), hidden=hidden)


def make_fusion(wl: Workload, seed: int, d_ff: int, device="cpu", layers=None) -> dict:
    """Seeded SwiGLU fusion weights per layer (Eq. 10; the paper trains
    them): W_gate, W_up [L, d_ff, d_v] ~ N(0, 1/d_v) and W_down [L, d_h, d_ff]
    ~ N(0, 1/d_ff), in the workload's dtype; L = ``layers`` or the
    workload's layer count (at most 10)."""
    dev = torch.device(device)
    dt = TORCH_DTYPE[wl.dtype]
    base = 1000 * seed
    L = layers or wl.layers
    assert L <= 10
    gate = torch.empty((L, d_ff, wl.d_v), dtype=dt, device=dev)
    up = torch.empty((L, d_ff, wl.d_v), dtype=dt, device=dev)
    down = torch.empty((L, wl.d_h, d_ff), dtype=dt, device=dev)
    for l in range(L):
        gate[l] = _randn_rows(d_ff, wl.d_v, base + TID_FUS_GATE + l, dev, 1.0 / math.sqrt(wl.d_v), dt)
        up[l] = _randn_rows(d_ff, wl.d_v, base + TID_FUS_UP + l, dev, 1.0 / math.sqrt(wl.d_v), dt)
        down[l] = _randn_rows(wl.d_h, d_ff, base + TID_FUS_DOWN + l, dev, 1.0 / math.sqrt(d_ff), dt)
    return dict(w_gate=gate, w_up=up, w_down=down, d_ff=d_ff)


def make_propagation(wl: Workload, seed: int, steps: int, device="cpu") -> torch.Tensor:
    """Seeded propagation projections of Eq. 11 (trained in the paper), one
    per propagated layer (at most 10): W_p ~ N(0, 1/(4 d_v)), returned
    transposed (output-row-major) as w_p_t [steps, d_v, d_v] in the
    workload's dtype; the residual keeps R's scale within a factor of about
    1.1 a step."""
    assert 1 <= steps <= 10
    dev = torch.device(device)
    dt = TORCH_DTYPE[wl.dtype]
    out = torch.empty((steps, wl.d_v, wl.d_v), dtype=dt, device=dev)
    for j in range(steps):
        out[j] = _randn_rows(wl.d_v, wl.d_v, 1000 * seed + TID_PROP + j, dev,
                             0.5 / math.sqrt(wl.d_v), dt)
    return out


def make_multiscale(wl: Workload, seed: int, scales: int, device="cpu") -> dict:
    """Seeded inputs of multi-scale retrieval (Sec. 3.2, Eq. 8) over the
    workload's table split into ``scales`` scene partitions (at most 10):
    per-scale tokens x [M, n, d_in] iid N(0, 1) (features of M encoder
    layers), per-scale projections W^T [M, d_e, d_in] ~ N(0, 1/d_in) and the
    router projection W_{h->e} stored transposed, w_he_t [d_v, d_h] ~
    N(0, 1/d_h), in the workload's dtype (the paper trains them)."""
    assert 1 <= scales <= 10 and wl.scenes % scales == 0
    dev = torch.device(device)
    dt = TORCH_DTYPE[wl.dtype]
    base = 1000 * seed
    n = wl.n_tokens
    x = torch.empty((scales, n, wl.d_in), dtype=dt, device=dev)
    wt = torch.empty((scales, wl.d_e, wl.d_in), dtype=dt, device=dev)
    for m in range(scales):
        x[m] = _randn_rows(n, wl.d_in, base + TID_MS_X + m, dev, 1.0, dt)
        wt[m] = _randn_rows(wl.d_e, wl.d_in, base + TID_MS_W + m, dev, 1.0 / math.sqrt(wl.d_in), dt)
    w_he_t = _randn_rows(wl.d_v, wl.d_h, base + TID_MS_HE, dev, 1.0 / math.sqrt(wl.d_h), dt)
    return dict(x=x, wt=wt, w_he_t=w_he_t, scales=scales)


def make_gate(wl: Workload, seed: int, device="cpu", layers=None, tid: int = TID_GATE) -> torch.Tensor:
    """Seeded SKA gate projections (Eq. 9; trained in the paper), one column
    per layer: w_g [L, d_c] ~ N(0, 1/d_c) in the workload's dtype, so that
    z = Delta W_g is of the order of ||Delta|| / sqrt(d_c) and about half of
    the gates open on zero-mean Delta.  ``tid`` separates the pathways'
    gates."""
    dev = torch.device(device)
    dt = TORCH_DTYPE[wl.dtype]
    L = layers or wl.layers
    return _randn_rows(L, wl.crit_dim, 1000 * seed + tid, dev, 1.0 / math.sqrt(wl.crit_dim), dt)


def make_text(seed: int, vocab: int, d_t: int, pos: torch.Tensor, dtype: str = "bf16",
              device="cpu", value_std: float = 0.02) -> dict:
    """Seeded text pathway inputs (Sec. 3.2, Eq. 1): a text table
    [vocab, d_t] ~ N(0, value_std) and token ids uniform in [0, vocab) for
    the given text positions ``pos`` [n_text] (int32)."""
    dev = torch.device(device)
    dt = TORCH_DTYPE[dtype]
    table = _randn_rows(vocab, d_t, 1000 * seed + TID_TEXT_TAB, dev, value_std, dt)
    g = _gen(1000 * seed + TID_TEXT_IDS, 0, dev)
    ids = torch.randint(0, vocab, (pos.numel(),), generator=g, device=dev, dtype=torch.int64)
    return dict(table=table, pos=pos.to(device=dev, dtype=torch.int32).contiguous(),
                ids=ids.to(torch.int32), vocab=vocab, d_t=d_t)


def make_layer(wl: Workload, seed: int, text_before: int, text_after: int, vocab: int,
               d_t: int, cross_scenes: int, cross_prims: int, cross_k: int,
               device="cpu") -> dict:
    """One LookME layer's inputs (Eq. 2) over a sequence of text_before text
    positions, the workload's n_tokens image positions, then text_after text
    positions:
      image   the workload's inputs (make_inputs; its first layer is used)
              for the image block [text_before, text_before + n_tokens);
      h_dec   L_dec(H_in) [n_seq, d_h] iid N(0, 1);
      delta   Delta = Attn(H_in) [n_seq, d_c], rows a_t z_t with a_t
              log-normal and z_t ~ N(0, I / d_c) as for the image workload;
      text    make_text over the text positions, table [vocab, d_t];
      cross   the cross-modal pathway's own table: cross_scenes x cross_prims
              unit-norm keys of width d_e, rows [S P, d_h] ~ N(0, value_std),
              and its query projection W^T [d_e, d_h] ~ N(0, 1/d_h);
      gates   w_g [3, d_c] (text, image, cross) from make_gate.
    """
    dev = torch.device(device)
    dt = TORCH_DTYPE[wl.dtype]
    base = 1000 * seed
    img = make_inputs(wl.scaled(layers=1), seed, device)
    n_img = wl.n_tokens
    n_seq = text_before + n_img + text_after
    pos = torch.cat([torch.arange(0, text_before),
                     torch.arange(text_before + n_img, n_seq)]).to(torch.int32)
    text = make_text(seed, vocab, d_t, pos, wl.dtype, device, wl.value_std)
    h_dec = _randn_rows(n_seq, wl.d_h, base + TID_HDEC, dev, 1.0, dt)
    g = _gen(base + TID_SEQ_DELTA, 0, dev)
    a = torch.exp(torch.randn((n_seq, 1), generator=g, device=dev, dtype=torch.float32))
    z = _randn_rows(n_seq, wl.crit_dim, base + TID_SEQ_DELTA + 500, dev,
                    1.0 / math.sqrt(wl.crit_dim), torch.float32)
    delta = (a * z).to(dt)
    cross = dict(
        wt=_randn_rows(wl.d_e, wl.d_h, base + TID_CROSS_W, dev, 1.0 / math.sqrt(wl.d_h),
                       dt).unsqueeze(0),
        scene_keys=_randn_rows(cross_scenes, wl.d_e, base + TID_CROSS_K1, dev, 1.0, dt,
                               normalize=True),
        prim_keys=_randn_rows(cross_scenes * cross_prims, wl.d_e, base + TID_CROSS_K2, dev, 1.0,
                              dt, normalize=True).view(cross_scenes, cross_prims, wl.d_e),
        values=_randn_rows(cross_scenes * cross_prims, wl.d_h, base + TID_CROSS_V, dev,
                           wl.value_std, dt),
        k=cross_k)
    w_g = torch.cat([make_gate(wl, seed, device, 1, TID_GATE + 10 * p) for p in range(3)])
    return dict(workload=wl, image=img, start=text_before, n_seq=n_seq, h_dec=h_dec,
                delta=delta, text=text, cross=cross, w_g=w_g)
