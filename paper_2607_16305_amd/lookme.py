"""Thin ctypes binding of liblookme.so (the C ABI in include/lookme.h).

Argument marshalling only: every step of the path runs in the library's
gfx950 kernels.  If the library has not been built this module raises on
first use; there is no other implementation to fall back to.

The functions keep the C names and order of arguments; tensors are torch
tensors (device memory), converted to raw pointers here.
"""

from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblookme.so")

LOOKME_OK, LOOKME_ERR_INVALID, LOOKME_ERR_UNSUPPORTED, LOOKME_ERR_WORKSPACE, LOOKME_ERR_HIP = range(5)
LOOKME_F32, LOOKME_BF16 = 0, 1
LOOKME_SCORE_DOT, LOOKME_SCORE_COS = 0, 1
LOOKME_KMAX = 32
LOOKME_NOALLOC_MAX_ROWS = 131072

STATUS_NAMES = {0: "OK", 1: "INVALID", 2: "UNSUPPORTED", 3: "WORKSPACE", 4: "HIP"}

EXPORTED = ("lookme_create", "lookme_workspace_size", "lookme_set_workspace", "lookme_route",
            "lookme_lookup", "lookme_inject", "lookme_select", "lookme_inject_kept",
            "lookme_set_relevance", "lookme_lookup_relevance", "lookme_set_fusion",
            "lookme_inject_fused", "lookme_set_propagation", "lookme_inject_propagated",
            "lookme_set_multiscale", "lookme_inject_multiscale",
            "lookme_inject_multiscale_gated", "lookme_gate",
            "lookme_inject_gated", "lookme_inject_fused_gated", "lookme_inject_propagated_gated",
            "lookme_inject_text", "lookme_lookup_select", "lookme_lookup_gate",
            "lookme_scene_keys", "lookme_index_errors",
            "lookme_destroy", "lookme_last_error",
            "lookme_profile_enable", "lookme_profile_read", "lookme_inject_noalloc")

GROUPS = ("project", "route", "bucket", "score", "norm", "select", "inject")


class LookmeError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"LOOKME_ERR_{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class lookme_desc_t(ctypes.Structure):
    _fields_ = [("num_scenes", ctypes.c_int32), ("prims_per_scene", ctypes.c_int32),
                ("key_dim", ctypes.c_int32), ("value_dim", ctypes.c_int32),
                ("top_k", ctypes.c_int32), ("dtype", ctypes.c_int32), ("score", ctypes.c_int32)]


_lib = None
_vp = ctypes.c_void_p


def load():
    """Load liblookme.so once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2607_16305_amd.build` (no fallback path exists)")
    lib = ctypes.CDLL(LIB_PATH)
    st = ctypes.c_int
    sig = {
        "lookme_create": [ctypes.POINTER(lookme_desc_t), _vp, _vp, _vp, _vp, ctypes.POINTER(_vp)],
        "lookme_workspace_size": [_vp, ctypes.c_int32, ctypes.c_int64,
                                  ctypes.POINTER(ctypes.c_size_t)],
        "lookme_set_workspace": [_vp, _vp, ctypes.c_size_t],
        "lookme_route": [_vp, ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, _vp, _vp, _vp, _vp,
                         _vp],
        "lookme_lookup": [_vp, ctypes.c_int32, ctypes.c_int64, _vp, _vp, _vp, _vp, _vp],
        "lookme_inject": [_vp, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, _vp,
                          ctypes.c_int32, _vp, _vp, _vp, _vp, ctypes.c_int32, _vp, _vp],
        "lookme_select": [_vp, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, _vp,
                          ctypes.c_int32, _vp, _vp],
        "lookme_inject_noalloc": [_vp, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, _vp,
                                  ctypes.c_int32, _vp, _vp, _vp, _vp, ctypes.c_int32, _vp, _vp],
        "lookme_inject_kept": [_vp, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, _vp, _vp, _vp,
                               _vp, _vp, ctypes.c_int32, _vp],
        "lookme_set_relevance": [_vp, ctypes.c_int32, _vp, _vp, _vp, _vp],
        "lookme_lookup_relevance": [_vp, ctypes.c_int32, ctypes.c_int64, _vp, _vp, _vp, _vp, _vp,
                                    _vp],
        "lookme_set_fusion": [_vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp, _vp,
                              _vp],
        "lookme_inject_fused": [_vp, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, _vp, _vp,
                                _vp, _vp, _vp, ctypes.c_int32, _vp],
        "lookme_set_propagation": [_vp, ctypes.c_int32, _vp],
        "lookme_set_multiscale": [_vp, ctypes.c_int32, ctypes.c_int32, _vp],
        "lookme_inject_multiscale": [_vp, ctypes.c_int64, ctypes.c_int64, _vp, _vp, _vp, _vp, _vp,
                                     ctypes.c_int32, _vp],
        "lookme_inject_propagated": [_vp, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, _vp,
                                     _vp, _vp, _vp, _vp, ctypes.c_int32, _vp],
        "lookme_gate": [_vp, ctypes.c_int32, ctypes.c_int64, _vp, ctypes.c_int64, ctypes.c_int32,
                        _vp, _vp, _vp, _vp, _vp],
        "lookme_inject_multiscale_gated": [_vp, ctypes.c_int64, _vp, _vp, _vp, _vp, _vp, _vp,
                                           ctypes.c_int32, _vp],
        "lookme_inject_gated": [_vp, ctypes.c_int32, ctypes.c_int64, _vp, _vp, _vp, _vp, _vp,
                                _vp, ctypes.c_int32, _vp],
        "lookme_inject_fused_gated": [_vp, ctypes.c_int32, ctypes.c_int64, _vp, _vp, _vp, _vp,
                                      _vp, _vp, ctypes.c_int32, _vp],
        "lookme_inject_propagated_gated": [_vp, ctypes.c_int32, ctypes.c_int64, _vp, _vp, _vp,
                                           _vp, _vp, _vp, ctypes.c_int32, _vp],
        "lookme_scene_keys": [ctypes.POINTER(lookme_desc_t), _vp, _vp, _vp],
        "lookme_index_errors": [_vp, ctypes.POINTER(ctypes.c_uint64)],
        "lookme_inject_text": [ctypes.c_int32, _vp, ctypes.c_int64, ctypes.c_int32,
                               ctypes.c_int64, _vp, _vp, _vp, _vp, _vp, ctypes.c_int64,
                               ctypes.c_int32, _vp],
        "lookme_lookup_select": [_vp, ctypes.c_int32, ctypes.c_int64, _vp, _vp, _vp, _vp,
                                 ctypes.c_int64, _vp, ctypes.c_int32, _vp, _vp],
        "lookme_lookup_gate": [_vp, ctypes.c_int32, ctypes.c_int64, _vp, _vp, _vp, _vp, _vp,
                               ctypes.c_int32, _vp, _vp, _vp, _vp],
        "lookme_destroy": [_vp],
        "lookme_profile_enable": [_vp, ctypes.c_int32],
        "lookme_profile_read": [_vp, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64),
                                ctypes.POINTER(ctypes.c_double), ctypes.c_int32],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = st
    lib.lookme_last_error.argtypes = []
    lib.lookme_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int):
    if status != LOOKME_OK:
        raise LookmeError(status, load().lookme_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


DTYPE_CODE = {torch.float32: LOOKME_F32, torch.bfloat16: LOOKME_BF16}


def lookme_create(desc: lookme_desc_t, scene_keys, prim_keys, values, scene_bias=None):
    """Returns an opaque handle (int).  The table tensors are borrowed."""
    h = _vp()
    _check(load().lookme_create(ctypes.byref(desc), _ptr(scene_keys), _ptr(prim_keys),
                                _ptr(values), _ptr(scene_bias), ctypes.byref(h)))
    return h.value


def lookme_workspace_size(h, layers: int, n_tokens: int) -> int:
    out = ctypes.c_size_t()
    _check(load().lookme_workspace_size(h, layers, n_tokens, ctypes.byref(out)))
    return out.value


def lookme_set_workspace(h, ws, nbytes: int):
    _check(load().lookme_set_workspace(h, _ptr(ws), nbytes))


def lookme_route(h, layers, n, d_in, x, w_proj, q_out, scene_out, stream=None):
    _check(load().lookme_route(h, layers, n, d_in, _ptr(x), _ptr(w_proj), _ptr(q_out),
                               _ptr(scene_out), _stream(stream)))


def lookme_lookup(h, layers, n, q, scene, prim_out, w_out, stream=None):
    _check(load().lookme_lookup(h, layers, n, _ptr(q), _ptr(scene), _ptr(prim_out),
                                _ptr(w_out), _stream(stream)))


def lookme_inject(h, layers, n, n_keep, crit, d_c, scene, prim, w, hidden, d_h, kept_out=None,
                  stream=None):
    _check(load().lookme_inject(h, layers, n, n_keep, _ptr(crit), d_c, _ptr(scene), _ptr(prim),
                                _ptr(w), _ptr(hidden), d_h, _ptr(kept_out), _stream(stream)))


def lookme_inject_noalloc(h, layers, n, n_keep, crit, d_c, scene, prim, w, hidden, d_h,
                          kept_out=None, stream=None):
    _check(load().lookme_inject_noalloc(h, layers, n, n_keep, _ptr(crit), d_c, _ptr(scene),
                                        _ptr(prim), _ptr(w), _ptr(hidden), d_h, _ptr(kept_out),
                                        _stream(stream)))


def lookme_select(h, layers, n, n_keep, crit, d_c, kept_out, stream=None):
    _check(load().lookme_select(h, layers, n, n_keep, _ptr(crit), d_c, _ptr(kept_out),
                                _stream(stream)))


def lookme_inject_kept(h, layers, n, n_keep, kept, scene, prim, w, hidden, d_h, stream=None):
    _check(load().lookme_inject_kept(h, layers, n, n_keep, _ptr(kept), _ptr(scene), _ptr(prim),
                                     _ptr(w), _ptr(hidden), d_h, _stream(stream)))


def lookme_set_relevance(h, hidden, w1, b1, w2, b2):
    _check(load().lookme_set_relevance(h, hidden, _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2)))


def lookme_lookup_relevance(h, layers, n, q, scene, act_out, prim_out, w_out, stream=None):
    _check(load().lookme_lookup_relevance(h, layers, n, _ptr(q), _ptr(scene), _ptr(act_out),
                                          _ptr(prim_out), _ptr(w_out), _stream(stream)))


def lookme_set_fusion(h, layers, d_ff, d_h, w_gate, w_up, w_down):
    _check(load().lookme_set_fusion(h, layers, d_ff, d_h, _ptr(w_gate), _ptr(w_up),
                                    _ptr(w_down)))


def lookme_inject_fused(h, layers, n, n_keep, kept, scene, prim, w, hidden, d_h, stream=None):
    _check(load().lookme_inject_fused(h, layers, n, n_keep, _ptr(kept), _ptr(scene), _ptr(prim),
                                      _ptr(w), _ptr(hidden), d_h, _stream(stream)))


def lookme_set_propagation(h, steps, w_p_t):
    _check(load().lookme_set_propagation(h, steps, _ptr(w_p_t)))


def lookme_inject_propagated(h, steps, n, n_keep, kept, scene, prim, w, hidden, d_h,
                             stream=None):
    _check(load().lookme_inject_propagated(h, steps, n, n_keep, _ptr(kept), _ptr(scene),
                                           _ptr(prim), _ptr(w), _ptr(hidden), d_h,
                                           _stream(stream)))


def lookme_set_multiscale(h, scales, d_h, w_he_t):
    _check(load().lookme_set_multiscale(h, scales, d_h, _ptr(w_he_t)))


def lookme_inject_multiscale(h, n, n_keep, kept, scene, prim, w, hidden, d_h, stream=None):
    _check(load().lookme_inject_multiscale(h, n, n_keep, _ptr(kept), _ptr(scene), _ptr(prim),
                                           _ptr(w), _ptr(hidden), d_h, _stream(stream)))


def lookme_lookup_select(h, layers, n, q, scene, prim_out, w_out, n_keep, crit, d_c, kept_out,
                         stream=None):
    _check(load().lookme_lookup_select(h, layers, n, _ptr(q), _ptr(scene), _ptr(prim_out),
                                       _ptr(w_out), n_keep, _ptr(crit), d_c, _ptr(kept_out),
                                       _stream(stream)))


def lookme_lookup_gate(h, layers, n, q, scene, prim_out, w_out, delta, d_c, w_g, kept_out,
                       count_out, stream=None):
    _check(load().lookme_lookup_gate(h, layers, n, _ptr(q), _ptr(scene), _ptr(prim_out),
                                     _ptr(w_out), _ptr(delta), d_c, _ptr(w_g), _ptr(kept_out),
                                     _ptr(count_out), _stream(stream)))


def lookme_gate(h, layers, n, delta, delta_rows, d_c, pos, w_g, kept_out, count_out,
                stream=None):
    _check(load().lookme_gate(h, layers, n, _ptr(delta), delta_rows, d_c, _ptr(pos), _ptr(w_g),
                              _ptr(kept_out), _ptr(count_out), _stream(stream)))


def lookme_inject_gated(h, layers, n, kept, count, scene, prim, w, hidden, d_h, stream=None):
    _check(load().lookme_inject_gated(h, layers, n, _ptr(kept), _ptr(count), _ptr(scene),
                                      _ptr(prim), _ptr(w), _ptr(hidden), d_h, _stream(stream)))


def lookme_inject_multiscale_gated(h, n, kept, count, scene, prim, w, hidden, d_h, stream=None):
    _check(load().lookme_inject_multiscale_gated(h, n, _ptr(kept), _ptr(count), _ptr(scene),
                                                 _ptr(prim), _ptr(w), _ptr(hidden), d_h,
                                                 _stream(stream)))


def lookme_inject_fused_gated(h, layers, n, kept, count, scene, prim, w, hidden, d_h,
                              stream=None):
    _check(load().lookme_inject_fused_gated(h, layers, n, _ptr(kept), _ptr(count), _ptr(scene),
                                            _ptr(prim), _ptr(w), _ptr(hidden), d_h,
                                            _stream(stream)))


def lookme_inject_propagated_gated(h, steps, n, kept, count, scene, prim, w, hidden, d_h,
                                   stream=None):
    _check(load().lookme_inject_propagated_gated(h, steps, n, _ptr(kept), _ptr(count),
                                                 _ptr(scene), _ptr(prim), _ptr(w), _ptr(hidden),
                                                 d_h, _stream(stream)))


def lookme_index_errors(stream=None):
    """Kept entries left out for an index out of range since the last call
    (read and reset; synchronises the stream)."""
    v = ctypes.c_uint64(0)
    _check(load().lookme_index_errors(_stream(stream), ctypes.byref(v)))
    return v.value


def lookme_scene_keys(desc, prim_keys, scene_keys, stream=None):
    _check(load().lookme_scene_keys(ctypes.byref(desc) if desc is not None else None,
                                    _ptr(prim_keys), _ptr(scene_keys), _stream(stream)))


def scene_keys(prim_keys, stream=None):
    """lookme_scene_keys on a torch tensor prim_keys [S, P, d_e]: returns the
    [S, d_e] scene keys of Eq. 4 (a new tensor of the same dtype)."""
    import torch
    S, P, d_e = prim_keys.shape
    out = torch.empty((S, d_e), dtype=prim_keys.dtype, device=prim_keys.device)
    desc = lookme_desc_t(S, P, d_e, d_e, 1, DTYPE_CODE[prim_keys.dtype], 0)
    lookme_scene_keys(desc, prim_keys, out, stream)
    return out


def lookme_inject_text(dtype, table, vocab, d_t, n_text, pos, ids, kept, count, hidden, n, d_h,
                       stream=None):
    _check(load().lookme_inject_text(dtype, _ptr(table), vocab, d_t, n_text, _ptr(pos),
                                     _ptr(ids), _ptr(kept), _ptr(count), _ptr(hidden), n, d_h,
                                     _stream(stream)))


def inject_text(table, pos, ids, hidden, kept=None, count=None, stream=None):
    """lookme_inject_text on torch tensors: table [V, d_t], pos and ids
    [n_text] int32, hidden [n, d_h] (updated in place)."""
    lookme_inject_text(DTYPE_CODE[table.dtype], table, table.shape[0], table.shape[1],
                       pos.numel(), pos, ids, kept, count, hidden, hidden.shape[0],
                       hidden.shape[1], stream)


def lookme_destroy(h):
    if h:
        _check(load().lookme_destroy(h))


def lookme_profile_enable(h, enabled: bool):
    _check(load().lookme_profile_enable(h, 1 if enabled else 0))


def lookme_profile_read(h, group: int, reset: bool = False):
    """(number of timed launches, total milliseconds) of one kernel group."""
    c = ctypes.c_int64()
    ms = ctypes.c_double()
    _check(load().lookme_profile_read(h, group, ctypes.byref(c), ctypes.byref(ms),
                                      1 if reset else 0))
    return c.value, ms.value


def lookme_last_error() -> str:
    return load().lookme_last_error().decode()


class Table:
    """Convenience owner of a handle plus its workspace (torch device memory)."""

    def __init__(self, scene_keys, prim_keys, values, top_k, scene_bias=None,
                 score=LOOKME_SCORE_DOT):
        S, P, d_e = prim_keys.shape
        self.desc = lookme_desc_t(S, P, d_e, values.shape[1], top_k,
                                  DTYPE_CODE[prim_keys.dtype], score)
        self.tensors = (scene_keys, prim_keys, values, scene_bias)   # keep alive
        self.handle = lookme_create(self.desc, scene_keys, prim_keys, values, scene_bias)
        self.ws = None
        self.ws_rows = (0, 0)
        self.device = prim_keys.device

    def reserve(self, layers: int, n: int):
        need = lookme_workspace_size(self.handle, layers, n)
        if self.ws is None or self.ws.numel() < need:
            self.ws = torch.empty(need, dtype=torch.uint8, device=self.device)
            lookme_set_workspace(self.handle, self.ws, self.ws.numel())
        return need

    def route(self, x, w_proj, q_out, scene_out, layers=1, stream=None):
        n, d_in = x.shape
        self.reserve(layers, n)
        lookme_route(self.handle, layers, n, d_in, x, w_proj, q_out, scene_out, stream)

    def lookup(self, q, scene, prim_out, w_out, layers=1, stream=None):
        n = scene.numel() // layers
        self.reserve(layers, n)
        lookme_lookup(self.handle, layers, n, q, scene, prim_out, w_out, stream)

    def inject(self, crit, scene, prim, w, hidden, n_keep, kept_out=None, layers=1, stream=None):
        n = scene.numel() // layers
        self.reserve(layers, n)
        lookme_inject(self.handle, layers, n, n_keep, crit, crit.shape[-1], scene, prim, w,
                      hidden, hidden.shape[-1], kept_out, stream)

    def lookup_select(self, q, scene, prim_out, w_out, crit, kept_out, n_keep, layers=1,
                      stream=None):
        n = scene.numel() // layers
        self.reserve(layers, n)
        lookme_lookup_select(self.handle, layers, n, q, scene, prim_out, w_out, n_keep, crit,
                             crit.shape[-1], kept_out, stream)

    def lookup_gate(self, q, scene, prim_out, w_out, delta, w_g, kept_out, count_out, layers=1,
                    stream=None):
        n = scene.numel() // layers
        self.reserve(layers, n)
        lookme_lookup_gate(self.handle, layers, n, q, scene, prim_out, w_out, delta,
                           delta.shape[-1], w_g, kept_out, count_out, stream)

    def select(self, crit, kept_out, n_keep, layers=1, stream=None):
        n = crit.numel() // (layers * crit.shape[-1])
        self.reserve(layers, n)
        lookme_select(self.handle, layers, n, n_keep, crit, crit.shape[-1], kept_out, stream)

    def inject_kept(self, kept, scene, prim, w, hidden, n_keep, layers=1, stream=None):
        n = scene.numel() // layers
        lookme_inject_kept(self.handle, layers, n, n_keep, kept, scene, prim, w, hidden,
                           hidden.shape[-1], stream)

    def set_relevance(self, w1, b1, w2, b2):
        self.relevance = (w1, b1, w2, b2)      # keep alive
        lookme_set_relevance(self.handle, w1.shape[0], w1, b1, w2, b2)

    def lookup_relevance(self, q, scene, act_out, prim_out, w_out, layers=1, stream=None):
        n = scene.numel() // layers
        self.reserve(layers, n)
        lookme_lookup_relevance(self.handle, layers, n, q, scene, act_out, prim_out, w_out,
                                stream)

    def set_fusion(self, w_gate, w_up, w_down):
        self.fusion = (w_gate, w_up, w_down)     # keep alive
        L, d_ff, _ = w_gate.shape
        lookme_set_fusion(self.handle, L, d_ff, w_down.shape[1], w_gate, w_up, w_down)

    def inject_fused(self, kept, scene, prim, w, hidden, n_keep, layers=1, stream=None):
        n = scene.numel() // layers
        self.reserve(layers, n)
        lookme_inject_fused(self.handle, layers, n, n_keep, kept, scene, prim, w, hidden,
                            hidden.shape[-1], stream)

    def set_propagation(self, w_p_t):
        self.propagation = w_p_t                 # keep alive
        lookme_set_propagation(self.handle, w_p_t.shape[0], w_p_t)

    def inject_propagated(self, kept, scene, prim, w, hidden, n_keep, steps, stream=None):
        n = scene.numel()
        self.reserve(steps + 1, n)
        lookme_inject_propagated(self.handle, steps, n, n_keep, kept, scene, prim, w, hidden,
                                 hidden.shape[-1], stream)

    def scale_view(self, m: int, scales: int) -> "Table":
        """A table over scale m's partition (scenes [m S/M, (m+1) S/M)) of
        this table's tensors (views, no copies), for that scale's routing and
        lookup."""
        scene_keys, prim_keys, values, _ = self.tensors
        S, P = prim_keys.shape[0], prim_keys.shape[1]
        Sm = S // scales
        return Table(scene_keys[m * Sm:(m + 1) * Sm], prim_keys[m * Sm:(m + 1) * Sm],
                     values[m * Sm * P:(m + 1) * Sm * P], self.desc.top_k)

    def set_multiscale(self, scales, w_he_t):
        self.multiscale = w_he_t                 # keep alive
        lookme_set_multiscale(self.handle, scales, w_he_t.shape[1], w_he_t)

    def inject_multiscale(self, kept, scene, prim, w, hidden, n_keep, stream=None):
        n = hidden.shape[0]
        self.reserve(1, n)
        lookme_inject_multiscale(self.handle, n, n_keep, kept, scene, prim, w, hidden,
                                 hidden.shape[-1], stream)

    def inject_multiscale_gated(self, kept, count, scene, prim, w, hidden, stream=None):
        n = hidden.shape[0]
        self.reserve(1, n)
        lookme_inject_multiscale_gated(self.handle, n, kept, count, scene, prim, w, hidden,
                                       hidden.shape[-1], stream)

    def gate(self, delta, w_g, kept_out, count_out, pos=None, layers=1, stream=None):
        """lookme_gate: delta [layers, rows, d_c] (or [rows, d_c]); pos [n] or
        None (n = rows); w_g [layers, d_c]; kept_out [layers, n]; count_out
        [layers]."""
        rows = delta.numel() // (layers * delta.shape[-1])
        n = rows if pos is None else pos.numel()
        self.reserve(layers, n)
        lookme_gate(self.handle, layers, n, delta, rows, delta.shape[-1], pos, w_g, kept_out,
                    count_out, stream)

    def inject_gated(self, kept, count, scene, prim, w, hidden, layers=1, stream=None):
        n = scene.numel() // layers
        lookme_inject_gated(self.handle, layers, n, kept, count, scene, prim, w, hidden,
                            hidden.shape[-1], stream)

    def inject_fused_gated(self, kept, count, scene, prim, w, hidden, layers=1, stream=None):
        n = scene.numel() // layers
        self.reserve(layers, n)
        lookme_inject_fused_gated(self.handle, layers, n, kept, count, scene, prim, w, hidden,
                                  hidden.shape[-1], stream)

    def inject_propagated_gated(self, kept, count, scene, prim, w, hidden, steps, stream=None):
        n = scene.numel()
        self.reserve(steps + 1, n)
        lookme_inject_propagated_gated(self.handle, steps, n, kept, count, scene, prim, w, hidden,
                                       hidden.shape[-1], stream)

    def close(self):
        if self.handle:
            lookme_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
