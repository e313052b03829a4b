"""C-ABI checks that need no GPU: the library loads, exports every entry
point declared in include/lookme.h, and rejects bad arguments before
anything is launched (fake, aligned device addresses are never touched)."""

import ctypes
import os
import re

import pytest

from paper_2607_16305_amd import lookme as lk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lookme.h")
FAKE = 0x7F0000100000          # 256-byte aligned stand-in address, never dereferenced


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"\b(lookme_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(lk.LIB_PATH):
        pytest.fail("liblookme.so is not built (run __graft_entry__.build())")
    return lk.load()


def test_exports_every_declared_entry_point(lib):
    names = _declared()
    assert set(lk.EXPORTED) == set(names)
    for name in names:
        assert hasattr(lib, name), name


def _desc(**kw):
    d = dict(num_scenes=16, prims_per_scene=64, key_dim=256, value_dim=256, top_k=4,
             dtype=lk.LOOKME_F32, score=lk.LOOKME_SCORE_DOT)
    d.update(kw)
    return lk.lookme_desc_t(**d)


def _status(fn):
    try:
        fn()
    except lk.LookmeError as e:
        return e.status, str(e)
    return lk.LOOKME_OK, ""


@pytest.mark.parametrize("kw,status", [
    (dict(top_k=0), lk.LOOKME_ERR_INVALID),
    (dict(top_k=65), lk.LOOKME_ERR_INVALID),                  # k > P
    (dict(prims_per_scene=64, top_k=33), lk.LOOKME_ERR_UNSUPPORTED),   # k > KMAX
    (dict(num_scenes=0), lk.LOOKME_ERR_INVALID),
    (dict(dtype=7), lk.LOOKME_ERR_INVALID),
    (dict(key_dim=250), lk.LOOKME_ERR_UNSUPPORTED),           # 1000 B, not a multiple of 64
    (dict(key_dim=1024), lk.LOOKME_ERR_UNSUPPORTED),          # 4096 B > 2048 B (fp32)
    (dict(value_dim=3), lk.LOOKME_ERR_UNSUPPORTED),
    (dict(num_scenes=20000), lk.LOOKME_ERR_UNSUPPORTED),
    (dict(score=5), lk.LOOKME_ERR_INVALID),
])
def test_create_rejects(lib, kw, status):
    st, msg = _status(lambda: lk.lookme_create(_desc(**kw), FAKE, FAKE, FAKE))
    assert st == status, msg
    assert msg


def test_create_rejects_null_and_misaligned(lib):
    assert _status(lambda: lk.lookme_create(_desc(), None, FAKE, FAKE))[0] == lk.LOOKME_ERR_INVALID
    assert _status(lambda: lk.lookme_create(_desc(), FAKE, FAKE + 8, FAKE))[0] == \
        lk.LOOKME_ERR_INVALID


def test_create_destroy_and_workspace_size(lib):
    h = lk.lookme_create(_desc(), FAKE, FAKE, FAKE)
    try:
        a = lk.lookme_workspace_size(h, 1, 256)
        b = lk.lookme_workspace_size(h, 4, 256)
        assert 0 < a < b
        assert lk.lookme_workspace_size(h, 1, 0) >= 256
        assert _status(lambda: lk.lookme_workspace_size(h, 0, 5))[0] == lk.LOOKME_ERR_INVALID
        assert _status(lambda: lk.lookme_workspace_size(h, 1, -1))[0] == lk.LOOKME_ERR_INVALID
    finally:
        lk.lookme_destroy(h)


def test_calls_validate_before_launch(lib):
    bf = _desc(dtype=lk.LOOKME_BF16, key_dim=512, value_dim=2048, prims_per_scene=1024,
               top_k=8, num_scenes=256)
    h = lk.lookme_create(bf, FAKE, FAKE, FAKE)
    try:
        S = lambda f: _status(f)[0]
        # n == 0 is a no-op, even with null pointers
        assert S(lambda: lk.lookme_route(h, 1, 0, 2048, None, FAKE, None, None, 0)) == lk.LOOKME_OK
        assert S(lambda: lk.lookme_lookup(h, 1, 0, None, None, None, None, 0)) == lk.LOOKME_OK
        # null and misaligned pointers
        assert S(lambda: lk.lookme_route(h, 1, 8, 2048, None, FAKE, FAKE, FAKE, 0)) == \
            lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_route(h, 1, 8, 2048, FAKE + 4, FAKE, FAKE, FAKE, 0)) == \
            lk.LOOKME_ERR_INVALID
        # no projection needs d_in == d_e
        assert S(lambda: lk.lookme_route(h, 1, 8, 2048, FAKE, None, FAKE, FAKE, 0)) == \
            lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_route(h, 1, 8, 100, FAKE, FAKE, FAKE, FAKE, 0)) == \
            lk.LOOKME_ERR_UNSUPPORTED
        assert S(lambda: lk.lookme_route(h, 0, 8, 2048, FAKE, FAKE, FAKE, FAKE, 0)) == \
            lk.LOOKME_ERR_INVALID
        # route, lookup and inject need a workspace
        assert S(lambda: lk.lookme_route(h, 1, 8, 2048, FAKE, FAKE, FAKE, FAKE, 0)) == \
            lk.LOOKME_ERR_WORKSPACE
        assert S(lambda: lk.lookme_lookup(h, 1, 8, FAKE, FAKE, FAKE, FAKE, 0)) == \
            lk.LOOKME_ERR_WORKSPACE
        assert S(lambda: lk.lookme_inject(h, 1, 8, 2, FAKE, 2048, FAKE, FAKE, FAKE, FAKE, 2048,
                                          None, 0)) == lk.LOOKME_ERR_WORKSPACE
        # inject argument ranges
        assert S(lambda: lk.lookme_inject(h, 1, 8, 9, FAKE, 2048, FAKE, FAKE, FAKE, FAKE, 2048,
                                          None, 0)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_inject(h, 1, 8, -1, FAKE, 2048, FAKE, FAKE, FAKE, FAKE, 2048,
                                          None, 0)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_inject(h, 1, 8, 2, FAKE, 2048, FAKE, FAKE, FAKE, FAKE, 1024,
                                          None, 0)) == lk.LOOKME_ERR_INVALID     # d_v > d_h
        assert S(lambda: lk.lookme_inject(h, 1, 8, 2, FAKE, 2047, FAKE, FAKE, FAKE, FAKE, 2048,
                                          None, 0)) == lk.LOOKME_ERR_UNSUPPORTED
        msg = _status(lambda: lk.lookme_inject(h, 1, 8, 9, FAKE, 2048, FAKE, FAKE, FAKE, FAKE,
                                               2048, None, 0))[1]
        assert "n_keep" in msg and "n_keep" in lk.lookme_last_error()
        # select alone: ranges, the kept output, the workspace; n_keep = 0 does nothing
        assert S(lambda: lk.lookme_select(h, 1, 8, 9, FAKE, 2048, FAKE, 0)) == \
            lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_select(h, 1, 8, 2, FAKE, 2047, FAKE, 0)) == \
            lk.LOOKME_ERR_UNSUPPORTED
        assert S(lambda: lk.lookme_select(h, 1, 8, 2, FAKE, 2048, None, 0)) == \
            lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_select(h, 1, 8, 2, FAKE, 2048, FAKE, 0)) == \
            lk.LOOKME_ERR_WORKSPACE
        assert S(lambda: lk.lookme_select(h, 1, 8, 0, None, 2048, None, 0)) == lk.LOOKME_OK
        # inject of a given kept set: ranges and pointers (it needs no workspace)
        assert S(lambda: lk.lookme_inject_kept(h, 1, 8, 9, FAKE, FAKE, FAKE, FAKE, FAKE, 2048,
                                               0)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_inject_kept(h, 1, 8, 2, FAKE, FAKE, FAKE, FAKE, FAKE, 1024,
                                               0)) == lk.LOOKME_ERR_INVALID     # d_v > d_h
        assert S(lambda: lk.lookme_inject_kept(h, 1, 8, 2, None, FAKE, FAKE, FAKE, FAKE, 2048,
                                               0)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_inject_kept(h, 1, 8, 0, None, None, None, None, None, 2048,
                                               0)) == lk.LOOKME_OK
    finally:
        lk.lookme_destroy(h)


def test_inject_noalloc_validates_before_launch(lib):
    """The entry point that allocates nothing: the same argument checks as
    lookme_inject, no workspace needed, and a batch beyond its scratch
    rejected before anything runs."""
    bf = _desc(dtype=lk.LOOKME_BF16, key_dim=512, value_dim=2048, prims_per_scene=1024,
               top_k=8, num_scenes=256)
    h = lk.lookme_create(bf, FAKE, FAKE, FAKE)
    try:
        S = lambda f: _status(f)[0]
        inj = lambda layers, n, n_keep, d_c=2048, d_h=2048, crit=FAKE, kept=None: \
            lk.lookme_inject_noalloc(h, layers, n, n_keep, crit, d_c, FAKE, FAKE, FAKE, FAKE,
                                     d_h, kept, 0)
        assert S(lambda: inj(1, 0, 0, crit=None)) == lk.LOOKME_OK
        assert S(lambda: inj(1, 8, 9)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: inj(1, 8, 2, d_h=1024)) == lk.LOOKME_ERR_INVALID      # d_v > d_h
        assert S(lambda: inj(1, 8, 2, d_c=2047)) == lk.LOOKME_ERR_UNSUPPORTED
        assert S(lambda: inj(1, 8, 2, crit=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: inj(1, 8, 2, kept=FAKE + 4)) == lk.LOOKME_ERR_INVALID
        big = lk.LOOKME_NOALLOC_MAX_ROWS
        st, msg = _status(lambda: inj(2, big // 2 + 1, 4))
        assert st == lk.LOOKME_ERR_UNSUPPORTED and "scratch" in msg
        assert S(lambda: inj(1, big + 1, 4)) == lk.LOOKME_ERR_UNSUPPORTED
    finally:
        lk.lookme_destroy(h)


def test_relevance_entry_points_validate(lib):
    bf = _desc(dtype=lk.LOOKME_BF16, key_dim=512, value_dim=2048, prims_per_scene=1024,
               top_k=8, num_scenes=256)
    h = lk.lookme_create(bf, FAKE, FAKE, FAKE)
    try:
        S = lambda f: _status(f)[0]
        # lookup before any MLP is registered
        assert S(lambda: lk.lookme_lookup_relevance(h, 1, 8, FAKE, FAKE, FAKE, FAKE, FAKE, 0)) \
            == lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_set_relevance(h, 0, FAKE, None, FAKE, None)) == \
            lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_set_relevance(h, 96, FAKE, None, FAKE, None)) == \
            lk.LOOKME_ERR_UNSUPPORTED        # 192 bytes: not whole 128-byte stages
        assert S(lambda: lk.lookme_set_relevance(h, 512, None, None, FAKE, None)) == \
            lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_set_relevance(h, 512, FAKE, FAKE + 2, FAKE, None)) == \
            lk.LOOKME_ERR_INVALID
        base = lk.lookme_workspace_size(h, 1, 1000)
        assert S(lambda: lk.lookme_set_relevance(h, 512, FAKE, None, FAKE, None)) == lk.LOOKME_OK
        # the logits of the rows now go through the workspace
        assert lk.lookme_workspace_size(h, 1, 1000) >= base + 1000 * 1024 * 4
        assert S(lambda: lk.lookme_lookup_relevance(h, 1, 0, None, None, None, None, None, 0)) \
            == lk.LOOKME_OK
        assert S(lambda: lk.lookme_lookup_relevance(h, 1, 8, FAKE, FAKE, FAKE, FAKE, FAKE, 0)) \
            == lk.LOOKME_ERR_WORKSPACE
        assert S(lambda: lk.lookme_lookup_relevance(h, 1, 8, FAKE, None, FAKE, FAKE, FAKE, 0)) \
            == lk.LOOKME_ERR_INVALID
    finally:
        lk.lookme_destroy(h)
    # the first layer needs key rows in whole 128-byte stages
    h = lk.lookme_create(_desc(dtype=lk.LOOKME_BF16, key_dim=32), FAKE, FAKE, FAKE)
    try:
        assert _status(lambda: lk.lookme_set_relevance(h, 64, FAKE, None, FAKE, None))[0] == \
            lk.LOOKME_ERR_UNSUPPORTED
    finally:
        lk.lookme_destroy(h)


def test_fusion_entry_points_validate(lib):
    bf = _desc(dtype=lk.LOOKME_BF16, key_dim=512, value_dim=2048, prims_per_scene=1024,
               top_k=8, num_scenes=256)
    h = lk.lookme_create(bf, FAKE, FAKE, FAKE)
    try:
        S = lambda f: _status(f)[0]
        assert S(lambda: lk.lookme_inject_fused(h, 1, 8, 2, FAKE, FAKE, FAKE, FAKE, FAKE, 2048,
                                                0)) == lk.LOOKME_ERR_INVALID     # none set
        assert S(lambda: lk.lookme_set_fusion(h, 1, 0, 2048, FAKE, FAKE, FAKE)) == \
            lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_set_fusion(h, 1, 96, 2048, FAKE, FAKE, FAKE)) == \
            lk.LOOKME_ERR_UNSUPPORTED       # 192 bytes: not whole 128-byte stages
        assert S(lambda: lk.lookme_set_fusion(h, 1, 2048, 2048, FAKE, None, FAKE)) == \
            lk.LOOKME_ERR_INVALID
        base = lk.lookme_workspace_size(h, 1, 100)
        assert S(lambda: lk.lookme_set_fusion(h, 2, 2048, 2048, FAKE, FAKE, FAKE)) == \
            lk.LOOKME_OK
        assert lk.lookme_workspace_size(h, 1, 100) >= base + 100 * (2048 + 2048) * 2
        assert S(lambda: lk.lookme_inject_fused(h, 3, 8, 2, FAKE, FAKE, FAKE, FAKE, FAKE, 2048,
                                                0)) == lk.LOOKME_ERR_INVALID     # 3 > 2 layers
        assert S(lambda: lk.lookme_inject_fused(h, 1, 8, 2, FAKE, FAKE, FAKE, FAKE, FAKE, 1024,
                                                0)) == lk.LOOKME_ERR_INVALID     # wrong d_h
        assert S(lambda: lk.lookme_inject_fused(h, 1, 8, 9, FAKE, FAKE, FAKE, FAKE, FAKE, 2048,
                                                0)) == lk.LOOKME_ERR_INVALID     # n_keep > n
        assert S(lambda: lk.lookme_inject_fused(h, 1, 8, 0, None, None, None, None, None, 2048,
                                                0)) == lk.LOOKME_OK
        assert S(lambda: lk.lookme_inject_fused(h, 1, 8, 2, FAKE, FAKE, FAKE, FAKE, FAKE, 2048,
                                                0)) == lk.LOOKME_ERR_WORKSPACE
    finally:
        lk.lookme_destroy(h)


def test_propagation_entry_points_validate(lib):
    bf = _desc(dtype=lk.LOOKME_BF16, key_dim=512, value_dim=2048, prims_per_scene=1024,
               top_k=8, num_scenes=256)
    h = lk.lookme_create(bf, FAKE, FAKE, FAKE)
    try:
        S = lambda f: _status(f)[0]
        call = lambda steps, n=8, n_keep=2, d_h=2048, p=FAKE: lk.lookme_inject_propagated(
            h, steps, n, n_keep, p, p, p, p, p, d_h, 0)
        assert S(lambda: call(1)) == lk.LOOKME_ERR_INVALID          # no fusion
        assert S(lambda: lk.lookme_set_propagation(h, 0, FAKE)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_set_propagation(h, 2, None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_set_fusion(h, 3, 2048, 2048, FAKE, FAKE, FAKE)) == lk.LOOKME_OK
        assert S(lambda: call(-1)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call(1)) == lk.LOOKME_ERR_INVALID          # no projections
        assert S(lambda: lk.lookme_set_propagation(h, 2, FAKE)) == lk.LOOKME_OK
        assert S(lambda: call(3)) == lk.LOOKME_ERR_INVALID          # 4 layers > fusion's 3
        assert S(lambda: call(2, d_h=1024)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call(2, n_keep=9)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call(2, n_keep=0, p=None)) == lk.LOOKME_OK
        assert S(lambda: call(2, p=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call(2)) == lk.LOOKME_ERR_WORKSPACE
        f32 = _desc(dtype=lk.LOOKME_F32, key_dim=512, value_dim=40, prims_per_scene=64,
                    top_k=4, num_scenes=16)
        h2 = lk.lookme_create(f32, FAKE, FAKE, FAKE)
        try:   # 160-byte rows: not whole 128-byte stages
            assert S(lambda: lk.lookme_set_propagation(h2, 1, FAKE)) == lk.LOOKME_ERR_UNSUPPORTED
        finally:
            lk.lookme_destroy(h2)
    finally:
        lk.lookme_destroy(h)


def test_multiscale_entry_points_validate(lib):
    bf = _desc(dtype=lk.LOOKME_BF16, key_dim=512, value_dim=2048, prims_per_scene=1024,
               top_k=8, num_scenes=256)
    h = lk.lookme_create(bf, FAKE, FAKE, FAKE)
    try:
        S = lambda f: _status(f)[0]
        call = lambda n=8, n_keep=2, d_h=2048, p=FAKE: lk.lookme_inject_multiscale(
            h, n, n_keep, p, p, p, p, p, d_h, 0)
        gated = lambda n=8, c=FAKE, d_h=2048, p=FAKE: lk.lookme_inject_multiscale_gated(
            h, n, p, c, p, p, p, p, d_h, 0)
        assert S(lambda: call()) == lk.LOOKME_ERR_INVALID                    # none registered
        assert S(lambda: gated()) == lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_set_multiscale(h, 0, 2048, FAKE)) == lk.LOOKME_ERR_UNSUPPORTED
        assert S(lambda: lk.lookme_set_multiscale(h, 9, 2048, FAKE)) == lk.LOOKME_ERR_UNSUPPORTED
        assert S(lambda: lk.lookme_set_multiscale(h, 3, 2048, FAKE)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_set_multiscale(h, 2, 1024, FAKE)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_set_multiscale(h, 2, 2056, FAKE)) == lk.LOOKME_ERR_UNSUPPORTED
        assert S(lambda: lk.lookme_set_multiscale(h, 2, 2048, None)) == lk.LOOKME_ERR_INVALID
        base = lk.lookme_workspace_size(h, 1, 100)
        assert S(lambda: lk.lookme_set_multiscale(h, 2, 2048, FAKE)) == lk.LOOKME_OK
        assert lk.lookme_workspace_size(h, 1, 100) >= base + 3 * 100 * 2048 * 2
        assert S(lambda: call(d_h=4096)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call(n_keep=9)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call(n_keep=0, p=None)) == lk.LOOKME_OK
        assert S(lambda: call(p=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call()) == lk.LOOKME_ERR_WORKSPACE
        assert S(lambda: gated(d_h=4096)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: gated(c=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: gated(p=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: gated(n=0, c=None, p=None)) == lk.LOOKME_OK
        assert S(lambda: gated()) == lk.LOOKME_ERR_WORKSPACE
    finally:
        lk.lookme_destroy(h)


def test_null_handle(lib):
    assert _status(lambda: lk.lookme_workspace_size(None, 1, 1))[0] == lk.LOOKME_ERR_INVALID
    assert _status(lambda: lk.lookme_route(None, 1, 1, 1, FAKE, FAKE, FAKE, FAKE, 0))[0] == \
        lk.LOOKME_ERR_INVALID
    lk.lookme_destroy(None)


def test_gate_and_text_entry_points_validate(lib):
    bf = _desc(dtype=lk.LOOKME_BF16, key_dim=512, value_dim=2048, prims_per_scene=1024,
               top_k=8, num_scenes=256)
    h = lk.lookme_create(bf, FAKE, FAKE, FAKE)
    try:
        S = lambda f: _status(f)[0]
        gate = lambda n=8, rows=8, d_c=2048, pos=None, p=FAKE, c=FAKE: lk.lookme_gate(
            h, 1, n, p, rows, d_c, pos, p, p, c, 0)
        assert S(lambda: gate(c=None)) == lk.LOOKME_ERR_INVALID          # count_out needed
        assert S(lambda: gate(d_c=1001)) == lk.LOOKME_ERR_UNSUPPORTED     # 2002 B rows
        assert S(lambda: gate(rows=4)) == lk.LOOKME_ERR_INVALID          # rows < n, no pos
        assert S(lambda: gate(rows=0)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: gate(p=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: gate(pos=FAKE + 4)) == lk.LOOKME_ERR_INVALID     # misaligned
        assert S(lambda: gate()) == lk.LOOKME_ERR_WORKSPACE
        assert S(lambda: gate(rows=4, pos=FAKE)) == lk.LOOKME_ERR_WORKSPACE
        inj = lambda n=8, d_h=2048, c=FAKE, p=FAKE: lk.lookme_inject_gated(
            h, 1, n, p, c, p, p, p, p, d_h, 0)
        assert S(lambda: inj(d_h=1024)) == lk.LOOKME_ERR_INVALID          # d_v > d_h
        assert S(lambda: inj(c=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: inj(p=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: inj(n=0, p=None, c=None)) == lk.LOOKME_OK
        fus = lambda n=8, c=FAKE: lk.lookme_inject_fused_gated(h, 1, n, FAKE, c, FAKE, FAKE,
                                                               FAKE, FAKE, 2048, 0)
        assert S(lambda: fus()) == lk.LOOKME_ERR_INVALID                  # no fusion
        prop = lambda steps=1: lk.lookme_inject_propagated_gated(h, steps, 8, FAKE, FAKE, FAKE,
                                                                 FAKE, FAKE, FAKE, 2048, 0)
        assert S(lambda: prop(-1)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: lk.lookme_set_fusion(h, 2, 2048, 2048, FAKE, FAKE, FAKE)) == lk.LOOKME_OK
        assert S(lambda: fus(c=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: fus()) == lk.LOOKME_ERR_WORKSPACE
        assert S(lambda: prop(1)) == lk.LOOKME_ERR_INVALID                # no projections
    finally:
        lk.lookme_destroy(h)
    txt = lambda dt=lk.LOOKME_BF16, V=100, d_t=64, n_text=5, d_h=64, n=9, p=FAKE, kept=None: \
        lk.lookme_inject_text(dt, p, V, d_t, n_text, p, p, kept, None, p, n, d_h, 0)
    S = lambda f: _status(f)[0]
    assert S(lambda: txt(dt=5)) == lk.LOOKME_ERR_INVALID
    assert S(lambda: txt(V=0)) == lk.LOOKME_ERR_INVALID
    assert S(lambda: txt(d_t=128)) == lk.LOOKME_ERR_INVALID             # d_t > d_h
    assert S(lambda: txt(d_t=4)) == lk.LOOKME_ERR_UNSUPPORTED            # 8-byte rows
    assert S(lambda: txt(n=0)) == lk.LOOKME_ERR_INVALID
    assert S(lambda: txt(p=None)) == lk.LOOKME_ERR_INVALID
    assert S(lambda: txt(kept=FAKE + 8)) == lk.LOOKME_ERR_INVALID
    assert S(lambda: txt(n_text=0, p=None)) == lk.LOOKME_OK


def test_lookup_select_validates(lib):
    bf = _desc(dtype=lk.LOOKME_BF16, key_dim=512, value_dim=2048, prims_per_scene=1024,
               top_k=8, num_scenes=256)
    h = lk.lookme_create(bf, FAKE, FAKE, FAKE)
    try:
        S = lambda f: _status(f)[0]
        call = lambda n=8, n_keep=2, d_c=2048, p=FAKE, crit=FAKE, kept=FAKE: \
            lk.lookme_lookup_select(h, 1, n, p, p, p, p, n_keep, crit, d_c, kept, 0)
        assert S(lambda: call(n_keep=9)) == lk.LOOKME_ERR_INVALID        # n_keep > n
        assert S(lambda: call(n_keep=-1)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call(d_c=1001)) == lk.LOOKME_ERR_UNSUPPORTED    # 2002-byte rows
        assert S(lambda: call(p=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call(crit=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call(kept=FAKE + 4)) == lk.LOOKME_ERR_INVALID   # misaligned
        assert S(lambda: call(n_keep=0, crit=None, kept=None)) == lk.LOOKME_ERR_WORKSPACE
        assert S(lambda: call()) == lk.LOOKME_ERR_WORKSPACE
        assert S(lambda: call(n=0, n_keep=0, p=None, crit=None, kept=None)) == lk.LOOKME_OK
    finally:
        lk.lookme_destroy(h)


def test_lookup_gate_validates(lib):
    bf = _desc(dtype=lk.LOOKME_BF16, key_dim=512, value_dim=2048, prims_per_scene=1024,
               top_k=8, num_scenes=256)
    h = lk.lookme_create(bf, FAKE, FAKE, FAKE)
    try:
        S = lambda f: _status(f)[0]
        call = lambda n=8, d_c=2048, p=FAKE, wg=FAKE, cnt=FAKE: lk.lookme_lookup_gate(
            h, 1, n, p, p, p, p, p, d_c, wg, p, cnt, 0)
        assert S(lambda: call(d_c=1001)) == lk.LOOKME_ERR_UNSUPPORTED
        assert S(lambda: call(wg=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call(cnt=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call(p=None)) == lk.LOOKME_ERR_INVALID
        assert S(lambda: call()) == lk.LOOKME_ERR_WORKSPACE
        assert S(lambda: call(n=0, p=None, wg=None, cnt=None)) == lk.LOOKME_OK
    finally:
        lk.lookme_destroy(h)


def test_scene_keys_validates(lib):
    """lookme_scene_keys (Eq. 4) rejects bad descriptors and pointers before
    any launch (no GPU needed)."""
    S = lambda f: _status(f)[0]
    sk = lambda p=FAKE, o=FAKE, **kw: lk.lookme_scene_keys(_desc(**kw), p, o, 0)
    assert S(lambda: lk.lookme_scene_keys(None, FAKE, FAKE, 0)) == lk.LOOKME_ERR_INVALID
    assert S(lambda: sk(dtype=7)) == lk.LOOKME_ERR_INVALID
    assert S(lambda: sk(num_scenes=0)) == lk.LOOKME_ERR_INVALID
    assert S(lambda: sk(prims_per_scene=0)) == lk.LOOKME_ERR_INVALID
    assert S(lambda: sk(key_dim=0)) == lk.LOOKME_ERR_INVALID
    assert S(lambda: sk(key_dim=6, dtype=lk.LOOKME_BF16)) == lk.LOOKME_ERR_UNSUPPORTED  # 12 B
    assert S(lambda: sk(num_scenes=1 << 16, prims_per_scene=1 << 16)) == \
        lk.LOOKME_ERR_UNSUPPORTED
    assert S(lambda: sk(p=None)) == lk.LOOKME_ERR_INVALID
    assert S(lambda: sk(o=FAKE + 4)) == lk.LOOKME_ERR_INVALID


def test_index_errors_validates(lib):
    """lookme_index_errors needs somewhere to write the count."""
    assert lib.lookme_index_errors(None, None) == lk.LOOKME_ERR_INVALID
