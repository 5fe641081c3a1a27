"""The C ABI library loads, exports every function include/rgcn.h declares, and rejects
invalid arguments on the host before touching the GPU (no GPU needed)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2406_06022_amd import rgcn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(rgcn.LIB_PATH):
        from paper_2406_06022_amd import build
        build.build()
    return rgcn.load_library()


def _declared():
    text = open(os.path.join(ROOT, "include", "rgcn.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rgcn_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert set(names) == set(rgcn.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n
    assert "gfx950" in rgcn.rgcn_version()


class _FakeBlock:
    """A structurally valid block whose device pointers are fake: only host validation may
    run on it."""

    def __init__(self, n_src, n_dst, rels, grad=0):
        self.n_src_a = (ctypes.c_int64 * len(n_src))(*n_src)
        self.n_dst_a = (ctypes.c_int64 * len(n_dst))(*n_dst)
        self.rels_a = (rgcn._Relation * max(len(rels), 1))()
        for i, (s, t, nnz) in enumerate(rels):
            self.rels_a[i] = rgcn._Relation(s, t, nnz, 0x10000, 0x20000)
        self.c = rgcn._Block(len(n_src), len(rels), self.n_src_a, self.n_dst_a, self.rels_a, grad)


def _params(d_in=8, d_out=8, dtype=rgcn.RGCN_F32, nrel=1, ntypes=1):
    w_rel = (ctypes.c_void_p * max(nrel, 1))(*([0x40000] * nrel))
    w_self = (ctypes.c_void_p * ntypes)(*([0x40000] * ntypes))
    p = rgcn._Params(dtype, d_in, d_out, w_rel, w_self, None)
    p._keep = (w_rel, w_self)
    return p


def _ws_size(lib, blk, p):
    out = ctypes.c_size_t(0)
    st = lib.rgcn_block_workspace_size(ctypes.byref(blk.c), ctypes.byref(p), ctypes.byref(out))
    return st, out.value


def test_workspace_size_and_host_validation(lib):
    good = _FakeBlock([20], [10], [(0, 0, 30)])
    st, n = _ws_size(lib, good, _params())
    assert st == 0 and n > 0
    cases = [
        (_FakeBlock([20], [10], [(0, 0, 30)], grad=0b10), _params(), 1),   # grad bit past types
        (_FakeBlock([5], [10], [(0, 0, 30)]), _params(), 2),               # n_dst > n_src
        (_FakeBlock([20], [10], [(0, 3, 30)]), _params(), 1),              # bad dst type
        (_FakeBlock([20], [10], [(0, 0, -1)]), _params(), 7),              # negative nnz
        (good, _params(dtype=5), 3),                                       # dtype
        (good, _params(d_in=6), 7),                                        # d_in not multiple of 4
        (good, _params(d_in=8, d_out=12, dtype=rgcn.RGCN_BF16), 7),        # bf16 needs 8
        (good, _params(d_in=0), 1),
    ]
    for blk, p, want in cases:
        st, _ = _ws_size(lib, blk, p)
        assert st == want, (st, want, lib.rgcn_last_error())
        assert lib.rgcn_last_error()


def test_null_and_small_workspace_rejected(lib):
    blk = _FakeBlock([20], [10], [(0, 0, 30)])
    p = _params()
    st = lib.rgcn_block_plan(ctypes.byref(blk.c), ctypes.byref(p), None, 0, 0, None)
    assert st == 1
    st = lib.rgcn_block_plan(ctypes.byref(blk.c), ctypes.byref(p), 0x100000, 16, 0, None)
    assert st == 6
    st = lib.rgcn_block_plan(ctypes.byref(blk.c), ctypes.byref(p), 0x100008, 1 << 40, 0, None)
    assert st == 1  # misaligned
    _, n = _ws_size(lib, blk, p)
    # forward: NULL inputs, then NULL outputs
    st = lib.rgcn_block_forward(ctypes.byref(blk.c), None, ctypes.byref(p), None, None,
                                0x100000, n, 0, None)
    assert st == 1
    inp = (rgcn._Input * 1)(rgcn._Input(0x40000, None, 20, 8))
    st = lib.rgcn_block_forward(ctypes.byref(blk.c), inp, ctypes.byref(p), None, None, 0x100000,
                                n, 0, None)
    assert st == 1
    bad_ld = (rgcn._Input * 1)(rgcn._Input(0x40000, None, 20, 6))
    y = (ctypes.c_void_p * 1)(0x80000)
    st = lib.rgcn_block_forward(ctypes.byref(blk.c), bad_ld, ctypes.byref(p), y, None, 0x100000,
                                n, 0, None)
    assert st == 2
    # sign-mask outputs: only with RGCN_FUSE_RELU, and 8-byte aligned
    mask = (ctypes.c_void_p * 1)(0xA0000)
    st = lib.rgcn_block_forward(ctypes.byref(blk.c), inp, ctypes.byref(p), y, mask, 0x100000, n,
                                0, None)
    assert st == 1 and "RGCN_FUSE_RELU" in lib.rgcn_last_error().decode()
    st = lib.rgcn_block_transform(ctypes.byref(blk.c), ctypes.byref(p), y, mask, 0x100000, n, 0,
                                  None)
    assert st == 1 and "RGCN_FUSE_RELU" in lib.rgcn_last_error().decode()
    odd = (ctypes.c_void_p * 1)(0xA0004)
    st = lib.rgcn_block_forward(ctypes.byref(blk.c), inp, ctypes.byref(p), y, odd, 0x100000, n,
                                rgcn.RGCN_FUSE_RELU, None)
    assert st == 1 and "8-byte" in lib.rgcn_last_error().decode()
    # backward: a gradient of a type that is not in grad_src_types
    dy = (ctypes.c_void_p * 1)(0x80000)
    dh = (ctypes.c_void_p * 1)(0x90000)
    st = lib.rgcn_block_backward(ctypes.byref(blk.c), inp, ctypes.byref(p), dy, None, None, None,
                                 dh, None, 0x100000, n, 0, None)
    assert st == 1
    assert "grad_src_types" in lib.rgcn_last_error().decode()


def test_sparse_adagrad_host_validation(lib):
    """The standalone step rejects bad sizes, dtypes, flags and pointers before any launch;
    an empty row list is a no-op."""
    f = lib.rgcn_sparse_adagrad
    A, B, C, D = 0x100000, 0x200000, 0x300000, 0x400000
    good = dict(n=4, rows=A, num_rows=10, d=8, grad=B, state=C, table=D, ld=8,
                dtype=rgcn.RGCN_F32, lr=0.1, eps=1e-8, flags=0)

    def call(**kw):
        a = dict(good, **kw)
        return f(a["n"], a["rows"], a["num_rows"], a["d"], a["grad"], a["state"], a["table"],
                 a["ld"], a["dtype"], a["lr"], a["eps"], a["flags"], None)

    assert call(n=0) == 0
    cases = [(dict(dtype=5), 3), (dict(d=6), 2), (dict(ld=4), 2), (dict(dtype=rgcn.RGCN_BF16, d=4, ld=8), 2),
             (dict(dtype=rgcn.RGCN_BF16, d=8, ld=12), 2), (dict(n=-1), 2), (dict(flags=0x1), 1),
             (dict(lr=float("nan")), 1), (dict(rows=None), 1), (dict(table=None), 1),
             (dict(rows=A + 4), 1), (dict(state=C + 8), 1)]
    for kw, want in cases:
        assert call(**kw) == want, (kw, lib.rgcn_last_error())
        assert lib.rgcn_last_error()


def test_fused_adagrad_host_validation(lib):
    """The fused step needs RGCN_IDS_UNIQUE, a table equal to the input base, the type's
    gradient bit, no ReLU-input flag and no demb for the same type."""
    blk = _FakeBlock([20], [10], [(0, 0, 30)], grad=1)
    p = _params()
    _, n = _ws_size(lib, blk, p)
    inp = (rgcn._Input * 1)(rgcn._Input(0x40000, None, 20, 8))
    f = lib.rgcn_block_backward_sparse_adagrad

    def call(state=0x50000, table=0x40000, flags=rgcn.RGCN_IDS_UNIQUE, demb=None, block=blk,
             opt=True, eps=1e-8):
        st = (ctypes.c_void_p * 1)(state)
        tb = (ctypes.c_void_p * 1)(table)
        o = rgcn._Adagrad(0.1, eps, st, tb)
        de = None if demb is None else (ctypes.c_void_p * 1)(demb)
        return f(ctypes.byref(block.c), inp, ctypes.byref(p), None, de,
                 ctypes.byref(o) if opt else None, 0x100000, n, flags, None)

    cases = [(dict(opt=False), "opt is NULL"), (dict(flags=0), "RGCN_IDS_UNIQUE"),
             (dict(flags=rgcn.RGCN_IDS_UNIQUE | rgcn.RGCN_INPUT_RELU), "RGCN_INPUT_RELU"),
             (dict(table=0x60000), "writable base"), (dict(demb=0x70000), "both demb"),
             (dict(state=0x50004), "aligned"), (dict(eps=float("nan")), "NaN"),
             (dict(block=_FakeBlock([20], [10], [(0, 0, 30)], grad=0)), "grad_src_types")]
    for kw, msg in cases:
        assert call(**kw) == 1, kw
        assert msg in lib.rgcn_last_error().decode(), (kw, lib.rgcn_last_error())


def test_sampling_host_validation(lib):
    """Sampling rejects bad graphs, fanouts and arrays before any launch."""
    nodes = (ctypes.c_int64 * 2)(100, 50)
    rels = (rgcn._GraphRel * 2)(rgcn._GraphRel(0, 1, 0x10000, 0x20000),
                                rgcn._GraphRel(1, 0, 0x30000, 0x40000))
    g = rgcn._Graph(2, 2, nodes, rels)
    nd = (ctypes.c_int64 * 2)(10, 5)
    out = ctypes.c_size_t(0)
    assert lib.rgcn_sample_workspace_size(ctypes.byref(g), nd, 8, ctypes.byref(out)) == 0
    assert out.value > 0
    for fo in (0, 65):
        assert lib.rgcn_sample_workspace_size(ctypes.byref(g), nd, fo, ctypes.byref(out)) == 7
    bad = rgcn._Graph(2, 2, nodes, (rgcn._GraphRel * 2)(rgcn._GraphRel(0, 2, 0x10000, 0x20000),
                                                        rgcn._GraphRel(1, 0, 0x30000, 0x40000)))
    assert lib.rgcn_sample_workspace_size(ctypes.byref(bad), nd, 8, ctypes.byref(out)) == 1
    neg = (ctypes.c_int64 * 2)(-1, 5)
    assert lib.rgcn_sample_workspace_size(ctypes.byref(g), neg, 8, ctypes.byref(out)) == 2
    huge = (ctypes.c_int64 * 2)(1 << 27, 1 << 27)
    assert lib.rgcn_sample_workspace_size(ctypes.byref(g), huge, 64, ctypes.byref(out)) == 7
    ws = out.value
    lib.rgcn_sample_workspace_size(ctypes.byref(g), nd, 8, ctypes.byref(out))
    p2 = (ctypes.c_void_p * 2)(0x50000, 0x60000)
    p3 = (ctypes.c_void_p * 2)(0x70000, 0x80000)
    f = lib.rgcn_sample_block
    # workspace too small, misaligned workspace, NULL counts, NULL destination ids
    assert f(ctypes.byref(g), p2, nd, 8, 1, 0, p3, p3, p2, None, 0x90000, 0x100000, 16, 0, None) == 6
    assert f(ctypes.byref(g), p2, nd, 8, 1, 0, p3, p3, p2, None, 0x90000, 0x100010, out.value, 0,
             None) == 1
    assert f(ctypes.byref(g), p2, nd, 8, 1, 0, p3, p3, p2, None, None, 0x100000, out.value, 0,
             None) == 1
    nul = (ctypes.c_void_p * 2)(None, 0x60000)
    assert f(ctypes.byref(g), nul, nd, 8, 1, 0, p3, p3, p2, None, 0x90000, 0x100000, out.value, 0,
             None) == 1
    assert "dst_ids[0]" in lib.rgcn_last_error().decode()
    odd = (ctypes.c_void_p * 2)(0x90004, None)     # per-edge source ids misaligned
    assert f(ctypes.byref(g), p2, nd, 8, 1, 0, p3, p3, p2, odd, 0x90000, 0x100000, out.value, 0,
             None) == 1
    assert "out_src_rows[0]" in lib.rgcn_last_error().decode()
    assert f(ctypes.byref(g), p2, nd, 8, 1, 0, p3, p3, p2, None, 0x90000, 0x100000, out.value, 0x4,
             None) == 1


def test_link_prediction_host_validation(lib):
    """The decoder rejects bad widths, modes, strides and pointers before any launch."""
    def batch(**kw):
        a = dict(dtype=rgcn.RGCN_BF16, d=64, n_rows=100, ld=64, emb=0x100000, rel=0x200000,
                 neg_mode=0, loss=2, batch=8, src=0x300000, dst=0x400000, k=4, neg=0x500000,
                 pos_weight=None)
        a.update(kw)
        return rgcn._LpBatch(a["dtype"], a["d"], a["n_rows"], a["ld"], a["emb"], a["rel"],
                             a["neg_mode"], a["loss"], a["batch"], a["src"], a["dst"], a["k"],
                             a["neg"], a["pos_weight"])
    out = ctypes.c_size_t(0)
    assert lib.rgcn_lp_workspace_size(ctypes.byref(batch()), ctypes.byref(out)) == 0
    cases = [(dict(dtype=9), 3), (dict(d=60), 7), (dict(d=4096), 7), (dict(ld=32), 2),
             (dict(neg_mode=3), 1), (dict(loss=5), 1), (dict(k=0), 2), (dict(batch=-1), 2),
             (dict(emb=0x100008), 1), (dict(neg=None), 1), (dict(loss=1), 1),
             (dict(neg_mode=2, batch=50000), 7)]
    for kw, want in cases:
        # pointer checks run in the workspace query too
        got = lib.rgcn_lp_workspace_size(ctypes.byref(batch(**kw)), ctypes.byref(out))
        assert got == want, (kw, got, lib.rgcn_last_error())
    # in-batch needs no negative array
    assert lib.rgcn_lp_workspace_size(ctypes.byref(batch(neg_mode=2, neg=None)),
                                      ctypes.byref(out)) == 0
    b = batch()
    lib.rgcn_lp_workspace_size(ctypes.byref(b), ctypes.byref(out))
    f = lib.rgcn_lp_loss
    assert f(ctypes.byref(b), None, None, None, None, None, 0x600000, out.value, 0, None) == 1
    assert f(ctypes.byref(b), 0x700000, None, None, None, None, 0x600000, 16, 0, None) == 6
    assert f(ctypes.byref(b), 0x700000, None, None, None, None, 0x600000, out.value, 0x8,
             None) == 1
    nodot = batch(rel=None)
    lib.rgcn_lp_workspace_size(ctypes.byref(nodot), ctypes.byref(out))
    assert f(ctypes.byref(nodot), 0x700000, None, None, None, 0x800000, 0x600000, out.value, 0,
             None) == 1
    assert "d_rel" in lib.rgcn_last_error().decode()
    g = lib.rgcn_lp_negatives
    assert g(2, 10, 100, 1, 0x900000, None) == 1
    assert g(0, 10, 0, 1, 0x900000, None) == 2
    assert g(0, 0, 10, 1, None, None) == 0


def test_binding_constants_match_header():
    """Every numeric #define of the C header that the binding also names has the same value
    there (flags, limits, workspace sizes)."""
    import os
    import re
    from paper_2406_06022_amd import rgcn
    hdr = open(os.path.join(os.path.dirname(__file__), "..", "include", "rgcn.h")).read()
    seen = 0
    for name, val in re.findall(r"^#define\s+(RGCN_\w+)\s+\(?(0x[0-9a-fA-F]+|\d+)u?\)?", hdr, re.M):
        if hasattr(rgcn, name):
            assert getattr(rgcn, name) == int(val, 0), name
            seen += 1
    assert seen >= 8 and rgcn.RGCN_PLAN_FORWARD != rgcn.RGCN_PLAN_BACKWARD
