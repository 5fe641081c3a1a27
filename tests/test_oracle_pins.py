"""Pins of the CPU oracle against things other than itself (no GPU needed).

* a block worked by hand in exact rationals (tests/golden/hand_worked_block.json);
* dense brute force: the layer written as dense normalised-adjacency products and
  evaluated with numpy matmul, on tiny random blocks (duplicates, zero degrees, empty
  relations, several node types);
* the single-relation case reduces to the right-normalised GCN with a self-loop,
  evaluated with scipy.sparse;
* invariants: mean of a constant feature is that constant (exactly, for dyadic values);
  zero-degree destinations get the self-loop (+bias) only; edge order inside a segment
  and consistent source relabelling do not matter;
* calculus: central finite differences (exact up to rounding, the layer is affine in
  every single parameter) for every weight, bias, input and embedding entry; the adjoint
  identity <dY, F(dH)> = <B(dY), dH>; the ReLU-input mask against differences taken
  through max(0, .);
* the integer plan: CSC against scipy's CSR->CSC conversion and the ordering rule
  against Python's stable sort; an integer "index probe" that exposes a wrong gathered row.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.sparse as sp

from paper_2406_06022_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _frac(x):
    return float(Fraction(str(x)))


def _arr(x):
    return np.vectorize(_frac, otypes=[np.float64])(np.array(x, dtype=object))


class _B:
    def __init__(self, n_src, n_dst, rels):
        self.n_src, self.n_dst, self.rels = n_src, n_dst, rels


class _R:
    def __init__(self, s, t, indptr, indices):
        self.src_type, self.dst_type = s, t
        self.indptr = np.asarray(indptr, dtype=np.int32)
        self.indices = np.asarray(indices, dtype=np.int32)


def _rand_inputs(rng, blk, d_in, d_out, bias=True):
    T, R = len(blk.n_src), len(blk.rels)
    h = [rng.standard_normal((blk.n_src[t], d_in)) for t in range(T)]
    w_rel = [rng.standard_normal((d_in, d_out)) for _ in range(R)]
    w_self = [rng.standard_normal((d_in, d_out)) for _ in range(T)]
    b = [rng.standard_normal(d_out) for _ in range(T)] if bias else None
    dy = [rng.standard_normal((blk.n_dst[t], d_out)) for t in range(T)]
    return h, w_rel, w_self, b, dy


def _dense_norm_adj(rel, n_dst, n_src):
    """Dense A_hat[i, j] = (#edges i<-j) / deg(i), built edge by edge."""
    a = np.zeros((n_dst, n_src))
    for i in range(n_dst):
        lo, hi = int(rel.indptr[i]), int(rel.indptr[i + 1])
        for k in range(lo, hi):
            a[i, int(rel.indices[k])] += 1.0 / (hi - lo)
    return a


def _dense_forward(blk, h, w_rel, w_self, b):
    ys = []
    for t in range(len(blk.n_src)):
        nd = blk.n_dst[t]
        if nd == 0:
            ys.append(None)
            continue
        y = h[t][:nd] @ w_self[t] + (b[t] if b is not None else 0.0)
        for r, rel in enumerate(blk.rels):
            if rel.dst_type == t:
                y = y + _dense_norm_adj(rel, nd, blk.n_src[rel.src_type]) @ h[rel.src_type] @ w_rel[r]
        ys.append(y)
    return ys


def _dense_backward(blk, h, w_rel, w_self, dy):
    T = len(blk.n_src)
    out = {"dw_rel": [], "dw_self": [], "dbias": [], "dh_src": []}
    adj = [_dense_norm_adj(rel, blk.n_dst[rel.dst_type], blk.n_src[rel.src_type])
           for rel in blk.rels]
    for t in range(T):
        nd = blk.n_dst[t]
        out["dbias"].append(dy[t].sum(axis=0))
        out["dw_self"].append(h[t][:nd].T @ dy[t])
    for r, rel in enumerate(blk.rels):
        out["dw_rel"].append((adj[r] @ h[rel.src_type]).T @ dy[rel.dst_type])
    for s in range(T):
        g = np.zeros_like(h[s])
        g[: blk.n_dst[s]] += dy[s] @ w_self[s].T
        for r, rel in enumerate(blk.rels):
            if rel.src_type == s:
                g += adj[r].T @ (dy[rel.dst_type] @ w_rel[r].T)
        out["dh_src"].append(g)
    return out


def _relerr(a, b):
    a, b = np.asarray(a, dtype=np.float64), np.asarray(b, dtype=np.float64)
    if b.size == 0:
        return 0.0
    scale = max(np.abs(b).max(), np.sqrt(np.mean(b * b)), 1e-300)
    return float(np.abs(a - b).max() / scale)


def _tiny_blocks():
    rng = np.random.default_rng(7)
    yield "one-type", synth.random_block(rng, [9], [5], [(0, 0), (0, 0)], 4)
    yield "three-types", synth.random_block(rng, [7, 6, 8], [3, 4, 0],
                                            [(0, 1), (1, 0), (2, 0), (2, 1), (0, 0)], 5)
    yield "empty-relation", synth.random_block(rng, [6, 5], [4, 2], [(0, 1), (1, 0)], 0)
    yield "all-zero-type", _B([4, 3], [2, 3], [_R(0, 1, [0, 0, 0, 0], [])])
    yield "no-dst", synth.random_block(rng, [5, 4], [0, 0], [(0, 1), (1, 0)], 3)


# --------------------------------------------------------------------------------------
def test_hand_worked_block(orc):
    g = json.load(open(os.path.join(GOLDEN, "hand_worked_block.json")))
    blk = _B(g["n_src"], g["n_dst"], [_R(r["src_type"], r["dst_type"], r["indptr"],
                                         r["indices"]) for r in g["rels"]])
    h = [_arr(g["h"])]
    w_rel = [_arr(w) for w in g["w_rel"]]
    w_self = [_arr(g["w_self"])]
    bias = [_arr(g["bias"])]
    y = orc.block_forward(blk, h, w_rel, w_self, bias)
    np.testing.assert_allclose(y[0], _arr(g["y"]), rtol=0, atol=1e-14)
    gr = orc.block_backward(blk, h, w_rel, w_self, [_arr(g["dy"])])
    np.testing.assert_allclose(gr["dbias"][0], _arr(g["dbias"]), rtol=0, atol=1e-14)
    np.testing.assert_allclose(gr["dw_self"][0], _arr(g["dw_self"]), rtol=0, atol=1e-14)
    for r in range(2):
        np.testing.assert_allclose(gr["dw_rel"][r], _arr(g["dw_rel"][r]), rtol=0, atol=1e-14)
    np.testing.assert_allclose(gr["dh_src"][0], _arr(g["dh"]), rtol=0, atol=1e-14)
    for r, c in enumerate(g["csc"]):
        cip, cd, ce = orc.csc(3, blk.rels[r].indptr, blk.rels[r].indices)
        assert cip.tolist() == c["indptr"] and cd.tolist() == c["dst"] and ce.tolist() == c["eid"]
    demb = np.zeros((g["emb_rows"], 2))
    orc.scatter_add(np.array(g["emb_ids"]), gr["dh_src"][0], demb)
    for row in range(g["emb_rows"]):
        want = _arr(g["demb_nonzero"][str(row)]) if str(row) in g["demb_nonzero"] else np.zeros(2)
        np.testing.assert_allclose(demb[row], want, rtol=0, atol=1e-14)


@pytest.mark.parametrize("name,blk", list(_tiny_blocks()))
def test_dense_brute_force(orc, name, blk):
    rng = np.random.default_rng(11)
    for d_in, d_out in ((3, 4), (5, 2)):
        h, w_rel, w_self, b, dy = _rand_inputs(rng, blk, d_in, d_out)
        ys = orc.block_forward(blk, h, w_rel, w_self, b)
        want = _dense_forward(blk, h, w_rel, w_self, b)
        for t, (y, w) in enumerate(zip(ys, want)):
            assert (y is None) == (w is None)
            if y is not None:
                assert _relerr(y, w) < 1e-12, (name, t)
        # ReLU epilogue is max(0, .) of the same values
        yr = orc.block_forward(blk, h, w_rel, w_self, b, relu=True)
        for y, w in zip(yr, want):
            if y is not None:
                assert _relerr(y, np.maximum(w, 0.0)) < 1e-12
        got = orc.block_backward(blk, h, w_rel, w_self, dy)
        ref = _dense_backward(blk, h, w_rel, w_self, dy)
        for key in ("dw_rel", "dw_self", "dbias", "dh_src"):
            for a, bref in zip(got[key], ref[key]):
                assert _relerr(a, bref) < 1e-12, (name, key)


def test_single_relation_is_normalised_gcn(orc):
    rng = np.random.default_rng(3)
    n_src, n_dst, d_in, d_out = 40, 25, 6, 5
    blk = synth.random_block(rng, [n_src], [n_dst], [(0, 0)], 7, zero_frac=0.0)
    rel = blk.rels[0]
    a = sp.csr_matrix((np.ones(rel.nnz), rel.indices, rel.indptr), shape=(n_dst, n_src))
    deg = np.asarray(a.sum(axis=1)).ravel()
    inv = np.divide(1.0, deg, out=np.zeros_like(deg), where=deg > 0)  # zero-degree rows: 0
    a_norm = sp.diags(inv) @ a
    h = rng.standard_normal((n_src, d_in))
    w, ws = rng.standard_normal((d_in, d_out)), rng.standard_normal((d_in, d_out))
    want = a_norm @ h @ w + h[:n_dst] @ ws
    y = orc.block_forward(blk, [h], [w], [ws])[0]
    assert _relerr(y, want) < 1e-12


def test_constant_feature_mean_is_exact(orc):
    rng = np.random.default_rng(5)
    blk = synth.random_block(rng, [50], [30], [(0, 0)], 13)
    rel = blk.rels[0]
    deg = orc.degrees(rel.indptr)
    for c in (0.5, -2.0, 1.0, 0.375):
        h = np.full((50, 4), c)
        m = orc.mean_aggregate(rel.indptr, rel.indices, h)
        assert np.all(m[deg > 0] == c)
        assert np.all(m[deg == 0] == 0.0)


def test_zero_degree_rows_get_self_loop_only(orc):
    rng = np.random.default_rng(9)
    blk = synth.random_block(rng, [12, 10], [8, 6], [(0, 0), (1, 0), (0, 1)], 4, zero_frac=0.5)
    h, w_rel, w_self, b, _ = _rand_inputs(rng, blk, 4, 3)
    ys = orc.block_forward(blk, h, w_rel, w_self, b)
    self_only = _B(blk.n_src, blk.n_dst, [])
    ys0 = orc.block_forward(self_only, h, [], w_self, b)
    for t in range(2):
        into = [rel for rel in blk.rels if rel.dst_type == t]
        zero_all = np.ones(blk.n_dst[t], dtype=bool)
        for rel in into:
            zero_all &= orc.degrees(rel.indptr) == 0
        assert zero_all.any()
        assert np.array_equal(ys[t][zero_all], ys0[t][zero_all])
        np.testing.assert_allclose(ys0[t], h[t][: blk.n_dst[t]] @ w_self[t] + b[t], rtol=1e-13)
    # a relation whose rows all have degree zero contributes nothing
    rel = blk.rels[0]
    empty = _R(rel.src_type, rel.dst_type, np.zeros_like(rel.indptr), [])
    with_empty = _B(blk.n_src, blk.n_dst, [empty] + list(blk.rels[1:]))
    without = _B(blk.n_src, blk.n_dst, list(blk.rels[1:]))
    a = orc.block_forward(with_empty, h, w_rel, w_self, b)
    c = orc.block_forward(without, h, w_rel[1:], w_self, b)
    for t in range(2):
        assert np.array_equal(a[t], c[t])


def _loss(orc, blk, h, w_rel, w_self, b, g):
    ys = orc.block_forward(blk, h, w_rel, w_self, b)
    return sum(float((y * gg).sum()) for y, gg in zip(ys, g) if y is not None)


def test_finite_differences_every_entry(orc):
    rng = np.random.default_rng(21)
    blk = synth.random_block(rng, [5, 4], [3, 2], [(0, 0), (1, 0), (0, 1), (0, 1)], 3)
    d_in, d_out = 3, 2
    h, w_rel, w_self, b, dy = _rand_inputs(rng, blk, d_in, d_out)
    got = orc.block_backward(blk, h, w_rel, w_self, dy)
    eps = 0.5  # the loss is affine in each single entry: any step is exact up to rounding

    def fd(arrs, idx):
        a = arrs[idx[0]]
        old = a[idx[1:]]
        a[idx[1:]] = old + eps
        lp = _loss(orc, blk, h, w_rel, w_self, b, dy)
        a[idx[1:]] = old - eps
        lm = _loss(orc, blk, h, w_rel, w_self, b, dy)
        a[idx[1:]] = old
        return (lp - lm) / (2 * eps)

    for name, arrs in (("dw_rel", w_rel), ("dw_self", w_self), ("dbias", b), ("dh_src", h)):
        for p, a in enumerate(arrs):
            for idx in np.ndindex(*a.shape):
                want = fd(arrs, (p,) + idx)
                assert abs(got[name][p][idx] - want) <= 1e-9 * max(1.0, abs(want)), (name, p, idx)


def test_finite_differences_embedding_scatter(orc):
    """Gradient w.r.t. a learnable table read through (possibly repeated) ids."""
    rng = np.random.default_rng(23)
    blk = synth.random_block(rng, [6], [3], [(0, 0), (0, 0)], 3)
    rows, d_in, d_out = 9, 2, 3
    ids = np.array([4, 1, 7, 4, 0, 8])
    table = rng.standard_normal((rows, d_in))
    _, w_rel, w_self, b, dy = _rand_inputs(rng, blk, d_in, d_out)
    got = orc.block_backward(blk, [table[ids]], w_rel, w_self, dy)
    demb = np.zeros((rows, d_in))
    orc.scatter_add(ids, got["dh_src"][0], demb)
    eps = 0.25
    for idx in np.ndindex(rows, d_in):
        old = table[idx]
        table[idx] = old + eps
        lp = _loss(orc, blk, [table[ids]], w_rel, w_self, b, dy)
        table[idx] = old - eps
        lm = _loss(orc, blk, [table[ids]], w_rel, w_self, b, dy)
        table[idx] = old
        want = (lp - lm) / (2 * eps)
        assert abs(demb[idx] - want) <= 1e-9 * max(1.0, abs(want)), idx
    assert np.all(demb[[2, 3, 5, 6]] == 0.0)


def test_relu_input_mask_matches_differences(orc):
    rng = np.random.default_rng(29)
    blk = synth.random_block(rng, [6, 5], [4, 3], [(0, 1), (1, 0), (0, 0)], 3)
    d_in, d_out = 3, 2
    pre, w_rel, w_self, b, dy = _rand_inputs(rng, blk, d_in, d_out)
    for p in pre:  # keep every pre-activation well away from the kink
        p[np.abs(p) < 0.2] += 0.5
    got = orc.block_backward(blk, [np.maximum(p, 0) for p in pre], w_rel, w_self, dy,
                             input_relu=True)
    eps = 0.05
    for t, p in enumerate(pre):
        for idx in np.ndindex(*p.shape):
            old = p[idx]
            p[idx] = old + eps
            lp = _loss(orc, blk, [np.maximum(q, 0) for q in pre], w_rel, w_self, b, dy)
            p[idx] = old - eps
            lm = _loss(orc, blk, [np.maximum(q, 0) for q in pre], w_rel, w_self, b, dy)
            p[idx] = old
            want = (lp - lm) / (2 * eps)
            assert abs(got["dh_src"][t][idx] - want) <= 1e-9 * max(1.0, abs(want))


def test_adjoint_identity(orc):
    rng = np.random.default_rng(31)
    blk = synth.random_block(rng, [30, 20, 25], [10, 12, 0], [(0, 1), (1, 0), (2, 0), (2, 1),
                                                              (0, 0), (1, 1)], 6)
    d_in, d_out = 7, 5
    dh, w_rel, w_self, _, dy = _rand_inputs(rng, blk, d_in, d_out, bias=False)
    ys = orc.block_forward(blk, dh, w_rel, w_self, None)
    lhs = sum(float((y * g).sum()) for y, g in zip(ys, dy) if y is not None)
    back = orc.block_backward(blk, dh, w_rel, w_self, dy)
    rhs = sum(float((a * bb).sum()) for a, bb in zip(back["dh_src"], dh))
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))


def test_permutation_invariance_and_index_probe(orc):
    rng = np.random.default_rng(37)
    n_src, n_dst = 300, 120
    blk = synth.random_block(rng, [n_src], [n_dst], [(0, 0)], 9)
    rel = blk.rels[0]
    ids = rng.permutation(1 << 20)[:n_src].astype(np.int64)
    # integer probe: column c holds byte c of the row's global id, plus one
    probe = np.stack([((ids >> (8 * c)) & 0xFF) + 1 for c in range(3)], axis=1).astype(np.float64)
    m = orc.mean_aggregate(rel.indptr, rel.indices, probe)
    deg = orc.degrees(rel.indptr)
    for i in range(n_dst):
        lo, hi = rel.indptr[i], rel.indptr[i + 1]
        want = sum(probe[rel.indices[k]] for k in range(lo, hi)) if hi > lo else np.zeros(3)
        assert np.array_equal(np.rint(m[i] * max(deg[i], 1)), want)
    # shuffle edges inside every segment: identical integer sums
    perm_idx = rel.indices.copy()
    for i in range(n_dst):
        lo, hi = rel.indptr[i], rel.indptr[i + 1]
        perm_idx[lo:hi] = rng.permutation(perm_idx[lo:hi])
    m2 = orc.mean_aggregate(rel.indptr, perm_idx, probe)
    assert np.array_equal(np.rint(m2 * np.maximum(deg, 1)[:, None]),
                          np.rint(m * np.maximum(deg, 1)[:, None]))
    # consistent relabelling of the non-destination sources
    perm = np.arange(n_src)
    perm[n_dst:] = n_dst + rng.permutation(n_src - n_dst)
    probe2 = np.empty_like(probe)
    probe2[perm] = probe
    m3 = orc.mean_aggregate(rel.indptr, perm[rel.indices], probe2)
    assert np.array_equal(m3, m)


def test_csc_against_scipy(orc):
    rng = np.random.default_rng(41)
    for (ns, nd, md) in ((50, 40, 6), (7, 30, 9), (300, 1, 40), (1, 5, 3)):
        blk = synth.random_block(rng, [ns], [nd], [(0, 0)], md)
        rel = blk.rels[0]
        nnz = rel.nnz
        cip, cd, ce = orc.csc(ns, rel.indptr, rel.indices)
        eid = np.arange(nnz)
        a = sp.csr_matrix((eid + 1, rel.indices, rel.indptr), shape=(nd, ns))
        c = a.tocsc()  # keeps duplicates, rows ascending inside a column
        assert np.array_equal(cip, c.indptr)
        assert np.array_equal(ce, c.data - 1)
        assert np.array_equal(cd, c.indices)
        dst_of = np.repeat(np.arange(nd), np.diff(rel.indptr))
        assert np.array_equal(cd, dst_of[ce])


def test_invalid_blocks_are_rejected(orc):
    good = _B([4], [2], [_R(0, 0, [0, 1, 3], [0, 3, 1])])
    assert orc.check_block(good)
    assert not orc.check_block(_B([4], [2], [_R(0, 0, [0, 1, 3], [0, 4, 1])]))  # index >= n_src
    assert not orc.check_block(_B([4], [2], [_R(0, 0, [0, 2, 1], [0, 1, 1])]))  # decreasing
    assert not orc.check_block(_B([4], [2], [_R(0, 0, [1, 2, 3], [0, 1, 1])]))  # indptr[0] != 0
    assert not orc.check_block(_B([1], [2], []))                                  # n_dst > n_src


def test_relu_epilogue_exact_small_values(orc):
    """max(0, .) on exactly representable outputs straddling zero."""
    vals = np.array([-2.0 ** -12, 0.0, 2.0 ** -12, 1.0, -1.0, -2.0 ** -30])
    d = vals.shape[0]
    blk = _B([1], [1], [])
    h = [np.ones((1, 1))]
    w_self = [vals.reshape(1, d)]
    y = orc.block_forward(blk, h, [], w_self, None, relu=True)[0]
    assert y.ravel().tolist() == [0.0, 0.0, 2.0 ** -12, 1.0, 0.0, 0.0]


def test_sub_block_preserves_kept_rows(orc):
    """Outputs of kept rows, and input gradients of sources referenced only by kept rows,
    equal those of the whole block."""
    rng = np.random.default_rng(51)
    blk = synth.random_block(rng, [60, 45], [30, 20], [(0, 1), (1, 0), (0, 0)], 5)
    h, w_rel, w_self, b, dy = _rand_inputs(rng, blk, 3, 4)
    keep = [np.array([2, 5, 11, 29]), np.array([0, 7])]
    sub, src_map = orc.sub_block(blk, keep)
    y = orc.block_forward(blk, h, w_rel, w_self, b)
    ys = orc.block_forward(sub, [h[t][src_map[t]] for t in range(2)], w_rel, w_self, b)
    for t in range(2):
        np.testing.assert_allclose(ys[t], y[t][keep[t]], rtol=1e-13, atol=1e-13)
    # gradient: zero dY outside the kept rows on the full block
    dy_full = [np.zeros_like(x) for x in dy]
    for t in range(2):
        dy_full[t][keep[t]] = dy[t][keep[t]]
    g = orc.block_backward(blk, h, w_rel, w_self, dy_full)
    gs = orc.block_backward(sub, [h[t][src_map[t]] for t in range(2)], w_rel, w_self,
                            [dy[t][keep[t]] for t in range(2)])
    for t in range(2):
        np.testing.assert_allclose(gs["dh_src"][t], g["dh_src"][t][src_map[t]], rtol=1e-12,
                                   atol=1e-12)
    for r in range(3):
        np.testing.assert_allclose(gs["dw_rel"][r], g["dw_rel"][r], rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- sparse Adagrad step
def test_sparse_adagrad_matches_torch_adagrad_when_every_row_is_touched(orc):
    """With every row listed, the step is torch.optim.Adagrad's dense rule (no decay, zero
    initial accumulator): state += g^2, w -= lr g / (sqrt(state) + eps); three steps."""
    import torch
    rng = np.random.default_rng(3)
    w0 = rng.standard_normal((7, 5))
    lr, eps = 0.05, 1e-10
    w = torch.tensor(w0.copy(), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adagrad([w], lr=lr, eps=eps)
    table, state = w0.copy(), np.zeros_like(w0)
    for step in range(3):
        g = rng.standard_normal(w0.shape)
        w.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        orc.sparse_adagrad(np.arange(7), g, state, table, lr, eps)
        np.testing.assert_allclose(table, w.detach().numpy(), rtol=1e-14, atol=1e-15)
        np.testing.assert_allclose(state, opt.state[w]["sum"].numpy(), rtol=1e-14, atol=0)


def test_sparse_adagrad_first_step_closed_form_and_untouched_rows(orc):
    """From a zero state the first step is w - lr g / (|g| + eps) = w - lr sign(g) (up to
    eps); rows not listed keep their bits; a repeated row is rejected."""
    rng = np.random.default_rng(5)
    table0 = rng.standard_normal((10, 4))
    g = np.zeros_like(table0)
    rows = np.array([7, 2, 5])
    g[rows] = np.array([[0.5, -2.0, 4.0, -0.25], [1.0, 1.0, -1.0, 8.0], [-3.0, 0.125, 2.0, -1.0]])
    table, state = table0.copy(), np.zeros_like(table0)
    orc.sparse_adagrad(rows, g, state, table, 0.1, 0.0)
    np.testing.assert_array_equal(state[rows], g[rows] ** 2)
    np.testing.assert_allclose(table[rows], table0[rows] - 0.1 * np.sign(g[rows]), rtol=0,
                               atol=1e-15)
    others = np.setdiff1d(np.arange(10), rows)
    assert np.array_equal(table[others], table0[others]) and not state[others].any()
    with pytest.raises(ValueError):
        orc.sparse_adagrad(np.array([1, 1]), g, state, table, 0.1, 0.0)


def test_sparse_adagrad_on_scattered_gradient_of_a_block(orc):
    """The fused form (update each touched row from its own dH row) equals the two-pass form
    (scatter-add dH into a zeroed table-shaped gradient, then step the listed rows) when the
    block's source ids are distinct."""
    rng = np.random.default_rng(8)
    blk = synth.random_block(rng, [40, 30], [12, 9], [(0, 1), (1, 0), (0, 0)], 6)
    d_in, d_out = 4, 3
    h = [rng.standard_normal((n, d_in)) for n in blk.n_src]
    w_rel = [rng.standard_normal((d_in, d_out)) for _ in blk.rels]
    w_self = [rng.standard_normal((d_in, d_out)) for _ in blk.n_src]
    dy = [rng.standard_normal((n, d_out)) for n in blk.n_dst]
    g = orc.block_backward(blk, h, w_rel, w_self, dy)
    ids = rng.permutation(100)[: blk.n_src[0]]
    table0, state0 = rng.standard_normal((100, d_in)), rng.random((100, d_in))
    dE = np.zeros((100, d_in))
    orc.scatter_add(ids, g["dh_src"][0], dE)
    t2, s2 = table0.copy(), state0.copy()
    orc.sparse_adagrad(ids, dE, s2, t2, 0.02, 1e-8)
    for j, e in enumerate(ids):   # per touched row, straight from dH
        s = state0[e] + g["dh_src"][0][j] ** 2
        np.testing.assert_allclose(s2[e], s, rtol=1e-15)
        np.testing.assert_allclose(t2[e], table0[e] - 0.02 * g["dh_src"][0][j] / (np.sqrt(s) + 1e-8),
                                   rtol=1e-15)


def test_results_do_not_depend_on_the_thread_count(orc):
    """The oracle's parallel loops give every output element to one thread, which adds its
    terms in the written order: forward and backward are bit-identical on 1 and 5 threads."""
    rng = np.random.default_rng(77)
    blk = synth.random_block(rng, [300, 200], [120, 80], [(0, 1), (1, 0), (0, 0), (1, 1)], 9)
    h, w_rel, w_self, b, dy = _rand_inputs(rng, blk, 6, 5)
    before = orc.get_threads()
    runs = []
    try:
        for n in (1, 5):
            orc.set_threads(n)
            y = orc.block_forward(blk, h, w_rel, w_self, b)
            g = orc.block_backward(blk, h, w_rel, w_self, dy, input_relu=True)
            runs.append((y, g))
    finally:
        orc.set_threads(before)
    (y1, g1), (y5, g5) = runs
    for a, c in zip(y1, y5):
        assert np.array_equal(a, c)
    for key in ("dw_rel", "dw_self", "dbias", "dh_src"):
        for a, c in zip(g1[key], g5[key]):
            assert np.array_equal(a, c), key
