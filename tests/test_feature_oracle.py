"""Pins of the featureless-feature oracle (CPU): the mean over in-neighbours equals the
row-normalised sparse adjacency times the features (scipy), constant features stay
constant, nodes without neighbours get zeros, and repeated edges count twice."""
import numpy as np
import pytest
import scipy.sparse as sp

import oracle
from paper_2406_06022_amd import synth


def _rels(seed, n_dst=300, srcs=(500, 200), d=7):
    rng = np.random.default_rng(seed)
    g = synth.random_graph(rng, [n_dst] + list(srcs), [(1 + k, 0) for k in range(len(srcs))], 1.0,
                           heavy=3, heavy_deg=90)
    feats = [rng.standard_normal((n, d)) for n in srcs]
    return [(r.indptr, r.indices, feats[k]) for k, r in enumerate(g.rels)], feats, n_dst


def test_matches_normalised_adjacency():
    rels, feats, n = _rels(1)
    got = oracle.featureless_mean(rels, n)
    # one sparse matrix over the concatenated source rows; duplicates are summed by scipy
    offs = np.cumsum([0] + [f.shape[0] for f in feats])
    rows, cols = [], []
    for k, (ip, ix, _) in enumerate(rels):
        rows.append(np.repeat(np.arange(n), np.diff(ip)))
        cols.append(ix + offs[k])
    A = sp.csr_matrix((np.ones(sum(len(c) for c in cols)), (np.concatenate(rows),
                                                           np.concatenate(cols))),
                      shape=(n, offs[-1]))
    deg = np.asarray(A.sum(1)).ravel()
    want = (A @ np.vstack(feats)) / np.maximum(deg, 1)[:, None]
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)
    assert (deg == 0).any() and not got[deg == 0].any()


def test_constant_features_and_repeats():
    ip = np.array([0, 3, 3, 5], dtype=np.int64)
    ix = np.array([2, 2, 0, 1, 1], dtype=np.int64)
    f = np.array([[1.0, 2.0], [4.0, -2.0], [7.0, 8.0]])
    got = oracle.featureless_mean([(ip, ix, f)], 3)
    np.testing.assert_array_equal(got, [[5.0, 6.0], [0.0, 0.0], [4.0, -2.0]])
    c = np.full((3, 2), 0.375)
    np.testing.assert_array_equal(oracle.featureless_mean([(ip, ix, c)], 3)[[0, 2]], 0.375)


def test_out_of_range_rejected():
    with pytest.raises(ValueError):
        oracle.featureless_mean([(np.array([0, 1]), np.array([5]), np.zeros((3, 2)))], 1)
