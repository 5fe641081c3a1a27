"""Pins of the sampling oracle (CPU): the Philox4x64-10 stream against numpy's
implementation of the same generator, Floyd's sampler against the distribution it must
have, and block construction against a brute-force relabelling written with dicts."""
import itertools

import numpy as np
import pytest

import oracle
from paper_2406_06022_amd import synth

M64 = (1 << 64) - 1


def test_philox_matches_numpy():
    """numpy's Philox bit generator (the same 4x64, 10-round function) advances its counter
    before each block, so a generator set at counter c - 1 yields the block of c."""
    rng = np.random.default_rng(0)
    for _ in range(300):
        c = rng.integers(0, 1 << 62, size=4, dtype=np.uint64) * np.uint64(4) + np.uint64(1)
        k = rng.integers(0, 1 << 62, size=2, dtype=np.uint64) * np.uint64(3)
        prev = c.copy()
        prev[0] -= np.uint64(1)
        want = np.random.Philox(counter=prev, key=k).random_raw(4)
        assert np.array_equal(oracle.philox4x64(c, k), want)
    # counter 0: numpy wraps an all-ones counter to zero before generating
    want0 = np.random.Philox(counter=[M64] * 4, key=[0, 0]).random_raw(4)
    assert np.array_equal(oracle.philox4x64([0, 0, 0, 0], [0, 0]), want0)


def test_draws_are_the_stream_words():
    """Draw k of (v, r) is word k mod 4 of the block at counter (v, r, k // 4, 0), key
    (seed, layer)."""
    for (seed, layer, v, r) in ((7, 0, 1, 0), (2 ** 40 + 3, 2, 123456789, 11), (1, 1, 5, 63)):
        for k in range(9):
            want = np.random.Philox(counter=[v - 1, r, k // 4, 0], key=[seed, layer]).random_raw(4)
            assert oracle.sample_draw(seed, layer, v, r, k) == int(want[k % 4])


def test_small_segments_take_every_edge():
    for n in range(0, 6):
        assert oracle.sample_segment(n, 5, 1, 0, 42, 3).tolist() == list(range(n))


def test_floyd_subsets_are_uniform():
    """n = 7, fanout 3: each of the 35 subsets is equally likely.  35,000 segments
    (distinct v) give 1,000 expected per subset; the chi-square statistic (34 degrees of
    freedom) stays far below the 1e-6 tail (about 83)."""
    n, f, trials = 7, 3, 35_000
    counts = {c: 0 for c in itertools.combinations(range(n), f)}
    for v in range(trials):
        pos = oracle.sample_segment(n, f, 99, 1, v, 2)
        assert len(pos) == f and list(pos) == sorted(set(pos.tolist()))
        assert 0 <= pos[0] and pos[-1] < n
        counts[tuple(pos.tolist())] += 1
    exp = trials / len(counts)
    chi2 = sum((c - exp) ** 2 / exp for c in counts.values())
    assert chi2 < 83, chi2


def test_floyd_inclusion_probability_on_a_large_segment():
    """n = 1000, fanout 25: every position is taken with probability 1/40; the first, last
    and middle tenths of the positions each collect 10 % of the picks."""
    n, f, trials = 1000, 25, 8000
    hits = np.zeros(n)
    for v in range(trials):
        pos = oracle.sample_segment(n, f, 5, 0, v, 0)
        assert len(np.unique(pos)) == f
        hits[pos] += 1
    total = trials * f
    for lo in (0, 450, 900):
        share = hits[lo:lo + 100].sum() / total
        assert abs(share - 0.1) < 0.006, (lo, share)
    assert hits.max() < 4 * total / n


def _brute_block(graph, dst_ids, fanout, seed, layer):
    """Relabelling with dicts, sampling positions through the oracle's segment sampler."""
    T, R = len(graph.num_nodes), len(graph.rels)
    cand = []
    indptr = []
    for r, rel in enumerate(graph.rels):
        ip, got = [0], []
        for v in dst_ids[rel.dst_type]:
            b, e = int(rel.indptr[v]), int(rel.indptr[v + 1])
            pos = oracle.sample_segment(e - b, fanout, seed, layer, int(v), r)
            got += [int(rel.indices[b + p]) for p in pos]
            ip.append(len(got))
        cand.append(got)
        indptr.append(ip)
    src_ids, local = [], []
    for s in range(T):
        seen = {}
        for v in list(dst_ids[s]) + [x for r in range(R) if graph.rels[r].src_type == s
                                     for x in cand[r]]:
            if int(v) not in seen:
                seen[int(v)] = len(seen)
        src_ids.append(list(seen.keys()))
        local.append(seen)
    indices = [[local[graph.rels[r].src_type][x] for x in cand[r]] for r in range(R)]
    return indptr, indices, src_ids


@pytest.mark.parametrize("fanout", [1, 3, 10])
def test_block_construction_matches_brute_force(fanout):
    rng = np.random.default_rng(fanout)
    g = synth.random_graph(rng, [300, 200, 120], [(0, 1), (1, 0), (2, 0), (0, 0), (1, 2)], 4.0,
                           heavy=3, heavy_deg=80)
    dst = [rng.choice(300, 40, replace=False), rng.choice(200, 25, replace=False),
           np.zeros(0, dtype=np.int64)]
    blk = oracle.sample_block(g, dst, fanout, seed=11, layer=1)
    ip, ix, src = _brute_block(g, dst, fanout, 11, 1)
    for r in range(len(g.rels)):
        assert blk.rels[r].indptr.tolist() == ip[r]
        assert blk.rels[r].indices.tolist() == ix[r]
    for t in range(3):
        assert blk.src_ids[t].tolist() == src[t]
        assert blk.src_ids[t][: len(dst[t])].tolist() == list(dst[t])   # destination prefix
    # the block is a valid input of the layer
    assert oracle.check_block(blk)


def test_sampled_edges_are_graph_edges_and_respect_the_fanout():
    rng = np.random.default_rng(3)
    g = synth.random_graph(rng, [500, 400], [(0, 1), (1, 0), (1, 1)], 9.0, heavy=5,
                           heavy_deg=300)
    dst = [rng.choice(500, 60, replace=False), rng.choice(400, 70, replace=False)]
    blk = oracle.sample_block(g, dst, 7, seed=5, layer=0)
    for r, rel in enumerate(g.rels):
        srel = blk.rels[r]
        for i, v in enumerate(dst[rel.dst_type]):
            nb = rel.indices[rel.indptr[v]:rel.indptr[v + 1]]
            got = blk.src_ids[rel.src_type][srel.indices[srel.indptr[i]:srel.indptr[i + 1]]]
            assert len(got) == min(len(nb), 7)
            # a multiset drawn from the neighbour list without reusing a position
            vals, cnt = np.unique(got, return_counts=True)
            nv, ncnt = np.unique(nb, return_counts=True)
            have = dict(zip(nv.tolist(), ncnt.tolist()))
            assert all(have.get(int(x), 0) >= c for x, c in zip(vals, cnt))


def test_invalid_destinations_rejected():
    rng = np.random.default_rng(4)
    g = synth.random_graph(rng, [50, 40], [(0, 1), (1, 0)], 3.0)
    with pytest.raises(ValueError):
        oracle.sample_block(g, [np.array([1, 2, 1]), np.array([0])], 3, 1, 0)
    with pytest.raises(ValueError):
        oracle.sample_block(g, [np.array([1, 50]), np.array([0])], 3, 1, 0)
