"""The seeded workload generator produces valid blocks with the stated structure."""
import numpy as np
import pytest

from paper_2406_06022_amd import synth


@pytest.mark.parametrize("index", range(5))
def test_small_configs_are_valid_minibatches(orc, index):
    spec = synth.small_config(index)
    mb = synth.sample_minibatch(spec)
    assert len(mb.blocks) == spec.num_layers
    T = len(spec.ntype_names)
    for l, blk in enumerate(mb.blocks):
        assert orc.check_block(blk)
        if l + 1 < len(mb.blocks):  # block l's destinations are block l+1's sources
            assert blk.n_dst == mb.blocks[l + 1].n_src
        for r, rel in enumerate(blk.rels):
            assert (rel.src_type, rel.dst_type) == spec.rels[r]
            deg = np.diff(rel.indptr)
            assert deg.max(initial=0) <= spec.fanouts[l]
            if spec.degree in ("exact", "zipf") and deg.size:
                assert deg.min() >= 1
            for i in range(min(blk.n_dst[rel.dst_type], 200)):
                seg = rel.indices[rel.indptr[i]:rel.indptr[i + 1]]
                assert np.unique(seg).size == seg.size  # without replacement
    # seeds: last block's destinations
    last = mb.blocks[-1]
    for t in range(T):
        assert last.n_dst[t] == (spec.n_seeds if t in spec.seed_types else 0)
    for t in range(T):
        ids = mb.input_ids[t]
        assert ids.shape[0] == mb.blocks[0].n_src[t]
        assert np.unique(ids).size == ids.size
        assert ids.size == 0 or (ids.min() >= 0 and ids.max() < spec.type_rows[t])


def test_generator_is_deterministic():
    a = synth.sample_minibatch(synth.small_config(1))
    b = synth.sample_minibatch(synth.small_config(1))
    for x, y in zip(a.blocks, b.blocks):
        for r1, r2 in zip(x.rels, y.rels):
            assert np.array_equal(r1.indptr, r2.indptr) and np.array_equal(r1.indices, r2.indices)


def test_pareto_zero_degree_fraction():
    spec = synth.config(3)
    rng = np.random.Generator(np.random.PCG64(1))
    d0 = synth._degrees(rng, spec, 0, 200000, 30)
    assert abs((d0 == 0).mean() - (1 - (1 / 3) ** 1.5)) < 0.01
    d19 = synth._degrees(rng, spec, 19, 20000, 30)
    assert (d19 == 30).all()


def test_skewed_sources_are_distinct_and_in_range():
    rng = np.random.Generator(np.random.PCG64(2))
    deg = rng.integers(0, 20, size=500)
    src = synth._draw_sources(rng, deg, 10000, 0.8)
    assert src.min() >= 0 and src.max() < 10000
    off = np.concatenate([[0], np.cumsum(deg)])
    for i in range(500):
        seg = src[off[i]:off[i + 1]]
        assert np.unique(seg).size == seg.size


@pytest.mark.parametrize("index", [1, 3])
def test_sources_numbered_by_first_appearance(index):
    """Past the destination prefix, source rows are numbered in order of first use over the
    relations' edge lists (relations in order, edges in CSR order)."""
    mb = synth.sample_minibatch(synth.small_config(index))
    for blk in mb.blocks:
        for s in range(len(blk.n_src)):
            seen = []
            for rel in blk.rels:
                if rel.src_type == s:
                    seen.append(rel.indices.astype(np.int64))
            if not seen:
                assert blk.n_src[s] == blk.n_dst[s]
                continue
            edges = np.concatenate(seen)
            fresh = edges[edges >= blk.n_dst[s]]
            _, first = np.unique(fresh, return_index=True)
            order = fresh[np.sort(first)]
            assert np.array_equal(order, np.arange(blk.n_dst[s], blk.n_src[s]))
