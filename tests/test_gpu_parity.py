"""HIP path vs the CPU oracle, through the C ABI, on seeded inputs.

Random small blocks (ragged degrees, zero-degree rows, empty relations, repeated edges,
types without destination rows, several dims), the five workload configurations at a
size the oracle evaluates in seconds (every block of every mini-batch), the integer plan
bit for bit, an integer index probe, determinism, and the device-side validation errors.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
from harness import BlockRun, sign_words, TOL, rel_err, to64
from paper_2406_06022_amd import rgcn, synth

pytestmark = pytest.mark.gpu


def _random_blocks():
    rng = np.random.default_rng(1234)
    yield "one-type-dup", synth.random_block(rng, [300], [170], [(0, 0), (0, 0)], 9)
    yield "three-types", synth.random_block(rng, [400, 260, 333], [130, 257, 0],
                                            [(0, 1), (1, 0), (2, 0), (2, 1), (0, 0), (1, 1)], 12)
    yield "zero-heavy", synth.random_block(rng, [500, 90], [200, 77], [(0, 0), (1, 0), (0, 1)], 40,
                                           zero_frac=0.7)
    yield "empty-rel", synth.random_block(rng, [64, 50], [40, 33], [(0, 1), (1, 0)], 0)
    yield "wide-deg", synth.random_block(rng, [2000], [129], [(0, 0)], 300)


@pytest.mark.parametrize("dtype,d_in,d_out", [("f32", 32, 64), ("f32", 12, 20), ("bf16", 128, 256),
                                              ("bf16", 24, 40), ("bf16", 512, 128),
                                              ("f32", 256, 64)])
@pytest.mark.parametrize("name,blk", list(_random_blocks()))
def test_random_block_parity(name, blk, dtype, d_in, d_out):
    run = BlockRun(blk, dtype, d_in, d_out, seed=zlib.crc32(f"{name}-{d_in}".encode()) % 1000, bias=True,
                   use_ids=True)
    print(f"case {name} {dtype} {d_in}->{d_out}", flush=True)
    run.run_gpu()
    run.run_oracle()
    run.assert_parity()


# Destination types whose input-side product has at most 128 gradient columns (one slot of
# d_in <= 128, or two to four narrower ones) take, in bf16 with d_out 256 or 512, the
# streamed kernel that splits K over the waves of a workgroup (other d_out: the
# register-staged kernel).  Type 0 has a gradient and only its self slot (no degree
# division); type 1 takes k relation slots from type 0 (divided by the degree, zero-degree
# rows included).  Row counts cover a few 16-row blocks, a ragged last block, and many
# blocks per workgroup (past the register prefetch depth); N = 96 leaves 16-column tiles
# empty.
@pytest.mark.parametrize("d_in,d_out,n0,n1,k", [(128, 512, 2_500, 2_500, 1),
                                                (32, 512, 25_001, 25_000, 4),
                                                (64, 256, 40_000, 3_000, 2),
                                                (32, 512, 77, 77, 4),
                                                (96, 256, 2_500, 2_500, 1),
                                                (128, 64, 66_000, 700, 1),
                                                (64, 192, 4_133, 4_133, 2),
                                                (32, 128, 1_000, 1_000, 1)])
def test_input_side_narrow_slots(d_in, d_out, n0, n1, k):
    rng = np.random.default_rng(d_in * 7 + d_out + k)
    rels = [(0, 1)] * k + [(1, 0), (1, 1)]
    blk = synth.random_block(rng, [n0 + 40, n1 + n1 // 3 + 5], [n0, n1], rels, 6, zero_frac=0.3)
    print(f"case narrow input side {d_in}->{d_out} rows {n0}, {n1} slots {k}", flush=True)
    run = BlockRun(blk, "bf16", d_in, d_out, seed=d_out + k, use_ids=True, grad_types=(0,))
    run.run_gpu()
    run.run_oracle()
    run.assert_parity()


def _claimed_runs_block():
    # Large enough that the gather's runs outnumber its resident lane groups (runs are then
    # claimed from the shared counter), with forward segments heavy enough to span several
    # runs, so some claimed runs hold no segment start at all.
    rng = np.random.default_rng(4242)
    n_src, n_dst = [300_000, 60_000], [90_000, 20_000]
    rels = []
    for s_t, d_t, mx in ((0, 0, 24), (1, 0, 8), (0, 1, 30)):
        nd = n_dst[d_t]
        deg = rng.integers(0, mx + 1, size=nd)
        heavy = rng.choice(nd, size=6, replace=False)
        deg[heavy] = rng.integers(3000, 9000, size=6)
        indptr = np.zeros(nd + 1, dtype=np.int64)
        np.cumsum(deg, out=indptr[1:])
        idx = rng.integers(0, n_src[s_t], size=int(indptr[-1]))
        rels.append(synth.Relation(s_t, d_t, indptr.astype(np.int32), idx.astype(np.int32)))
    return synth.Block(n_src, n_dst, rels)


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f32", 64)])
def test_claimed_runs_and_heavy_segments(dtype, d):
    blk = _claimed_runs_block()
    print(f"claimed runs {dtype} d={d}: nnz {sum(r.nnz for r in blk.rels)}", flush=True)
    run = BlockRun(blk, dtype, d, 64, seed=31, use_ids=True)
    run.run_gpu(repeat=2)
    run.run_oracle()
    run.assert_parity()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_relu_flags_and_embedding_scatter(dtype):
    rng = np.random.default_rng(77)
    blk = synth.random_block(rng, [700, 300], [250, 100], [(0, 1), (1, 0), (0, 0)], 14)
    d = 32 if dtype == "f32" else 64
    for unique in (True, False):
        run = BlockRun(blk, dtype, d, d, seed=5, use_ids=True, input_relu=True, fwd_relu=True,
                       emb_types=(0,), grad_types=(0, 1), ids_unique=unique, dup_ids=not unique)
        run.run_gpu()
        run.run_oracle()
        run.assert_parity()


# ReLU sign bits: the forward writes them beside y (bit-exact against y > 0 on the stored
# values, words fully written, bits past d_out zero), and a backward that reads them gives
# bit for bit the results of one that reads the input rows (and matches the oracle).
# d_out 40 and 136 leave a part-filled last word; 512 is whole words in every tile.
@pytest.mark.parametrize("dtype,d_in,d_out", [("bf16", 64, 40), ("bf16", 128, 136),
                                              ("bf16", 128, 512), ("f32", 32, 40),
                                              ("f32", 64, 136)])
def test_relu_sign_bits(dtype, d_in, d_out):
    rng = np.random.default_rng(d_in + d_out)
    blk = synth.random_block(rng, [700, 333], [517, 100], [(0, 1), (1, 0), (0, 0)], 9)
    print(f"case relu sign bits {dtype} {d_in}->{d_out}", flush=True)
    fwd = BlockRun(blk, dtype, d_in, d_out, seed=11, use_ids=True, fwd_relu=True, bias=True,
                   mask_out=True)
    fwd.run_gpu()
    for t, y in enumerate(fwd.gpu["y"]):
        if y is None:
            continue
        want = sign_words(y)
        got = fwd.gpu["y_mask"][t]
        assert torch.equal(got, want), f"type {t}: sign words differ"
    runs = []
    for mask_in in (False, True):
        run = BlockRun(blk, dtype, d_in, d_out, seed=12, use_ids=True, input_relu=True,
                       grad_types=(0, 1), emb_types=(0,), mask_in=mask_in)
        run.run_gpu()
        runs.append(run)
    runs[1].run_oracle()
    runs[1].assert_parity()
    for key in ("dh", "demb"):
        for a, b in zip(runs[0].gpu[key], runs[1].gpu[key]):
            if a is not None:
                assert torch.equal(a, b), f"{key} differs when read through the sign bits"


@pytest.mark.parametrize("index", range(5))
def test_small_config_blocks_parity(index):
    spec = synth.small_config(index)
    mb = synth.sample_minibatch(spec)
    for l, blk in enumerate(mb.blocks):
        d_in, d_out = spec.dims[l], spec.dims[l + 1]
        emb = [t for t in range(len(spec.ntype_names)) if spec.featureless[t]] if l == 0 else []
        grad = list(range(len(spec.ntype_names))) if l > 0 else []
        print(f"config {spec.name} block {l} nnz {blk.nnz} {d_in}->{d_out}", flush=True)
        run = BlockRun(blk, spec.dtype, d_in, d_out, seed=100 + 10 * index + l,
                       use_ids=(l == 0), input_relu=(l > 0), emb_types=emb, grad_types=grad)
        run.run_gpu()
        run.run_oracle()
        errs = run.assert_parity()
        print({k: f"{v:.2e}" for k, v in errs.items()}, flush=True)


def _plan_arrays(run):
    lay = rgcn.rgcn_block_plan_layout(run.dblk, run.params)
    ws = run.ws.cpu().numpy()

    def arr(off, n):
        return np.frombuffer(ws[off:off + 4 * n].tobytes(), dtype=np.int32)

    fwd = arr(lay["fwd_order"], lay["n_fwd_segments"])
    bwd = arr(lay["bwd_order"], lay["n_bwd_rows"])
    csc = {}
    for r, rel in enumerate(run.blk.rels):
        if lay["csc_indptr"][r] is not None:
            ns = run.blk.n_src[rel.src_type]
            ip = arr(lay["csc_indptr"][r], ns + 1)
            csc[r] = (ip - ip[0], arr(lay["csc_dst"][r], len(rel.indices)))
    return fwd, bwd, csc


def _check_schedules(run, fwd, bwd):
    """The schedules are library policy (no passage of the paper orders the work): all a
    caller may rely on is that each is a permutation of the items it covers."""
    lay = rgcn.rgcn_block_plan_layout(run.dblk, run.params)
    assert np.array_equal(np.sort(fwd), np.arange(lay["n_fwd_segments"]))
    base = 0
    for t in sorted(set(run.grad_types)):
        n = run.blk.n_src[t]
        assert np.array_equal(np.sort(bwd[base:base + n]), np.arange(n)), t
        base += n
    assert base == len(bwd)


def _check_csc(run, csc):
    for r, (cip, cdst) in csc.items():
        rel = run.blk.rels[r]
        want_ip, want_dst, _ = oracle.csc(run.blk.n_src[rel.src_type], rel.indptr, rel.indices)
        assert np.array_equal(cip, want_ip), r
        assert np.array_equal(cdst, want_dst), r


@pytest.mark.parametrize("index", [1, 2, 3, 4])
def test_plan_is_bit_exact(index):
    """CSC transposes bit for bit against the oracle's stable counting sort; schedules are
    permutations."""
    spec = synth.small_config(index)
    mb = synth.sample_minibatch(spec)
    for blk in mb.blocks:
        T = len(blk.n_src)
        run = BlockRun(blk, spec.dtype, 8 if spec.dtype == "bf16" else 4, 8, seed=1,
                       grad_types=[t for t in range(T) if blk.n_src[t] > 0])
        run.run_gpu()
        fwd, bwd, csc = _plan_arrays(run)
        _check_schedules(run, fwd, bwd)
        _check_csc(run, csc)


def _skewed_block():
    spec = synth.WorkloadSpec("skewed", "bf16", ("A", "B"), (300000, 5000), (False, False),
                              ((0, 1), (1, 0), (0, 0)), (1,), 3000, (25,), "zipf", (8, 8),
                              synth.BASE_SEED + 50, skew=0.9)
    return synth.sample_minibatch(spec).blocks[0]


def test_plan_skewed_sources_bit_exact():
    """Power-law source popularity: long transpose segments (hub sources), so the
    backward schedule is reordered; RGCN_PLAN_ENUMERATION_ORDER keeps enumeration order."""
    blk = _skewed_block()
    run = BlockRun(blk, "bf16", 8, 8, seed=3, grad_types=[0, 1])
    run.run_gpu()
    fwd, bwd, csc = _plan_arrays(run)
    _check_schedules(run, fwd, bwd)
    _check_csc(run, csc)
    longest = max(int(np.diff(oracle.csc(blk.n_src[r.src_type], r.indptr, r.indices)[0]).max(initial=0))
                  for r in blk.rels)
    assert longest > 32  # hub sources exist ...
    assert not np.array_equal(bwd, np.concatenate([np.arange(n) for n in blk.n_src]))  # ... and moved
    run.run_gpu(plan_flags=rgcn.RGCN_PLAN_ENUMERATION_ORDER)
    fwd, bwd, csc = _plan_arrays(run)
    assert np.array_equal(fwd, np.arange(len(fwd)))
    assert np.array_equal(bwd, np.concatenate([np.arange(n) for n in blk.n_src]))
    _check_csc(run, csc)


def _bitwise_equal(a, b):
    for key in a:
        if a[key] is None:
            assert b[key] is None, key
            continue
        for x, z in zip(a[key], b[key]):
            if x is None:
                assert z is None
                continue
            if x.dtype in (torch.bfloat16, torch.float32):
                x = x.view(torch.int16) if x.dtype == torch.bfloat16 else x.view(torch.int32)
                z = z.view(torch.int16) if z.dtype == torch.bfloat16 else z.view(torch.int32)
            assert torch.equal(x, z), key


@pytest.mark.parametrize("case", ["skewed-bf16", "claimed-runs-bf16", "claimed-runs-f32"])
def test_results_do_not_depend_on_the_schedule(case):
    """Every output and gradient is bit-identical whether the kernels walk the degree-sorted
    schedules or plain enumeration order (blocks with segments of more than 32 edges in both
    directions, so the sorted schedules differ from enumeration order); and both match the
    oracle."""
    if case.startswith("skewed"):
        blk, dtype, d, ids = _skewed_block(), "bf16", 64, True
    else:
        blk, dtype = _claimed_runs_block(), case.split("-")[-1]
        d, ids = (128 if dtype == "bf16" else 64), True
    T = len(blk.n_src)
    run = BlockRun(blk, dtype, d, 64, seed=17, use_ids=ids, bias=True, emb_types=(0,),
                   grad_types=list(range(T)))
    print(f"case {case} nnz {sum(r.nnz for r in blk.rels)}", flush=True)
    sorted_out = run.run_gpu()[0]
    fwd, bwd, _ = _plan_arrays(run)
    enum_bwd = np.concatenate([np.arange(blk.n_src[t]) for t in sorted(set(run.grad_types))])
    # the forward segments are heavy in the claimed-runs block, the transpose segments in the
    # skewed one: the sorted schedule differs from enumeration order in that direction
    if case.startswith("skewed"):
        assert not np.array_equal(bwd, enum_bwd)
    else:
        assert not np.array_equal(fwd, np.arange(len(fwd)))
    enum_out = run.run_gpu(plan_flags=rgcn.RGCN_PLAN_ENUMERATION_ORDER)[0]
    fwd2, bwd2, _ = _plan_arrays(run)
    assert np.array_equal(fwd2, np.arange(len(fwd2))) and np.array_equal(bwd2, enum_bwd)
    _bitwise_equal(sorted_out, enum_out)
    run.run_oracle()
    run.assert_parity()


@pytest.mark.parametrize("n_src", [900, 5000, 1_200_000])
def test_plan_csc_hubs_beyond_lds(n_src):
    """Transpose segments of every length class: 2, up to 16, up to 16384 (sorted in LDS)
    and one hub source with more than 16384 edges, which sends the whole transpose down the
    radix-sort path; source counts giving 1, 2 and 3 radix passes."""
    rng = np.random.default_rng(n_src)
    n_dst = min(n_src, 20000)
    per_row = max(1, -(-17000 // n_dst))          # hub-0 edges per destination row
    rows = []
    for i in range(n_dst):
        e = [0] * per_row
        if i % 4 == 0:
            e.append(1)                            # hub 1: ~n_dst / 4 edges
        e += rng.integers(2, n_src, size=int(rng.integers(0, 6))).tolist()
        rng.shuffle(e)
        rows.append(e)
    indptr = np.zeros(n_dst + 1, dtype=np.int32)
    np.cumsum([len(e) for e in rows], out=indptr[1:])
    indices = np.concatenate([np.asarray(e, dtype=np.int32) for e in rows])
    blk = synth.Block([n_src], [n_dst], [synth.Relation(0, 0, indptr, indices)])
    print(f"case csc hubs n_src {n_src} nnz {len(indices)}", flush=True)
    run = BlockRun(blk, "f32", 4, 8, seed=5, grad_types=[0])
    run.run_gpu()
    _, _, csc = _plan_arrays(run)
    cip, cdst = csc[0]
    want_ip, want_dst, _ = oracle.csc(n_src, indptr, indices)
    assert int(np.diff(want_ip).max()) > 16384
    assert np.array_equal(cip, want_ip) and np.array_equal(cdst, want_dst)


def test_index_probe_is_exact():
    """fp32 integer features encoding the global id bytes; W_self = 0 and W_r = I, so every
    output is a gathered-row sum divided by the degree; times the degree it must equal the
    oracle's integer sums exactly (any wrong row would show)."""
    rng = np.random.default_rng(99)
    blk = synth.random_block(rng, [5000], [1500], [(0, 0)], 25)
    rows = 1 << 16
    ids = torch.randperm(rows)[:5000].to(torch.int64)
    allid = torch.arange(rows, dtype=torch.int64)
    cols = [((allid >> (8 * c)) & 0xFF) + 1 for c in range(2)] + [torch.ones(rows, dtype=torch.int64)] * 2
    table = torch.stack(cols, dim=1).to(torch.float32)
    d = 4
    dev = "cuda"
    dblk = rgcn.DeviceBlock(blk, 0, dev)
    eye = torch.eye(d, dtype=torch.float32, device=dev)
    zero = torch.zeros((d, d), dtype=torch.float32, device=dev)
    params = rgcn.Params("f32", d, d, [eye], [zero])
    inputs = rgcn.Inputs([table.to(dev)], [ids.to(dev)])
    ws = rgcn.new_workspace(dblk, params)
    y = torch.empty((1500, d), dtype=torch.float32, device=dev)
    rgcn.rgcn_block_plan(dblk, params, ws)
    rgcn.rgcn_block_forward(dblk, inputs, params, [y], ws)
    torch.cuda.synchronize()
    deg = oracle.degrees(blk.rels[0].indptr)
    got = np.rint(to64(y.cpu()) * np.maximum(deg, 1)[:, None])
    h = table[ids].to(torch.float64).numpy()
    m = oracle.mean_aggregate(blk.rels[0].indptr, blk.rels[0].indices, h)
    want = np.rint(m * np.maximum(deg, 1)[:, None])
    assert np.array_equal(got, want)


def test_deterministic_bitwise():
    spec = synth.small_config(2)
    blk = synth.sample_minibatch(spec).blocks[0]
    run = BlockRun(blk, "bf16", 128, 256, seed=8, use_ids=True, emb_types=(0,), grad_types=())
    a, b = run.run_gpu(repeat=2)
    for key in ("y", "dw_rel", "dw_self", "demb"):
        for x, z in zip(a[key], b[key]):
            if x is not None:
                assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x,
                                   z.view(torch.int16) if z.dtype == torch.bfloat16 else z), key


def test_degenerate_blocks():
    # no destination rows at all; no edges at all; one row one edge
    cases = [
        synth.Block([10, 5], [0, 0], [synth.Relation(0, 1, np.zeros(1, np.int32),
                                                     np.zeros(0, np.int32))]),
        synth.Block([10, 5], [4, 5], [synth.Relation(0, 1, np.zeros(6, np.int32),
                                                     np.zeros(0, np.int32)),
                                      synth.Relation(1, 0, np.zeros(5, np.int32),
                                                     np.zeros(0, np.int32))]),
        synth.Block([1], [1], [synth.Relation(0, 0, np.array([0, 1], np.int32),
                                              np.array([0], np.int32))]),
    ]
    for blk in cases:
        for dtype, d in (("f32", 8), ("bf16", 16)):
            run = BlockRun(blk, dtype, d, d, seed=2, bias=True)
            run.run_gpu()
            run.run_oracle()
            run.assert_parity()


def test_device_validation_reports_errors():
    blk = synth.Block([20], [10], [synth.Relation(0, 0, np.arange(11, dtype=np.int32),
                                                  np.arange(10, dtype=np.int32))])
    run = BlockRun(blk, "f32", 8, 8, seed=4)
    run.run_gpu(validate=True)  # valid block passes validation
    bad_idx = synth.Block([20], [10], [synth.Relation(0, 0, np.arange(11, dtype=np.int32),
                                                      np.array([0] * 9 + [20], np.int32))])
    run = BlockRun(bad_idx, "f32", 8, 8, seed=4)
    with pytest.raises(rgcn.RgcnError) as e:
        run.run_gpu(validate=True)
    assert e.value.status == 4
    ip = np.arange(11, dtype=np.int32)
    ip[5] = 2  # not monotone
    bad_csr = synth.Block([20], [10], [synth.Relation(0, 0, ip, np.arange(10, dtype=np.int32))])
    run = BlockRun(bad_csr, "f32", 8, 8, seed=4)
    with pytest.raises(rgcn.RgcnError) as e:
        run.run_gpu(validate=True)
    assert e.value.status == 5
    # out-of-range row id of the input table
    run = BlockRun(blk, "f32", 8, 8, seed=4, use_ids=True)
    run.ids[0][3] = run.tables[0].shape[0]
    with pytest.raises(rgcn.RgcnError) as e:
        run.run_gpu(validate=True)
    assert e.value.status == 4


def test_workspace_too_small_and_bad_dims():
    blk = synth.Block([20], [10], [synth.Relation(0, 0, np.arange(11, dtype=np.int32),
                                                  np.arange(10, dtype=np.int32))])
    dblk = rgcn.DeviceBlock(blk, 0)
    w = torch.zeros((8, 8), device="cuda")
    params = rgcn.Params("f32", 8, 8, [w], [w])
    ws = torch.empty(64, dtype=torch.uint8, device="cuda")
    with pytest.raises(rgcn.RgcnError) as e:
        rgcn.rgcn_block_plan(dblk, params, ws)
    assert e.value.status == 6
    with pytest.raises(rgcn.RgcnError) as e:
        rgcn.rgcn_block_workspace_size(dblk, rgcn.Params("f32", 6, 8, [w], [w]))
    assert e.value.status == 7


# transpose degrees around the split threshold of the backward (128 edges per piece) and
# far beyond it: one piece plus one edge, whole pieces, a ragged last piece, and in bf16 a
# hub past the LDS sort of the plan.  (fp32 stops at 3,000: each fp32 input-side term
# carries a rounding error of about sqrt(d_out) 2^-24 of its size, and over 17,000
# cancelling terms that alone reaches the 1e-5 bar at elements of rms size, whatever the
# order of summation.)
HUBS = {"f32": [129, 256, 257, 1000, 3000], "bf16": [129, 256, 257, 1000, 3000, 17000]}


@pytest.mark.parametrize("dtype,d_in,d_out", [("f32", 64, 32), ("bf16", 128, 64),
                                              ("f32", 32, 16), ("bf16", 264, 40)])
def test_split_hub_rows(dtype, d_in, d_out):
    """Source rows whose transpose holds more than one piece of edges are summed piecewise
    by several lane groups and then reduced; their input and embedding gradients, with the
    ReLU mask and with repeated edges, against the oracle.  d 32 fp32 leaves more relations
    per type than lanes per group (the non-pipelined sum)."""
    rng = np.random.default_rng(d_in + d_out)
    rels = [(0, 0), (0, 1), (1, 0), (0, 0)] + ([(0, 1)] * 6 if d_in == 32 else [])
    blk = synth.random_block(rng, [6000, 900], [2000, 700], rels, 6)
    blk = synth.with_hub_sources(rng, blk, 0, HUBS[dtype])
    refs = np.zeros(6000, np.int64)
    for rel in blk.rels:
        if rel.src_type == 0:
            refs += np.bincount(np.asarray(rel.indices, np.int64), minlength=6000)
    assert refs.max() >= HUBS[dtype][-1] and (refs > 128).sum() >= len(HUBS[dtype])
    print(f"case split hubs {dtype} {d_in}->{d_out}: nnz {sum(r.nnz for r in blk.rels)}",
          flush=True)
    for relu in (False, True):
        run = BlockRun(blk, dtype, d_in, d_out, seed=13, use_ids=True, input_relu=relu,
                       emb_types=(0,), grad_types=(0, 1))
        run.run_gpu()
        run.run_oracle()
        run.assert_parity()


@pytest.mark.parametrize("index", [1, 2, 3, 4])
def test_per_edge_source_rows_match_id_resolution(index):
    """The input layer given each edge's table row (as the sampler emits it) gathers the
    same rows in the same order as resolving indices through the row ids: every output and
    gradient bit for bit, and both at the oracle's bar; a wrong per-edge row is reported
    under device validation."""
    spec = synth.small_config(index)
    blk = synth.sample_minibatch(spec).blocks[0]
    T = len(spec.ntype_names)
    emb = [t for t in range(T) if spec.featureless[t]]
    run = BlockRun(blk, spec.dtype, spec.dims[0], spec.dims[1], seed=300 + index, use_ids=True,
                   emb_types=emb, grad_types=emb)
    print(f"case per-edge rows {spec.name} nnz {blk.nnz}", flush=True)
    by_ids = run.run_gpu()[0]
    run.edge_rows = True
    by_rows = run.run_gpu(validate=True)[0]
    _bitwise_equal(by_ids, by_rows)
    run.run_oracle()
    run.assert_parity()
    # corrupt one per-edge row: validation reports it
    r = next(i for i, rel in enumerate(blk.rels) if len(rel.indices))
    run.device_setup()
    run.dblk.src_rows[r][0] += 1
    with pytest.raises(rgcn.RgcnError) as e:
        rgcn.rgcn_block_plan(run.dblk, run.params, run.ws, rgcn.RGCN_VALIDATE_DEVICE)
        rgcn.rgcn_block_aggregate(run.dblk, run.inputs, run.params, run.ws,
                                  rgcn.RGCN_VALIDATE_DEVICE)
    assert e.value.status == 4
