"""Sparse Adagrad step of learnable embedding tables on the GPU vs the oracle's step.

Two forms: fused into the backward transposed sum (each table row of the block takes its
step straight from its input-gradient row), and the standalone pass over a table-shaped
gradient.  Inputs are seeded; the oracle runs on the same decoded values in fp64.

Bars of the fused form.  The GPU's gradient g' meets the gradient bar of the dtype
(harness metric: |g' - g| <= tol max(|g|, rms g), tol 1e-5 fp32 / 2e-2 bf16), which is
asserted on the dh output of the same launch.  Each step is a monotone increasing
function of g': after m steps on the same gradient
  state_m = s0 + m g'^2,   w_m = w0 - sum_{k=1..m} lr g' / (sqrt(s0 + k g'^2) + eps),
so state and table must lie in the images of the interval [g - d, g + d], d = tol max(|g|,
rms g), widened by the fp32 rounding of the kernel's few operations and, for bf16 tables,
by half a bf16 ulp per step (round to nearest even of the fp32 result).  Every bound comes
from the oracle's gradient and the inputs alone; near g = 0 with an empty state the step
is steep (lr g / (|g| + eps)), which is why a relative bar on the step does not hold there.
The standalone pass reads the same fp32 gradient the oracle reads, so its bars are fp32
rounding only (1e-5 in the harness metric), plus the bf16 half ulp of the table.
"""
import numpy as np
import pytest
import torch

import oracle
from harness import BlockRun, TOL, rel_err, to64
from paper_2406_06022_amd import rgcn, synth

pytestmark = pytest.mark.gpu

LR = 0.0625          # exact in fp32, so both sides use the same constant
EPS = 2.0 ** -20


def _half_ulp_bf16(x):
    a = np.maximum(np.abs(x), 2.0 ** -126)
    return np.exp2(np.floor(np.log2(a)) - 8)


def _check_table(got, w0, want, dtype, tol_step, what):
    """got: table after the GPU step; w0: before; want: the oracle's table after."""
    step_want = want - w0
    if dtype == "f32":
        err = rel_err(got - w0, step_want)
        assert err <= tol_step, f"{what}: step error {err}"
        return
    rms = float(np.sqrt(np.mean(step_want * step_want))) if step_want.size else 0.0
    bound = _half_ulp_bf16(np.maximum(np.abs(got), np.abs(want))) + tol_step * np.maximum(
        np.abs(step_want), rms)
    over = np.abs(got - want) - bound
    assert not (over > 0).any(), f"{what}: {int((over > 0).sum())} elements over the bound"


def _adagrad_block(kind):
    rng = np.random.default_rng({"mixed": 7, "many-rels": 8, "hubs": 9}[kind])
    if kind == "hubs":
        # learnable rows whose transposes span several pieces of the split backward
        blk = synth.random_block(rng, [3000, 500], [800, 200], [(0, 0), (0, 1), (1, 0)], 8)
        return synth.with_hub_sources(rng, blk, 0, [129, 700, 5000]), [0]
    if kind == "mixed":
        # type 0 learnable (ids into a larger table), type 1 featured; zero-degree rows,
        # source rows without out-edges, a heavy destination row
        blk = synth.random_block(rng, [900, 500], [300, 200], [(0, 0), (0, 1), (1, 0), (1, 1)],
                                 14, zero_frac=0.3)
        return blk, [0]
    # one type with more relations leaving it than a lane group is wide (the non-pipelined
    # transposed sum at d = 32)
    rels = [(0, 0)] * 6 + [(0, 1)] * 5 + [(1, 0)]
    blk = synth.random_block(rng, [700, 300], [250, 120], rels, 6)
    return synth.with_hub_sources(rng, blk, 0, [300, 2000]), [0, 1]   # split rows too


@pytest.mark.parametrize("kind", ["mixed", "many-rels", "hubs"])
@pytest.mark.parametrize("dtype,d_in,d_out", [("f32", 32, 48), ("bf16", 32, 64),
                                              ("bf16", 128, 64), ("f32", 264, 40)])
def test_fused_adagrad_matches_oracle(kind, dtype, d_in, d_out):
    blk, opt_types = _adagrad_block(kind)
    T = len(blk.n_src)
    print(f"case fused {kind} {dtype} {d_in}->{d_out}", flush=True)
    run = BlockRun(blk, dtype, d_in, d_out, seed=31 + d_in, use_ids=True, emb_types=opt_types,
                   grad_types=[0])
    run.device_setup()
    dev = "cuda"
    gen = torch.Generator().manual_seed(5 + d_in)
    state0 = []
    for t in range(T):
        s = torch.rand((run.tables[t].shape[0], d_in), generator=gen) * 2.0
        s[: s.shape[0] // 4] = 0.0          # rows never stepped before
        state0.append(s)
    d_state = [state0[t].to(dev) if t in opt_types else None for t in range(T)]
    tdt = synth.torch_dtype(dtype)
    y = [torch.empty((n, d_out), dtype=tdt, device=dev) if n else None for n in blk.n_dst]
    dy = [x.to(dev) for x in run.dy]
    dh = [torch.full((blk.n_src[0], d_in), float("nan"), device=dev)] + [None] * (T - 1)
    rgcn.rgcn_block_plan(run.dblk, run.params, run.ws)
    rgcn.rgcn_block_forward(run.dblk, run.inputs, run.params, y, run.ws)
    rgcn.rgcn_block_backward_dense(run.dblk, run.params, dy, workspace=run.ws)
    steps = []
    for _ in range(2):   # the second step reads the state the first one wrote
        rgcn.rgcn_block_backward_sparse_adagrad(run.dblk, run.inputs, run.params, d_state, LR,
                                                EPS, dh_src=dh, workspace=run.ws,
                                                flags=rgcn.RGCN_IDS_UNIQUE)
        torch.cuda.synchronize()
        steps.append(([to64(t) for t in run.d_tables],
                      [to64(s) if s is not None else None for s in d_state]))

    ref = run.run_oracle()
    tol = TOL[dtype]
    assert rel_err(to64(dh[0]), ref["dh"][0]) <= tol
    for t in opt_types:
        ids = run.ids[t].numpy()
        touched = np.zeros(run.tables[t].shape[0], dtype=bool)
        touched[ids] = True
        w0, s0 = to64(run.tables[t]), state0[t].double().numpy()
        for k, (tabs, states) in enumerate(steps):
            got_w, got_s = tabs[t], states[t]
            # rows outside the block keep their bits
            assert np.array_equal(got_w[~touched], w0[~touched]), (t, k)
            assert np.array_equal(got_s[~touched], s0[~touched]), (t, k)
            _check_steps(ref["demb"][t][ids], s0[ids], w0[ids], got_s[ids], got_w[ids], k + 1,
                         tol, dtype, f"type {t} step {k}")


def _check_steps(g, s0, w0, got_s, got_w, m, tol, dtype, what):
    """State and table after m fused steps on gradient g' within the interval images."""
    rms = float(np.sqrt(np.mean(g * g))) if g.size else 0.0
    d = tol * np.maximum(np.abs(g), rms)
    lo, hi = g - d, g + d
    sq_max = np.maximum(lo * lo, hi * hi)
    sq_min = np.where((lo <= 0) & (hi >= 0), 0.0, np.minimum(lo * lo, hi * hi))
    r32 = 2.0 ** -22                      # a few fp32 roundings, relative
    s_lo = (s0 + m * sq_min) * (1 - m * r32)
    s_hi = (s0 + m * sq_max) * (1 + m * r32)
    bad = (got_s < s_lo) | (got_s > s_hi)
    assert not bad.any(), f"{what}: {int(bad.sum())} state elements outside the bound"

    def total_step(x):
        return sum(LR * x / (np.sqrt(s0 + k * x * x) + EPS) for k in range(1, m + 1))

    u_lo, u_hi = total_step(lo), total_step(hi)      # monotone in x: u_lo <= u_hi
    mag = np.maximum(np.abs(w0), np.abs(got_w)) + np.abs(u_lo) + np.abs(u_hi)
    if dtype == "f32":
        slack = m * (mag * 2.0 ** -23 + (np.abs(u_lo) + np.abs(u_hi)) * r32)
    else:
        # the fp32 sum is rounded once more, to bf16: a near-tie may go either way
        slack = m * (_half_ulp_bf16(mag) + mag * 2.0 ** -23) + (np.abs(u_lo) + np.abs(u_hi)) * r32
    bad = (got_w < w0 - u_hi - slack) | (got_w > w0 - u_lo + slack)
    assert not bad.any(), f"{what}: {int(bad.sum())} table elements outside the bound"


def test_fused_adagrad_identity_rows():
    """row_ids NULL: the block's source rows are the table's first rows."""
    rng = np.random.default_rng(11)
    blk = synth.random_block(rng, [600], [240], [(0, 0), (0, 0)], 10, zero_frac=0.2)
    run = BlockRun(blk, "f32", 64, 32, seed=3, use_ids=False, emb_types=[0], grad_types=[])
    run.device_setup()
    state = torch.zeros((run.tables[0].shape[0], 64), device="cuda")
    y = [torch.empty((240, 32), device="cuda")]
    rgcn.rgcn_block_plan(run.dblk, run.params, run.ws)
    rgcn.rgcn_block_forward(run.dblk, run.inputs, run.params, y, run.ws)
    rgcn.rgcn_block_backward_dense(run.dblk, run.params, [run.dy[0].cuda()], workspace=run.ws)
    rgcn.rgcn_block_backward_sparse_adagrad(run.dblk, run.inputs, run.params, [state], LR, EPS,
                                            workspace=run.ws, flags=rgcn.RGCN_IDS_UNIQUE)
    torch.cuda.synchronize()
    ref = run.run_oracle()
    _check_steps(ref["demb"][0], np.zeros((600, 64)), to64(run.tables[0]), to64(state),
                 to64(run.d_tables[0]), 1, TOL["f32"], "f32", "identity rows")


@pytest.mark.parametrize("dtype,d,n,num_rows,clear", [("f32", 36, 1500, 5000, True),
                                                      ("bf16", 264, 900, 2000, False),
                                                      ("bf16", 8, 3, 10, True),
                                                      ("f32", 128, 600_000, 1_000_000, True)])
def test_standalone_adagrad_matches_oracle(dtype, d, n, num_rows, clear):
    print(f"case standalone {dtype} d={d} n={n}", flush=True)
    gen = torch.Generator().manual_seed(n + d)
    tdt = synth.torch_dtype(dtype)
    ld = d + (8 if dtype == "bf16" else 4)        # a padded table
    table0 = torch.randn((num_rows, ld), generator=gen).to(tdt)
    grad0 = torch.randn((num_rows, d), generator=gen)
    state0 = torch.rand((num_rows, d), generator=gen)
    rows = torch.randperm(num_rows, generator=gen)[:n]
    # out-of-range rows are skipped by the kernel (and not given to the oracle)
    rows_dev = torch.cat([rows, torch.tensor([-1, num_rows, num_rows + 7])]).cuda()
    table, grad, state = table0.cuda(), grad0.cuda(), state0.cuda()
    rgcn.rgcn_sparse_adagrad(rows_dev, grad, state, table, LR, EPS,
                             flags=rgcn.RGCN_CLEAR_GRAD if clear else 0)
    torch.cuda.synchronize()
    w = to64(table0)[:, :d].copy()
    s = state0.double().numpy().copy()
    oracle.sparse_adagrad(rows.numpy(), grad0.double().numpy(), s, w, LR, EPS)
    got_w, got_s, got_g = to64(table), to64(state), to64(grad)
    assert np.array_equal(got_w[:, d:], to64(table0)[:, d:])      # padding untouched
    assert rel_err(got_s, s) <= TOL["f32"]
    _check_table(got_w[:, :d], to64(table0)[:, :d], w, dtype, TOL["f32"], "standalone")
    listed = np.zeros(num_rows, dtype=bool)
    listed[rows.numpy()] = True
    if clear:
        assert not got_g[listed].any()
    else:
        assert np.array_equal(got_g[listed], grad0.double().numpy()[listed])
    assert np.array_equal(got_g[~listed], grad0.double().numpy()[~listed])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_chain_adagrad_with_repeated_ids(dtype):
    """The chain driver declared with repeated input ids (ids_unique=False): the embedding
    gradient is scatter-added with atomics, then each distinct table row takes one step
    from the summed gradient (the fused step, which would race, is not used).  Rows named
    twice or more must have stepped on their summed gradient, rows never named keep their
    bits, and the gradient buffer is left cleared for the next step."""
    from paper_2406_06022_amd import chain

    blk, _ = _adagrad_block("mixed")
    T, R = len(blk.n_src), len(blk.rels)
    d_in, d_out = 32, 48
    tdt = synth.torch_dtype(dtype)
    gen = torch.Generator().manual_seed(71)
    rows0 = blk.n_src[0] // 2 + 5
    ids = [torch.randint(0, rows0, (blk.n_src[0],), generator=gen),      # repeats
           torch.randperm(blk.n_src[1] + 40, generator=gen)[: blk.n_src[1]]]
    assert torch.unique(ids[0]).numel() < blk.n_src[0]
    tables = [torch.randn((rows0, d_in), generator=gen).to(tdt),
              torch.randn((blk.n_src[1] + 40, d_in), generator=gen).to(tdt)]
    w_rel, w_self, _ = synth.block_weights(T, R, d_in, d_out, tdt, 19)
    dy = [torch.randn((n, d_out), generator=gen) for n in blk.n_dst]
    dev = "cuda"
    d_tables = [x.to(dev) for x in tables]
    stack = chain.MiniBatchStack([blk], d_tables, [x.to(dev) for x in ids],
                                 [([w.to(dev) for w in w_rel], [w.to(dev) for w in w_self], None)],
                                 dtype, [d_in, d_out], emb_types=[0], device=dev,
                                 ids_unique=False)
    stack.attach_adagrad(LR, EPS)
    stack.step([x.to(dev) for x in dy])
    torch.cuda.synchronize()

    h = [to64(tables[t])[ids[t].numpy()] for t in range(T)]
    g = oracle.block_backward(blk, h, [to64(w) for w in w_rel], [to64(w) for w in w_self],
                              [to64(x) for x in dy], want_dh=[True, False])
    grad = np.zeros((rows0, d_in))
    oracle.scatter_add(ids[0].numpy(), g["dh_src"][0], grad)
    rows = np.unique(ids[0].numpy())
    w0 = to64(tables[0])
    got_w = to64(d_tables[0])
    got_s = to64(stack.adagrad[2][0])
    named = np.zeros(rows0, dtype=bool)
    named[rows] = True
    assert np.array_equal(got_w[~named], w0[~named])
    assert not got_s[~named].any()
    assert not to64(stack.demb[0]).any()          # cleared by the step
    _check_steps(grad[rows], np.zeros((rows.size, d_in)), w0[rows], got_s[rows], got_w[rows], 1,
                 TOL[dtype], dtype, f"repeated ids {dtype}")
