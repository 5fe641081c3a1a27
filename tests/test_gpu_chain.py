"""Multi-layer mini-batch through the chain driver the benchmark uses, against the oracle
applied layer by layer (ReLU between layers, last layer linear, backward from the top).

ReLU's derivative is a decision taken on a floating-point value, so both sides must see
the same sign at every pre-activation.  Each layer gets a bias of +c or -c per output
column (seeded signs) with c = 1.5 * 2^k and 2^k above twice the largest |pre-activation|
z the oracle computes without bias: every pre-activation is then at least 2^k away from
zero and its sign is the bias's, on both sides; the positive ones stay inside the binade
[2^k, 2^(k+1)), so their rounding to the block dtype has one spacing.  c is exact in bf16.  The oracle computes c, so no expected value comes
from the GPU.  Between layers the oracle stores each block's output in the block dtype
(round to nearest even), as the block's output is defined; inside a block it keeps fp64.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2406_06022_amd import chain, rgcn, synth
from tests.harness import TOL, rel_err, to64

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _margin_biases(blocks, h0, w64, T, seed, quant):
    """Per-layer biases (fp64 lists per type, exact in the block dtype via ``quant``) and the
    oracle's forward outputs."""
    rng = np.random.default_rng(seed)
    h = h0
    biases, ys = [], []
    L = len(blocks)
    for l, blk in enumerate(blocks):
        w_rel, w_self = w64[l]
        z = oracle.block_forward(blk, h, w_rel, w_self)
        d_out = w_self[0].shape[1]
        if l < L - 1:
            zmax = max((np.abs(x).max() for x in z if x is not None and x.size), default=1.0)
            c = 1.5 * 2.0 ** math.ceil(math.log2(2.0 * zmax + 1.0))
            sign = np.where(rng.random(d_out) < 0.5, -1.0, 1.0)
            b = [c * sign for _ in range(T)]
        else:
            b = [quant(rng.uniform(-0.5, 0.5, d_out)) for _ in range(T)]
        y = oracle.block_forward(blk, h, w_rel, w_self, b, relu=l < L - 1)
        if l < L - 1:
            # a block's output is stored in the block dtype and is the next block's input
            y = [quant(x) if x is not None else None for x in y]
        biases.append(b)
        ys.append(y)
        h = [y[t] if y[t] is not None else np.zeros((0, d_out)) for t in range(T)]
    return biases, ys


@pytest.mark.parametrize("index", [1, 2, 4])
def test_chain_matches_layerwise_oracle(index):
    spec = synth.small_config(index)
    mb = synth.sample_minibatch(spec)
    T, R, L = len(spec.ntype_names), len(spec.rels), spec.num_layers
    tdt = synth.torch_dtype(spec.dtype)
    emb = [t for t in range(T) if spec.featureless[t]]
    tables = [synth.normal_table(spec.type_rows[t], spec.dims[0], tdt, 300 + t) for t in range(T)]
    ids = [torch.as_tensor(mb.input_ids[t]) for t in range(T)]
    w = [synth.block_weights(T, R, spec.dims[l], spec.dims[l + 1], tdt, 40 + l)[:2]
         for l in range(L)]
    w64 = [([to64(x) for x in wr], [to64(x) for x in wsf]) for wr, wsf in w]
    h0 = [to64(tables[t])[mb.input_ids[t]] for t in range(T)]
    def quant(x):
        return to64(torch.as_tensor(x).to(tdt))

    biases, ys = _margin_biases(mb.blocks, h0, w64, T, 77 + index, quant)
    b_dev = [[torch.as_tensor(b[t]).to(tdt) for t in range(T)] for b in biases]
    for l in range(L):  # every bias is exact in the block dtype
        for t in range(T):
            assert np.array_equal(to64(b_dev[l][t]), biases[l][t])

    gen = torch.Generator().manual_seed(90 + index)
    top = mb.blocks[-1]
    dy_top = [torch.randn((n, spec.dims[-1]), generator=gen) for n in top.n_dst]

    # ---- GPU through the chain driver
    weights = [([x.to(DEV) for x in w[l][0]], [x.to(DEV) for x in w[l][1]],
                [x.to(DEV) for x in b_dev[l]]) for l in range(L)]
    stack = chain.MiniBatchStack(mb.blocks, [x.to(DEV) for x in tables],
                                 [x.to(DEV) for x in ids], weights, spec.dtype, spec.dims,
                                 emb_types=emb, device=DEV)
    stack.step([x.to(DEV) if x.numel() else None for x in dy_top])
    torch.cuda.synchronize()

    # ---- oracle, layer by layer from the top
    hs = [h0] + [[ys[l][t] if ys[l][t] is not None else np.zeros((0, spec.dims[l + 1]))
                  for t in range(T)] for l in range(L - 1)]
    dy = [to64(x) for x in dy_top]
    grads = [None] * L
    for l in reversed(range(L)):
        blk = mb.blocks[l]
        want = [(t in emb) if l == 0 else blk.n_src[t] > 0 for t in range(T)]
        g = oracle.block_backward(blk, hs[l], w64[l][0], w64[l][1], dy, input_relu=l > 0,
                                  want_dh=want)
        grads[l] = g
        dy = [g["dh_src"][t] if g["dh_src"][t] is not None else np.zeros((0, spec.dims[l]))
              for t in range(T)]
    demb_ref = {}
    for t in emb:
        d = np.zeros((spec.type_rows[t], spec.dims[0]))
        oracle.scatter_add(mb.input_ids[t], grads[0]["dh_src"][t], d)
        demb_ref[t] = d

    tol = TOL[spec.dtype]
    errs = {}
    for t in range(T):
        if top.n_dst[t] > 0:
            errs[f"y_top[{t}]"] = rel_err(to64(stack.y[-1][t]), ys[-1][t])
    for l in range(L):
        for r in range(R):
            errs[f"dw_rel[{l}][{r}]"] = rel_err(to64(stack.dw_rel[l][r]), grads[l]["dw_rel"][r])
        for t in range(T):
            errs[f"dw_self[{l}][{t}]"] = rel_err(to64(stack.dw_self[l][t]), grads[l]["dw_self"][t])
            errs[f"dbias[{l}][{t}]"] = rel_err(to64(stack.dbias[l][t]), grads[l]["dbias"][t])
    for t in emb:
        errs[f"demb[{t}]"] = rel_err(to64(stack.demb[t]), demb_ref[t])
    bad = {k: v for k, v in errs.items() if not v <= tol}
    print(f"[chain] {spec.name}: worst {max(errs.values()):.3g} ({max(errs, key=errs.get)})")
    assert not bad, f"chain parity failures (tol {tol}): {bad}"


def poison_stack(stack):
    """Fill every workspace with 0xFF bytes (NaN in fp32 and bf16, -1 as int32) and every
    output buffer with NaN, so that nothing a step reads before writing survives from an
    earlier step."""
    for ws in stack.workspaces:
        ws.fill_(0xFF)
    for l in range(stack.L):
        for x in stack.y[l]:
            if x is not None:
                x.fill_(float("nan"))
        for grp in (stack.dw_rel[l], stack.dw_self[l], stack.dbias[l]):
            for x in grp or []:
                if x is not None:
                    x.fill_(float("nan"))
        if stack.dh[l] is not None:
            for x in stack.dh[l]:
                if x is not None:
                    x.fill_(float("nan"))


def step_outputs(stack, emb):
    out = [x.clone() for x in stack.y[-1] if x is not None]
    for l in range(stack.L):
        out += [x.clone() for x in stack.dw_rel[l]] + [x.clone() for x in stack.dw_self[l]]
        if stack.dh[l] is not None:
            out += [x.clone() for x in stack.dh[l] if x is not None]
    out += [stack.demb[t].clone() for t in emb]
    return out


@pytest.mark.parametrize("index", [1, 2, 4])
def test_overlapped_plan_matches_serial_step(index):
    """The step with the backward half of the plan on a second stream (from the end of the
    first aggregate stage) gives bit-identical outputs and gradients to the serial order.
    Every step starts from poisoned workspaces and outputs, and the overlapped step runs
    first, so a backward that read a transpose or schedule the side stream had not yet
    written (a missing wait, a plan part skipped) would show."""
    spec = synth.small_config(index)
    mb = synth.sample_minibatch(spec)
    T, R, L = len(spec.ntype_names), len(spec.rels), spec.num_layers
    tdt = synth.torch_dtype(spec.dtype)
    emb = [t for t in range(T) if spec.featureless[t]]
    tables = [synth.normal_table(spec.type_rows[t], spec.dims[0], tdt, 500 + t).to(DEV)
              for t in range(T)]
    ids = [torch.as_tensor(mb.input_ids[t]).to(DEV) for t in range(T)]
    weights = []
    for l in range(L):
        w_rel, w_self, _ = synth.block_weights(T, R, spec.dims[l], spec.dims[l + 1], tdt, 60 + l)
        weights.append(([x.to(DEV) for x in w_rel], [x.to(DEV) for x in w_self], None))
    stack = chain.MiniBatchStack(mb.blocks, tables, ids, weights, spec.dtype, spec.dims,
                                 emb_types=emb, device=DEV)
    gen = torch.Generator().manual_seed(95 + index)
    dy = [torch.randn((n, spec.dims[-1]), generator=gen).to(DEV) if n else None
          for n in mb.blocks[-1].n_dst]

    def run(overlap):
        poison_stack(stack)
        for t in emb:
            stack.demb[t].zero_()
        stack.step(dy, overlap_plan=overlap)
        torch.cuda.synchronize()
        return step_outputs(stack, emb)

    first = run(True)
    want = run(False)
    second = run(True)
    for rep, got in enumerate((first, second)):
        assert len(got) == len(want)
        for i, (g, w_) in enumerate(zip(got, want)):
            assert not torch.isnan(w_).any(), f"serial output {i} left unwritten"
            assert torch.equal(g, w_), f"overlapped step {rep}: output {i} differs"


@pytest.mark.parametrize("index", [1, 2, 4])
def test_hilo_gradients_between_blocks_match_fp32(index):
    """The chain with the gradients between bf16 blocks in the hi/lo form (the default) and
    with them in fp32 (hilo_grads=False): the forward and the top block's weight gradients
    bit for bit (the same operands reach the same kernels).  Below the top the results
    differ at fp32 rounding: a hidden block's input side adds its hi and lo sums in
    another order when the rows come in the hi/lo form (the persistent product), so its
    input gradient differs in the last bits, which now and then moves the bf16 rounding of
    a low part (2^-16 of the element) in the next block's operands; bias sums of hi + lo
    differ from fp32 sums by at most 2^-16 of each term.  Through a block whose sums
    cancel (the embedding gradient is judged per touched element) that reaches about 1e-4,
    so the bar below the top is 1e-3, twenty times under the oracle's bf16 bar; a wrong
    form anywhere (hi/lo bytes read as fp32, or the reverse) is off by order one."""
    spec = synth.small_config(index)
    assert spec.dtype == "bf16"
    mb = synth.sample_minibatch(spec)
    T, R, L = len(spec.ntype_names), len(spec.rels), spec.num_layers
    tdt = synth.torch_dtype(spec.dtype)
    emb = [t for t in range(T) if spec.featureless[t]]
    tables = [synth.normal_table(spec.type_rows[t], spec.dims[0], tdt, 700 + t).to(DEV)
              for t in range(T)]
    ids = [torch.as_tensor(mb.input_ids[t]).to(DEV) for t in range(T)]
    weights = []
    for l in range(L):
        w_rel, w_self, b = synth.block_weights(T, R, spec.dims[l], spec.dims[l + 1], tdt,
                                               80 + l, with_bias=True)
        weights.append(([x.to(DEV) for x in w_rel], [x.to(DEV) for x in w_self],
                        [x.to(DEV) for x in b]))
    gen = torch.Generator().manual_seed(170 + index)
    dy = [torch.randn((n, spec.dims[-1]), generator=gen).to(DEV) if n else None
          for n in mb.blocks[-1].n_dst]
    outs = []
    for hilo in (True, False):
        stack = chain.MiniBatchStack(mb.blocks, tables, ids, weights, spec.dtype, spec.dims,
                                     emb_types=emb, device=DEV, hilo_grads=hilo)
        assert stack.hilo_grads == hilo
        stack.step(dy)
        torch.cuda.synchronize()
        outs.append(stack)
    h, f = outs
    for t, (a, b) in enumerate(zip(h.y[-1], f.y[-1])):
        if a is not None:
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), f"y[{t}]"
    errs = {}
    for l in range(L):
        pairs = [(f"dw_rel[{l}][{r}]", h.dw_rel[l][r], f.dw_rel[l][r]) for r in range(R)]
        pairs += [(f"dw_self[{l}][{t}]", h.dw_self[l][t], f.dw_self[l][t]) for t in range(T)]
        pairs += [(f"dbias[{l}][{t}]", h.dbias[l][t], f.dbias[l][t]) for t in range(T)
                  if h.dbias[l][t] is not None]
        for name, a, b in pairs:
            if l == L - 1 and not name.startswith("dbias"):
                assert torch.equal(a.view(torch.int32), b.view(torch.int32)), name
            errs[name] = rel_err(to64(a), to64(b))
    for t in emb:
        errs[f"demb[{t}]"] = rel_err(to64(h.demb[t]), to64(f.demb[t]))
    bad = {k: v for k, v in errs.items() if not v <= 1e-3}
    print(f"[chain hilo] {spec.name}: worst {max(errs.values()):.3g} ({max(errs, key=errs.get)})",
          flush=True)
    assert not bad, f"hi/lo vs fp32 gradients between blocks: {bad}"
