"""The hi/lo gradient form of the bf16 backward, through the C ABI.

A bf16 block's backward products take an fp32 output gradient as two bf16 operands,
hi = bf16(g) and lo = bf16(g - hi).  With RGCN_DY_HILO the dense stage reads dy already in
that form (per row d_out high parts, then d_out low parts); with RGCN_DH_HILO the sparse
stage writes the input gradient in it.  Against the same block run on fp32 gradients:

- y and the weight gradients are bit for bit the same (the weight-side product sees the
  same bf16 operands in the same order);
- the input-side products see the same operands too; where d_in is a multiple of 64 and
  more than 128 columns take gradients, the hi/lo rows go through the persistent product
  as one bf16 row of 2 d_out values, so the hi and lo sums are added in another order:
  embedding gradients agree to the fp32 bar, and dh, decoded, to that plus the form's
  2^-16 relative representation bound; elsewhere dh is bit for bit the host's split of the
  fp32 result (both round to nearest even);
- the bias gradient is the column sum of hi + lo, at the fp32 summation bar against an
  fp64 sum of those values;
- everything, dh decoded, is at the oracle's bf16 bar.

The cases reach every kernel that reads or writes the form: the persistent, the
register-staged and the streamed input-side products (narrow gradient slots at d_out 256
and 512), the weight gradient, the bias sums, and the transposed sum at one, two and four
chunks per lane, with and without the ReLU sign bits, and its split path for hub rows.
"""
import numpy as np
import pytest
import torch

from harness import BlockRun, TOL, hilo_decode, hilo_split, rel_err, to64
from paper_2406_06022_amd import rgcn, synth

pytestmark = pytest.mark.gpu

HILO = rgcn.RGCN_DY_HILO | rgcn.RGCN_DH_HILO
# decoded hi/lo rows against the fp32 run: 2^-16 of the form plus fp32 reassociation
TOL_FORM = 2.5e-5


def _bits(x: torch.Tensor) -> torch.Tensor:
    return x.contiguous().view(torch.int16 if x.element_size() == 2 else torch.int32)


def _persistent_input_side(run: BlockRun) -> bool:
    """Whether some destination type's input side takes the persistent product."""
    blk = run.blk
    want = set(run.grad_types) | set(run.emb_types)
    for t in range(len(blk.n_dst)):
        if blk.n_dst[t] == 0:
            continue
        slots = (t in want) + sum(1 for r in blk.rels if r.dst_type == t and r.src_type in want)
        if run.d_in % 64 == 0 and slots * run.d_in > 128:
            return True
    return False


def _check_against_fp32_gradients(run: BlockRun) -> None:
    ref = run.run_gpu()[0]
    got = run.run_gpu(hilo_flags=HILO)[0]
    exact = not _persistent_input_side(run)
    for key in ("y", "dw_rel", "dw_self") + (("demb",) if exact else ()):
        for i, (a, b) in enumerate(zip(ref[key], got[key])):
            if a is not None:
                assert torch.equal(_bits(a), _bits(b)), f"{key}[{i}] differs from the fp32 run"
    if not exact:
        for t, a in enumerate(ref["demb"]):
            if a is not None:
                err = rel_err(to64(got["demb"][t]), to64(a))
                assert err <= TOL["f32"], f"demb[{t}]: {err:.3g} against the fp32 run"
    for t, x in enumerate(ref["dh"]):
        if x is None:
            continue
        if exact:
            assert torch.equal(_bits(got["dh"][t]), _bits(hilo_split(x))), \
                f"dh[{t}] is not the split of the fp32 result"
        else:
            err = rel_err(hilo_decode(got["dh"][t]), to64(x))
            assert err <= TOL_FORM, f"dh[{t}]: {err:.3g} against the fp32 run"
    for t, b in enumerate(got["dbias"]):
        if b is not None:
            want = hilo_decode(hilo_split(run.dy[t])).sum(axis=0)
            err = rel_err(to64(b), want)
            assert err <= TOL["f32"], f"dbias[{t}]: {err:.3g} against the sum of hi + lo"
    # the oracle's bar, dh decoded
    run.gpu = dict(got)
    run.gpu["dh"] = [torch.from_numpy(hilo_decode(x)) if x is not None else None
                     for x in got["dh"]]
    run.run_oracle()
    run.assert_parity()


# (192, 136) and (64, 520) take the persistent input side with a part-filled last column
# tile and a K of 2 d_out that ends inside a K step, the hi/lo boundary inside a step
@pytest.mark.parametrize("d_in,d_out", [(128, 256), (24, 40), (512, 128), (264, 40), (64, 64),
                                        (192, 136), (64, 520)])
@pytest.mark.parametrize("relu", ["none", "rows", "bits"])
def test_hilo_gradients_random_blocks(d_in, d_out, relu):
    rng = np.random.default_rng(d_in * 3 + d_out)
    blk = synth.random_block(rng, [900, 333, 260], [517, 100, 0],
                             [(0, 1), (1, 0), (0, 0), (2, 0), (2, 1)], 11, zero_frac=0.2)
    print(f"case hilo {d_in}->{d_out} relu {relu}", flush=True)
    run = BlockRun(blk, "bf16", d_in, d_out, seed=d_in + d_out, use_ids=True, bias=True,
                   input_relu=relu != "none", mask_in=relu == "bits", emb_types=(2,),
                   grad_types=(0, 1))
    _check_against_fp32_gradients(run)


@pytest.mark.parametrize("d_in,d_out,n0,n1,k", [(128, 512, 2_500, 2_500, 1),
                                                (32, 512, 25_001, 25_000, 4),
                                                (64, 256, 40_000, 3_000, 2),
                                                (96, 256, 2_500, 2_500, 1)])
def test_hilo_streamed_input_side(d_in, d_out, n0, n1, k):
    rng = np.random.default_rng(d_in * 7 + d_out + k)
    rels = [(0, 1)] * k + [(1, 0), (1, 1)]
    blk = synth.random_block(rng, [n0 + 40, n1 + n1 // 3 + 5], [n0, n1], rels, 6, zero_frac=0.3)
    print(f"case hilo streamed {d_in}->{d_out} rows {n0}, {n1} slots {k}", flush=True)
    run = BlockRun(blk, "bf16", d_in, d_out, seed=d_out + k, use_ids=True, grad_types=(0,),
                   bias=True)
    _check_against_fp32_gradients(run)


@pytest.mark.parametrize("d_in,d_out", [(128, 64), (264, 40)])
def test_hilo_split_hub_rows(d_in, d_out):
    rng = np.random.default_rng(d_in + d_out + 1)
    blk = synth.random_block(rng, [6000, 900], [2000, 700], [(0, 0), (0, 1), (1, 0), (0, 0)], 6)
    blk = synth.with_hub_sources(rng, blk, 0, [129, 256, 257, 1000, 3000])
    print(f"case hilo hubs {d_in}->{d_out}", flush=True)
    run = BlockRun(blk, "bf16", d_in, d_out, seed=17, use_ids=True, input_relu=True,
                   grad_types=(0, 1))
    _check_against_fp32_gradients(run)


@pytest.mark.parametrize("flag", [rgcn.RGCN_DY_HILO, rgcn.RGCN_DH_HILO])
def test_hilo_flags_need_bf16(flag):
    rng = np.random.default_rng(5)
    blk = synth.random_block(rng, [100], [60], [(0, 0)], 5)
    run = BlockRun(blk, "f32", 16, 16, seed=3)
    with pytest.raises(rgcn.RgcnError) as e:
        run.run_gpu(hilo_flags=flag)
    assert e.value.status == 7
