"""rgcn_lp_loss_noalloc -- the link-prediction decoder with its temporaries in the
library's fixed per-device array instead of a caller workspace -- against rgcn_lp_loss
with a workspace, through the C ABI on the same inputs.  Two calls in a row on one device,
the second with a smaller batch (the array still holds the first call's temporaries), each
compared with the workspace entry point: scores, loss and relation gradient bit for bit
(their kernels are deterministic), the embedding gradient (fp32 atomics, order varies)
within the fp32 bar.  A batch whose temporaries exceed the array is rejected on the host
before any work."""
import numpy as np
import pytest
import torch

from harness import rel_err, to64
from paper_2406_06022_amd import rgcn, synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _batch(seed, dtype, n, d, B, k, mode):
    gen = torch.Generator().manual_seed(seed)
    tdt = synth.torch_dtype(dtype)
    emb = (torch.randn((n, d), generator=gen) * 0.5).to(tdt).to(DEV)
    rel = torch.randn(d, generator=gen).to(tdt).to(DEV)
    src = torch.randint(0, n, (B,), generator=gen, dtype=torch.int32).to(DEV)
    dst = torch.randint(0, n, (B,), generator=gen, dtype=torch.int32).to(DEV)
    if mode == rgcn.RGCN_LP_NEG_PER_EDGE:
        neg = torch.randint(0, n, (B * k,), generator=gen, dtype=torch.int32).to(DEV)
    elif mode == rgcn.RGCN_LP_NEG_JOINT:
        neg = torch.randint(0, n, (((B + k - 1) // k) * k,), generator=gen,
                            dtype=torch.int32).to(DEV)
    else:
        neg = None
    w = (torch.rand(B, generator=gen) * 2.0 + 0.25).to(DEV)
    return emb, rel, src, dst, neg, w


def _outputs(B, nn, n, d):
    return (torch.full((1,), float("nan"), device=DEV),
            torch.full((B,), float("nan"), device=DEV),
            torch.full((max(B * nn, 1),), float("nan"), device=DEV),
            torch.zeros((n, d), device=DEV),
            torch.full((d,), float("nan"), device=DEV))


CASES = [  # (seed, dtype, rows, d, B, k, negative mode, loss): the second is smaller
    (1, "bf16", 5000, 256, 1024, 0, rgcn.RGCN_LP_NEG_IN_BATCH, rgcn.RGCN_LP_CONTRASTIVE),
    (2, "f32", 300, 40, 37, 5, rgcn.RGCN_LP_NEG_JOINT, rgcn.RGCN_LP_WEIGHTED_CE),
]


def test_noalloc_matches_workspace_entry_point():
    for seed, dtype, n, d, B, k, mode, kind in CASES:
        print(f"case noalloc {dtype} rows {n} d {d} B {B} k {k} mode {mode} loss {kind}",
              flush=True)
        emb, rel, src, dst, neg, w = _batch(seed, dtype, n, d, B, k, mode)
        nn = B - 1 if mode == rgcn.RGCN_LP_NEG_IN_BATCH else k
        b = rgcn.lp_batch(emb, rel, mode, kind, src, dst, k, neg, w)
        assert rgcn.rgcn_lp_workspace_size(b) <= rgcn.RGCN_LP_NOALLOC_MAX_SCRATCH
        ws = torch.full((rgcn.rgcn_lp_workspace_size(b),), 0xFF, dtype=torch.uint8, device=DEV)
        want = _outputs(B, nn, n, d)
        rgcn.rgcn_lp_loss(b, *want, workspace=ws)
        got = _outputs(B, nn, n, d)
        rgcn.rgcn_lp_loss_noalloc(b, *got)
        torch.cuda.synchronize()
        for name, g, x in zip(("loss", "pos_score", "neg_score", "d_rel"),
                              (got[0], got[1], got[2], got[4]), (want[0], want[1], want[2], want[4])):
            assert not torch.isnan(x[: B * nn if name == "neg_score" else x.numel()]).any(), name
            assert torch.equal(g, x) or (name == "neg_score" and nn == 0), name
        assert rel_err(to64(got[3]), to64(want[3])) <= 1e-5


def test_noalloc_rejects_a_batch_above_the_array():
    emb, rel, src, dst, neg, w = _batch(3, "bf16", 100_000, 512, 65536, 32,
                                        rgcn.RGCN_LP_NEG_PER_EDGE)
    b = rgcn.lp_batch(emb, rel, rgcn.RGCN_LP_NEG_PER_EDGE, rgcn.RGCN_LP_CONTRASTIVE, src, dst,
                      32, neg)
    assert rgcn.rgcn_lp_workspace_size(b) > rgcn.RGCN_LP_NOALLOC_MAX_SCRATCH
    loss = torch.zeros(1, device=DEV)
    with pytest.raises(rgcn.RgcnError) as e:
        rgcn.rgcn_lp_loss_noalloc(b, loss)
    assert e.value.status == 7
    assert "scratch" in rgcn.rgcn_last_error()
