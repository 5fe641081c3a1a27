"""Link-prediction decoder on the GPU vs the oracle: scores, loss and gradients for the
three negative modes x three losses x dot / DistMult, fp32 and bf16 embeddings (decoded
exactly, so both sides see the same values), ragged widths and batches; a paper-sized
in-batch batch and a large per-edge batch; negative ids bit for bit; device validation.

The GPU computes in fp32 from the same inputs.  Scores and the loss are held to the fp32
bar of the harness metric (max |got - want| / max(|want|, rms(want)) <= 1e-5; the loss
relatively).

Gradients are held per element to the fp32 bar plus the propagated score error.  A d-term
fp32 dot product (DistMult: a product of three factors) errs by at most
ds_e = (d + 2) 2^-24 sum_c |a_c v_c| on scored edge e.  The loss derivative g_e = dL/ds_e
is a sigmoid (cross entropy) or softmax (contrastive) weight, so that absolute score error
becomes an error of g_e: |dg_e| <= w_e / N * max sigma'(s) ds_e over the score interval for
cross entropy, and <= p_e (exp(ds_e + max_f ds_f) - 1) / B for the softmax over a positive's
scores, plus the fp32 rounding of exp and the normaliser.  Each gradient element is a sum
of g_e times another row's element, so its error bound is
    1e-5 max(|want|, rms(want)) + sum_e (|dg_e| + 2^-23 |g_e|) |x_e[c]|
with x_e the row the derivative multiplies (rel * h_v or h_v for the source row, u_i for
the destination row; h_src * h_v for the relation vector).  Everything in the bound comes
from the inputs and the oracle's fp64 scores."""
import numpy as np
import pytest
import scipy.sparse as sp
import torch

import oracle
from harness import rel_err, to64
from paper_2406_06022_amd import rgcn, synth

pytestmark = pytest.mark.gpu

TOL = 1e-5
U32 = 2.0 ** -24


def _scored_edges(mode, B, k, src, dst, neg):
    """(positive index, scored row, label) of every scored edge: the B positives, then each
    positive's negatives in order."""
    nn = (B - 1 if B > 0 else 0) if mode == rgcn.RGCN_LP_NEG_IN_BATCH else k
    i = np.repeat(np.arange(B), nn)
    kk = np.tile(np.arange(nn), B)
    if mode == rgcn.RGCN_LP_NEG_PER_EDGE:
        v = neg[i * k + kk]
    elif mode == rgcn.RGCN_LP_NEG_JOINT:
        v = neg[(i // k) * k + kk]
    else:
        v = dst[np.where(kk < i, kk, kk + 1)]
    ii = np.concatenate([np.arange(B), i])
    vv = np.concatenate([dst, v])
    lab = np.concatenate([np.ones(B), np.zeros(i.size)])
    return ii, vv, lab, nn


def _grad_bounds(emb, rel, mode, kind, src, dst, k, neg, w, ref):
    """Per-element error bounds of d_emb and d_rel beyond the fp32 bar: the score error of
    every scored edge carried through the loss derivative (see the module docstring)."""
    n, d = emb.shape
    B = src.size
    ii, vv, lab, nn = _scored_edges(mode, B, k, src, dst, neg)
    s = np.concatenate([ref["pos_score"], ref["neg_score"].ravel()])
    r = rel if rel is not None else np.ones(d)
    a = emb[src] * r                                   # u_i
    absdot = np.einsum("ec,ec->e", np.abs(a[ii]), np.abs(emb[vv])) if ii.size else np.zeros(0)
    ds = (d + 2) * U32 * absdot
    if kind == rgcn.RGCN_LP_CONTRASTIVE:
        S = np.concatenate([ref["pos_score"][:, None], ref["neg_score"].reshape(B, nn)], axis=1)
        DS = np.concatenate([ds[:B, None], ds[B:].reshape(B, nn)], axis=1)
        m = S.max(axis=1, keepdims=True)
        p = np.exp(S - m)
        p /= p.sum(axis=1, keepdims=True)
        Y = np.zeros_like(S)
        Y[:, 0] = 1.0
        g = (p - Y) / B
        dg = (p * np.expm1(DS + DS.max(axis=1, keepdims=True)) +
              p * U32 * (2.0 * np.abs(S - m) + nn + 8) + U32) / B
        g = np.concatenate([g[:, 0], g[:, 1:].ravel()])
        dg = np.concatenate([dg[:, 0], dg[:, 1:].ravel()])
    else:
        wt = np.ones_like(s)
        if kind == rgcn.RGCN_LP_WEIGHTED_CE:
            wt[:B] = w
        N = s.size
        sig = 1.0 / (1.0 + np.exp(-s))
        g = wt * (sig - lab) / N
        smin = np.maximum(np.abs(s) - ds, 0.0)
        dsig = np.exp(-smin) / (1.0 + np.exp(-smin)) ** 2
        dg = wt / N * (dsig * ds + 8 * U32)
    c = dg + 2 * U32 * np.abs(g)
    y_abs = np.abs(emb * r)                            # rel * h_v (or h_v): source side
    s1 = sp.coo_matrix((c, (src[ii], vv)), shape=(n, n)).tocsr()
    s2 = sp.coo_matrix((c, (vv, ii)), shape=(n, B)).tocsr()
    p_emb = s1 @ y_abs + s2 @ np.abs(a)
    p_rel = None
    if rel is not None:
        s3 = sp.coo_matrix((c, (ii, vv)), shape=(B, n)).tocsr()
        p_rel = (np.abs(emb[src]) * (s3 @ np.abs(emb))).sum(axis=0)
    return p_emb, p_rel


def _within(got, want, extra, what):
    rms = float(np.sqrt(np.mean(want * want))) if want.size else 0.0
    bound = TOL * np.maximum(np.abs(want), rms) + extra
    over = np.abs(got - want) - bound
    assert not (over > 0).any(), (f"{what}: {int((over > 0).sum())} elements over the derived "
                                  f"bound, worst excess {float(over.max()):.3g}")


def _case(seed, dtype, n, d, B, k, mode):
    gen = torch.Generator().manual_seed(seed)
    tdt = synth.torch_dtype(dtype)
    emb = (torch.randn((n, d), generator=gen) * 0.5).to(tdt)
    rel = torch.randn(d, generator=gen).to(tdt)
    src = torch.randint(0, n, (B,), generator=gen, dtype=torch.int32)
    dst = torch.randint(0, n, (B,), generator=gen, dtype=torch.int32)
    if mode == rgcn.RGCN_LP_NEG_PER_EDGE:
        neg = torch.randint(0, n, (B * k,), generator=gen, dtype=torch.int32)
    elif mode == rgcn.RGCN_LP_NEG_JOINT:
        neg = torch.randint(0, n, (((B + k - 1) // k) * k,), generator=gen, dtype=torch.int32)
    else:
        neg = None
    w = torch.rand(B, generator=gen) * 2.0 + 0.25
    return emb, rel, src, dst, neg, w


def _run(emb, rel, mode, kind, src, dst, k, neg, w, d_rel=True):
    dev = "cuda"
    e, r = emb.to(dev), (rel.to(dev) if rel is not None else None)
    s_, d_ = src.to(dev), dst.to(dev)
    n_ = neg.to(dev) if neg is not None else None
    w_ = w.to(dev)
    B = src.numel()
    nn = B - 1 if mode == rgcn.RGCN_LP_NEG_IN_BATCH else k
    b = rgcn.lp_batch(e, r, mode, kind, s_, d_, k, n_, w_)
    loss = torch.full((1,), float("nan"), device=dev)
    pos = torch.full((B,), float("nan"), device=dev)
    negs = torch.full((max(B * nn, 1),), float("nan"), device=dev)
    d_emb = torch.zeros((emb.shape[0], emb.shape[1]), device=dev)
    d_r = torch.full((emb.shape[1],), float("nan"), device=dev) if (r is not None and d_rel) else None
    rgcn.rgcn_lp_loss(b, loss, pos, negs, d_emb, d_r)
    torch.cuda.synchronize()
    return (float(loss.item()), to64(pos), to64(negs)[: B * nn].reshape(B, nn), to64(d_emb),
            to64(d_r) if d_r is not None else None)


def _check(got, emb, rel, mode, kind, src, dst, k, neg, w):
    e64, r64 = to64(emb), (to64(rel) if rel is not None else None)
    s_, d_ = src.numpy().astype(np.int64), dst.numpy().astype(np.int64)
    n_ = neg.numpy().astype(np.int64) if neg is not None else None
    ref = oracle.lp_loss(e64, r64, mode, kind, s_, d_, k, n_, to64(w))
    assert got[0] == pytest.approx(ref["loss"], rel=TOL, abs=1e-7)
    assert rel_err(got[1], ref["pos_score"]) <= TOL
    assert rel_err(got[2], ref["neg_score"]) <= TOL
    p_emb, p_rel = _grad_bounds(e64, r64, mode, kind, s_, d_, k, n_, to64(w), ref)
    _within(got[3], ref["d_emb"], p_emb, "d_emb")
    if rel is not None:
        _within(got[4], ref["d_rel"], p_rel, "d_rel")


@pytest.mark.parametrize("mode", [0, 1, 2])
@pytest.mark.parametrize("kind", [0, 1, 2])
@pytest.mark.parametrize("dtype,d", [("f32", 40), ("bf16", 264)])
@pytest.mark.parametrize("distmult", [False, True])
def test_decoder_matches_oracle(mode, kind, dtype, d, distmult):
    emb, rel, src, dst, neg, w = _case(mode * 9 + kind * 3 + d, dtype, 300, d, 37, 5, mode)
    rel = rel if distmult else None
    print(f"case lp mode={mode} loss={kind} {dtype} d={d} distmult={distmult}", flush=True)
    got = _run(emb, rel, mode, kind, src, dst, 5, neg, w)
    _check(got, emb, rel, mode, kind, src, dst, 5, neg, w)


@pytest.mark.parametrize("dtype,d", [("bf16", 1032), ("f32", 1024), ("bf16", 8)])
def test_wide_and_narrow_rows(dtype, d):
    emb, rel, src, dst, neg, w = _case(d, dtype, 200, d, 19, 3, rgcn.RGCN_LP_NEG_JOINT)
    got = _run(emb, rel, rgcn.RGCN_LP_NEG_JOINT, rgcn.RGCN_LP_CONTRASTIVE, src, dst, 3, neg, w)
    _check(got, emb, rel, rgcn.RGCN_LP_NEG_JOINT, rgcn.RGCN_LP_CONTRASTIVE, src, dst, 3, neg, w)


def test_paper_sized_in_batch_and_joint():
    """Local batch of 1,024 positives (the paper's link-prediction runs), d = 256 bf16:
    in-batch (1,023 negatives each) and joint-32, contrastive and cross entropy."""
    for mode, k in ((rgcn.RGCN_LP_NEG_IN_BATCH, 0), (rgcn.RGCN_LP_NEG_JOINT, 32)):
        for kind in (rgcn.RGCN_LP_CONTRASTIVE, rgcn.RGCN_LP_CE):
            emb, rel, src, dst, neg, w = _case(40 + mode + kind, "bf16", 5000, 256, 1024, k, mode)
            print(f"case lp paper mode={mode} loss={kind}", flush=True)
            got = _run(emb, rel, mode, kind, src, dst, k, neg, w)
            _check(got, emb, rel, mode, kind, src, dst, k, neg, w)


def test_large_per_edge_batch():
    """65,536 positives x 32 negatives over a 1M-row table, d = 256 bf16 (the benchmark's
    gather-bound shape), DistMult, contrastive."""
    emb, rel, src, dst, neg, w = _case(5, "bf16", 1_000_000, 256, 65536, 32, 0)
    got = _run(emb, rel, 0, rgcn.RGCN_LP_CONTRASTIVE, src, dst, 32, neg, w)
    _check(got, emb, rel, 0, rgcn.RGCN_LP_CONTRASTIVE, src, dst, 32, neg, w)


def test_edge_cases():
    # a single positive in-batch has no negatives; an empty batch has loss 0
    emb, rel, src, dst, neg, w = _case(3, "f32", 50, 16, 1, 0, 2)
    got = _run(emb, rel, 2, rgcn.RGCN_LP_CONTRASTIVE, src, dst, 0, None, w)
    _check(got, emb, rel, 2, rgcn.RGCN_LP_CONTRASTIVE, src, dst, 0, None, w)
    e = torch.zeros((4, 16), device="cuda")
    z = torch.zeros(0, dtype=torch.int32, device="cuda")
    b = rgcn.lp_batch(e, None, 0, 0, z, z, 2, z)
    loss = torch.full((1,), float("nan"), device="cuda")
    rgcn.rgcn_lp_loss(b, loss)
    assert loss.item() == 0.0


@pytest.mark.parametrize("mode,slots", [(0, 1000), (1, 37), (0, 3)])
def test_negative_ids_bit_exact(mode, slots):
    out = torch.full((slots,), -1, dtype=torch.int64, device="cuda")
    rgcn.rgcn_lp_negatives(mode, slots, 123457, 99, out)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy(), oracle.lp_negatives(mode, slots, 123457, 99))


def test_out_of_range_rows_reported():
    emb, rel, src, dst, neg, w = _case(8, "f32", 50, 16, 10, 2, 0)
    neg[5] = 50
    e = emb.cuda()
    b = rgcn.lp_batch(e, None, 0, 0, src.cuda(), dst.cuda(), 2, neg.cuda())
    loss = torch.zeros(1, device="cuda")
    with pytest.raises(rgcn.RgcnError) as ex:
        rgcn.rgcn_lp_loss(b, loss, flags=rgcn.RGCN_VALIDATE_DEVICE)
    assert ex.value.status == 4
