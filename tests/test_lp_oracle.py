"""Pins of the link-prediction oracle (CPU): its losses against torch's library losses on
the same scores, its gradients against torch autograd and central differences, the
negative enumeration against the paper's worked in-batch example, and the negative-id
stream against numpy's Philox."""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "in_batch_negatives.json")
M64 = (1 << 64) - 1


def _batch(seed, n=40, d=6, B=8, k=4, mode=oracle.NEG_PER_EDGE):
    rng = np.random.default_rng(seed)
    emb = rng.standard_normal((n, d))
    rel = rng.standard_normal(d)
    src = rng.integers(0, n, B)
    dst = rng.integers(0, n, B)
    if mode == oracle.NEG_PER_EDGE:
        neg = rng.integers(0, n, B * k)
    elif mode == oracle.NEG_JOINT:
        neg = rng.integers(0, n, ((B + k - 1) // k) * k)
    else:
        neg = None
    w = rng.uniform(0.2, 3.0, B)
    return emb, rel, src, dst, neg, w


def _neg_rows(mode, src, dst, k, neg):
    B = len(src)
    if mode == oracle.NEG_PER_EDGE:
        return np.asarray(neg).reshape(B, k)
    if mode == oracle.NEG_JOINT:
        return np.stack([np.asarray(neg)[(i // k) * k:(i // k) * k + k] for i in range(B)])
    return np.stack([np.delete(np.asarray(dst), i) for i in range(B)])


def _torch_loss(emb, rel, mode, kind, src, dst, k, neg, w):
    """The loss through torch's own loss functions (scores written directly)."""
    e = torch.tensor(emb, dtype=torch.float64, requires_grad=True)
    r = torch.tensor(rel, dtype=torch.float64, requires_grad=True) if rel is not None else None
    rows = torch.as_tensor(_neg_rows(mode, src, dst, k, neg))
    s_ = torch.as_tensor(src)
    u = e[s_] * (r if r is not None else 1.0)
    pos = (u * e[torch.as_tensor(dst)]).sum(-1)
    negs = (u[:, None, :] * e[rows]).sum(-1)
    if kind == oracle.LOSS_CONTRASTIVE:
        logits = torch.cat([pos[:, None], negs], 1)
        loss = F.cross_entropy(logits, torch.zeros(len(src), dtype=torch.long))
    else:
        logits = torch.cat([pos, negs.reshape(-1)])
        lab = torch.cat([torch.ones_like(pos), torch.zeros(negs.numel(), dtype=torch.float64)])
        wt = None
        if kind == oracle.LOSS_WEIGHTED_CE:
            wt = torch.cat([torch.as_tensor(w), torch.ones(negs.numel(), dtype=torch.float64)])
        loss = F.binary_cross_entropy_with_logits(logits, lab, weight=wt)
    loss.backward()
    return loss.item(), pos.detach().numpy(), negs.detach().numpy(), e.grad.numpy(), \
        (r.grad.numpy() if r is not None else None)


@pytest.mark.parametrize("mode", [oracle.NEG_PER_EDGE, oracle.NEG_JOINT, oracle.NEG_IN_BATCH])
@pytest.mark.parametrize("kind", [oracle.LOSS_CE, oracle.LOSS_WEIGHTED_CE, oracle.LOSS_CONTRASTIVE])
@pytest.mark.parametrize("distmult", [False, True])
def test_loss_scores_and_grads_match_torch(mode, kind, distmult):
    emb, rel, src, dst, neg, w = _batch(7 + mode * 3 + kind, B=9, k=4, mode=mode)
    rel = rel if distmult else None
    got = oracle.lp_loss(emb, rel, mode, kind, src, dst, 4, neg,
                         w if kind == oracle.LOSS_WEIGHTED_CE else None)
    want = _torch_loss(emb, rel, mode, kind, src, dst, 4, neg, w)
    assert got["loss"] == pytest.approx(want[0], rel=1e-13)
    np.testing.assert_allclose(got["pos_score"], want[1], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(got["neg_score"], want[2], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(got["d_emb"], want[3], rtol=1e-11, atol=1e-14)
    if distmult:
        np.testing.assert_allclose(got["d_rel"], want[4], rtol=1e-11, atol=1e-14)


def test_gradients_by_central_differences():
    emb, rel, src, dst, neg, w = _batch(3, n=12, d=3, B=5, k=3, mode=oracle.NEG_JOINT)
    for kind in (oracle.LOSS_WEIGHTED_CE, oracle.LOSS_CONTRASTIVE):
        g = oracle.lp_loss(emb, rel, oracle.NEG_JOINT, kind, src, dst, 3, neg, w)
        h = 1e-6
        for (a, b) in [(0, 0), (int(src[1]), 2), (int(dst[2]), 1), (int(neg[4]), 0)]:
            ep, em = emb.copy(), emb.copy()
            ep[a, b] += h
            em[a, b] -= h
            fp = oracle.lp_loss(ep, rel, oracle.NEG_JOINT, kind, src, dst, 3, neg, w, grads=False)
            fm = oracle.lp_loss(em, rel, oracle.NEG_JOINT, kind, src, dst, 3, neg, w, grads=False)
            assert g["d_emb"][a, b] == pytest.approx((fp["loss"] - fm["loss"]) / (2 * h), abs=1e-8)
        for c in range(3):
            rp, rm = rel.copy(), rel.copy()
            rp[c] += h
            rm[c] -= h
            fp = oracle.lp_loss(emb, rp, oracle.NEG_JOINT, kind, src, dst, 3, neg, w, grads=False)
            fm = oracle.lp_loss(emb, rm, oracle.NEG_JOINT, kind, src, dst, 3, neg, w, grads=False)
            assert g["d_rel"][c] == pytest.approx((fp["loss"] - fm["loss"]) / (2 * h), abs=1e-8)


def test_in_batch_negatives_follow_the_worked_example():
    """Embeddings that identify the pair: u rows are all ones, v_j has j + 1 in column 0
    and zeros elsewhere, so score(u_i, v_j) = j + 1."""
    ex = json.load(open(GOLDEN))
    names = [p[1] for p in ex["positives"]]
    emb = np.zeros((6, 3))
    emb[:3] = 1.0
    for j in range(3):
        emb[3 + j, 0] = j + 1
    got = oracle.lp_loss(emb, None, oracle.NEG_IN_BATCH, oracle.LOSS_CONTRASTIVE, [0, 1, 2],
                         [3, 4, 5], grads=False)
    for i, (u, _) in enumerate(ex["positives"]):
        want = [names.index(v) + 1 for v in ex["negatives"][u]]
        assert got["neg_score"][i].tolist() == want


def test_joint_groups_share_their_negatives():
    """K = 2 over 5 positives: positives 0-1 use neg[0:2], 2-3 use neg[2:4], 4 uses neg[4:6]."""
    emb = np.zeros((20, 2))
    emb[:5] = 1.0
    emb[5:, 0] = np.arange(15) + 1.0
    neg = np.array([5, 9, 12, 6, 19, 8])
    got = oracle.lp_loss(emb, None, oracle.NEG_JOINT, oracle.LOSS_CE, np.arange(5),
                         np.arange(5), 2, neg, grads=False)
    want = [[1, 5], [1, 5], [8, 2], [8, 2], [15, 4]]
    assert got["neg_score"].tolist() == want


def test_distmult_with_unit_relation_is_the_dot_product():
    emb, rel, src, dst, neg, w = _batch(11)
    a = oracle.lp_loss(emb, np.ones(emb.shape[1]), oracle.NEG_PER_EDGE, oracle.LOSS_CE, src,
                       dst, 4, neg)
    b = oracle.lp_loss(emb, None, oracle.NEG_PER_EDGE, oracle.LOSS_CE, src, dst, 4, neg)
    assert a["loss"] == b["loss"]
    np.testing.assert_array_equal(a["d_emb"], b["d_emb"])


def test_weighted_ce_with_unit_weights_is_ce():
    emb, rel, src, dst, neg, w = _batch(12)
    a = oracle.lp_loss(emb, rel, oracle.NEG_PER_EDGE, oracle.LOSS_WEIGHTED_CE, src, dst, 4, neg,
                       np.ones(len(src)))
    b = oracle.lp_loss(emb, rel, oracle.NEG_PER_EDGE, oracle.LOSS_CE, src, dst, 4, neg)
    assert a["loss"] == b["loss"]


def test_negative_ids_are_the_philox_stream_and_uniform():
    for mode in (0, 1):
        ids = oracle.lp_negatives(mode, 400, 1000, 77)
        for q in range(4, 400, 37):
            w = np.random.Philox(counter=[q // 4 - 1, mode, 0, 0], key=[77, 0x6E6567]).random_raw(4)
            assert ids[q] == (int(w[q % 4]) * 1000) >> 64
    ids = oracle.lp_negatives(0, 100_000, 10, 5)
    assert ids.min() >= 0 and ids.max() < 10
    cnt = np.bincount(ids, minlength=10)
    chi2 = float(((cnt - 10_000) ** 2 / 10_000).sum())
    assert chi2 < 40, chi2   # 9 degrees of freedom: P(chi2 > 40) is below 1e-5
