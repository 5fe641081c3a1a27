"""Feature construction for featureless nodes on the GPU vs the oracle (eq. 1, the
average of the featured in-neighbours): small graphs with several relations, heavy and
zero-degree nodes, fp32 and bf16 tables of several widths, every output element; a
tenth-scale billion-edge graph on sampled nodes; indices out of range reported.

fp32: the harness bar (1e-5).  bf16: the output is the fp32 mean rounded to nearest even,
so it may differ from the exact mean by half a bf16 ulp of the larger magnitude plus the
fp32 error (1e-5 of the row scale)."""
import numpy as np
import pytest
import torch

import oracle
from harness import rel_err, to64
from paper_2406_06022_amd import rgcn, synth

pytestmark = pytest.mark.gpu


def _half_ulp_bf16(x):
    a = np.maximum(np.abs(x), 2.0 ** -126)
    return np.exp2(np.floor(np.log2(a)) - 8)


def _compare(got, want, dtype):
    if dtype == "f32":
        assert rel_err(got, want) <= 1e-5
        return
    rms = float(np.sqrt(np.mean(want * want))) if want.size else 0.0
    bound = _half_ulp_bf16(np.maximum(np.abs(got), np.abs(want))) + 1e-5 * np.maximum(np.abs(want), rms)
    over = np.abs(got - want) - bound
    assert not (over > 0).any(), f"{int((over > 0).sum())} elements over the bound"


def _graph(seed, n=2000, srcs=(3000, 800, 50), mean=2.0):
    rng = np.random.default_rng(seed)
    return synth.random_graph(rng, [n] + list(srcs), [(1 + k, 0) for k in range(len(srcs))],
                              mean, heavy=5, heavy_deg=5000)


@pytest.mark.parametrize("dtype,d", [("f32", 40), ("bf16", 128), ("bf16", 264), ("f32", 1024),
                                     ("bf16", 8)])
def test_matches_oracle(dtype, d):
    g = _graph(d)
    gen = torch.Generator().manual_seed(d)
    tdt = synth.torch_dtype(dtype)
    pad = 8 if dtype == "bf16" else 4
    feats = [torch.randn((n, d + pad), generator=gen).to(tdt) for n in g.num_nodes[1:]]
    rels = [(torch.as_tensor(r.indptr).cuda(), torch.as_tensor(r.indices).cuda(),
             feats[k].cuda()) for k, r in enumerate(g.rels)]
    out_full = torch.full((g.num_nodes[0], d + pad), float("nan"), dtype=tdt, device="cuda")
    out = out_full[:, :d]
    print(f"case featureless {dtype} d={d}", flush=True)
    rgcn.rgcn_featureless_mean(rels, g.num_nodes[0], out, flags=rgcn.RGCN_VALIDATE_DEVICE)
    torch.cuda.synchronize()
    want = oracle.featureless_mean([(r.indptr, r.indices, to64(feats[k])[:, :d])
                                    for k, r in enumerate(g.rels)], g.num_nodes[0])
    _compare(to64(out), want, dtype)
    assert torch.isnan(out_full[:, d:]).all()      # the padding is not written


def test_many_relations():
    """20 relations into the type (more than the 2 chunks of a 16-wide bf16 row), so the
    lane group is as wide as the relation count; some sources with no rows at all."""
    rng = np.random.default_rng(20)
    srcs = [int(x) for x in rng.integers(0, 400, size=20)]
    srcs[3] = 0
    g = synth.random_graph(rng, [1500] + srcs, [(1 + k, 0) for k in range(20)], 0.8,
                           heavy=2, heavy_deg=300)
    gen = torch.Generator().manual_seed(20)
    feats = [torch.randn((max(n, 0), 16), generator=gen).to(torch.bfloat16) for n in srcs]
    # the library takes non-NULL index arrays: an edgeless relation passes one dummy entry
    rels = [(torch.as_tensor(r.indptr).cuda(),
             torch.as_tensor(r.indices if len(r.indices) else np.zeros(1, np.int64)).cuda(),
             feats[k].cuda()) for k, r in enumerate(g.rels)]
    out = torch.full((1500, 16), float("nan"), dtype=torch.bfloat16, device="cuda")
    print("case featureless 20 relations", flush=True)
    rgcn.rgcn_featureless_mean(rels, 1500, out, flags=rgcn.RGCN_VALIDATE_DEVICE)
    torch.cuda.synchronize()
    want = oracle.featureless_mean([(r.indptr, r.indices, to64(feats[k]) if srcs[k] else
                                     np.zeros((0, 16))) for k, r in enumerate(g.rels)], 1500)
    _compare(to64(out), want, "bf16")


def test_out_of_range_reported_and_skipped():
    ip = torch.tensor([0, 2, 3], dtype=torch.int64, device="cuda")
    ix = torch.tensor([1, 7, 0], dtype=torch.int64, device="cuda")
    f = torch.tensor([[1.0, 2.0, 3.0, 4.0], [5.0, 6.0, 7.0, 8.0]], device="cuda")
    out = torch.zeros((2, 4), device="cuda")
    with pytest.raises(rgcn.RgcnError) as e:
        rgcn.rgcn_featureless_mean([(ip, ix, f)], 2, out, flags=rgcn.RGCN_VALIDATE_DEVICE)
    assert e.value.status == 4


def test_workload_graph_sampled_nodes():
    """The billion-edge workload's graph at a tenth of its node counts: the features of
    type U (10M nodes) from its in-neighbours of V, W and X (d = 128 bf16)."""
    spec = synth.config(4)
    g = synth.device_graph(spec, device="cuda", node_scale=0.1)
    feats = [synth.normal_table(g.num_nodes[t], 128, torch.bfloat16, 50 + t, device="cuda")
             for t in range(4)]
    into = [r for r in g.rels if r.dst_type == 0]
    rels = [(r.indptr, r.indices, feats[r.src_type]) for r in into]
    out = torch.empty((g.num_nodes[0], 128), dtype=torch.bfloat16, device="cuda")
    print("case featureless workload graph", flush=True)
    rgcn.rgcn_featureless_mean(rels, g.num_nodes[0], out)
    torch.cuda.synchronize()
    deg = sum((r.indptr[1:] - r.indptr[:-1]) for r in into)
    rng = np.random.default_rng(2)
    nodes = {int(torch.argmax(deg))} | set(rng.integers(0, g.num_nodes[0], 40).tolist())
    zero = torch.nonzero(deg == 0)
    if zero.numel():
        nodes.add(int(zero[0]))
    for v in sorted(nodes):
        sub = []
        for r in into:
            b, e = int(r.indptr[v]), int(r.indptr[v + 1])
            ids = r.indices[b:e]
            rows = to64(feats[r.src_type][ids]) if e > b else np.zeros((0, 128))
            sub.append((np.array([0, e - b]), np.arange(e - b), rows if e > b else np.zeros((1, 128))))
        want = oracle.featureless_mean(sub, 1)
        _compare(to64(out[v:v + 1]), want, "bf16")
