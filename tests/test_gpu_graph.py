"""A training step recorded into a HIP graph and replayed: every replay, with eager steps
and synchronisations between the replays, gives the eager step's outputs and gradients bit
for bit (the non-atomic paths are deterministic), on the multi-layer workloads at a size the
oracle also runs, including the embedding scatter of a learnable table and the backward plans
on a second stream."""
import pytest
import torch

from paper_2406_06022_amd import chain, synth
from tests.test_gpu_chain import poison_stack, step_outputs

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("index", [2, 4])
def test_graph_replays_match_eager_step(index):
    spec = synth.small_config(index)
    mb = synth.sample_minibatch(spec)
    T, R, L = len(spec.ntype_names), len(spec.rels), spec.num_layers
    tdt = synth.torch_dtype(spec.dtype)
    emb = [t for t in range(T) if spec.featureless[t]]
    tables = [synth.normal_table(spec.type_rows[t], spec.dims[0], tdt, 700 + t).to(DEV)
              for t in range(T)]
    ids = [torch.as_tensor(mb.input_ids[t]).to(DEV) for t in range(T)]
    weights = []
    for l in range(L):
        w_rel, w_self, _ = synth.block_weights(T, R, spec.dims[l], spec.dims[l + 1], tdt, 80 + l)
        weights.append(([x.to(DEV) for x in w_rel], [x.to(DEV) for x in w_self], None))
    stack = chain.MiniBatchStack(mb.blocks, tables, ids, weights, spec.dtype, spec.dims,
                                 emb_types=emb, device=DEV)
    gen = torch.Generator().manual_seed(55 + index)
    dy = [torch.randn((n, spec.dims[-1]), generator=gen).to(DEV) if n else None
          for n in mb.blocks[-1].n_dst]

    def eager():
        poison_stack(stack)
        for t in emb:
            stack.demb[t].zero_()
        stack.step(dy)
        torch.cuda.synchronize()
        return step_outputs(stack, emb)

    want = eager()
    graph = stack.capture_step(dy)
    torch.cuda.synchronize()
    for rep in range(3):
        print(f"case graph {spec.name} replay {rep}", flush=True)
        poison_stack(stack)
        for t in emb:
            stack.demb[t].zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = step_outputs(stack, emb)
        for i, (g, w_) in enumerate(zip(got, want)):
            assert torch.equal(g, w_), f"replay {rep}: output {i} differs from the eager step"
        assert all(torch.equal(a, b) for a, b in zip(eager(), want))   # eager work between
