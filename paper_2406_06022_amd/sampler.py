"""Mini-batch sampling on the device: one rgcn_sample_block call per layer, top-down from
the seeds (the paper's on-the-fly sampling with a fanout per layer, one block per GNN
layer).  Each layer's source ids become the next layer's destination ids; the host reads
the counts between layers to size the blocks.  Argument marshalling and slicing only."""
from __future__ import annotations

from typing import List, Sequence

import torch

from . import rgcn


def sample_minibatch(graph: "rgcn.DeviceGraph", seeds: Sequence[torch.Tensor],
                     fanouts: Sequence[int], seed: int, grad_src_types=None,
                     flags: int = 0, stream=None, src_rows: bool = False):
    """Blocks (blocks[0] nearest the input, fanouts[l] for block l, as DeviceBlockView) and
    the input layer's source ids per type.  ``seeds[t]``: device int64 ids (may be empty).
    ``grad_src_types[l]``: the grad mask given to block l (default 0).  With ``src_rows``
    the input-side block also carries each edge's global source id (its table row)."""
    T = graph.num_types
    L = len(fanouts)
    frontier = [x.to(torch.int64).contiguous() for x in seeds]
    blocks: List[rgcn.DeviceBlockView] = []
    for layer in reversed(range(L)):
        want_rows = src_rows and layer == 0
        out = rgcn.rgcn_sample_block(graph, frontier, fanouts[layer], seed, layer, flags=flags,
                                     stream=stream, src_rows=want_rows)
        ip, ix, src, counts = out[:4]
        c = counts.cpu().tolist()   # synchronises: the block's sizes
        R = graph.num_rels
        rels = [(graph.types[r][0], graph.types[r][1], ip[r], ix[r][: c[r]],
                 out[4][r][: c[r]] if want_rows and c[r] > 0 else None)
                for r in range(R)]
        n_src = c[R:R + T]
        n_dst = [int(x.numel()) for x in frontier]
        mask = 0 if grad_src_types is None else int(grad_src_types[layer])
        blocks.insert(0, rgcn.DeviceBlockView(n_src, n_dst, rels, mask))
        frontier = [src[t][: n_src[t]] for t in range(T)]
    return blocks, frontier
