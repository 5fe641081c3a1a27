"""Seeded synthetic mini-batch workloads for the relational graph-convolution block.

This module draws *inputs* only: the structure of sampled mini-batch blocks (one bipartite
message-flow graph per GNN layer, stored as a per-relation CSR) and the values of feature
tables, learnable-embedding tables, weights and output gradients.  It holds none of the
layer's arithmetic; both the HIP path and the CPU oracle consume what it produces.

Workload shapes follow the heterogeneous-graph setting of the paper: several node types,
canonical edge types (src type, relation, dst type), featureless node types backed by a
learnable embedding table (Sec. 3.3.2), and on-the-fly neighbour sampling with a per-layer
fanout that yields one block per layer (Sec. 3.1.1; the per-layer loop over ``blocks`` of
the customised-model figure in the programming-interface appendix).  The paper's datasets
are not used; the generator reproduces only their scale and structure.

Block convention: the destination nodes of type t are the first ``n_dst[t]`` source nodes
of type t, so the self-loop term reads rows ``[0, n_dst[t])`` of the source input.
``fanouts[l]`` applies to block ``l``; block 0 is nearest the input and the seed-adjacent
block uses the last fanout.  Sources are drawn uniformly without replacement per
(destination, relation) segment.  Source rows after the destination prefix are numbered
in order of first appearance over the relations' edge lists (relations in order, edges in
CSR order), the compaction order of the block construction in DGL, on which the paper's
system builds its mini-batches.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Callable, List, Optional, Sequence, Tuple

import numpy as np

BASE_SEED = 20240600


# --------------------------------------------------------------------------------------
# Workload specifications
# --------------------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class WorkloadSpec:
    name: str
    dtype: str                        # "f32" or "bf16": storage/compute type of the forward
    ntype_names: Tuple[str, ...]
    type_rows: Tuple[int, ...]        # rows of each type's feature / embedding table
    featureless: Tuple[bool, ...]     # True: the table is a learnable embedding (needs dE)
    rels: Tuple[Tuple[int, int], ...]  # (src_type, dst_type) per relation
    seed_types: Tuple[int, ...]       # node types that receive seeds
    n_seeds: int                      # seeds per seed type
    fanouts: Tuple[int, ...]          # fanouts[l] applies to block l
    degree: str                       # "exact", "zipf" or "pareto"
    dims: Tuple[int, ...]             # d_0 (input) ... d_L (output)
    seed: int
    skew: float = 0.0                 # >0: sources drawn by popularity rank^-skew

    @property
    def num_layers(self) -> int:
        return len(self.fanouts)

    def scaled(self, name: str, type_rows: Sequence[int], n_seeds: int,
               seed_offset: int = 100) -> "WorkloadSpec":
        """Same structure, smaller tables/batch (for parity runs the oracle finishes fast)."""
        return dataclasses.replace(self, name=name, type_rows=tuple(type_rows),
                                   n_seeds=n_seeds, seed=self.seed + seed_offset)


def _cfg1() -> WorkloadSpec:
    # Tiny 1-layer block, fp32: A,B (5,000 each), r0 A->A, r1 B->A, r2 A->B,
    # 1,000 destination seeds per type, exactly 5 sources per (dst, relation), 32 -> 64.
    return WorkloadSpec("tiny_fp32", "f32", ("A", "B"), (5000, 5000), (False, False),
                        ((0, 0), (1, 0), (0, 1)), (0, 1), 1000, (5,), "exact", (32, 64),
                        BASE_SEED + 0)


def _cfg2() -> WorkloadSpec:
    # 2-layer mini-batch, bf16: T0..T3 (1M each), 8 relations, 1,024 seeds of T0,
    # fanouts [15, 10], Zipf(1.5) degrees capped at the fanout, 128 -> 256 -> 256.
    rels = ((1, 0), (0, 1), (2, 0), (0, 2), (3, 1), (1, 3), (0, 0), (2, 3))
    return WorkloadSpec("minibatch_2layer_bf16", "bf16", ("T0", "T1", "T2", "T3"),
                        (1_000_000,) * 4, (False,) * 4, rels, (0,), 1024, (15, 10), "zipf",
                        (128, 256, 256), BASE_SEED + 1)


def _cfg3() -> WorkloadSpec:
    # Academic-style graph: author (featureless, learnable 1.9M x 128 table), paper (2M),
    # field (1M), institution (1M); 7 relations with reverse edges; 4,096 paper seeds;
    # fanouts [25, 15]; 128 -> 256 -> 256.
    # types: 0=A(author) 1=P(paper) 2=F(field) 3=I(institution)
    rels = ((0, 1), (1, 0), (1, 1), (1, 2), (2, 1), (0, 3), (3, 0))
    return WorkloadSpec("academic_2layer_bf16", "bf16", ("author", "paper", "field", "inst"),
                        (1_900_000, 2_000_000, 1_000_000, 1_000_000),
                        (True, False, False, False), rels, (1,), 4096, (25, 15), "zipf",
                        (128, 256, 256), BASE_SEED + 2)


def _cfg4() -> WorkloadSpec:
    # Wide-relation block: 20 relations S_{r mod 4} -> D of mixed density (mean degree
    # log-spaced 1..200, Pareto(1.5)), 8,192 destination nodes, fanout 30, 512 -> 512.
    rels = tuple((r % 4, 4) for r in range(20))
    return WorkloadSpec("wide_20rel_bf16", "bf16", ("S0", "S1", "S2", "S3", "D"),
                        (2_000_000,) * 4 + (1_000_000,), (False,) * 5, rels, (4,), 8192,
                        (30,), "pareto", (512, 512), BASE_SEED + 3)


def _cfg5() -> WorkloadSpec:
    # Single-GPU share of a billion-edge graph: U (100M, featureless, 100M x 128 bf16
    # learnable table), V (20M), W (10M), X (1M); 12 relations; 4,096 seeds of V;
    # fanouts [25, 20, 15]; 128 -> 512 -> 512 -> 512; embedding gradient for U.
    # types: 0=U 1=V 2=W 3=X
    rels = ((1, 0), (2, 0), (3, 0), (0, 1), (1, 1), (1, 1), (2, 1), (0, 2), (1, 2), (3, 2),
            (2, 3), (0, 3))
    return WorkloadSpec("billion_share_3layer_bf16", "bf16", ("U", "V", "W", "X"),
                        (100_000_000, 20_000_000, 10_000_000, 1_000_000),
                        (True, False, False, False), rels, (1,), 4096, (25, 20, 15), "zipf",
                        (128, 512, 512, 512), BASE_SEED + 4)


CONFIGS: Tuple[Callable[[], WorkloadSpec], ...] = (_cfg1, _cfg2, _cfg3, _cfg4, _cfg5)


def config(index: int) -> WorkloadSpec:
    return CONFIGS[index]()


def skewed_config(index: int, skew: float = 0.8) -> WorkloadSpec:
    """The workload with sources drawn by popularity rank, p(rank k) proportional to
    (k + 1)^-skew, mapped to ids by a fixed bijection: power-law source degrees, so the
    backward's transpose segments are uncapped (hub sources with tens of thousands of
    edges)."""
    spec = config(index)
    return dataclasses.replace(spec, name=f"{spec.name}_skewed", skew=skew)


def small_config(index: int) -> WorkloadSpec:
    """Each configuration's structure at a size the oracle evaluates in seconds.

    Tables shrink (keeping several thousand rows so indices span many tiles) and the seed
    batch shrinks; relations, fanouts, degree laws and dimensions are unchanged.
    """
    spec = config(index)
    if index == 0:
        return spec.scaled("tiny_fp32_small", (2000, 1500), 333)
    if index == 1:
        return spec.scaled("minibatch_2layer_small", (20000, 15000, 12000, 9000), 37)
    if index == 2:
        return spec.scaled("academic_2layer_small", (30000, 25000, 9000, 7000), 41)
    if index == 3:
        return spec.scaled("wide_20rel_small", (9000, 8000, 7000, 6000, 5000), 300)
    return spec.scaled("billion_share_3layer_small", (60000, 40000, 20000, 3000), 5)


# --------------------------------------------------------------------------------------
# Block structure
# --------------------------------------------------------------------------------------
@dataclasses.dataclass
class Relation:
    src_type: int
    dst_type: int
    indptr: np.ndarray    # int32 [n_dst[dst_type] + 1]
    indices: np.ndarray   # int32 [nnz], local source rows in [0, n_src[src_type])
    # int64 [nnz] global id of each edge's source as drawn (the sampler's output before
    # relabelling: the input-table row of the source at the input layer), or None
    src_rows: Optional[np.ndarray] = None

    @property
    def nnz(self) -> int:
        return int(self.indices.shape[0])


@dataclasses.dataclass
class Block:
    n_src: List[int]
    n_dst: List[int]
    rels: List[Relation]

    @property
    def num_types(self) -> int:
        return len(self.n_src)

    @property
    def nnz(self) -> int:
        return sum(r.nnz for r in self.rels)


@dataclasses.dataclass
class MiniBatch:
    spec: WorkloadSpec
    blocks: List[Block]          # blocks[0] is nearest the input
    input_ids: List[np.ndarray]  # int64 global table rows of block 0's sources, per type

    @property
    def nnz(self) -> int:
        return sum(b.nnz for b in self.blocks)


def _degrees(rng: np.random.Generator, spec: WorkloadSpec, rel_index: int, n: int,
             fanout: int) -> np.ndarray:
    if n == 0:
        return np.zeros(0, dtype=np.int64)
    if spec.degree == "exact":
        return np.full(n, fanout, dtype=np.int64)
    if spec.degree == "zipf":
        return np.minimum(rng.zipf(1.5, n), fanout).astype(np.int64)
    if spec.degree == "pareto":
        # Full-graph mean degree log-spaced from 1 to 200 over the relations; degree is
        # floor(Pareto(alpha=1.5, x_m=mu/3)) and the sampled degree is capped at the fanout.
        nrel = len(spec.rels)
        mu = 200.0 ** (rel_index / max(nrel - 1, 1))
        xm = mu / 3.0
        raw = np.floor((rng.pareto(1.5, n) + 1.0) * xm)
        return np.minimum(raw, fanout).astype(np.int64)
    raise ValueError(spec.degree)


def _popularity_map(rows: int, skew: float, rng: np.random.Generator, n: int) -> np.ndarray:
    """Draw n ids with p(rank k) proportional to (k+1)^-skew, ranks scattered over the ids."""
    # inverse-CDF of the continuous power law on [1, rows+1)
    u = rng.random(n)
    a = 1.0 - skew
    lo, hi = 1.0, float(rows) + 1.0
    x = (lo ** a + u * (hi ** a - lo ** a)) ** (1.0 / a)
    rank = np.minimum(np.floor(x).astype(np.int64) - 1, rows - 1)
    # fixed bijection rank -> id: multiplication by an odd constant modulo a power of two,
    # restricted to [0, rows) by cycle walking
    p2 = 1 << max(1, int(math.ceil(math.log2(rows))))
    ids = rank.copy()
    mult = np.int64(0x9E3779B1 | 1)
    todo = np.ones(n, dtype=bool)
    while True:
        ids[todo] = (ids[todo] * mult + 0x7F4A7C15) % p2
        todo = ids >= rows
        if not todo.any():
            return ids


def _draw_sources(rng: np.random.Generator, deg: np.ndarray, rows: int,
                  skew: float, device="cpu") -> np.ndarray:
    """Sources per segment, uniform (or popularity-skewed) and distinct within a segment.

    Draws come from ``rng`` (so the result does not depend on ``device``); the duplicate
    search (a sort of segment-major keys) runs with torch on ``device``."""
    import torch
    total = int(deg.sum())
    if total == 0:
        return np.zeros(0, dtype=np.int64)
    if int(deg.max()) > rows:
        raise ValueError("segment degree exceeds the source population")
    seg = torch.repeat_interleave(torch.arange(deg.shape[0], dtype=torch.int64, device=device),
                                  torch.as_tensor(deg, dtype=torch.int64, device=device))

    def draw(n: int) -> np.ndarray:
        if skew > 0.0:
            return _popularity_map(rows, skew, rng, n)
        return rng.integers(0, rows, size=n, dtype=np.int64)

    src = draw(total)
    while True:
        s_t = torch.as_tensor(src, device=device)
        key = seg * rows + s_t
        sk, order = torch.sort(key, stable=True)
        dup_sorted = torch.zeros(total, dtype=torch.bool, device=device)
        dup_sorted[1:] = sk[1:] == sk[:-1]
        dup = order[dup_sorted].cpu().numpy()
        if dup.shape[0] == 0:
            return src
        src[dup] = draw(dup.shape[0])


def _unique_first_appearance(x):
    """Distinct values of the 1-D tensor ``x`` in order of their first occurrence."""
    import torch
    if x.numel() == 0:
        return x
    uniq, inv = torch.unique(x, return_inverse=True)
    pos = torch.arange(x.numel(), dtype=torch.int64, device=x.device)
    first = torch.full((uniq.numel(),), x.numel(), dtype=torch.int64, device=x.device)
    first.scatter_reduce_(0, inv, pos, reduce="amin")
    return uniq[torch.argsort(first)]


def _relabel(global_ids, table):
    """Position of each global id inside ``table`` (torch tensors; every id is present)."""
    import torch
    sorted_table, order = torch.sort(table, stable=True)
    pos = torch.searchsorted(sorted_table, global_ids)
    return order[pos]


def sample_minibatch(spec: WorkloadSpec, seed_ids: Optional[List[np.ndarray]] = None,
                     device="cpu") -> MiniBatch:
    """Sample a multi-layer mini-batch top-down from the seeds, one block per layer.

    Random draws use numpy's PCG64 stream seeded by the spec; sorting, de-duplication and
    relabelling run with torch on ``device``.  The result is the same on every device."""
    import torch
    rng = np.random.Generator(np.random.PCG64(spec.seed))
    T = len(spec.ntype_names)
    frontier: List[np.ndarray] = [np.zeros(0, dtype=np.int64) for _ in range(T)]
    for t in spec.seed_types:
        if seed_ids is not None:
            frontier[t] = np.asarray(seed_ids[t], dtype=np.int64)
        else:
            frontier[t] = rng.choice(spec.type_rows[t], size=spec.n_seeds, replace=False
                                     ).astype(np.int64)
    blocks: List[Block] = []
    for layer in reversed(range(spec.num_layers)):
        fanout = spec.fanouts[layer]
        dst_ids = frontier
        drawn: List[Tuple[np.ndarray, np.ndarray]] = []
        per_type_new: List[List[np.ndarray]] = [[] for _ in range(T)]
        for r, (s, t) in enumerate(spec.rels):
            deg = _degrees(rng, spec, r, dst_ids[t].shape[0], fanout)
            src = _draw_sources(rng, deg, spec.type_rows[s], spec.skew, device)
            drawn.append((deg, src))
            per_type_new[s].append(src)
        src_t = []
        for s in range(T):
            dst_t = torch.as_tensor(dst_ids[s], device=device)
            if per_type_new[s]:
                pool = _unique_first_appearance(
                    torch.as_tensor(np.concatenate(per_type_new[s]), device=device))
                fresh = pool[~torch.isin(pool, dst_t)]
            else:
                fresh = torch.zeros(0, dtype=torch.int64, device=device)
            src_t.append(torch.cat([dst_t, fresh]))
        rels: List[Relation] = []
        for r, (s, t) in enumerate(spec.rels):
            deg, src = drawn[r]
            indptr = np.zeros(deg.shape[0] + 1, dtype=np.int64)
            np.cumsum(deg, out=indptr[1:])
            if src.shape[0]:
                local = _relabel(torch.as_tensor(src, device=device), src_t[s]).cpu().numpy()
            else:
                local = np.zeros(0, np.int64)
            rels.append(Relation(s, t, indptr.astype(np.int32), local.astype(np.int32),
                                 np.asarray(src, dtype=np.int64)))
        src_ids = [x.cpu().numpy().astype(np.int64) for x in src_t]
        blocks.insert(0, Block([int(x.shape[0]) for x in src_ids],
                               [int(x.shape[0]) for x in dst_ids], rels))
        frontier = src_ids
    return MiniBatch(spec, blocks, frontier)


def random_block(rng: np.random.Generator, n_src: Sequence[int], n_dst: Sequence[int],
                 rels: Sequence[Tuple[int, int]], max_deg: int, zero_frac: float = 0.2,
                 allow_duplicates: bool = True) -> Block:
    """A small random block for property tests: ragged degrees, zero-degree rows,
    empty relations and (optionally) repeated (dst, src) edges."""
    out: List[Relation] = []
    for (s, t) in rels:
        nd = int(n_dst[t])
        deg = rng.integers(0, max_deg + 1, size=nd)
        deg[rng.random(nd) < zero_frac] = 0
        if n_src[s] == 0:
            deg[:] = 0
        indptr = np.zeros(nd + 1, dtype=np.int64)
        np.cumsum(deg, out=indptr[1:])
        nnz = int(indptr[-1])
        if allow_duplicates:
            idx = rng.integers(0, max(int(n_src[s]), 1), size=nnz)
        else:
            idx = _draw_sources(rng, deg, int(n_src[s]), 0.0)
        out.append(Relation(s, t, indptr.astype(np.int32), idx.astype(np.int32)))
    return Block([int(x) for x in n_src], [int(x) for x in n_dst], out)


def with_hub_sources(rng: np.random.Generator, blk: Block, src_type: int,
                     hub_degrees: Sequence[int]) -> Block:
    """``blk`` with extra edges from source rows 0, 1, ... of ``src_type``: source row h
    gains about hub_degrees[h] in-edges over the relations leaving the type, spread over
    random destination rows (repeated edges included), kept in CSR order."""
    rels = [r for r in blk.rels if r.src_type == src_type and blk.n_dst[r.dst_type] > 0]
    if not rels:
        return blk
    extra = {id(r): [] for r in rels}
    for h, dh in enumerate(hub_degrees):
        which = rng.integers(0, len(rels), size=int(dh))
        for k, rel in enumerate(rels):
            m = int((which == k).sum())
            rows = rng.integers(0, blk.n_dst[rel.dst_type], size=m)
            extra[id(rel)].append(np.stack([rows, np.full(m, h)], axis=1))
    out = []
    for rel in blk.rels:
        if id(rel) not in extra:
            out.append(rel)
            continue
        nd = blk.n_dst[rel.dst_type]
        ip = np.asarray(rel.indptr, np.int64)
        rows = np.repeat(np.arange(nd), np.diff(ip))
        add = np.concatenate(extra[id(rel)]) if extra[id(rel)] else np.zeros((0, 2), np.int64)
        all_rows = np.concatenate([rows, add[:, 0]])
        all_src = np.concatenate([np.asarray(rel.indices, np.int64), add[:, 1]])
        order = np.argsort(all_rows, kind="stable")
        indptr = np.zeros(nd + 1, dtype=np.int64)
        np.cumsum(np.bincount(all_rows, minlength=nd), out=indptr[1:])
        out.append(Relation(rel.src_type, rel.dst_type, indptr.astype(np.int32),
                            all_src[order].astype(np.int32)))
    return Block(list(blk.n_src), list(blk.n_dst), out)


# --------------------------------------------------------------------------------------
# Full graphs to sample from (in-edge CSR per relation, global ids)
# --------------------------------------------------------------------------------------
@dataclasses.dataclass
class GraphRel:
    src_type: int
    dst_type: int
    indptr: object    # int64 [num_nodes[dst_type] + 1] (numpy array or torch tensor)
    indices: object   # int64 [nnz] global source ids of type src_type


@dataclasses.dataclass
class Graph:
    num_nodes: List[int]
    rels: List[GraphRel]

    @property
    def nnz(self) -> int:
        return sum(int(r.indices.shape[0]) for r in self.rels)


def random_graph(rng: np.random.Generator, num_nodes: Sequence[int],
                 rels: Sequence[Tuple[int, int]], mean_deg: float, heavy: int = 0,
                 heavy_deg: int = 0) -> Graph:
    """A small full graph for tests: in-degrees Poisson(mean_deg) (zeros included), plus
    ``heavy`` destination nodes per relation with ``heavy_deg`` in-edges; sources uniform
    (repeats allowed, as in a multigraph)."""
    out = []
    for (s, t) in rels:
        n = int(num_nodes[t])
        deg = rng.poisson(mean_deg, size=n).astype(np.int64)
        if heavy and n:
            deg[rng.choice(n, size=min(heavy, n), replace=False)] = heavy_deg
        if num_nodes[s] == 0:
            deg[:] = 0
        indptr = np.zeros(n + 1, dtype=np.int64)
        np.cumsum(deg, out=indptr[1:])
        idx = rng.integers(0, max(int(num_nodes[s]), 1), size=int(indptr[-1]), dtype=np.int64)
        out.append(GraphRel(s, t, indptr, idx))
    return Graph([int(x) for x in num_nodes], out)


def device_graph(spec: WorkloadSpec, mean_deg: float = 5.0, max_deg: int = 100_000,
                 device="cuda", node_scale: float = 1.0) -> Graph:
    """The full graph behind a workload's mini-batches, drawn on ``device``: node counts of
    the spec's types (times ``node_scale``), and per relation in-degrees
    floor(Pareto(alpha = 2, x_m = (mean_deg + 0.5) / 2)) (mean about ``mean_deg``, power-law
    tail, capped at ``max_deg``), sources uniform over the source type.  Seeded by the
    spec."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(spec.seed * 31 + 7)
    nodes = [max(1, int(round(n * node_scale))) for n in spec.type_rows]
    out = []
    for (s, t) in spec.rels:
        n = nodes[t]
        u = torch.rand(n, generator=gen, device=device, dtype=torch.float64)
        deg = torch.floor(((mean_deg + 0.5) / 2.0) / torch.sqrt(1.0 - u)).clamp_(max=max_deg)
        indptr = torch.zeros(n + 1, dtype=torch.int64, device=device)
        torch.cumsum(deg.to(torch.int64), 0, out=indptr[1:])
        nnz = int(indptr[-1])
        idx = torch.randint(0, nodes[s], (nnz,), generator=gen, device=device, dtype=torch.int64)
        out.append(GraphRel(s, t, indptr, idx))
    return Graph(nodes, out)


# --------------------------------------------------------------------------------------
# Values
# --------------------------------------------------------------------------------------
def torch_dtype(name: str):
    import torch
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def normal_table(rows: int, cols: int, dtype, seed: int, device="cpu",
                 chunk_rows: int = 1 << 21):
    """rows x cols table of N(0,1) values rounded to ``dtype``, drawn in row chunks from a
    seeded torch generator on ``device`` (so multi-GB tables never sit in host memory)."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    out = torch.empty((rows, cols), dtype=dtype, device=device)
    for r0 in range(0, rows, chunk_rows):
        r1 = min(rows, r0 + chunk_rows)
        out[r0:r1] = torch.randn((r1 - r0, cols), generator=gen, device=device,
                                 dtype=torch.float32).to(dtype)
    return out


def glorot(d_in: int, d_out: int, dtype, seed: int):
    """Xavier-uniform U(-a, a), a = sqrt(6 / (d_in + d_out)), on the CPU."""
    import torch
    gen = torch.Generator(device="cpu")
    gen.manual_seed(int(seed))
    a = math.sqrt(6.0 / (d_in + d_out))
    w = (torch.rand((d_in, d_out), generator=gen, dtype=torch.float64) * 2.0 - 1.0) * a
    return w.to(dtype)


def block_weights(num_types: int, num_rels: int, d_in: int, d_out: int, dtype, seed: int,
                  with_bias: bool = False):
    """Per-relation W_r, per-type self-loop W_self and (optional) bias for one block."""
    import torch
    w_rel = [glorot(d_in, d_out, dtype, seed * 1000 + r) for r in range(num_rels)]
    w_self = [glorot(d_in, d_out, dtype, seed * 1000 + 500 + t) for t in range(num_types)]
    if with_bias:
        gen = torch.Generator(device="cpu")
        gen.manual_seed(int(seed) * 7 + 3)
        bias = [(torch.rand(d_out, generator=gen, dtype=torch.float64) - 0.5).to(dtype)
                for _ in range(num_types)]
    else:
        bias = [None] * num_types
    return w_rel, w_self, bias
