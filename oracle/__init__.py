"""CPU oracle of the RGCN block (forward, backward, integer plan) -- TEST INFRASTRUCTURE.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import this package.  It shares no code with the HIP library: the arithmetic lives in
``rgcn_oracle.c`` (plain loops, IEEE double), and this wrapper only marshals numpy
arrays into it.  Block objects are duck-typed: anything with ``n_src``, ``n_dst`` and
``rels`` (each with ``src_type``, ``dst_type``, ``indptr``, ``indices``) is accepted.

Which passage each function follows is stated in ``rgcn_oracle.c``.  The order in which
the library processes segments is library policy, not the method's arithmetic, so it has
no counterpart here: the tests check that the library's schedules are permutations and that
results do not depend on them.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "rgcn_oracle.c")
_SRC_SAMPLE = os.path.join(_HERE, "sample_oracle.c")
_SRC_LP = os.path.join(_HERE, "lp_oracle.c")
_SRC_FEAT = os.path.join(_HERE, "feature_oracle.c")
# ORACLE_SANITIZE=1 selects an AddressSanitizer / UndefinedBehaviorSanitizer build of the
# same sources (host code; loading it needs the ASan runtime preloaded)
_LIB_PATH = os.path.join(_HERE, "liboracle_san.so" if os.environ.get("ORACLE_SANITIZE") == "1"
                         else "liboracle.so")
_lib = None


def _flags():
    """gcc flags of the oracle: plain IEEE double (no fast-math, no contraction into fused
    multiply-adds), OpenMP for the loops that hand whole output elements to one thread.
    ORACLE_SANITIZE=1 adds AddressSanitizer and UndefinedBehaviorSanitizer (host code)."""
    f = ["-O2", "-std=c99", "-fno-fast-math", "-ffp-contract=off", "-fopenmp"]
    if os.environ.get("ORACLE_SANITIZE") == "1":
        f += ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
              "-fno-omit-frame-pointer", "-g"]
    return f


def build(force: bool = True) -> str:
    """Compile the oracle with the host C compiler (plain IEEE double, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.run(["gcc", *_flags(), "-fPIC", "-shared", _SRC, _SRC_SAMPLE, _SRC_LP,
                        _SRC_FEAT, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Rel(ctypes.Structure):
    _fields_ = [("src_type", ctypes.c_int32), ("dst_type", ctypes.c_int32),
                ("indptr", ctypes.c_void_p), ("indices", ctypes.c_void_p)]


class _Block(ctypes.Structure):
    _fields_ = [("num_types", ctypes.c_int32), ("num_rels", ctypes.c_int32),
                ("n_src", ctypes.c_void_p), ("n_dst", ctypes.c_void_p),
                ("rels", ctypes.POINTER(_Rel))]


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        lib.orc_set_threads.argtypes = [ctypes.c_int]
        lib.orc_get_threads.restype = ctypes.c_int
        lib.orc_check_block.argtypes = [vp]
        lib.orc_check_block.restype = ctypes.c_int
        lib.orc_degrees.argtypes = [vp, i64, vp]
        lib.orc_mean_aggregate.argtypes = [vp, vp, i64, vp, i64, vp]
        lib.orc_block_forward.argtypes = [vp, i64, i64, vp, vp, vp, vp, ctypes.c_int, vp]
        lib.orc_block_forward.restype = ctypes.c_int
        lib.orc_block_backward.argtypes = [vp, i64, i64, vp, vp, vp, vp, ctypes.c_int,
                                           vp, vp, vp, vp]
        lib.orc_block_backward.restype = ctypes.c_int
        lib.orc_scatter_add.argtypes = [i64, i64, vp, vp, vp]
        lib.orc_sparse_adagrad.argtypes = [i64, i64, i64, vp, vp, vp, vp, ctypes.c_double,
                                           ctypes.c_double]
        lib.orc_sparse_adagrad.restype = ctypes.c_int
        lib.orc_csc.argtypes = [i64, i64, vp, vp, vp, vp, vp]
        lib.orc_csc.restype = ctypes.c_int
        u64 = ctypes.c_uint64
        lib.orc_philox4x64.argtypes = [vp, vp, vp]
        lib.orc_sample_draw.argtypes = [u64, u64, u64, u64, u64]
        lib.orc_sample_draw.restype = u64
        lib.orc_sample_segment.argtypes = [i64, i64, u64, i32, i64, i32, vp]
        lib.orc_sample_segment.restype = i64
        lib.orc_sample_block.argtypes = [i32, i32, vp, vp, vp, vp, vp, vp, vp, i64, u64, i32,
                                         vp, vp, vp, vp]
        lib.orc_sample_block.restype = ctypes.c_int
        lib.orc_lp_loss.argtypes = [i64, i64, vp, vp, i32, i32, i64, vp, vp, i64, vp, vp, vp, vp,
                                    vp, vp, vp]
        lib.orc_lp_loss.restype = ctypes.c_int
        lib.orc_lp_negatives.argtypes = [i32, i64, i64, u64, vp]
        lib.orc_featureless_mean.argtypes = [i32, vp, vp, vp, vp, i64, i64, vp]
        lib.orc_featureless_mean.restype = ctypes.c_int
        _lib = lib
    return _lib


def set_threads(n: int) -> None:
    """Threads of the oracle's parallel loops (results do not depend on it)."""
    _load().orc_set_threads(int(n))


def get_threads() -> int:
    return int(_load().orc_get_threads())


def _ptr(a: Optional[np.ndarray]) -> Optional[int]:
    return None if a is None else a.ctypes.data


class _Marshal:
    """Holds the ctypes mirror of a block (and keeps its arrays alive)."""

    def __init__(self, block):
        self.keep = []
        T = len(block.n_src)
        self.n_src = np.asarray(block.n_src, dtype=np.int64)
        self.n_dst = np.asarray(block.n_dst, dtype=np.int64)
        rels = (_Rel * max(len(block.rels), 1))()
        for r, rel in enumerate(block.rels):
            ip = np.ascontiguousarray(rel.indptr, dtype=np.int32)
            ix = np.ascontiguousarray(rel.indices, dtype=np.int32)
            if ix.size == 0:
                ix = np.zeros(1, dtype=np.int32)
            self.keep += [ip, ix]
            rels[r] = _Rel(rel.src_type, rel.dst_type, ip.ctypes.data, ix.ctypes.data)
        self.rels = rels
        self.c = _Block(T, len(block.rels), self.n_src.ctypes.data, self.n_dst.ctypes.data,
                        ctypes.cast(rels, ctypes.POINTER(_Rel)))

    def ptrs(self, arrays: Sequence[Optional[np.ndarray]]):
        arr = (ctypes.c_void_p * max(len(arrays), 1))()
        for i, a in enumerate(arrays):
            if a is not None:
                a = np.ascontiguousarray(a, dtype=np.float64)
                self.keep.append(a)
                arr[i] = a.ctypes.data
        self.keep.append(arr)
        return ctypes.cast(arr, ctypes.c_void_p)

    def out_ptrs(self, arrays: Sequence[Optional[np.ndarray]]):
        arr = (ctypes.c_void_p * max(len(arrays), 1))()
        for i, a in enumerate(arrays):
            if a is not None:
                assert a.dtype == np.float64 and a.flags.c_contiguous
                arr[i] = a.ctypes.data
        self.keep.append(arr)
        return ctypes.cast(arr, ctypes.c_void_p)


def check_block(block) -> bool:
    m = _Marshal(block)
    return _load().orc_check_block(ctypes.byref(m.c)) == 0


def degrees(indptr: np.ndarray) -> np.ndarray:
    ip = np.ascontiguousarray(indptr, dtype=np.int32)
    n = ip.shape[0] - 1
    out = np.zeros(max(n, 1), dtype=np.int32)
    _load().orc_degrees(ip.ctypes.data, n, out.ctypes.data)
    return out[:n]


def mean_aggregate(indptr, indices, h_src: np.ndarray) -> np.ndarray:
    ip = np.ascontiguousarray(indptr, dtype=np.int32)
    ix = np.ascontiguousarray(indices, dtype=np.int32)
    if ix.size == 0:
        ix = np.zeros(1, dtype=np.int32)
    h = np.ascontiguousarray(h_src, dtype=np.float64)
    n = ip.shape[0] - 1
    d = h.shape[1]
    out = np.zeros((n, d), dtype=np.float64)
    _load().orc_mean_aggregate(ip.ctypes.data, ix.ctypes.data, n, _ptr(h) or 0, d,
                               out.ctypes.data)
    return out


def block_forward(block, h_src: Sequence[Optional[np.ndarray]], w_rel, w_self, bias=None,
                  relu: bool = False) -> List[Optional[np.ndarray]]:
    """Y_t for every type with n_dst[t] > 0 (None otherwise), in float64."""
    m = _Marshal(block)
    T = len(block.n_src)
    d_in = int(np.asarray(w_rel[0] if len(w_rel) else w_self[0]).shape[0])
    d_out = int(np.asarray(w_rel[0] if len(w_rel) else w_self[0]).shape[1])
    ys = [np.zeros((block.n_dst[t], d_out), dtype=np.float64) if block.n_dst[t] > 0 else None
          for t in range(T)]
    bias = bias if bias is not None else [None] * T
    rc = _load().orc_block_forward(ctypes.byref(m.c), d_in, d_out, m.ptrs(h_src),
                                   m.ptrs(w_rel), m.ptrs(w_self),
                                   m.ptrs(bias) if any(b is not None for b in bias) else None,
                                   int(relu), m.out_ptrs(ys))
    if rc != 0:
        raise ValueError("oracle: invalid block")
    return ys


def block_backward(block, h_src, w_rel, w_self, dy, input_relu: bool = False,
                   want_dh: Optional[Sequence[bool]] = None, want_dw: bool = True):
    """Gradients of one block in float64: dict with dw_rel, dw_self, dbias, dh_src."""
    m = _Marshal(block)
    T, R = len(block.n_src), len(block.rels)
    d_in = int(np.asarray(w_self[0]).shape[0])
    d_out = int(np.asarray(w_self[0]).shape[1])
    want_dh = [True] * T if want_dh is None else list(want_dh)
    dw_rel = [np.zeros((d_in, d_out)) for _ in range(R)] if want_dw else []
    dw_self = [np.zeros((d_in, d_out)) for _ in range(T)] if want_dw else []
    dbias = [np.zeros(d_out) for _ in range(T)] if want_dw else []
    dh = [np.zeros((block.n_src[t], d_in)) if want_dh[t] else None for t in range(T)]
    rc = _load().orc_block_backward(
        ctypes.byref(m.c), d_in, d_out, m.ptrs(h_src), m.ptrs(w_rel), m.ptrs(w_self),
        m.ptrs(dy), int(input_relu),
        m.out_ptrs(dw_rel) if want_dw else None, m.out_ptrs(dw_self) if want_dw else None,
        m.out_ptrs(dbias) if want_dw else None, m.out_ptrs(dh))
    if rc != 0:
        raise ValueError("oracle: invalid block")
    return {"dw_rel": dw_rel, "dw_self": dw_self, "dbias": dbias, "dh_src": dh}


def scatter_add(ids: np.ndarray, dh: np.ndarray, demb: np.ndarray) -> None:
    """demb[ids[j]] += dh[j] in ascending j (in place; demb float64, C-contiguous)."""
    ids = np.ascontiguousarray(ids, dtype=np.int64)
    dh = np.ascontiguousarray(dh, dtype=np.float64)
    assert demb.dtype == np.float64 and demb.flags.c_contiguous
    if ids.size == 0:
        return
    if ids.min() < 0 or ids.max() >= demb.shape[0]:
        raise IndexError("oracle: scatter id out of range")
    _load().orc_scatter_add(ids.shape[0], dh.shape[1], ids.ctypes.data, dh.ctypes.data,
                            demb.ctypes.data)


def sparse_adagrad(rows: np.ndarray, grad: np.ndarray, state: np.ndarray, table: np.ndarray,
                   lr: float, eps: float) -> None:
    """Sparse Adagrad step on the listed (distinct) rows, in place on float64 C-contiguous
    state and table; grad is table-shaped float64."""
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    grad = np.ascontiguousarray(grad, dtype=np.float64)
    for a in (state, table):
        assert a.dtype == np.float64 and a.flags.c_contiguous and a.shape == grad.shape
    rc = _load().orc_sparse_adagrad(rows.shape[0], grad.shape[1], grad.shape[0],
                                    rows.ctypes.data, grad.ctypes.data, state.ctypes.data,
                                    table.ctypes.data, float(lr), float(eps))
    if rc != 0:
        raise ValueError("oracle: adagrad rows out of range or repeated")


def csc(n_src: int, indptr, indices):
    """(csc_indptr [n_src+1], csc_dst [nnz], csc_eid [nnz]) as int32."""
    ip = np.ascontiguousarray(indptr, dtype=np.int32)
    ix = np.ascontiguousarray(indices, dtype=np.int32)
    nnz = int(ip[-1])
    ix1 = ix if ix.size else np.zeros(1, dtype=np.int32)
    cip = np.zeros(n_src + 1, dtype=np.int32)
    cd = np.zeros(max(nnz, 1), dtype=np.int32)
    ce = np.zeros(max(nnz, 1), dtype=np.int32)
    rc = _load().orc_csc(n_src, ip.shape[0] - 1, ip.ctypes.data, ix1.ctypes.data,
                         cip.ctypes.data, cd.ctypes.data, ce.ctypes.data)
    if rc != 0:
        raise MemoryError
    return cip, cd[:nnz], ce[:nnz]


class _SubRel:
    def __init__(self, s, t, indptr, indices):
        self.src_type, self.dst_type, self.indptr, self.indices = s, t, indptr, indices


class _SubBlock:
    def __init__(self, n_src, n_dst, rels):
        self.n_src, self.n_dst, self.rels = n_src, n_dst, rels


def sub_block(block, dst_rows):
    """The part of ``block`` that determines the outputs of the listed destination rows.

    dst_rows[t]: sorted int array of destination rows of type t to keep.  Each kept row
    keeps its whole segment in every relation, so its aggregates and outputs, and the
    input gradient of every source row that only kept rows reference, are unchanged.
    Returns (sub, src_map): sub is a block whose destination rows of type t are the kept
    rows in the given order (the prefix of the type's sources), and src_map[t] lists, for
    each source row of the sub-block, its row in ``block``."""
    T = len(block.n_src)
    keep = [np.asarray(dst_rows[t], dtype=np.int64) for t in range(T)]
    used = [[keep[t]] for t in range(T)]
    segs = []
    for rel in block.rels:
        rows = keep[rel.dst_type]
        ip = np.asarray(rel.indptr, dtype=np.int64)
        lo, hi = ip[rows], ip[rows + 1]
        deg = hi - lo
        idx = np.concatenate([np.arange(a, b) for a, b in zip(lo, hi)]) if rows.size else np.zeros(0, np.int64)
        src = np.asarray(rel.indices, dtype=np.int64)[idx] if idx.size else np.zeros(0, np.int64)
        segs.append((deg, src))
        used[rel.src_type].append(src)
    src_map = []
    for t in range(T):
        others = np.unique(np.concatenate(used[t][1:])) if len(used[t]) > 1 else np.zeros(0, np.int64)
        others = others[~np.isin(others, keep[t])]
        src_map.append(np.concatenate([keep[t], others]))
    rels = []
    for rel, (deg, src) in zip(block.rels, segs):
        m = src_map[rel.src_type]
        order = np.argsort(m, kind="stable")
        local = order[np.searchsorted(m[order], src)] if src.size else np.zeros(0, np.int64)
        indptr = np.zeros(deg.size + 1, dtype=np.int64)
        np.cumsum(deg, out=indptr[1:])
        rels.append(_SubRel(rel.src_type, rel.dst_type, indptr.astype(np.int32),
                            local.astype(np.int32)))
    sub = _SubBlock([int(m.size) for m in src_map], [int(k.size) for k in keep], rels)
    return sub, src_map


# ------------------------------------------------------------------------------------
# Neighbour sampling and block construction (sample_oracle.c states the reading)
# ------------------------------------------------------------------------------------
def philox4x64(ctr, key) -> np.ndarray:
    """The Philox4x64-10 block function: 4 counter words, 2 key words -> 4 words."""
    c = np.ascontiguousarray(ctr, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    _load().orc_philox4x64(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def sample_draw(seed: int, layer: int, v: int, r: int, k: int) -> int:
    return int(_load().orc_sample_draw(seed, layer, v, r, k))


def sample_segment(n: int, fanout: int, seed: int, layer: int, v: int, r: int) -> np.ndarray:
    """Positions (ascending) taken from a segment of n in-edges."""
    pos = np.zeros(max(min(n, fanout), 1), dtype=np.int64)
    c = _load().orc_sample_segment(n, fanout, seed, layer, v, r, pos.ctypes.data)
    return pos[:c]


class SampledBlock:
    def __init__(self, n_src, n_dst, rels, src_ids):
        self.n_src, self.n_dst, self.rels, self.src_ids = n_src, n_dst, rels, src_ids


class _SRel:
    def __init__(self, src_type, dst_type, indptr, indices):
        self.src_type, self.dst_type, self.indptr, self.indices = src_type, dst_type, indptr, indices


def sample_block(graph, dst_ids: Sequence[np.ndarray], fanout: int, seed: int,
                 layer: int) -> SampledBlock:
    """One layer's block sampled from ``graph`` (``num_nodes`` per type; ``rels`` with
    ``src_type``, ``dst_type`` and the in-edge CSR ``indptr``/``indices``, int64 global
    ids) for the destination nodes ``dst_ids`` (per type, distinct)."""
    T, R = len(graph.num_nodes), len(graph.rels)
    dst = [np.ascontiguousarray(x, dtype=np.int64) for x in dst_ids]
    n_dst = np.array([x.shape[0] for x in dst], dtype=np.int64)
    num_nodes = np.ascontiguousarray(graph.num_nodes, dtype=np.int64)
    rel_src = np.array([r.src_type for r in graph.rels], dtype=np.int32)
    rel_dst = np.array([r.dst_type for r in graph.rels], dtype=np.int32)
    gi = [np.ascontiguousarray(r.indptr, dtype=np.int64) for r in graph.rels]
    gx = [np.ascontiguousarray(r.indices, dtype=np.int64) for r in graph.rels]
    out_ip = [np.zeros(n_dst[rel_dst[r]] + 1, dtype=np.int32) for r in range(R)]
    out_ix = [np.zeros(max(int(n_dst[rel_dst[r]]) * fanout, 1), dtype=np.int32) for r in range(R)]
    cap = [int(n_dst[t]) + sum(int(n_dst[rel_dst[r]]) * fanout for r in range(R)
                               if rel_src[r] == t) for t in range(T)]
    out_src = [np.zeros(max(c, 1), dtype=np.int64) for c in cap]
    counts = np.zeros(R + T, dtype=np.int64)

    def parr(xs):
        a = (ctypes.c_void_p * max(len(xs), 1))()
        for i, x in enumerate(xs):
            a[i] = x.ctypes.data
        return a

    rc = _load().orc_sample_block(T, R, rel_src.ctypes.data, rel_dst.ctypes.data, parr(gi),
                                  parr(gx), num_nodes.ctypes.data, parr(dst),
                                  n_dst.ctypes.data, fanout, seed, layer, parr(out_ip),
                                  parr(out_ix), parr(out_src), counts.ctypes.data)
    if rc == -1:
        raise ValueError("destination id out of range")
    if rc == -2:
        raise ValueError("repeated destination ids")
    rels = [_SRel(int(rel_src[r]), int(rel_dst[r]), out_ip[r], out_ix[r][:counts[r]])
            for r in range(R)]
    src_ids = [out_src[t][:counts[R + t]] for t in range(T)]
    return SampledBlock([int(x.shape[0]) for x in src_ids], [int(x) for x in n_dst], rels,
                        src_ids)


# ------------------------------------------------------------------------------------
# Link-prediction decoder (lp_oracle.c states the readings)
# ------------------------------------------------------------------------------------
NEG_PER_EDGE, NEG_JOINT, NEG_IN_BATCH = 0, 1, 2
LOSS_CE, LOSS_WEIGHTED_CE, LOSS_CONTRASTIVE = 0, 1, 2


def lp_loss(emb: np.ndarray, rel: Optional[np.ndarray], neg_mode: int, loss_kind: int,
            src, dst, k: int = 0, neg=None, pos_weight=None, grads: bool = True) -> dict:
    """Scores, loss and gradients of one batch of positive edges (rows of ``emb``)."""
    emb = np.ascontiguousarray(emb, dtype=np.float64)
    n, d = emb.shape
    src = np.ascontiguousarray(src, dtype=np.int64)
    dst = np.ascontiguousarray(dst, dtype=np.int64)
    B = src.shape[0]
    nn = B - 1 if neg_mode == NEG_IN_BATCH else k
    negv = np.ascontiguousarray(neg if neg is not None else np.zeros(1), dtype=np.int64)
    relv = None if rel is None else np.ascontiguousarray(rel, dtype=np.float64)
    w = None if pos_weight is None else np.ascontiguousarray(pos_weight, dtype=np.float64)
    loss = np.zeros(1)
    pos = np.zeros(max(B, 1))
    negs = np.zeros(max(B * nn, 1))
    d_emb = np.zeros((n, d)) if grads else None
    d_rel = np.zeros(d) if (grads and rel is not None) else None
    rc = _load().orc_lp_loss(n, d, emb.ctypes.data, _ptr(relv), neg_mode, loss_kind, B,
                             src.ctypes.data, dst.ctypes.data, k, negv.ctypes.data, _ptr(w),
                             loss.ctypes.data, pos.ctypes.data, negs.ctypes.data, _ptr(d_emb),
                             _ptr(d_rel))
    if rc != 0:
        raise ValueError("invalid link-prediction batch")
    return {"loss": float(loss[0]), "pos_score": pos[:B], "neg_score": negs[:B * nn].reshape(B, nn),
            "d_emb": d_emb, "d_rel": d_rel}


def lp_negatives(neg_mode: int, slots: int, num_nodes: int, seed: int) -> np.ndarray:
    out = np.zeros(max(slots, 1), dtype=np.int64)
    _load().orc_lp_negatives(neg_mode, slots, num_nodes, seed, out.ctypes.data)
    return out[:slots]


# ------------------------------------------------------------------------------------
# Feature construction for featureless nodes (feature_oracle.c states the reading)
# ------------------------------------------------------------------------------------
def featureless_mean(rels, num_nodes: int) -> np.ndarray:
    """rels: list of (indptr int64 [num_nodes + 1], indices int64, source features
    [rows x d]).  Returns the mean of each node's in-neighbours' features (fp64)."""
    R = len(rels)
    d = int(rels[0][2].shape[1]) if R else 0
    ips = [np.ascontiguousarray(r[0], dtype=np.int64) for r in rels]
    ixs = [np.ascontiguousarray(r[1] if len(r[1]) else np.zeros(1), dtype=np.int64) for r in rels]
    fts = [np.ascontiguousarray(r[2], dtype=np.float64) for r in rels]
    rows = np.array([f.shape[0] for f in fts], dtype=np.int64)
    out = np.zeros((num_nodes, d))

    def parr(xs):
        a = (ctypes.c_void_p * max(len(xs), 1))()
        for i, x in enumerate(xs):
            a[i] = x.ctypes.data
        return a

    rc = _load().orc_featureless_mean(R, parr(ips), parr(ixs), parr(fts),
                                      rows.ctypes.data if R else None, num_nodes, d,
                                      out.ctypes.data)
    if rc != 0:
        raise ValueError("neighbour index out of range")
    return out
