"""Python binding of librgcn (include/rgcn.h): argument marshalling only.

Every function here passes device pointers and sizes across the C ABI and raises
``RgcnError`` on a non-OK status.  No arithmetic of the layer happens in Python; there is
no CPU fallback.  Tensors are torch tensors used as device memory; the stream is torch's
current stream unless one is given.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# RGCN_LIB_SANITIZE=1 loads the host-sanitized build of the same sources (CPU-side checks
# of the argument validation; needs the ASan runtime preloaded)
LIB_PATH = os.path.join(_HERE, "librgcn_san.so" if os.environ.get("RGCN_LIB_SANITIZE") == "1"
                        else "librgcn.so")

RGCN_F32, RGCN_BF16 = 0, 1
RGCN_MAX_TYPES, RGCN_MAX_RELS = 16, 64
RGCN_VALIDATE_DEVICE = 0x1
RGCN_FUSE_RELU = 0x2
RGCN_INPUT_RELU = 0x4
RGCN_IDS_UNIQUE = 0x8
RGCN_CLEAR_GRAD = 0x10
RGCN_PLAN_FORWARD = 0x20
RGCN_PLAN_BACKWARD = 0x40
RGCN_PLAN_ENUMERATION_ORDER = 0x80
RGCN_DY_HILO = 0x100
RGCN_DH_HILO = 0x200
STATUS_NAMES = {0: "RGCN_OK", 1: "RGCN_ERR_INVALID_ARG", 2: "RGCN_ERR_SHAPE",
                3: "RGCN_ERR_DTYPE", 4: "RGCN_ERR_INDEX_OOB", 5: "RGCN_ERR_BAD_CSR",
                6: "RGCN_ERR_WORKSPACE_TOO_SMALL", 7: "RGCN_ERR_UNSUPPORTED", 8: "RGCN_ERR_HIP"}
EXPORTED = ("rgcn_block_workspace_size", "rgcn_block_plan_layout", "rgcn_block_plan",
            "rgcn_block_forward", "rgcn_block_backward", "rgcn_block_aggregate",
            "rgcn_block_transform", "rgcn_block_backward_dense", "rgcn_block_backward_sparse",
            "rgcn_block_backward_sparse_adagrad", "rgcn_sparse_adagrad",
            "rgcn_sample_workspace_size", "rgcn_sample_block", "rgcn_lp_workspace_size",
            "rgcn_lp_loss", "rgcn_lp_loss_noalloc", "rgcn_lp_negatives", "rgcn_featureless_mean", "rgcn_last_error",
            "rgcn_version")
RGCN_FEATURELESS_WORKSPACE = 256
RGCN_LP_NEG_PER_EDGE, RGCN_LP_NEG_JOINT, RGCN_LP_NEG_IN_BATCH = 0, 1, 2
RGCN_LP_CE, RGCN_LP_WEIGHTED_CE, RGCN_LP_CONTRASTIVE = 0, 1, 2
RGCN_LP_NOALLOC_MAX_SCRATCH = 32 << 20
RGCN_MAX_FANOUT = 64


class RgcnError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class _Relation(ctypes.Structure):
    _fields_ = [("src_type", ctypes.c_int32), ("dst_type", ctypes.c_int32),
                ("nnz", ctypes.c_int64), ("indptr", ctypes.c_void_p),
                ("indices", ctypes.c_void_p), ("src_rows", ctypes.c_void_p)]


class _Block(ctypes.Structure):
    _fields_ = [("num_types", ctypes.c_int32), ("num_rels", ctypes.c_int32),
                ("n_src", ctypes.POINTER(ctypes.c_int64)), ("n_dst", ctypes.POINTER(ctypes.c_int64)),
                ("rels", ctypes.POINTER(_Relation)), ("grad_src_types", ctypes.c_uint32)]


class _Input(ctypes.Structure):
    _fields_ = [("base", ctypes.c_void_p), ("row_ids", ctypes.c_void_p),
                ("num_rows", ctypes.c_int64), ("ld", ctypes.c_int64),
                ("relu_mask", ctypes.c_void_p)]


class _Params(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("d_in", ctypes.c_int32), ("d_out", ctypes.c_int32),
                ("w_rel", ctypes.POINTER(ctypes.c_void_p)),
                ("w_self", ctypes.POINTER(ctypes.c_void_p)),
                ("bias", ctypes.POINTER(ctypes.c_void_p))]


class _Adagrad(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("eps", ctypes.c_float),
                ("state", ctypes.POINTER(ctypes.c_void_p)),
                ("table", ctypes.POINTER(ctypes.c_void_p))]


class _GraphRel(ctypes.Structure):
    _fields_ = [("src_type", ctypes.c_int32), ("dst_type", ctypes.c_int32),
                ("indptr", ctypes.c_void_p), ("indices", ctypes.c_void_p)]


class _Graph(ctypes.Structure):
    _fields_ = [("num_types", ctypes.c_int32), ("num_rels", ctypes.c_int32),
                ("num_nodes", ctypes.POINTER(ctypes.c_int64)), ("rels", ctypes.POINTER(_GraphRel))]


class _LpBatch(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("d", ctypes.c_int32), ("n_rows", ctypes.c_int64),
                ("ld", ctypes.c_int64), ("emb", ctypes.c_void_p), ("rel", ctypes.c_void_p),
                ("neg_mode", ctypes.c_int32), ("loss", ctypes.c_int32), ("batch", ctypes.c_int64),
                ("src", ctypes.c_void_p), ("dst", ctypes.c_void_p), ("k", ctypes.c_int32),
                ("neg", ctypes.c_void_p), ("pos_weight", ctypes.c_void_p)]


class _FeatureRel(ctypes.Structure):
    _fields_ = [("indptr", ctypes.c_void_p), ("indices", ctypes.c_void_p),
                ("features", ctypes.c_void_p), ("rows", ctypes.c_int64), ("ld", ctypes.c_int64)]


class _PlanLayout(ctypes.Structure):
    _fields_ = [("n_fwd_segments", ctypes.c_int64), ("fwd_order", ctypes.c_size_t),
                ("n_bwd_rows", ctypes.c_int64), ("bwd_order", ctypes.c_size_t),
                ("csc_indptr", ctypes.c_size_t * RGCN_MAX_RELS),
                ("csc_dst", ctypes.c_size_t * RGCN_MAX_RELS),
                ("total_bytes", ctypes.c_size_t)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load librgcn.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with "
                               "`python -m paper_2406_06022_amd.build`")
        lib = ctypes.CDLL(path)
        vp, st = ctypes.c_void_p, ctypes.c_int
        lib.rgcn_block_workspace_size.argtypes = [vp, vp, ctypes.POINTER(ctypes.c_size_t)]
        lib.rgcn_block_workspace_size.restype = st
        lib.rgcn_block_plan_layout.argtypes = [vp, vp, vp]
        lib.rgcn_block_plan_layout.restype = st
        lib.rgcn_block_plan.argtypes = [vp, vp, vp, ctypes.c_size_t, ctypes.c_uint, vp]
        lib.rgcn_block_plan.restype = st
        lib.rgcn_block_forward.argtypes = [vp, vp, vp, vp, vp, vp, ctypes.c_size_t, ctypes.c_uint,
                                           vp]
        lib.rgcn_block_forward.restype = st
        lib.rgcn_block_backward.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                            ctypes.c_size_t, ctypes.c_uint, vp]
        lib.rgcn_block_backward.restype = st
        lib.rgcn_block_aggregate.argtypes = [vp, vp, vp, vp, ctypes.c_size_t, ctypes.c_uint, vp]
        lib.rgcn_block_aggregate.restype = st
        lib.rgcn_block_transform.argtypes = [vp, vp, vp, vp, vp, ctypes.c_size_t, ctypes.c_uint,
                                             vp]
        lib.rgcn_block_transform.restype = st
        lib.rgcn_block_backward_dense.argtypes = [vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t,
                                                  ctypes.c_uint, vp]
        lib.rgcn_block_backward_dense.restype = st
        lib.rgcn_block_backward_sparse.argtypes = [vp, vp, vp, vp, vp, vp, ctypes.c_size_t,
                                                   ctypes.c_uint, vp]
        lib.rgcn_block_backward_sparse.restype = st
        lib.rgcn_block_backward_sparse_adagrad.argtypes = [vp, vp, vp, vp, vp, vp, vp,
                                                           ctypes.c_size_t, ctypes.c_uint, vp]
        lib.rgcn_block_backward_sparse_adagrad.restype = st
        lib.rgcn_sparse_adagrad.argtypes = [ctypes.c_int64, vp, ctypes.c_int64, ctypes.c_int32,
                                            vp, vp, vp, ctypes.c_int64, ctypes.c_int,
                                            ctypes.c_float, ctypes.c_float, ctypes.c_uint, vp]
        lib.rgcn_sparse_adagrad.restype = st
        lib.rgcn_sample_workspace_size.argtypes = [vp, vp, ctypes.c_int32, vp]
        lib.rgcn_sample_workspace_size.restype = st
        lib.rgcn_sample_block.argtypes = [vp, vp, vp, ctypes.c_int32, ctypes.c_uint64,
                                          ctypes.c_int32, vp, vp, vp, vp, vp, vp,
                                          ctypes.c_size_t, ctypes.c_uint, vp]
        lib.rgcn_sample_block.restype = st
        lib.rgcn_lp_workspace_size.argtypes = [vp, vp]
        lib.rgcn_lp_workspace_size.restype = st
        lib.rgcn_lp_loss.argtypes = [vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, ctypes.c_uint, vp]
        lib.rgcn_lp_loss.restype = st
        lib.rgcn_lp_loss_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, ctypes.c_uint, vp]
        lib.rgcn_lp_loss_noalloc.restype = st
        lib.rgcn_lp_negatives.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_uint64, vp, vp]
        lib.rgcn_lp_negatives.restype = st
        lib.rgcn_featureless_mean.argtypes = [ctypes.c_int32, vp, ctypes.c_int64, ctypes.c_int32,
                                              ctypes.c_int, vp, ctypes.c_int64, vp, ctypes.c_uint,
                                              vp]
        lib.rgcn_featureless_mean.restype = st
        lib.rgcn_last_error.restype = ctypes.c_char_p
        lib.rgcn_version.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def _check(status: int) -> None:
    if status != 0:
        raise RgcnError(status, load_library().rgcn_last_error().decode())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _ptr_array(ptrs: Sequence[Optional[int]]):
    arr = (ctypes.c_void_p * max(len(ptrs), 1))()
    for i, p in enumerate(ptrs):
        arr[i] = p
    return arr


# ------------------------------------------------------------------------------------
class DeviceBlock:
    """A block's structure in device memory plus its C mirror.

    ``blk`` is anything with ``n_src``, ``n_dst`` and ``rels`` (each relation with
    ``src_type``, ``dst_type``, ``indptr`` and ``indices``); arrays are copied to
    ``device`` as int32.  With ``src_rows`` the relations' per-edge input-table rows
    (``rel.src_rows``, int64, the sampler's global source ids) go along too (the input
    layer only: they must equal row_ids[indices])."""

    def __init__(self, blk, grad_src_types: int = 0, device="cuda", src_rows: bool = False):
        self.n_src = [int(x) for x in blk.n_src]
        self.n_dst = [int(x) for x in blk.n_dst]
        self.num_types = len(self.n_src)
        self.grad_src_types = int(grad_src_types)
        self.indptr: List[torch.Tensor] = []
        self.indices: List[torch.Tensor] = []
        self.src_rows: List[Optional[torch.Tensor]] = []
        self.types = []
        for rel in blk.rels:
            ip = torch.as_tensor(np.ascontiguousarray(rel.indptr, dtype=np.int32)).to(device)
            ix = torch.as_tensor(np.ascontiguousarray(rel.indices, dtype=np.int32))
            ix = (ix if ix.numel() else torch.zeros(1, dtype=torch.int32)).to(device)
            self.indptr.append(ip)
            self.indices.append(ix)
            sr = getattr(rel, "src_rows", None) if src_rows else None
            if sr is not None and len(rel.indices):
                sr = torch.as_tensor(np.ascontiguousarray(sr, dtype=np.int64)).to(device)
            else:
                sr = None
            self.src_rows.append(sr)
            self.types.append((int(rel.src_type), int(rel.dst_type), int(len(rel.indices))))
        self.num_rels = len(self.types)
        self._n_src = (ctypes.c_int64 * self.num_types)(*self.n_src)
        self._n_dst = (ctypes.c_int64 * self.num_types)(*self.n_dst)
        self._rels = (_Relation * max(self.num_rels, 1))()
        for r, (s, t, nnz) in enumerate(self.types):
            self._rels[r] = _Relation(s, t, nnz, self.indptr[r].data_ptr(),
                                      self.indices[r].data_ptr(), _ptr(self.src_rows[r]))
        self.c = _Block(self.num_types, self.num_rels, self._n_src, self._n_dst, self._rels,
                        self.grad_src_types)

    @property
    def nnz(self) -> int:
        return sum(x[2] for x in self.types)


class DeviceBlockView(DeviceBlock):
    """A block whose CSR arrays are already device tensors (e.g. from rgcn_sample_block):
    rels = [(src_type, dst_type, indptr int32, indices int32[, src_rows int64 or None])]."""

    def __init__(self, n_src, n_dst, rels, grad_src_types: int = 0):
        self.n_src = [int(x) for x in n_src]
        self.n_dst = [int(x) for x in n_dst]
        self.num_types = len(self.n_src)
        self.grad_src_types = int(grad_src_types)
        self.indptr = [r[2] for r in rels]
        self.indices = [r[3] for r in rels]
        self.src_rows = [r[4] if len(r) > 4 else None for r in rels]
        self.types = [(int(r[0]), int(r[1]), int(r[3].numel())) for r in rels]
        self.num_rels = len(self.types)
        self._n_src = (ctypes.c_int64 * self.num_types)(*self.n_src)
        self._n_dst = (ctypes.c_int64 * self.num_types)(*self.n_dst)
        self._rels = (_Relation * max(self.num_rels, 1))()
        for r, (s, t, nnz) in enumerate(self.types):
            self._rels[r] = _Relation(s, t, nnz, self.indptr[r].data_ptr(),
                                      self.indices[r].data_ptr(), _ptr(self.src_rows[r]))
        self.c = _Block(self.num_types, self.num_rels, self._n_src, self._n_dst, self._rels,
                        self.grad_src_types)


class DeviceGraph:
    """A full graph in device memory (in-edge CSR per relation, int64) plus its C mirror.
    ``graph`` has ``num_nodes`` and ``rels`` (``src_type``, ``dst_type``, ``indptr``,
    ``indices``; numpy arrays or torch tensors)."""

    def __init__(self, graph, device="cuda"):
        self.num_nodes = [int(x) for x in graph.num_nodes]
        self.num_types = len(self.num_nodes)
        self.indptr, self.indices, self.types = [], [], []
        for rel in graph.rels:
            ip = torch.as_tensor(rel.indptr).to(device=device, dtype=torch.int64)
            ix = torch.as_tensor(rel.indices).to(device=device, dtype=torch.int64)
            if ix.numel() == 0:
                ix = torch.zeros(1, dtype=torch.int64, device=device)
            self.indptr.append(ip.contiguous())
            self.indices.append(ix.contiguous())
            self.types.append((int(rel.src_type), int(rel.dst_type)))
        self.num_rels = len(self.types)
        self._nodes = (ctypes.c_int64 * self.num_types)(*self.num_nodes)
        self._rels = (_GraphRel * max(self.num_rels, 1))()
        for r, (s, t) in enumerate(self.types):
            self._rels[r] = _GraphRel(s, t, self.indptr[r].data_ptr(), self.indices[r].data_ptr())
        self.c = _Graph(self.num_types, self.num_rels, self._nodes, self._rels)


class Params:
    """Weights of one block (device tensors in the block dtype)."""

    def __init__(self, dtype: str, d_in: int, d_out: int, w_rel, w_self, bias=None):
        self.dtype = dtype
        self.d_in, self.d_out = int(d_in), int(d_out)
        self.w_rel, self.w_self = list(w_rel), list(w_self)
        self.bias = list(bias) if bias is not None else None
        self._w_rel = _ptr_array([_ptr(w) for w in self.w_rel])
        self._w_self = _ptr_array([_ptr(w) for w in self.w_self])
        self._bias = _ptr_array([_ptr(b) for b in self.bias]) if self.bias is not None else None
        self.c = _Params(RGCN_BF16 if dtype == "bf16" else RGCN_F32, self.d_in, self.d_out,
                         self._w_rel, self._w_self, self._bias)


class Inputs:
    """Per-type input rows: (base table, optional int64 row ids) with base [rows x ld], and
    optionally the tables' ReLU sign bits (uint64 / int64 [rows x ceil(d / 64)], as
    rgcn_block_forward writes them)."""

    def __init__(self, bases: Sequence[Optional[torch.Tensor]],
                 row_ids: Optional[Sequence[Optional[torch.Tensor]]] = None,
                 relu_masks: Optional[Sequence[Optional[torch.Tensor]]] = None):
        self.bases = list(bases)
        self.row_ids = list(row_ids) if row_ids is not None else [None] * len(self.bases)
        self.relu_masks = (list(relu_masks) if relu_masks is not None
                           else [None] * len(self.bases))
        self.c = (_Input * max(len(self.bases), 1))()
        for t, (b, ids, mk) in enumerate(zip(self.bases, self.row_ids, self.relu_masks)):
            if b is None:
                self.c[t] = _Input(None, None, 0, 0, None)
            else:
                self.c[t] = _Input(b.data_ptr(), _ptr(ids), int(b.shape[0]), int(b.stride(0)),
                                   _ptr(mk))


# ------------------------------------------------------------------------------------
def rgcn_version() -> str:
    return load_library().rgcn_version().decode()


def rgcn_last_error() -> str:
    return load_library().rgcn_last_error().decode()


def rgcn_block_workspace_size(block: DeviceBlock, params: Params) -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().rgcn_block_workspace_size(ctypes.byref(block.c), ctypes.byref(params.c),
                                                    ctypes.byref(out)))
    return int(out.value)


def rgcn_block_plan_layout(block: DeviceBlock, params: Params) -> dict:
    lay = _PlanLayout()
    _check(load_library().rgcn_block_plan_layout(ctypes.byref(block.c), ctypes.byref(params.c),
                                                 ctypes.byref(lay)))
    none = (1 << (8 * ctypes.sizeof(ctypes.c_size_t))) - 1
    return {"n_fwd_segments": lay.n_fwd_segments, "fwd_order": lay.fwd_order,
            "n_bwd_rows": lay.n_bwd_rows, "bwd_order": lay.bwd_order,
            "csc_indptr": [None if x == none else x for x in lay.csc_indptr],
            "csc_dst": [None if x == none else x for x in lay.csc_dst],
            "total_bytes": lay.total_bytes}


def new_workspace(block: DeviceBlock, params: Params, device="cuda") -> torch.Tensor:
    return torch.empty(rgcn_block_workspace_size(block, params), dtype=torch.uint8, device=device)


def rgcn_block_plan(block: DeviceBlock, params: Params, workspace: torch.Tensor, flags: int = 0,
                    stream=None) -> None:
    _check(load_library().rgcn_block_plan(ctypes.byref(block.c), ctypes.byref(params.c),
                                          workspace.data_ptr(), workspace.numel(), flags,
                                          _stream(stream)))


def relu_mask_words(d: int) -> int:
    """uint64 words per row of a ReLU sign mask of width d."""
    return (d + 63) // 64


def rgcn_block_forward(block: DeviceBlock, inputs: Inputs, params: Params,
                       y: Sequence[Optional[torch.Tensor]], workspace: torch.Tensor,
                       flags: int = 0, stream=None,
                       relu_mask: Optional[Sequence[Optional[torch.Tensor]]] = None) -> None:
    ys = _ptr_array([_ptr(t) for t in y])
    ms = None if relu_mask is None else _ptr_array([_ptr(t) for t in relu_mask])
    _check(load_library().rgcn_block_forward(ctypes.byref(block.c), inputs.c,
                                             ctypes.byref(params.c), ys, ms, workspace.data_ptr(),
                                             workspace.numel(), flags, _stream(stream)))


def rgcn_block_backward(block: DeviceBlock, inputs: Inputs, params: Params,
                        dy: Sequence[Optional[torch.Tensor]],
                        dw_rel: Optional[Sequence[Optional[torch.Tensor]]] = None,
                        dw_self: Optional[Sequence[Optional[torch.Tensor]]] = None,
                        dbias: Optional[Sequence[Optional[torch.Tensor]]] = None,
                        dh_src: Optional[Sequence[Optional[torch.Tensor]]] = None,
                        demb: Optional[Sequence[Optional[torch.Tensor]]] = None,
                        workspace: torch.Tensor = None, flags: int = 0, stream=None) -> None:
    def arr(xs):
        return None if xs is None else _ptr_array([_ptr(t) for t in xs])

    keep = [arr(dy), arr(dw_rel), arr(dw_self), arr(dbias), arr(dh_src), arr(demb)]
    _check(load_library().rgcn_block_backward(
        ctypes.byref(block.c), inputs.c, ctypes.byref(params.c), *keep,
        workspace.data_ptr(), workspace.numel(), flags, _stream(stream)))


def rgcn_block_aggregate(block: DeviceBlock, inputs: Inputs, params: Params,
                         workspace: torch.Tensor, flags: int = 0, stream=None) -> None:
    _check(load_library().rgcn_block_aggregate(ctypes.byref(block.c), inputs.c,
                                               ctypes.byref(params.c), workspace.data_ptr(),
                                               workspace.numel(), flags, _stream(stream)))


def rgcn_block_transform(block: DeviceBlock, params: Params, y: Sequence[Optional[torch.Tensor]],
                         workspace: torch.Tensor, flags: int = 0, stream=None,
                         relu_mask: Optional[Sequence[Optional[torch.Tensor]]] = None) -> None:
    ys = _ptr_array([_ptr(t) for t in y])
    ms = None if relu_mask is None else _ptr_array([_ptr(t) for t in relu_mask])
    _check(load_library().rgcn_block_transform(ctypes.byref(block.c), ctypes.byref(params.c), ys,
                                               ms, workspace.data_ptr(), workspace.numel(), flags,
                                               _stream(stream)))


def rgcn_block_backward_dense(block: DeviceBlock, params: Params,
                              dy: Sequence[Optional[torch.Tensor]], dw_rel=None, dw_self=None,
                              dbias=None, workspace: torch.Tensor = None, flags: int = 0,
                              stream=None) -> None:
    def arr(xs):
        return None if xs is None else _ptr_array([_ptr(t) for t in xs])

    keep = [arr(dy), arr(dw_rel), arr(dw_self), arr(dbias)]
    _check(load_library().rgcn_block_backward_dense(
        ctypes.byref(block.c), ctypes.byref(params.c), *keep, workspace.data_ptr(),
        workspace.numel(), flags, _stream(stream)))


def rgcn_block_backward_sparse(block: DeviceBlock, inputs: Inputs, params: Params, dh_src=None,
                               demb=None, workspace: torch.Tensor = None, flags: int = 0,
                               stream=None) -> None:
    def arr(xs):
        return None if xs is None else _ptr_array([_ptr(t) for t in xs])

    keep = [arr(dh_src), arr(demb)]
    _check(load_library().rgcn_block_backward_sparse(
        ctypes.byref(block.c), inputs.c, ctypes.byref(params.c), *keep, workspace.data_ptr(),
        workspace.numel(), flags, _stream(stream)))


def rgcn_block_backward_sparse_adagrad(block: DeviceBlock, inputs: Inputs, params: Params,
                                       state: Sequence[Optional[torch.Tensor]], lr: float,
                                       eps: float, dh_src=None, demb=None,
                                       workspace: torch.Tensor = None, flags: int = 0,
                                       stream=None) -> None:
    """Transposed sum with the Adagrad step fused in: for every type t with state[t] given,
    the table ``inputs.bases[t]`` and ``state[t]`` are updated in place."""
    def arr(xs):
        return None if xs is None else _ptr_array([_ptr(t) for t in xs])

    states = list(state) + [None] * (block.num_types - len(state))
    tables = [inputs.bases[t] if states[t] is not None else None for t in range(block.num_types)]
    st_arr, tb_arr = arr(states), arr(tables)
    opt = _Adagrad(float(lr), float(eps), st_arr, tb_arr)
    keep = [arr(dh_src), arr(demb)]
    _check(load_library().rgcn_block_backward_sparse_adagrad(
        ctypes.byref(block.c), inputs.c, ctypes.byref(params.c), *keep, ctypes.byref(opt),
        workspace.data_ptr(), workspace.numel(), flags, _stream(stream)))


def rgcn_sparse_adagrad(rows: torch.Tensor, grad: torch.Tensor, state: torch.Tensor,
                        table: torch.Tensor, lr: float, eps: float, flags: int = 0,
                        stream=None) -> None:
    """Adagrad step of the listed rows of ``table`` (rows int64; grad and state fp32
    [num_rows x d]; table [num_rows x ld], bf16 or fp32), all updated in place."""
    dt = RGCN_BF16 if table.dtype == torch.bfloat16 else RGCN_F32
    _check(load_library().rgcn_sparse_adagrad(
        int(rows.numel()), rows.data_ptr(), int(table.shape[0]), int(grad.shape[1]),
        grad.data_ptr(), state.data_ptr(), table.data_ptr(), int(table.stride(0)), dt,
        float(lr), float(eps), int(flags), _stream(stream)))


def rgcn_sample_workspace_size(graph: DeviceGraph, n_dst: Sequence[int], fanout: int) -> int:
    out = ctypes.c_size_t(0)
    nd = (ctypes.c_int64 * graph.num_types)(*[int(x) for x in n_dst])
    _check(load_library().rgcn_sample_workspace_size(ctypes.byref(graph.c), nd, int(fanout),
                                                     ctypes.byref(out)))
    return int(out.value)


def rgcn_sample_block(graph: DeviceGraph, dst_ids: Sequence[torch.Tensor], fanout: int,
                      seed: int, layer: int, workspace: Optional[torch.Tensor] = None,
                      flags: int = 0, stream=None, src_rows: bool = False):
    """One layer's block for destination ids ``dst_ids[t]`` (device int64).  Returns
    (out_indptr, out_indices, out_src_ids, counts) -- capacity-sized device tensors and the
    device int64 counts [num_rels + num_types] -- and, with ``src_rows``, a fifth element:
    the global source id of every sampled edge per relation."""
    T, R = graph.num_types, graph.num_rels
    dev = graph.indptr[0].device if R else dst_ids[0].device
    n_dst = [int(x.numel()) for x in dst_ids]
    if workspace is None:
        workspace = torch.empty(rgcn_sample_workspace_size(graph, n_dst, fanout),
                                dtype=torch.uint8, device=dev)
    out_ip = [torch.empty(n_dst[t] + 1, dtype=torch.int32, device=dev) for (_, t) in graph.types]
    out_ix = [torch.empty(max(n_dst[t] * fanout, 1), dtype=torch.int32, device=dev)
              for (_, t) in graph.types]
    cap = [n_dst[t] + sum(n_dst[d] * fanout for (s, d) in graph.types if s == t) for t in range(T)]
    out_src = [torch.empty(max(c, 1), dtype=torch.int64, device=dev) for c in cap]
    out_rows = ([torch.empty(max(n_dst[t] * fanout, 1), dtype=torch.int64, device=dev)
                 for (_, t) in graph.types] if src_rows else None)
    counts = torch.zeros(R + T, dtype=torch.int64, device=dev)
    ids = [x.contiguous() for x in dst_ids]
    keep = [_ptr_array([_ptr(x) for x in ids]), _ptr_array([_ptr(x) for x in out_ip]),
            _ptr_array([_ptr(x) for x in out_ix]), _ptr_array([_ptr(x) for x in out_src]),
            _ptr_array([_ptr(x) for x in out_rows]) if src_rows else None]
    nd = (ctypes.c_int64 * T)(*n_dst)
    _check(load_library().rgcn_sample_block(
        ctypes.byref(graph.c), keep[0], nd, int(fanout), int(seed), int(layer), keep[1],
        keep[2], keep[3], keep[4], counts.data_ptr(), workspace.data_ptr(), workspace.numel(),
        flags, _stream(stream)))
    if src_rows:
        return out_ip, out_ix, out_src, counts, out_rows
    return out_ip, out_ix, out_src, counts


def lp_batch(emb: torch.Tensor, rel: Optional[torch.Tensor], neg_mode: int, loss_kind: int,
             src: torch.Tensor, dst: torch.Tensor, k: int = 0, neg: Optional[torch.Tensor] = None,
             pos_weight: Optional[torch.Tensor] = None, d: Optional[int] = None):
    """The C description of a link-prediction batch (tensors must stay alive)."""
    dt = RGCN_BF16 if emb.dtype == torch.bfloat16 else RGCN_F32
    return _LpBatch(dt, int(d if d is not None else emb.shape[1]), int(emb.shape[0]),
                    int(emb.stride(0)), emb.data_ptr(), _ptr(rel), int(neg_mode), int(loss_kind),
                    int(src.numel()), src.data_ptr(), dst.data_ptr(), int(k), _ptr(neg),
                    _ptr(pos_weight))


def rgcn_lp_workspace_size(batch: "_LpBatch") -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().rgcn_lp_workspace_size(ctypes.byref(batch), ctypes.byref(out)))
    return int(out.value)


def rgcn_lp_loss(batch: "_LpBatch", loss: torch.Tensor, pos_score=None, neg_score=None,
                 d_emb=None, d_rel=None, workspace: Optional[torch.Tensor] = None, flags: int = 0,
                 stream=None) -> None:
    if workspace is None:
        workspace = torch.empty(rgcn_lp_workspace_size(batch), dtype=torch.uint8,
                                device=loss.device)
    _check(load_library().rgcn_lp_loss(ctypes.byref(batch), loss.data_ptr(), _ptr(pos_score),
                                       _ptr(neg_score), _ptr(d_emb), _ptr(d_rel),
                                       workspace.data_ptr(), workspace.numel(), flags,
                                       _stream(stream)))


def rgcn_lp_loss_noalloc(batch: "_LpBatch", loss: torch.Tensor, pos_score=None,
                         neg_score=None, d_emb=None, d_rel=None, flags: int = 0,
                         stream=None) -> None:
    """rgcn_lp_loss with the library's fixed per-device scratch array instead of a
    workspace (allocates nothing)."""
    _check(load_library().rgcn_lp_loss_noalloc(ctypes.byref(batch), loss.data_ptr(),
                                               _ptr(pos_score), _ptr(neg_score), _ptr(d_emb),
                                               _ptr(d_rel), flags, _stream(stream)))


def rgcn_lp_negatives(neg_mode: int, slots: int, num_nodes: int, seed: int, out: torch.Tensor,
                      stream=None) -> None:
    _check(load_library().rgcn_lp_negatives(int(neg_mode), int(slots), int(num_nodes), int(seed),
                                            out.data_ptr(), _stream(stream)))


def rgcn_featureless_mean(rels, num_nodes: int, out: torch.Tensor,
                          workspace: Optional[torch.Tensor] = None, flags: int = 0,
                          stream=None) -> None:
    """rels: list of (indptr int64, indices int64, features [rows x ld]) device tensors;
    out: [num_nodes x >= d] in the features' dtype (d = out.shape[1])."""
    dt = RGCN_BF16 if out.dtype == torch.bfloat16 else RGCN_F32
    arr = (_FeatureRel * max(len(rels), 1))()
    for i, (ip, ix, f) in enumerate(rels):
        arr[i] = _FeatureRel(ip.data_ptr(), ix.data_ptr(), f.data_ptr(), int(f.shape[0]),
                             int(f.stride(0)))
    if workspace is None:
        workspace = torch.empty(RGCN_FEATURELESS_WORKSPACE, dtype=torch.uint8, device=out.device)
    _check(load_library().rgcn_featureless_mean(len(rels), arr, int(num_nodes), int(out.shape[1]),
                                                dt, out.data_ptr(), int(out.stride(0)),
                                                workspace.data_ptr(), int(flags), _stream(stream)))
