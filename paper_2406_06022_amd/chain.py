"""Multi-block mini-batch driver: one RGCN layer per sampled block, input side first.

Follows the model loop of the paper's programming interface (customised-model figure in
the appendix): representations are kept per node type and layer i is applied to
blocks[i].  Between layers the output goes through a ReLU (fused into the producing
transform); the last layer has no activation.  Backward runs from the last block to the
first: block l+1's input gradient is block l's output gradient, masked by the ReLU.  At
the first block the featureless node types read learnable embedding tables (Sec. 3.3.2)
and their gradient is scatter-added into table-shaped buffers, or, once an Adagrad state
is attached, applied to the tables at once (the sparse optimizer step fused into the
first block's transposed sum).

This module only allocates buffers and sequences calls of the C ABI.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import torch

from . import rgcn


class MiniBatchStack:
    def __init__(self, blocks, input_tables: Sequence[Optional[torch.Tensor]],
                 input_ids: Sequence[Optional[torch.Tensor]], weights, dtype: str,
                 dims: Sequence[int], emb_types: Sequence[int] = (), device="cuda",
                 want_weight_grads: bool = True, ids_unique: bool = True,
                 edge_rows: bool = True, relu_masks: bool = True,
                 hilo_grads: Optional[bool] = None):
        """blocks: host blocks (blocks[0] nearest the input); input_tables[t] / input_ids[t]:
        layer-0 table and int64 global row ids of each type; weights[l] = (w_rel, w_self,
        bias) device tensors of layer l; emb_types: types whose table is learnable.
        edge_rows: give the first block's per-edge source rows (``rel.src_rows``, the
        sampler's global source ids) to the library when the blocks carry them and every
        type has row ids, so its gather reads each edge's table row directly.
        relu_masks: the transforms followed by a ReLU also write the signs of their output
        as bits, and the next block's backward reads those instead of the activation rows.
        hilo_grads (default: on for bf16): the gradients passed between blocks (dh[l],
        l >= 1) are written and read in the hi/lo form, per row d_l bf16 high parts then
        d_l bf16 low parts (hi = bf16(g), lo = bf16(g - hi)), which is what the bf16
        backward products take; the buffers keep their fp32 shape and size."""
        self.L = len(blocks)
        self.dtype = dtype
        self.tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.dims = list(dims)
        self.device = device
        self.emb_types = list(emb_types)
        self.ids_unique = ids_unique
        self.hilo_grads = (dtype == "bf16") if hilo_grads is None else bool(hilo_grads)
        self.blocks: List[rgcn.DeviceBlock] = []
        rows0 = edge_rows and all(x is not None for x in input_ids)
        for l, blk in enumerate(blocks):
            if l == 0:
                mask = 0
                for t in self.emb_types:
                    mask |= 1 << t
            else:
                mask = 0
                for t in range(len(blk.n_src)):
                    if blk.n_src[t] > 0:
                        mask |= 1 << t
            self.blocks.append(rgcn.DeviceBlock(blk, mask, device, src_rows=rows0 and l == 0))
        self.params = [rgcn.Params(dtype, dims[l], dims[l + 1], *weights[l]) for l in range(self.L)]
        self.workspaces = [rgcn.new_workspace(b, p, device) for b, p in zip(self.blocks, self.params)]
        # activations: y[l][t] = output of block l, [n_dst x d_{l+1}]
        self.y = [[torch.empty((n, dims[l + 1]), dtype=self.tdtype, device=device) if n > 0 else None
                   for n in b.n_dst] for l, b in enumerate(self.blocks)]
        # ReLU sign bits of y[l] for l < L - 1 (the inputs of the next block's backward)
        words = [rgcn.relu_mask_words(dims[l + 1]) for l in range(self.L)]
        self.y_mask = [[torch.empty((n, words[l]), dtype=torch.int64, device=device)
                        if n > 0 and relu_masks and l < self.L - 1 else None
                        for n in b.n_dst] for l, b in enumerate(self.blocks)]
        self.inputs = [rgcn.Inputs(list(input_tables), list(input_ids))]
        for l in range(1, self.L):
            self.inputs.append(rgcn.Inputs(self.y[l - 1], None, self.y_mask[l - 1]))
        # gradients
        f32 = torch.float32
        self.want_weight_grads = want_weight_grads
        self.dw_rel = [[torch.empty((dims[l], dims[l + 1]), dtype=f32, device=device)
                        for _ in b.types] if want_weight_grads else None
                       for l, b in enumerate(self.blocks)]
        self.dw_self = [[torch.empty((dims[l], dims[l + 1]), dtype=f32, device=device)
                         for _ in range(b.num_types)] if want_weight_grads else None
                        for l, b in enumerate(self.blocks)]
        self.dbias = [[torch.empty((dims[l + 1],), dtype=f32, device=device)
                       if weights[l][2] is not None and weights[l][2][t] is not None else None
                       for t in range(b.num_types)] if want_weight_grads else None
                      for l, b in enumerate(self.blocks)]
        # dh[l][t]: gradient w.r.t. block l's input (l >= 1) = output gradient of block l-1
        # (in the hi/lo form with hilo_grads)
        self.dh = [None] + [[torch.empty((n, dims[l]), dtype=f32, device=device) if n > 0 else None
                             for n in b.n_src] for l, b in enumerate(self.blocks) if l >= 1]
        self.demb = [None] * len(self.blocks[0].n_src)
        for t in self.emb_types:
            tab = input_tables[t]
            self.demb[t] = torch.zeros((tab.shape[0], dims[0]), dtype=f32, device=device)
        self.adagrad = None   # (lr, eps, state per type) once attached
        self._side = None     # stream of the overlapped backward plans (created on first use)

    def attach_adagrad(self, lr: float, eps: float) -> None:
        """Zero Adagrad state per learnable table; from now on backward steps the tables
        in place instead of filling demb.  With distinct row ids (ids_unique) the step is
        fused into the first block's transposed sum; with repeated ids the gradient is
        first scatter-added into demb (cleared here) and the standalone step then runs once
        over the distinct rows, clearing the gradient rows it reads."""
        states = [None] * len(self.demb)
        self._ada_rows = [None] * len(self.demb)
        for t in self.emb_types:
            tab = self.inputs[0].bases[t]
            states[t] = torch.zeros((tab.shape[0], self.dims[0]), dtype=torch.float32,
                                    device=self.device)
            if not self.ids_unique:
                self.demb[t].zero_()
                ids = self.inputs[0].row_ids[t]
                self._ada_rows[t] = (torch.unique(ids) if ids is not None else
                                     torch.arange(self.blocks[0].n_src[t], dtype=torch.int64,
                                                  device=self.device))
        self.adagrad = (float(lr), float(eps), states)

    def release(self) -> None:
        """Drop every buffer the stack allocated (workspaces, activations, gradients,
        optimizer state); the stack cannot step afterwards."""
        self.workspaces = []
        self.y = []
        self.y_mask = []
        self.inputs = []
        self.dh = []
        self.dw_rel = self.dw_self = self.dbias = []
        self.demb = []
        self.adagrad = None

    @property
    def nnz(self) -> int:
        return sum(b.nnz for b in self.blocks)

    def plan(self, flags: int = 0, timer=None) -> None:
        for l, (b, p, ws) in enumerate(zip(self.blocks, self.params, self.workspaces)):
            _mark(timer, ("plan", l), 0)
            rgcn.rgcn_block_plan(b, p, ws, flags)
            _mark(timer, ("plan", l), 1)

    def forward(self, flags: int = 0, timer=None, after_first_aggregate=None
                ) -> List[Optional[torch.Tensor]]:
        """Forward through all blocks (each as its aggregate and transform stages).
        after_first_aggregate, if given, is called once the first block's aggregate stage is
        enqueued."""
        for l in range(self.L):
            f = flags | (rgcn.RGCN_FUSE_RELU if l < self.L - 1 else 0)
            _mark(timer, ("aggregate", l), 0)
            rgcn.rgcn_block_aggregate(self.blocks[l], self.inputs[l], self.params[l],
                                      self.workspaces[l], f)
            _mark(timer, ("aggregate", l), 1)
            if l == 0 and after_first_aggregate is not None:
                after_first_aggregate()
            _mark(timer, ("transform", l), 0)
            rgcn.rgcn_block_transform(self.blocks[l], self.params[l], self.y[l],
                                      self.workspaces[l], f & ~rgcn.RGCN_VALIDATE_DEVICE,
                                      relu_mask=self.y_mask[l] if l < self.L - 1 else None)
            _mark(timer, ("transform", l), 1)
        return self.y[-1]

    def backward(self, dy_top: Sequence[Optional[torch.Tensor]], flags: int = 0,
                 timer=None) -> None:
        """Backward from the last block to the first (dense then sparse stage per block)."""
        for l in reversed(range(self.L)):
            dy = dy_top if l == self.L - 1 else self.dh[l + 1]
            f = flags
            if self.hilo_grads and l < self.L - 1:
                f |= rgcn.RGCN_DY_HILO
            if l > 0:
                f |= rgcn.RGCN_INPUT_RELU | (rgcn.RGCN_DH_HILO if self.hilo_grads else 0)
                dh, demb = self.dh[l], None
            else:
                dh = None
                demb = self.demb if any(x is not None for x in self.demb) else None
                if self.ids_unique:
                    f |= rgcn.RGCN_IDS_UNIQUE
            _mark(timer, ("dense", l), 0)
            rgcn.rgcn_block_backward_dense(self.blocks[l], self.params[l], dy, self.dw_rel[l],
                                           self.dw_self[l], self.dbias[l],
                                           self.workspaces[l], f)
            _mark(timer, ("dense", l), 1)
            _mark(timer, ("sparse", l), 0)
            if l == 0 and self.adagrad is not None and self.emb_types:
                self.sparse_adagrad_first_block(f)
            else:
                rgcn.rgcn_block_backward_sparse(self.blocks[l], self.inputs[l], self.params[l],
                                                dh, demb, self.workspaces[l], f)
            _mark(timer, ("sparse", l), 1)

    def sparse_adagrad_first_block(self, flags: int = 0) -> None:
        """First block's transposed sum with the Adagrad step of the learnable tables
        (after its dense backward stage)."""
        lr, eps, states = self.adagrad
        if self.ids_unique:
            rgcn.rgcn_block_backward_sparse_adagrad(self.blocks[0], self.inputs[0],
                                                    self.params[0], states, lr, eps,
                                                    workspace=self.workspaces[0],
                                                    flags=flags | rgcn.RGCN_IDS_UNIQUE)
            return
        # repeated ids: the fused step would race on a row listed twice
        rgcn.rgcn_block_backward_sparse(self.blocks[0], self.inputs[0], self.params[0], None,
                                        self.demb, self.workspaces[0],
                                        flags & ~rgcn.RGCN_IDS_UNIQUE)
        for t in self.emb_types:
            rgcn.rgcn_sparse_adagrad(self._ada_rows[t], self.demb[t], states[t],
                                     self.inputs[0].bases[t], lr, eps, rgcn.RGCN_CLEAR_GRAD)

    def step(self, dy_top, timer=None, overlap_plan: bool = True) -> None:
        """One pass of the whole path: plan, forward, backward.

        With overlap_plan the plan is split: the forward part of every block runs first;
        the backward part (CSC transposes and backward schedules) runs on a second stream
        from the end of the first block's aggregate stage, next to the MFMA-bound transforms,
        and the backward waits for it.  Same work and results as the serial order."""
        if not overlap_plan:
            self.plan(timer=timer)
            self.forward(timer=timer)
            self.backward(dy_top, timer=timer)
            return
        if self._side is None:
            self._side = torch.cuda.Stream(device=self.device)
        main = torch.cuda.current_stream(self.device)

        def backward_plans():
            self._side.wait_stream(main)
            with torch.cuda.stream(self._side):
                for l, (b, p, ws) in enumerate(zip(self.blocks, self.params, self.workspaces)):
                    _mark(timer, ("plan_bwd", l), 0)
                    rgcn.rgcn_block_plan(b, p, ws, rgcn.RGCN_PLAN_BACKWARD)
                    _mark(timer, ("plan_bwd", l), 1)

        self.plan(rgcn.RGCN_PLAN_FORWARD, timer=timer)
        self.forward(timer=timer, after_first_aggregate=backward_plans)
        main.wait_stream(self._side)
        self.backward(dy_top, timer=timer)


    def capture_step(self, dy_top, overlap_plan: bool = True) -> "torch.cuda.CUDAGraph":
        """Record one step (plan, forward, backward, and the optimizer step when attached)
        into a HIP graph; ``graph.replay()`` then reruns it with one launch from the host.
        Every buffer the step touches is allocated already, the library allocates nothing
        and clears no memory with memset nodes (its counters are cleared by kernels), and a
        step has no host synchronisation, so the recorded launches are the step.  One eager
        step on a side stream comes first (it creates the plan's second stream)."""
        side = torch.cuda.Stream(device=self.device)
        side.wait_stream(torch.cuda.current_stream(self.device))
        with torch.cuda.stream(side):
            self.step(dy_top, overlap_plan=overlap_plan)
        torch.cuda.current_stream(self.device).wait_stream(side)
        torch.cuda.synchronize(self.device)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, capture_error_mode="thread_local"):
            self.step(dy_top, overlap_plan=overlap_plan)
        return graph


def _mark(timer, tag, edge: int) -> None:
    if timer is not None:
        timer(tag, edge)
