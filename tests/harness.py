"""Shared helpers of the parity tests: seeded device inputs for one block, the HIP run
through the C ABI, the oracle run on the same values, and the error metric.

Error metric: max over elements of |got - want| / max(|want|, rms(want)) (elementwise
relative error with an RMS floor, so cancellation to ~0 is not over-weighted).  Bars:
1e-5 for fp32, 2e-2 for bf16.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2406_06022_amd import rgcn, synth

TOL = {"f32": 1e-5, "bf16": 2e-2}


def to64(t):
    if t is None:
        return None
    return t.detach().to("cpu").to(torch.float64).numpy()


def rel_err(got, want) -> float:
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    if want.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(want * want)))
    den = np.maximum(np.abs(want), rms)
    den = np.where(den > 0, den, 1.0)
    return float(np.max(np.abs(got - want) / den))


def hilo_split(x: torch.Tensor) -> torch.Tensor:
    """fp32 rows [n, d] in the library's hi/lo form: per row the d bf16 values hi = bf16(x)
    then the d values lo = bf16(x - hi), both rounded to nearest even (x - hi is exact in
    fp32), viewed as fp32 [n, d] (the same bytes per row)."""
    hi = x.to(torch.bfloat16)
    lo = (x - hi.to(torch.float32)).to(torch.bfloat16)
    return torch.cat([hi, lo], dim=1).contiguous().view(torch.float32)


def hilo_decode(x: torch.Tensor) -> np.ndarray:
    """hi + lo in fp64 of rows in the hi/lo form."""
    d = x.shape[1]
    b = x.detach().to("cpu").contiguous().view(torch.bfloat16).to(torch.float64)
    return (b[:, :d] + b[:, d:]).numpy()


def sign_words(t: torch.Tensor) -> torch.Tensor:
    """ReLU sign bits of a [rows x d] table as the library lays them out: int64 words
    [rows x ceil(d / 64)], bit c % 64 of word c / 64 set where element c is positive."""
    pos = (t.detach().to("cpu").to(torch.float32) > 0).numpy().astype(np.uint8)
    rows, d = pos.shape
    w = (d + 63) // 64
    pad = np.zeros((rows, w * 64), dtype=np.uint8)
    pad[:, :d] = pos
    by = np.packbits(pad.reshape(rows, w, 64), axis=2, bitorder="little")
    return torch.from_numpy(np.ascontiguousarray(by).view("<u8").reshape(rows, w).view(np.int64))


def gather_rows(table64: np.ndarray, ids) -> np.ndarray:
    """Input rows H[j] = table[ids[j]] (the oracle's first step at the input layer)."""
    if ids is None:
        return table64
    return table64[np.asarray(ids, dtype=np.int64)]


class BlockRun:
    """One block with seeded inputs, run on the GPU and (optionally) through the oracle."""

    def __init__(self, blk, dtype: str, d_in: int, d_out: int, seed: int, *,
                 grad_types=None, use_ids: bool = False, bias: bool = False,
                 input_relu: bool = False, fwd_relu: bool = False, emb_types=(),
                 ids_unique: bool = True, dup_ids: bool = False, device="cuda",
                 edge_rows: bool = False, mask_in: bool = False, mask_out: bool = False):
        self.blk, self.dtype, self.d_in, self.d_out = blk, dtype, d_in, d_out
        T, R = len(blk.n_src), len(blk.rels)
        tdt = synth.torch_dtype(dtype)
        gen = torch.Generator().manual_seed(seed)
        self.grad_types = list(range(T)) if grad_types is None else list(grad_types)
        self.emb_types = list(emb_types)
        self.input_relu, self.fwd_relu = input_relu, fwd_relu
        self.tables, self.ids = [], []
        for t in range(T):
            n = blk.n_src[t]
            if use_ids:
                rows = n + 17 + n // 3
                tab = torch.randn((rows, d_in), generator=gen).to(tdt)
                if dup_ids and n > 1:
                    ids = torch.randint(0, rows, (n,), generator=gen)
                else:
                    ids = torch.randperm(rows, generator=gen)[:n]
                self.ids.append(ids.to(torch.int64))
            else:
                tab = torch.randn((max(n, 1), d_in), generator=gen).to(tdt)
                self.ids.append(None)
            if input_relu:
                tab = torch.relu(tab)
            self.tables.append(tab)
        w_rel, w_self, b = synth.block_weights(T, R, d_in, d_out, tdt, seed, with_bias=bias)
        self.w_rel, self.w_self, self.bias = w_rel, w_self, b
        self.dy = [torch.randn((blk.n_dst[t], d_out), generator=gen, dtype=torch.float32)
                   for t in range(T)]
        mask = 0
        for t in set(self.grad_types) | set(self.emb_types):
            mask |= 1 << t
        self.flags_bwd = (rgcn.RGCN_INPUT_RELU if input_relu else 0) | (
            rgcn.RGCN_IDS_UNIQUE if ids_unique else 0)
        self.mask = mask
        self.device = device
        # give the library each edge's table row (ids[src][indices]) as a sampler would
        self.edge_rows = edge_rows
        # mask_in: the backward reads the input's ReLU signs as bits (from the tables);
        # mask_out: the forward also writes the signs of y (with fwd_relu)
        self.mask_in, self.mask_out = mask_in, mask_out

    # ------------------------------------------------------------------ GPU
    def device_setup(self):
        """Device copies of the block, weights, inputs and a NaN-filled workspace."""
        dev = self.device
        blk = self.blk
        if self.edge_rows:
            rels = []
            for rel in blk.rels:
                ix = np.asarray(rel.indices, dtype=np.int64)
                ids = self.ids[rel.src_type]
                rows = ids.numpy()[ix] if ids is not None else ix
                rels.append(synth.Relation(rel.src_type, rel.dst_type, rel.indptr, rel.indices,
                                           rows))
            self.dblk = rgcn.DeviceBlock(synth.Block(list(blk.n_src), list(blk.n_dst), rels),
                                         self.mask, dev, src_rows=True)
        else:
            self.dblk = rgcn.DeviceBlock(blk, self.mask, dev)
        d_wr = [w.to(dev) for w in self.w_rel]
        d_ws = [w.to(dev) for w in self.w_self]
        d_b = [x.to(dev) if x is not None else None for x in self.bias]
        self.params = rgcn.Params(self.dtype, self.d_in, self.d_out, d_wr, d_ws,
                                  d_b if any(x is not None for x in d_b) else None)
        self.d_tables = [t.to(dev) for t in self.tables]
        self.d_ids = [i.to(dev) if i is not None else None for i in self.ids]
        masks = [sign_words(t).to(dev) for t in self.tables] if self.mask_in else None
        self.inputs = rgcn.Inputs(self.d_tables, self.d_ids, masks)
        self.ws = rgcn.new_workspace(self.dblk, self.params, dev)
        # every byte the library reads before writing would show up as NaN (0xFF bytes are
        # NaN in fp32 and bf16)
        self.ws.fill_(0xFF)

    def run_gpu(self, validate: bool = False, repeat: int = 1, plan_flags: int = 0,
                hilo_flags: int = 0):
        """hilo_flags: RGCN_DY_HILO passes dy in the hi/lo form; RGCN_DH_HILO has dh written
        in it (returned as stored)."""
        dev = self.device
        blk = self.blk
        T = len(blk.n_src)
        self.device_setup()
        tdt = synth.torch_dtype(self.dtype)
        f32 = torch.float32
        flags = rgcn.RGCN_VALIDATE_DEVICE if validate else 0
        outs = []
        for _ in range(repeat):
            y = [torch.full((n, self.d_out), float("nan"), dtype=tdt, device=dev) if n > 0 else None
                 for n in blk.n_dst]
            dy = [(hilo_split(x) if hilo_flags & rgcn.RGCN_DY_HILO else x).to(dev)
                  for x in self.dy]
            dw_rel = [torch.full((self.d_in, self.d_out), float("nan"), dtype=f32, device=dev)
                      for _ in blk.rels]
            dw_self = [torch.full((self.d_in, self.d_out), float("nan"), dtype=f32, device=dev)
                       for _ in range(T)]
            dbias = [torch.full((self.d_out,), float("nan"), dtype=f32, device=dev)
                     if self.bias[t] is not None else None for t in range(T)]
            dh = [torch.full((blk.n_src[t], self.d_in), float("nan"), dtype=f32, device=dev)
                  if t in self.grad_types else None for t in range(T)]
            demb = [torch.zeros((self.tables[t].shape[0], self.d_in), dtype=f32, device=dev)
                    if t in self.emb_types else None for t in range(T)]
            # sign words start as all ones (0xFF bytes): every word must be written
            ym = ([torch.full((n, rgcn.relu_mask_words(self.d_out)), -1, dtype=torch.int64,
                              device=dev) if n > 0 else None for n in blk.n_dst]
                  if self.mask_out else None)
            rgcn.rgcn_block_plan(self.dblk, self.params, self.ws, flags | plan_flags)
            rgcn.rgcn_block_forward(self.dblk, self.inputs, self.params, y, self.ws,
                                    flags | (rgcn.RGCN_FUSE_RELU if self.fwd_relu else 0),
                                    relu_mask=ym)
            rgcn.rgcn_block_backward(self.dblk, self.inputs, self.params, dy, dw_rel, dw_self,
                                     dbias, dh, demb if self.emb_types else None, self.ws,
                                     flags | self.flags_bwd | hilo_flags)
            torch.cuda.synchronize()
            outs.append({"y": [x.cpu() if x is not None else None for x in y],
                         "dw_rel": [x.cpu() for x in dw_rel],
                         "dw_self": [x.cpu() for x in dw_self],
                         "dbias": [x.cpu() if x is not None else None for x in dbias],
                         "dh": [x.cpu() if x is not None else None for x in dh],
                         "demb": [x.cpu() if x is not None else None for x in demb],
                         "y_mask": ([x.cpu() if x is not None else None for x in ym]
                                    if ym is not None else None)})
        self.gpu = outs[0]
        return outs

    # ------------------------------------------------------------------ oracle
    def run_oracle(self):
        blk = self.blk
        T = len(blk.n_src)
        h = [gather_rows(to64(self.tables[t]), self.ids[t])[: blk.n_src[t]] for t in range(T)]
        w_rel = [to64(w) for w in self.w_rel]
        w_self = [to64(w) for w in self.w_self]
        bias = [to64(b) if b is not None else None for b in self.bias]
        dy = [to64(x) for x in self.dy]
        y = oracle.block_forward(blk, h, w_rel, w_self, bias, relu=self.fwd_relu)
        want_dh = [t in self.grad_types or t in self.emb_types for t in range(T)]
        g = oracle.block_backward(blk, h, w_rel, w_self, dy, input_relu=self.input_relu,
                                  want_dh=want_dh)
        demb = [None] * T
        for t in self.emb_types:
            d = np.zeros((self.tables[t].shape[0], self.d_in))
            ids = self.ids[t] if self.ids[t] is not None else np.arange(blk.n_src[t])
            oracle.scatter_add(np.asarray(ids), g["dh_src"][t], d)
            demb[t] = d
        self.ref = {"y": y, "dw_rel": g["dw_rel"], "dw_self": g["dw_self"],
                    "dbias": g["dbias"], "dh": g["dh_src"], "demb": demb}
        return self.ref

    def errors(self):
        """Per-output relative errors (GPU vs oracle)."""
        out = {}
        blk = self.blk
        T = len(blk.n_src)
        for t in range(T):
            if blk.n_dst[t] > 0:
                out[f"y[{t}]"] = rel_err(to64(self.gpu["y"][t]), self.ref["y"][t])
            out[f"dw_self[{t}]"] = rel_err(to64(self.gpu["dw_self"][t]), self.ref["dw_self"][t])
            if self.bias[t] is not None:
                out[f"dbias[{t}]"] = rel_err(to64(self.gpu["dbias"][t]), self.ref["dbias"][t])
            if t in self.grad_types and blk.n_src[t] > 0:
                out[f"dh[{t}]"] = rel_err(to64(self.gpu["dh"][t]), self.ref["dh"][t])
            if t in self.emb_types:
                out[f"demb[{t}]"] = rel_err(to64(self.gpu["demb"][t]), self.ref["demb"][t])
        for r in range(len(blk.rels)):
            out[f"dw_rel[{r}]"] = rel_err(to64(self.gpu["dw_rel"][r]), self.ref["dw_rel"][r])
        return out

    def assert_parity(self, tol=None):
        tol = TOL[self.dtype] if tol is None else tol
        errs = self.errors()
        bad = {k: v for k, v in errs.items() if not (v <= tol)}
        assert not bad, f"parity failures (tol {tol}): {bad}"
        return errs
