#!/usr/bin/env python3
"""Throughput of the RGCN mini-batch hot path on one MI355X.

One step = one pass of the whole path over one sampled mini-batch: for every block the
integer plan (degree-sorted schedules, CSC transpose), the forward (input gather +
per-relation segmented means, MFMA transform with self-loop and relation sum, ReLU
between layers) and the backward (weight/bias gradients, input-side products,
transposed sums, embedding-gradient scatter-add into the learnable table).

Default workload: the single-GPU share of a billion-edge graph -- 3 RGCN layers with
fanouts [25, 20, 15] from 4,096 seeds, 12 relations over 4 node types, a 100M x 128 bf16
learnable embedding table resident in HBM, 128 -> 512 -> 512 -> 512.  All inputs are
synthetic and seeded, generated on the device before timing.

Prints one JSON line: aggregated edges/s (sum of edges over all blocks / step time), ms
per step and per block, the roofline of the dominant kernel (HIP events around its
launches inside the timed steps), and the CPU oracle timed on a bounded sample.  The steps
run twice: launched eagerly, with HIP events around every stage (the per-stage times and
rooflines), then recorded once into a HIP graph and replayed (the headline step time; the
same launches, one host launch per step).
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16
METRIC = "aggregated edges/sec and ms per RGCN block fwd+bwd; % of HBM roofline"


# Files each timed kernel and its workload come from: the HBM-traffic figures recorded
# under profiles/ hold a digest of these files and count only while it still matches.
_COMMON_INPUTS = ["paper_2406_06022_amd/csrc/common.h", "include/rgcn.h",
                  "paper_2406_06022_amd/build.py", "paper_2406_06022_amd/synth.py"]
KERNEL_SOURCES = {
    "k_gather_flat": ["paper_2406_06022_amd/csrc/aggregate.hip"] + _COMMON_INPUTS,
    "k_transpose_pipe": ["paper_2406_06022_amd/csrc/aggregate.hip"] + _COMMON_INPUTS,
    "k_transpose_pipe_adagrad": ["paper_2406_06022_amd/csrc/aggregate.hip"] + _COMMON_INPUTS,
}
# Plain copy of known size run after the timed steps (an fp32 negation of a 1 GiB buffer:
# one read and one write of every byte per dispatch).  Its time gives the device's attainable
# streaming bandwidth; under rocprofv3 --pmc its HBM counters calibrate those of the timed
# kernels.
COPY_KERNEL = "neg_kernel"
COPY_BYTES = 1 << 30


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_digest(kernel: str) -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(rel.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def profile_path(kernel: str, workload: str, what: str) -> str:
    return os.path.join(ROOT, "profiles", f"{kernel}.{workload}.{what}.md")


def read_traffic(kernel: str, workload: str, position: int):
    """HBM bytes of one launch from the committed counter summary, or None when there is
    none for this kernel, workload and launch position, or the kernel's sources changed
    since the counters were taken."""
    path = profile_path(kernel, workload, "hbm")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            m = re.match(r"^- (\w+): (\S+)", line)
            if m:
                kv[m.group(1)] = m.group(2)
    if kv.get("source_digest") != source_digest(kernel):
        return None
    key = f"traffic_bytes_pos{position}"
    return float(kv[key]) if key in kv else None


def build_stack(index: int, device: str):
    import numpy as np
    import torch

    from paper_2406_06022_amd import chain, synth

    spec = synth.config(index)
    t0 = time.perf_counter()
    mb = synth.sample_minibatch(spec, device=device)
    log(f"sampled {spec.name}: blocks nnz {[b.nnz for b in mb.blocks]} in "
        f"{time.perf_counter() - t0:.1f}s")
    tdt = synth.torch_dtype(spec.dtype)
    T = len(spec.ntype_names)
    t0 = time.perf_counter()
    tables = [synth.normal_table(spec.type_rows[t], spec.dims[0], tdt, spec.seed * 10 + t,
                                 device=device) for t in range(T)]
    ids = [torch.as_tensor(mb.input_ids[t]).to(device) for t in range(T)]
    torch.cuda.synchronize()
    log(f"tables {[tuple(x.shape) for x in tables]} in {time.perf_counter() - t0:.1f}s")
    weights = []
    for l in range(spec.num_layers):
        w_rel, w_self, bias = synth.block_weights(T, len(spec.rels), spec.dims[l],
                                                  spec.dims[l + 1], tdt, spec.seed * 100 + l)
        weights.append(([w.to(device) for w in w_rel], [w.to(device) for w in w_self], None))
    emb = [t for t in range(T) if spec.featureless[t]]
    stack = chain.MiniBatchStack(mb.blocks, tables, ids, weights, spec.dtype, spec.dims,
                                 emb_types=emb, device=device)
    gen = torch.Generator(device=device)
    gen.manual_seed(spec.seed + 1)
    last = mb.blocks[-1]
    dy = [torch.randn((n, spec.dims[-1]), generator=gen, device=device, dtype=torch.float32)
          if n > 0 else None for n in last.n_dst]
    return spec, mb, tables, ids, weights, stack, dy


def method_bytes(spec, blk, dev_blk, stage: str, layer: int) -> float:
    """Algorithmic bytes of one launch of a stage's kernel as the method defines them (no
    cache reuse), the figures the roofline fractions use:
      aggregate (gather + segmented mean): per relation 4 (n_dst + 1) offsets, 4 nnz source
        indices, nnz gathered rows of d_in b bytes and one aggregate row of d_in b bytes per
        destination row written; at the input layer 8 bytes of global id per source row;
      sparse (transposed sum, embedding scatter-add): per relation leaving a type whose
        gradient is requested, one fp32 row of d_in per edge plus 8 bytes of transpose
        entry; per source row one fp32 gradient row written, and at the input layer, where
        the scatter-add into the embedding gradient is fused with the sum (distinct ids),
        that row read once more (the read half of its read-add-write)."""
    b = 2 if spec.dtype == "bf16" else 4
    d_in = spec.dims[layer]
    T = len(blk.n_src)
    if stage == "aggregate":
        tot = 0.0
        for rel in blk.rels:
            nd = blk.n_dst[rel.dst_type]
            nnz = len(rel.indices)
            tot += 4 * (nd + 1) + 4 * nnz + nnz * d_in * b + nd * d_in * b
        if layer == 0:
            tot += 8 * sum(blk.n_src)
        return tot
    if stage == "sparse":
        tot = 0.0
        for s in range(T):
            if not (dev_blk.grad_src_types >> s & 1) or blk.n_src[s] == 0:
                continue
            for rel in blk.rels:
                if rel.src_type == s and blk.n_dst[rel.dst_type] > 0:
                    tot += len(rel.indices) * (d_in * 4 + 8)
            tot += blk.n_src[s] * d_in * 4 * (2 if layer == 0 else 1)
        return tot
    raise ValueError(stage)


def algorithmic_bytes(spec, blk, dev_blk, stage: str, layer: int) -> float:
    """Bytes one launch of a stage's kernel moves in this implementation's data layout (no
    cache reuse): the method's bytes (method_bytes) plus what the layout adds -- the
    self-loop rows copied into the K-concatenated operand, an 8-byte id per gathered edge,
    the fp32 self-loop input-side rows and the ReLU sign bits the backward reads."""
    b = 2 if spec.dtype == "bf16" else 4
    d_in = spec.dims[layer]
    T = len(blk.n_src)
    if stage == "aggregate":
        # per relation: offsets, indices, one gathered row per edge (+ its 8-byte global id
        # at the input layer), one aggregate row written per destination row; per type:
        # the self-loop row read (+ id) and written
        ids = 8 if layer == 0 else 0
        tot = 0.0
        for rel in blk.rels:
            nd = blk.n_dst[rel.dst_type]
            nnz = len(rel.indices)
            tot += 4 * (nd + 1) + 4 * nnz + nnz * (d_in * b + ids) + nd * d_in * b
        for t in range(T):
            tot += blk.n_dst[t] * (2 * d_in * b + ids)
        return tot
    if stage in ("sparse", "sparse_adagrad"):
        # per requested source type: transpose offsets + destination ids + one fp32 input-
        # side row per edge, the fp32 self-loop row, the ReLU mask above the input layer
        # (the sign bits the producing transform wrote: ceil(d_in / 64) words per row),
        # and the fp32 output row (a read-add-write of the embedding-gradient row at the
        # input layer, else a write); with the fused Adagrad step the read-add-write is of
        # the fp32 state row and the table row
        tot = 0.0
        for s in range(T):
            if not (dev_blk.grad_src_types >> s & 1):
                continue
            ns = blk.n_src[s]
            out = 2 if layer == 0 else 1
            tot += ns * d_in * 4 * out + blk.n_dst[s] * d_in * 4 + (layer == 0) * 8 * ns
            tot += (layer > 0) * ns * 8 * ((d_in + 63) // 64)
            if stage == "sparse_adagrad":
                tot += ns * d_in * b * 2
            for rel in blk.rels:
                if rel.src_type == s:
                    tot += 4 * (ns + 1) + len(rel.indices) * (4 + d_in * 4)
        return tot
    raise ValueError(stage)


def transform_flops(spec, blk, layer: int) -> float:
    d_in, d_out = spec.dims[layer], spec.dims[layer + 1]
    tot = 0.0
    for t in range(len(blk.n_src)):
        if blk.n_dst[t] == 0:
            continue
        k = 1 + sum(1 for rel in blk.rels if rel.dst_type == t)
        tot += 2.0 * blk.n_dst[t] * k * d_in * d_out
    return tot


def backward_flops(spec, blk, grad_src_types: int, layer: int) -> float:
    """Flops of a block's dense backward products as the method defines them: the weight
    gradients (the forward product's flops) and the input-side products dMs = dY W^T for the
    self slot of every type whose input gradient is requested and every relation whose
    source type's is (the hi / lo split of dY doubles the MFMA work; it is not counted)."""
    d_in, d_out = spec.dims[layer], spec.dims[layer + 1]
    tot = transform_flops(spec, blk, layer)
    for t in range(len(blk.n_src)):
        if blk.n_dst[t] == 0:
            continue
        slots = 1 if grad_src_types >> t & 1 else 0
        slots += sum(1 for rel in blk.rels
                     if rel.dst_type == t and grad_src_types >> rel.src_type & 1)
        tot += 2.0 * blk.n_dst[t] * slots * d_in * d_out
    return tot


def host_info() -> dict:
    """The host the CPU baseline ran on."""
    info = {"nproc": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0))}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    info["cpu_model"] = line.split(":", 1)[1].strip()
                    break
        with open("/proc/meminfo") as f:
            for line in f:
                if line.startswith("MemTotal"):
                    info["ram_gib"] = round(int(line.split()[1]) / (1 << 20), 1)
                    break
    except OSError:
        pass
    return info


def oracle_threads() -> int:
    """Threads for the all-cores oracle run: the CPUs this process may use, at most 16 (a
    one-GPU machine's share of its host)."""
    return max(1, min(len(os.sched_getaffinity(0)), 16))


def cpu_baseline(spec, mb, tables, ids, weights, budget_s: float, threads: int):
    """The CPU oracle (fp64) on a bounded sample of block 0: the first n destination rows
    of every type with their full sampled segments, forward + backward (weight gradients
    and the embedding-type input gradient), on `threads` threads (the oracle's loops hand
    whole output elements to one thread, so results do not depend on it).  n grows until
    the run takes about budget_s seconds.  Returns edges/s of the sample."""
    import numpy as np
    import torch

    import oracle

    oracle.set_threads(threads)

    blk = mb.blocks[0]
    T = len(blk.n_src)
    emb = [t for t in range(T) if spec.featureless[t]]
    w_rel = [w.detach().cpu().to(torch.float64).numpy() for w in weights[0][0]]
    w_self = [w.detach().cpu().to(torch.float64).numpy() for w in weights[0][1]]
    n = 4
    result = None
    while True:
        keep = [np.arange(min(n, blk.n_dst[t])) for t in range(T)]
        sub, src_map = oracle.sub_block(blk, keep)
        h = []
        for t in range(T):
            rows = torch.as_tensor(mb.input_ids[t][src_map[t]], device=tables[t].device)
            h.append(tables[t].index_select(0, rows).to(torch.float64).cpu().numpy())
        gen = np.random.default_rng(5)
        dy = [gen.standard_normal((sub.n_dst[t], spec.dims[1])) for t in range(T)]
        t0 = time.perf_counter()
        oracle.block_forward(sub, h, w_rel, w_self)
        oracle.block_backward(sub, h, w_rel, w_self, dy, want_dh=[t in emb for t in range(T)])
        el = time.perf_counter() - t0
        nnz = sum(len(r.indices) for r in sub.rels)
        result = (nnz / el, nnz, el, sum(sub.n_dst))
        if el > budget_s / 3 or n >= 1 << 20:
            break
        n = int(n * max(2.0, min(8.0, budget_s / 2 / max(el, 1e-3))))
    return result


def _short_name(name: str) -> str:
    name = re.sub(r"^void ", "", name)
    name = name.replace("(anonymous namespace)::", "")
    name = re.sub(r"\(.*$", "", name)
    name = name.replace("rgcn::", "")
    return name[:90]


def _kernel_re(kernel: str) -> str:
    """Pattern of one library kernel template by its exact name (so that
    k_transpose_pipe does not also match k_transpose_pipe_adagrad)."""
    return r"\b" + re.escape(kernel) + "<"


def _dispatches(path: str, kernel_re: str, value_col=None, counter=None):
    """[(dispatch id, short name, value)] of the matching kernels, in dispatch order."""
    out = []
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            if not re.search(kernel_re, r["Kernel_Name"]):
                continue
            if counter is not None and r["Counter_Name"] != counter:
                continue
            if value_col is None:
                v = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
            else:
                v = float(r[value_col])
            out.append((int(r["Dispatch_Id"]), _short_name(r["Kernel_Name"]), v))
    out.sort()
    return out


def _by_position(rows, per_step: int, skip_steps: int, steps: int):
    """Average of each launch position over the first phase of the run: its first
    skip_steps + steps steps of per_step launches, the first skip_steps skipped (the
    training steps with the fused optimizer that follow launch the plain transposed sum
    once fewer per step, and are left out)."""
    rows = rows[skip_steps * per_step:(skip_steps + steps) * per_step]
    if per_step <= 0 or len(rows) % per_step:
        raise SystemExit(f"{len(rows)} dispatches are not a whole number of steps of {per_step}")
    pos = []
    for p in range(per_step):
        vals = [v for i, (_, _, v) in enumerate(rows) if i % per_step == p]
        pos.append((sum(vals) / len(vals), len(vals), rows[p][1]))
    return pos


def summarize_trace(args) -> str:
    """Per-kernel time of a kernel-trace run over the eagerly launched steps (warm-up and
    timed), and the launches of --kernel by position within a step.  The steps' window ends
    where the step after them starts: the gather launch that follows the last step's
    (--blocks launches per step)."""
    per, rest = {}, [0, 0.0]
    with open(args.summarize_trace, newline="") as f:
        rows = sorted(csv.DictReader(f), key=lambda r: float(r["Start_Timestamp"]))
    steps = args.steps + args.warmup
    gathers = [r for r in rows if re.search(_kernel_re("k_gather_flat"), r["Kernel_Name"])]
    lo = float(gathers[0]["Start_Timestamp"]) if gathers else 0.0
    hi = (float(gathers[steps * args.blocks]["Start_Timestamp"])
          if len(gathers) > steps * args.blocks else float("inf"))
    for r in rows:
        t0 = float(r["Start_Timestamp"])
        d = float(r["End_Timestamp"]) - t0
        if "rgcn::" in r["Kernel_Name"] and lo <= t0 < hi:
            a = per.setdefault(_short_name(r["Kernel_Name"]), [0, 0.0])
        else:
            a = rest
        a[0] += 1
        a[1] += d
    lines = [f"# {args.kernel}: kernel trace", "", "Command:", "", "```", args.command, "```", "",
             f"Launches of {args.kernel} by position within a step ({args.launches_per_step} "
             f"per step, first {args.warmup} of {steps} steps skipped):", ""]
    for p, (avg, n, name) in enumerate(_by_position(
            _dispatches(args.summarize_trace, _kernel_re(args.kernel)), args.launches_per_step,
            args.warmup, args.steps)):
        lines.append(f"- avg_us_pos{p}: {avg / 1e3:.1f} ({n} launches, {name})")
    ours = sum(v[1] for v in per.values())
    lines += ["", f"Library kernels of the {steps} eagerly launched steps (warm-up and timed): "
              f"{ours / 1e6:.3f} ms, {ours / steps / 1e6:.3f} ms per step (kernel time summed "
              f"over both streams: the plan's backward part runs beside the transforms).  "
              f"Everything else in the run (workload set-up, the graph-replayed steps, other "
              f"measurements): {rest[0]} launches, {rest[1] / 1e6:.3f} ms.", "",
              "| kernel | calls | total ms | avg us | ms per step |", "|---|---:|---:|---:|---:|"]
    for name, (n, tot) in sorted(per.items(), key=lambda x: -x[1][1]):
        lines.append(f"| `{name}` | {n} | {tot / 1e6:.3f} | {tot / n / 1e3:.1f} | "
                     f"{tot / steps / 1e6:.3f} |")
    return "\n".join(lines) + "\n"


def summarize_kernels(args) -> str:
    """Calls, total and average time of the kernels matching a pattern in a rocprofv3
    kernel_stats.csv, totals also divided by --per repetitions."""
    path, pat = args.summarize_kernels
    rows = []
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            if re.search(pat, r["Name"]):
                rows.append((_short_name(r["Name"]), int(r["Calls"]),
                             float(r["TotalDurationNs"]), float(r["AverageNs"])))
    rows.sort(key=lambda x: -x[2])
    tot = sum(x[2] for x in rows)
    lines = [f"# kernels matching `{pat}`", "", "Command:", "", "```", args.command, "```", "",
             f"Total {tot / 1e6:.3f} ms, {tot / args.per / 1e6:.3f} ms per repetition "
             f"({args.per} repetitions).", "",
             "| kernel | calls | total ms | avg us | ms per repetition |",
             "|---|---:|---:|---:|---:|"]
    for name, n, t, a in rows:
        lines.append(f"| `{name}` | {n} | {t / 1e6:.3f} | {a / 1e3:.1f} | "
                     f"{t / args.per / 1e6:.3f} |")
    return "\n".join(lines) + "\n"


LP_SETTINGS = ["contrastive / in-batch, B 1024", "cross entropy / in-batch, B 1024",
               "contrastive / joint-32, B 1024", "cross entropy / joint-32, B 1024",
               "contrastive / uniform-32, B 1024", "cross entropy / uniform-32, B 1024",
               "contrastive / uniform-32, B 65536 over 4M rows"]


def summarize_lp(args) -> str:
    """Kernel time per decoder call for each setting measure_lp runs (3 untimed and 50
    timed calls per B 1024 setting, 3 and 10 for the large batch, in that order; a call
    starts with its k_lp_scores launch)."""
    calls, cur = [], []
    for _, name, v in _dispatches(args.summarize_lp, r"rgcn::.*k_lp_"):
        base = re.sub(r"<.*$", "", name)
        if base == "k_lp_scores" and cur:
            calls.append(cur)
            cur = []
        cur.append((base, v / 1e3))
    calls.append(cur)
    keys = [("scores", ["k_lp_scores"]), ("gather", ["k_lp_gather"]), ("gemm (3)", ["k_lp_gemm"]),
            ("loss", ["k_lp_loss"]), ("sum", ["k_lp_sum"]), ("scatter", ["k_lp_scatter_cols"]),
            ("finish", ["k_lp_finish"]), ("d_rel", ["k_lp_rel_partial", "k_lp_rel_final"])]
    lines = ["# k_lp: decoder kernels per call", "", "Command:", "", "```", args.command, "```",
             "", "Per call, us (averages over the timed calls of each setting):", "",
             "| setting | " + " | ".join(k for k, _ in keys) + " | total |",
             "|---|" + "---:|" * (len(keys) + 1)]
    idx = 0
    for si, setting in enumerate(LP_SETTINGS):
        reps, warm = (53, 3) if si < 6 else (13, 3)
        grp = calls[idx + warm: idx + reps]
        idx += reps
        agg = {}
        for c in grp:
            for n, t in c:
                agg[n] = agg.get(n, 0.0) + t
        vals = [sum(agg.get(x, 0.0) for x in names) / max(len(grp), 1) for _, names in keys]
        lines.append(f"| {setting} | " + " | ".join(f"{v:.1f}" for v in vals) +
                     f" | {sum(vals):.1f} |")
    return "\n".join(lines) + "\n"


def summarize_counters(args) -> str:
    """Per-dispatch averages of hardware counters for the kernels matching each pattern,
    over the timed steps' launches (the first --warmup steps' launches skipped), from one
    or more rocprofv3 --pmc counter_collection.csv files, with derived ratios."""
    files = args.summarize_counters
    pats = [p for p in args.kernels.split(",") if p]
    per = {}   # pattern -> counter -> list of per-dispatch values
    names = {}
    for path in files:
        with open(path, newline="") as f:
            rows = list(csv.DictReader(f))
        # the timed eager steps: from the first gather launch of the first timed step to the
        # gather launch that follows the last step (--blocks gather launches per step)
        gstarts = sorted({float(r["Start_Timestamp"]) for r in rows
                          if re.search(_kernel_re("k_gather_flat"), r["Kernel_Name"])})
        nb = args.blocks
        lo = gstarts[args.warmup * nb] if len(gstarts) > args.warmup * nb else 0.0
        end_i = (args.warmup + args.steps) * nb
        hi = gstarts[end_i] if len(gstarts) > end_i else float("inf")
        for pat in pats:
            kre = _kernel_re(pat) if re.match(r"^\w+$", pat) else pat
            by_counter = {}
            for r in rows:
                if not re.search(kre, r["Kernel_Name"]):
                    continue
                if not lo <= float(r["Start_Timestamp"]) < hi:
                    continue
                nm = _short_name(r["Kernel_Name"])
                if nm not in names.setdefault(pat, []):
                    names[pat].append(nm)
                by_counter.setdefault(r["Counter_Name"], {}).setdefault(
                    int(r["Dispatch_Id"]), 0.0)
                by_counter[r["Counter_Name"]][int(r["Dispatch_Id"])] += float(r["Counter_Value"])
            for cn, d in by_counter.items():
                vals = list(d.values())
                per.setdefault(pat, {})[cn] = sum(vals) / len(vals)
                per[pat]["launches"] = len(vals)
    lines = [f"# hardware counters of {', '.join(pats)}", "", "Commands:", "", "```",
             args.command, "```", "",
             "Per-dispatch averages over the launches of the timed, eagerly launched steps "
             "(between the first gather launch of the first timed step and the gather launch "
             "after the last step), all blocks and node types of a step together, every form "
             "(template instance) of the kernel listed under its heading pooled.  Derived: `gpu_cycles` = GRBM_GUI_ACTIVE / 8 (the counter "
             "reads the sum over the 8 XCDs: 8x the kernel's cycles at the clock the trace "
             "durations imply); `mfma_busy` = SQ_VALU_MFMA_BUSY_CYCLES / (gpu_cycles x 256 "
             "CUs x 4 SIMDs); `valu_per_mfma` = SQ_INSTS_VALU / "
             "SQ_INSTS_MFMA (SQ_INSTS_VALU includes the MFMA instructions); `wait_share` = "
             "SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES (wave cycles spent waiting on "
             "s_waitcnt); `lds_conflict_per_lds_inst` = SQ_LDS_BANK_CONFLICT / "
             "SQ_INSTS_LDS; `fetch_GB`, `write_GB` = FETCH_SIZE and WRITE_SIZE (KiB) "
             "scaled as the plain copy calibrates them.", ""]
    f_scale = w_scale = None
    for path in files:
        with open(path, newline="") as f:
            rows = list(csv.DictReader(f))
        cf = [float(r["Counter_Value"]) for r in rows
              if re.search(COPY_KERNEL, r["Kernel_Name"]) and r["Counter_Name"] == "FETCH_SIZE"]
        cw = [float(r["Counter_Value"]) for r in rows
              if re.search(COPY_KERNEL, r["Kernel_Name"]) and r["Counter_Name"] == "WRITE_SIZE"]
        if cf:
            f_scale = COPY_BYTES / (sum(cf) / len(cf) * 1024.0)
        if cw:
            w_scale = COPY_BYTES / (sum(cw) / len(cw) * 1024.0)
    for pat in pats:
        c = per.get(pat, {})
        forms = names.get(pat, [pat])
        lines.append(f"## `{pat}`" + (f" ({len(forms)} forms)" if len(forms) > 1 else ""))
        lines.append("")
        for nm in forms:
            lines.append(f"- form: `{nm}`")
        for cn in sorted(c):
            lines.append(f"- {cn}: {c[cn]:.6g}")
        der = {}
        if "SQ_VALU_MFMA_BUSY_CYCLES" in c and c.get("GRBM_GUI_ACTIVE"):
            der["gpu_cycles"] = c["GRBM_GUI_ACTIVE"] / 8
            der["mfma_busy"] = c["SQ_VALU_MFMA_BUSY_CYCLES"] / (der["gpu_cycles"] * 256 * 4)
        if c.get("SQ_INSTS_MFMA"):
            der["valu_per_mfma"] = c.get("SQ_INSTS_VALU", 0.0) / c["SQ_INSTS_MFMA"]
        if c.get("SQ_WAVE_CYCLES"):
            der["wait_share"] = c.get("SQ_WAIT_INST_ANY", 0.0) / c["SQ_WAVE_CYCLES"]
        if c.get("SQ_INSTS_LDS"):
            der["lds_conflict_per_lds_inst"] = c.get("SQ_LDS_BANK_CONFLICT", 0.0) / c["SQ_INSTS_LDS"]
        if "FETCH_SIZE" in c and f_scale:
            der["fetch_GB"] = c["FETCH_SIZE"] * 1024.0 * f_scale / 1e9
        if "WRITE_SIZE" in c and w_scale:
            der["write_GB"] = c["WRITE_SIZE"] * 1024.0 * w_scale / 1e9
        for k, v in der.items():
            lines.append(f"- {k}: {v:.4g}")
        lines.append("")
    return "\n".join(lines) + "\n"


def summarize_pmc(args) -> str:
    """Per-launch HBM traffic of --kernel from FETCH_SIZE and WRITE_SIZE runs, each scaled
    by what the same counter reads for the plain copy of --copy-probe-mib MiB."""
    fetch_csv, write_csv = args.summarize_pmc
    copy_bytes = float(COPY_BYTES)
    cf = [v for _, _, v in _dispatches(fetch_csv, COPY_KERNEL, "Counter_Value", "FETCH_SIZE")]
    cw = [v for _, _, v in _dispatches(write_csv, COPY_KERNEL, "Counter_Value", "WRITE_SIZE")]
    if not cf or not cw:
        raise SystemExit("no calibration copy dispatches in the counter files")
    f_scale = copy_bytes / (sum(cf) / len(cf) * 1024.0)
    w_scale = copy_bytes / (sum(cw) / len(cw) * 1024.0)
    kre = _kernel_re(args.kernel)
    fpos = _by_position(_dispatches(fetch_csv, kre, "Counter_Value", "FETCH_SIZE"),
                        args.launches_per_step, args.warmup, args.steps)
    wpos = _by_position(_dispatches(write_csv, kre, "Counter_Value", "WRITE_SIZE"),
                        args.launches_per_step, args.warmup, args.steps)
    lines = [f"# {args.kernel}: HBM traffic per launch", "", "Commands:", "", "```",
             args.command, "```", "",
             f"Calibration: a plain copy of {COPY_BYTES >> 20} MiB (fp32 negation, kernel "
             f"matching '{COPY_KERNEL}', {len(cf)} dispatches) reads "
             f"FETCH_SIZE {sum(cf) / len(cf):.0f} KiB and WRITE_SIZE {sum(cw) / len(cw):.0f} KiB; "
             f"scale factors {f_scale:.3f} (fetch) and {w_scale:.3f} (write).", "",
             f"- source_digest: {source_digest(args.kernel)}",
             f"- fetch_scale: {f_scale:.4f}",
             f"- write_scale: {w_scale:.4f}"]
    for p, ((fk, n, name), (wk, _, _)) in enumerate(zip(fpos, wpos)):
        tb = fk * 1024.0 * f_scale + wk * 1024.0 * w_scale
        lines.append(f"- traffic_bytes_pos{p}: {tb:.0f}")
        lines.append(f"  - FETCH_SIZE {fk:.0f} KiB, WRITE_SIZE {wk:.0f} KiB per launch "
                     f"({n} launches, {name})")
    return "\n".join(lines) + "\n"


def full_graph(spec, dev):
    import torch

    from paper_2406_06022_amd import synth

    t0 = time.perf_counter()
    g = synth.device_graph(spec, device=dev)
    torch.cuda.synchronize()
    log(f"full graph: nodes {g.num_nodes}, {g.nnz} edges in {time.perf_counter() - t0:.1f}s")
    return g


def measure_sampling(spec, g, dev, args):
    """On-device mini-batch sampling from the workload's full graph: each mini-batch is
    the three layers top-down from 4,096 seeds (host reads of the counts between layers
    included), timed over several mini-batches with distinct random streams; the oracle
    samples the seed-adjacent layer on the host for a CPU rate."""
    import numpy as np
    import torch

    from paper_2406_06022_amd import rgcn, sampler

    dg = rgcn.DeviceGraph(g)
    gen = torch.Generator(device="cpu").manual_seed(spec.seed + 5)
    T = len(g.num_nodes)
    seeds = [torch.zeros(0, dtype=torch.int64, device=dev) for _ in range(T)]
    for t in spec.seed_types:
        seeds[t] = torch.randperm(g.num_nodes[t], generator=gen)[: spec.n_seeds].to(dev)
    runs, edges, per_layer = [], [], []
    n_batches = 10
    for k in range(2 + n_batches):
        torch.cuda.synchronize()
        a = time.perf_counter()
        blocks, _ = sampler.sample_minibatch(dg, seeds, spec.fanouts, seed=1000 + k)
        torch.cuda.synchronize()
        b = time.perf_counter()
        if k >= 2:
            runs.append((b - a) * 1e3)
            edges.append(sum(x.nnz for x in blocks))
            per_layer.append([x.nnz for x in blocks])
    ms = sum(runs) / len(runs)
    ne = sum(edges) / len(edges)
    out = {"graph": {"num_nodes": g.num_nodes, "edges": g.nnz,
                     "in_degree": "floor(Pareto(2, x_m = 2.75)), mean ~5 per relation, cap 1e5"},
           "seeds": spec.n_seeds, "fanouts": list(spec.fanouts),
           "ms_per_minibatch": round(ms, 3), "sampled_edges_per_minibatch": int(ne),
           "sampled_edges_per_layer": per_layer[0],
           "edges_per_s": ne / (ms * 1e-3), "minibatches": n_batches}
    if args.cpu_budget > 0:
        import oracle

        # host copy of the relations into the seed type (all the seed-adjacent layer reads)
        class _G:
            pass
        hg = _G()
        hg.num_nodes = g.num_nodes
        hg.rels = []
        seed_t = spec.seed_types[0]
        for r, (s_t, d_t) in enumerate(spec.rels):
            x = _G()
            x.src_type, x.dst_type = s_t, d_t
            if d_t == seed_t:
                x.indptr = g.rels[r].indptr.cpu().numpy()
                x.indices = g.rels[r].indices.cpu().numpy()
            else:
                x.indptr = np.zeros(g.num_nodes[d_t] + 1, dtype=np.int64)
                x.indices = np.zeros(1, dtype=np.int64)
            hg.rels.append(x)
        host_seeds = [x.cpu().numpy() for x in seeds]
        c0 = time.perf_counter()
        n_cpu, e_cpu = 0, 0
        while time.perf_counter() - c0 < min(args.cpu_budget, 10.0) or n_cpu == 0:
            blk = oracle.sample_block(hg, host_seeds, spec.fanouts[-1], 1000 + n_cpu,
                                      len(spec.fanouts) - 1)
            e_cpu += sum(int(r.indices.shape[0]) for r in blk.rels)
            n_cpu += 1
        el = time.perf_counter() - c0
        out["cpu_baseline"] = {"value": e_cpu / el, "unit": "sampled edges/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"{n_cpu} seed-adjacent blocks ({spec.n_seeds} seeds, "
                                         f"fanout {spec.fanouts[-1]}, {e_cpu} edges), {el:.1f}s"}
        # the GPU rate of the same seed-adjacent layer
        torch.cuda.synchronize()
        a = time.perf_counter()
        for k in range(20):
            ip, ix, src, counts = rgcn.rgcn_sample_block(dg, seeds, spec.fanouts[-1], 2000 + k,
                                                         len(spec.fanouts) - 1)
        torch.cuda.synchronize()
        out["seed_layer_gpu_ms"] = round((time.perf_counter() - a) * 1e3 / 20, 4)
    del dg
    torch.cuda.empty_cache()
    return out


def measure_featureless(spec, g, tables, dev, args):
    """Feature construction for the featureless type over the workload's whole graph: the
    mean of every node's featured in-neighbours (all relations into the type whose source
    type has a feature table), one call over all its nodes; the oracle runs the same
    construction for the first nodes of the type on the host."""
    import numpy as np
    import torch

    from paper_2406_06022_amd import rgcn

    T = len(g.num_nodes)
    fl = [t for t in range(T) if spec.featureless[t]]
    if not fl:
        return None
    t0 = fl[0]
    into = [r for r in g.rels if r.dst_type == t0 and not spec.featureless[r.src_type]]
    if not into:
        return None
    rels = [(r.indptr, r.indices, tables[r.src_type]) for r in into]
    n = g.num_nodes[t0]
    d = int(tables[into[0].src_type].shape[1])
    out_t = torch.empty((n, d), dtype=tables[into[0].src_type].dtype, device=dev)
    ws = torch.empty(rgcn.RGCN_FEATURELESS_WORKSPACE, dtype=torch.uint8, device=dev)
    esize = out_t.element_size()
    nnz = sum(int(r.indices.shape[0]) for r in into)
    byts = float(len(into) * 8 * (n + 1) + nnz * (8 + d * esize) + n * d * esize)
    rgcn.rgcn_featureless_mean(rels, n, out_t, ws)
    reps = 3
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        rgcn.rgcn_featureless_mean(rels, n, out_t, ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    gbs = byts / (ms * 1e-3) / 1e9
    res = {"type": spec.ntype_names[t0], "nodes": n, "d": d, "dtype": spec.dtype,
           "relations": [spec.ntype_names[r.src_type] for r in into], "edges": nnz,
           "kernel": "k_feature_mean", "ms": round(ms, 3), "bytes": byts,
           "GB/s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4),
           "edges_per_s": nnz / (ms * 1e-3)}
    if args.cpu_budget > 0:
        import oracle
        # the first nodes of the type with all their in-edges, copied to the host
        k = 100_000
        sub = []
        for r in into:
            ip = r.indptr[: k + 1].cpu().numpy()
            ix = r.indices[: int(ip[-1])].cpu().numpy()
            rows = np.unique(ix)
            feat = tables[r.src_type][torch.as_tensor(rows, device=dev)].float().cpu().numpy()
            sub.append((ip, np.searchsorted(rows, ix), feat))
        e_sub = sum(int(x[0][-1]) for x in sub)
        c0, reps_cpu = time.perf_counter(), 0
        while time.perf_counter() - c0 < min(args.cpu_budget, 5.0) or reps_cpu == 0:
            oracle.featureless_mean(sub, k)
            reps_cpu += 1
        el = time.perf_counter() - c0
        res["cpu_baseline"] = {"value": reps_cpu * e_sub / el, "unit": "edges/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"the first {k} nodes of the type ({e_sub} edges), "
                                         f"{reps_cpu} run(s), fp64, {el:.1f}s"}
    del out_t
    torch.cuda.empty_cache()
    return res


def lp_bytes(B: int, nn: int, d: int, esize: int, mode: int) -> float:
    """Algorithmic bytes of one decoder call (scores, loss and gradients): the source,
    destination and negative rows read once for the scores (shared negatives once per
    group), again for the gradients, u_i and its gradient written and read in fp32, the
    scores and their derivatives, and the gradient rows added into d_emb (read and
    written) for every row touched."""
    rows = 2 * B + (B * nn if mode == 0 else (((B + nn - 1) // max(nn, 1)) * nn if mode == 1 else 0))
    emb = rows * d * esize * 2
    u = B * d * 4 * 3
    sc = B * nn * 4 * 3 + B * 4 * 3
    grad = rows * d * 4 * 2
    return float(emb + u + sc + grad)


def measure_lp(dev, args):
    """The link-prediction decoder (scores, loss, gradients in one call): the paper's
    settings (local batch 1,024, in-batch / joint-32 / uniform-32 negatives, contrastive
    and cross entropy) at d = 512 bf16, and a large per-edge batch for the rate of the
    row gathers."""
    import numpy as np
    import torch

    from paper_2406_06022_amd import rgcn

    gen = torch.Generator(device=dev)
    gen.manual_seed(4242)
    d = 512
    out = {"d": d, "dtype": "bf16", "score": "DistMult"}

    def setup(n_rows, B, k, mode):
        emb = (torch.randn((n_rows, d), generator=gen, device=dev) * 0.1).to(torch.bfloat16)
        rel = torch.randn(d, generator=gen, device=dev).to(torch.bfloat16)
        src = torch.randint(0, n_rows, (B,), generator=gen, device=dev, dtype=torch.int32)
        dst = torch.randint(0, n_rows, (B,), generator=gen, device=dev, dtype=torch.int32)
        nneg = B * k if mode == 0 else (((B + k - 1) // k) * k if mode == 1 else 0)
        neg = torch.randint(0, n_rows, (max(nneg, 1),), generator=gen, device=dev,
                            dtype=torch.int32)
        return emb, rel, src, dst, neg

    def time_call(emb, rel, src, dst, neg, mode, kind, k, reps):
        b = rgcn.lp_batch(emb, rel, mode, kind, src, dst, k, neg)
        ws = torch.empty(rgcn.rgcn_lp_workspace_size(b), dtype=torch.uint8, device=dev)
        loss = torch.zeros(1, device=dev)
        d_emb = torch.zeros((emb.shape[0], d), device=dev)
        d_rel = torch.zeros(d, device=dev)
        for _ in range(3):
            rgcn.rgcn_lp_loss(b, loss, None, None, d_emb, d_rel, ws)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            rgcn.rgcn_lp_loss(b, loss, None, None, d_emb, d_rel, ws)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    paper = {}
    B = 1024
    for name, mode, k in (("in-batch", 2, 0), ("joint-32", 1, 32), ("uniform-32", 0, 32)):
        n_rows = 2 * B + (B * k if mode == 0 else k * (B // max(k, 1)) if mode == 1 else 0)
        t = setup(n_rows, B, k, mode)
        for lname, kind in (("contrastive", 2), ("cross-entropy", 0)):
            paper[f"{lname}/{name}"] = round(time_call(*t, mode, kind, k, 50), 4)
    out["paper_batch_1024_ms"] = paper
    # large per-edge batch: 65,536 positives x 32 negatives over 4M rows (4 GB)
    B, k, n_rows = 65536, 32, 4_000_000
    t = setup(n_rows, B, k, 0)
    ms = time_call(*t, 0, 2, k, 10)
    byts = lp_bytes(B, k, d, 2, 0)
    gbs = byts / (ms * 1e-3) / 1e9
    out["large_uniform"] = {"batch": B, "negatives": k, "rows": n_rows, "ms": round(ms, 4),
                            "bytes": byts, "GB/s": round(gbs, 1),
                            "frac": round(gbs / HBM_PEAK_GBS, 4),
                            "scored_edges_per_s": B * (k + 1) / (ms * 1e-3)}
    del t
    if args.cpu_budget > 0:
        import oracle
        rng = np.random.default_rng(3)
        n_rows, B, k = 2 * 1024 + 1024 * 32, 1024, 32
        emb = rng.standard_normal((n_rows, d)) * 0.1
        rel = rng.standard_normal(d)
        src, dst = rng.integers(0, n_rows, B), rng.integers(0, n_rows, B)
        neg = rng.integers(0, n_rows, B * k)
        c0, n = time.perf_counter(), 0
        while time.perf_counter() - c0 < min(args.cpu_budget, 5.0) or n == 0:
            oracle.lp_loss(emb, rel, 0, 2, src, dst, k, neg)
            n += 1
        el = time.perf_counter() - c0
        out["cpu_baseline"] = {"value": n * B * (k + 1) / el, "unit": "scored edges/s",
                               "cores": 1, "kind": "oracle",
                               "sample": f"{n} calls of the uniform-32 contrastive batch of "
                                         f"1,024 positives, d {d}, fp64, {el:.1f}s"}
    return out


def time_steps(stack, dy, steps: int, warmup: int) -> dict:
    """warmup untimed steps, then `steps` steps timed by the wall clock (synchronised on
    both sides) and by HIP events: one pair around each whole step on the stream the
    library launches on (the plan's second stream joins it before the step ends), and one
    pair around each stage.  Returns the wall ms per step, per-step event statistics and
    the mean ms of every (stage, block)."""
    import statistics

    import torch

    for _ in range(warmup):
        stack.step(dy)
    torch.cuda.synchronize()
    events = []

    def timer(tag, edge):
        ev = torch.cuda.Event(enable_timing=True)
        ev.record()
        events[-1].setdefault(tag, [None, None])[edge] = ev

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        events.append({})
        timer("step", 0)
        stack.step(dy, timer=timer)
        timer("step", 1)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps * 1e3
    stage = {}
    for ev in events:
        for tag, (a, b) in ev.items():
            stage.setdefault(tag, []).append(a.elapsed_time(b))
    per_step = stage.pop("step")
    q = sorted(per_step)
    stats = {"median": round(statistics.median(q), 4), "mean": round(statistics.fmean(q), 4),
             "min": round(q[0], 4), "max": round(q[-1], 4),
             "stdev": round(statistics.pstdev(q), 4), "n": len(q)}
    return {"wall_ms": wall, "step_stats": stats,
            "stage_avg": {tag: sum(v) / len(v) for tag, v in stage.items()}}


def time_graph(stack, dy, steps: int, warmup: int) -> dict:
    """The same step recorded once into a HIP graph and replayed: warmup untimed replays,
    then `steps` replays timed by the wall clock and by a HIP event pair around each."""
    import statistics

    import torch

    graph = stack.capture_step(dy)
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    evs = []
    t0 = time.perf_counter()
    for _ in range(steps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        graph.replay()
        b.record()
        evs.append((a, b))
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps * 1e3
    q = sorted(a.elapsed_time(b) for a, b in evs)
    del graph
    return {"wall_ms": wall, "step_stats": {"median": round(statistics.median(q), 4),
                                            "min": round(q[0], 4), "max": round(q[-1], 4),
                                            "n": len(q)}}


def block_ms(stack, avg) -> list:
    return [round(sum(avg.get((s, l), 0.0)
                      for s in ("plan", "aggregate", "transform", "dense", "sparse")), 4)
            for l in range(stack.L)]


def stage_rooflines(spec, mb, stack, avg) -> dict:
    """Every aggregate and sparse stage: its time, the method's bytes (method_bytes) and
    the fraction of the 8 TB/s peak they make, and this layout's bytes beside them."""
    out = {}
    for l in range(stack.L):
        for s in ("aggregate", "sparse"):
            if (s, l) not in avg:
                continue
            t_ms = avg[(s, l)]
            byts = method_bytes(spec, mb.blocks[l], stack.blocks[l], s, l)
            impl = algorithmic_bytes(spec, mb.blocks[l], stack.blocks[l], s, l)
            gbs = byts / (t_ms * 1e-3) / 1e9
            out[f"{s}[{l}]"] = {"ms": round(t_ms, 4), "bytes": byts, "GB/s": round(gbs, 1),
                                "frac": round(gbs / HBM_PEAK_GBS, 4), "impl_bytes": impl,
                                "impl_GB/s": round(impl / (t_ms * 1e-3) / 1e9, 1)}
    return out


def mfma_stages(spec, mb, stack, avg):
    mfma, mfma_bwd = {}, {}
    for l in range(stack.L):
        fl = transform_flops(spec, mb.blocks[l], l)
        tf = fl / (avg[("transform", l)] * 1e-3) / 1e12
        mfma[f"transform[{l}]"] = {"ms": round(avg[("transform", l)], 4), "TFLOP/s": round(tf, 1),
                                   "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4)}
        fl = backward_flops(spec, mb.blocks[l], stack.blocks[l].grad_src_types, l)
        tf = fl / (avg[("dense", l)] * 1e-3) / 1e12
        mfma_bwd[f"dense[{l}]"] = {"ms": round(avg[("dense", l)], 4), "TFLOP/s": round(tf, 1),
                                   "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4)}
    return mfma, mfma_bwd


def gather_by_ids(spec, mb, stack, reps: int = 10) -> dict:
    """Block 0's gather when each edge's table row is resolved through the block's row ids
    (indices -> ids -> row, a dependent random 8-byte read per edge) instead of read from
    the sampler's per-edge rows as the timed steps do: same segments, same bytes by the
    method's count, the id lookup on the critical path."""
    import torch

    from paper_2406_06022_amd import rgcn

    blk = mb.blocks[0]
    db = rgcn.DeviceBlock(blk, stack.blocks[0].grad_src_types, stack.device)
    p, ws, inp = stack.params[0], stack.workspaces[0], stack.inputs[0]
    rgcn.rgcn_block_plan(db, p, ws, rgcn.RGCN_PLAN_FORWARD)
    for _ in range(2):
        rgcn.rgcn_block_aggregate(db, inp, p, ws)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        rgcn.rgcn_block_aggregate(db, inp, p, ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    byts = method_bytes(spec, blk, stack.blocks[0], "aggregate", 0)
    gbs = byts / (ms * 1e-3) / 1e9
    return {"ms": round(ms, 4), "bytes": byts, "GB/s": round(gbs, 1),
            "frac": round(gbs / HBM_PEAK_GBS, 4)}


def measure_skewed(args, tables, dev):
    """The billion-edge workload with power-law sources (p(rank k) proportional to
    (k + 1)^-0.8 through a fixed id bijection), the backward's load-balance stress: the
    same tables and weights, a mini-batch sampled with skewed sources, full steps timed as
    the main workload is."""
    import numpy as np
    import torch

    from paper_2406_06022_amd import chain, synth

    spec = synth.skewed_config(args.config)
    t0 = time.perf_counter()
    mb = synth.sample_minibatch(spec, device=dev)
    log(f"sampled {spec.name}: blocks nnz {[b.nnz for b in mb.blocks]} in "
        f"{time.perf_counter() - t0:.1f}s")
    T = len(spec.ntype_names)
    tdt = synth.torch_dtype(spec.dtype)
    ids = [torch.as_tensor(mb.input_ids[t]).to(dev) for t in range(T)]
    weights = []
    for l in range(spec.num_layers):
        w_rel, w_self, _ = synth.block_weights(T, len(spec.rels), spec.dims[l],
                                               spec.dims[l + 1], tdt, spec.seed * 100 + l)
        weights.append(([w.to(dev) for w in w_rel], [w.to(dev) for w in w_self], None))
    emb = [t for t in range(T) if spec.featureless[t]]
    stack = chain.MiniBatchStack(mb.blocks, tables, ids, weights, spec.dtype, spec.dims,
                                 emb_types=emb, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(spec.seed + 1)
    dy = [torch.randn((n, spec.dims[-1]), generator=gen, device=dev, dtype=torch.float32)
          if n > 0 else None for n in mb.blocks[-1].n_dst]
    steps = max(3, args.steps // 2)
    run = time_steps(stack, dy, steps, min(args.warmup, 3))
    avg = run["stage_avg"]
    blk = mb.blocks[0]
    longest, hubs = 0, 0
    for rel in blk.rels:
        if stack.blocks[0].grad_src_types >> rel.src_type & 1 and rel.nnz:
            cnt = np.bincount(np.asarray(rel.indices))
            longest = max(longest, int(cnt.max()))
            hubs += int((cnt > 32).sum())
    roof = stage_rooflines(spec, mb, stack, avg)
    out = {"workload": spec.name, "skew": spec.skew, "blocks_nnz": [b.nnz for b in mb.blocks],
           "ms_per_step": round(run["wall_ms"], 4), "step_ms_events": run["step_stats"],
           "edges_per_s": stack.nnz / (run["wall_ms"] / 1e3),
           "ms_per_block": block_ms(stack, avg),
           "plan[0]": round(avg[("plan", 0)], 4), "plan_bwd[0]": round(avg[("plan_bwd", 0)], 4),
           "sparse[0]": dict(roof["sparse[0]"], kernel="k_transpose_pipe"),
           "aggregate[0]": roof["aggregate[0]"],
           "largest_transpose_degree": longest, "sources_over_32_edges": hubs,
           "csc_radix_path": longest > 16384}
    del stack
    torch.cuda.empty_cache()
    return out


def measure_configs(args, dev):
    """The other workloads (the parity configurations at full size): per-block ms of a
    full step and the gather's fraction of the HBM peak by the method's bytes."""
    import torch

    out = {}
    for index in range(5):
        if index == args.config:
            continue
        spec, mb, tables, ids, weights, stack, dy = build_stack(index, dev)
        run = time_steps(stack, dy, max(5, args.steps // 2), min(args.warmup, 3))
        avg = run["stage_avg"]
        roof = stage_rooflines(spec, mb, stack, avg)
        mf, mb_ = mfma_stages(spec, mb, stack, avg)
        gr = time_graph(stack, dy, max(5, args.steps // 2), min(args.warmup, 3))
        out[spec.name] = {"blocks_nnz": [b.nnz for b in mb.blocks],
                          "ms_per_step": round(run["wall_ms"], 4),
                          "ms_per_step_graph": round(gr["wall_ms"], 4),
                          "step_ms_median": run["step_stats"]["median"],
                          "edges_per_s": stack.nnz / (run["wall_ms"] / 1e3),
                          "ms_per_block": block_ms(stack, avg),
                          "aggregate_frac": {k: v["frac"] for k, v in roof.items()
                                             if k.startswith("aggregate")},
                          "sparse_frac": {k: v["frac"] for k, v in roof.items()
                                          if k.startswith("sparse")},
                          "transform_frac": {k: v["frac"] for k, v in mf.items()},
                          "dense_frac": {k: v["frac"] for k, v in mb_.items()}}
        del stack, tables, ids, weights, dy, mb
        torch.cuda.empty_cache()
    return out


def other_legs(args, spec, mb, tables, stack, dy, nnz, dev):
    """The measurement legs after the main steps: training steps with the fused sparse
    optimizer, the power-law-source workload, the other workloads, sampling, featureless
    feature construction and the link-prediction decoder."""
    import torch

    # the sparse optimizer step of the learnable tables fused into block 0's transposed sum:
    # full training steps (plan, forward, backward, table update) after the others, since
    # they change the tables
    stack.attach_adagrad(lr=0.01, eps=1e-10)
    ada = time_steps(stack, dy, args.steps, args.warmup)
    ada_ms = ada["wall_ms"]
    ada_sp_ms = ada["stage_avg"][("sparse", 0)]
    ada_bytes = algorithmic_bytes(spec, mb.blocks[0], stack.blocks[0], "sparse_adagrad", 0)
    ada_gbs = ada_bytes / (ada_sp_ms * 1e-3) / 1e9
    adagrad = {"ms_per_train_step": round(ada_ms, 4),
               "edges_per_s": nnz / (ada_ms / 1e3),
               "sparse[0]": {"kernel": "k_transpose_pipe_adagrad", "ms": round(ada_sp_ms, 4),
                             "bytes": ada_bytes, "GB/s": round(ada_gbs, 1),
                             "frac": round(ada_gbs / HBM_PEAK_GBS, 4)},
               "lr": 0.01, "eps": 1e-10}
    stack.release()
    torch.cuda.empty_cache()

    skewed = measure_skewed(args, tables, dev)
    torch.cuda.empty_cache()
    configs = measure_configs(args, dev)
    torch.cuda.empty_cache()

    g = full_graph(spec, dev)
    sampling = measure_sampling(spec, g, dev, args)
    featureless = measure_featureless(spec, g, tables, dev, args)
    del g
    torch.cuda.empty_cache()
    link_prediction = measure_lp(dev, args)

    return adagrad, skewed, configs, sampling, featureless, link_prediction


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=4, help="workload index 0..4 (default 4)")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle work for the CPU baseline (0 = skip)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="reduce two rocprofv3 --pmc counter_collection.csv files (FETCH_SIZE, "
                         "WRITE_SIZE) into the per-launch HBM traffic summary and exit")
    ap.add_argument("--summarize-counters", nargs="+", metavar="COUNTER_CSV",
                    help="reduce rocprofv3 --pmc counter_collection.csv files to per-dispatch "
                         "counter averages of the kernels in --kernels and exit")
    ap.add_argument("--kernels", default="k_gemm_dw,k_gemm_fwd,LoadRowsF32HiLo",
                    help="with --summarize-counters: comma-separated kernel names or patterns")
    ap.add_argument("--main-only", action="store_true",
                    help="time the main workload's steps (and the calibration copy) only: no "
                         "CPU baseline, training steps or other measurement legs")
    ap.add_argument("--summarize-trace", metavar="KERNEL_TRACE_CSV",
                    help="reduce a rocprofv3 kernel_trace.csv into a per-kernel summary and exit")
    ap.add_argument("--summarize-kernels", nargs=2, metavar=("KERNEL_STATS_CSV", "REGEX"),
                    help="reduce a rocprofv3 kernel_stats.csv to the kernels matching REGEX "
                         "and exit")
    ap.add_argument("--summarize-lp", metavar="KERNEL_TRACE_CSV",
                    help="per-setting kernel breakdown of a rocprofv3 kernel_trace.csv of "
                         "`bench.py --lp-only` and exit")
    ap.add_argument("--per", type=int, default=1,
                    help="with --summarize-kernels: divide totals by this many repetitions")
    ap.add_argument("--sampling-only", action="store_true",
                    help="run only the on-device mini-batch sampling measurement (12 "
                         "mini-batches of the workload) and print its JSON object")
    ap.add_argument("--featureless-only", action="store_true",
                    help="time only the featureless-type feature construction")
    ap.add_argument("--lp-only", action="store_true",
                    help="run only the link-prediction decoder measurement and print its JSON")
    ap.add_argument("--kernel", default="k_gather_flat")
    ap.add_argument("--blocks", type=int, default=3,
                    help="with --summarize-trace: blocks (gather launches) per step")
    ap.add_argument("--launches-per-step", type=int, default=3,
                    help="launches of --kernel per step (summaries split them by position)")
    ap.add_argument("--command", default="", help="command line recorded in a summary")
    args = ap.parse_args()
    if args.summarize_pmc:
        print(summarize_pmc(args), end="")
        return 0
    if args.summarize_counters:
        print(summarize_counters(args), end="")
        return 0
    if args.summarize_trace:
        print(summarize_trace(args), end="")
        return 0
    if args.summarize_kernels:
        print(summarize_kernels(args), end="")
        return 0
    if args.summarize_lp:
        print(summarize_lp(args), end="")
        return 0
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for --gpus {args.gpus}); the multi-GPU "
              "sharding of this path is a design note, not an implementation.", file=sys.stderr)
        return 2
    import torch

    from paper_2406_06022_amd import rgcn

    dev = "cuda:0"
    torch.cuda.set_device(0)
    rgcn.load_library()
    if args.lp_only:
        print(json.dumps(measure_lp(dev, args)), flush=True)
        return 0
    if args.sampling_only:
        from paper_2406_06022_amd import synth
        spec = synth.config(args.config)
        print(json.dumps(measure_sampling(spec, full_graph(spec, dev), dev, args)), flush=True)
        return 0
    if args.featureless_only:
        from paper_2406_06022_amd import synth
        spec = synth.config(args.config)
        g = full_graph(spec, dev)
        tables = [synth.normal_table(spec.type_rows[t], spec.dims[0],
                                     synth.torch_dtype(spec.dtype), spec.seed * 10 + t,
                                     device=dev) if not spec.featureless[t] else None
                  for t in range(len(spec.type_rows))]
        print(json.dumps(measure_featureless(spec, g, tables, dev, args)), flush=True)
        return 0
    spec, mb, tables, ids, weights, stack, dy = build_stack(args.config, dev)
    log(f"workspace bytes per block {[int(w.numel()) for w in stack.workspaces]}")
    run = time_steps(stack, dy, args.steps, args.warmup)
    log(f"warmup {args.warmup} and {args.steps} timed steps done")
    nnz = stack.nnz
    # the same step recorded into a HIP graph and replayed (one host launch per step); the
    # headline rate, unless recording fails, when the eagerly launched steps give it
    graph = None
    try:
        graph = time_graph(stack, dy, args.steps, args.warmup)
        log(f"{args.steps} graph replays: {graph['wall_ms']:.3f} ms per step")
    except Exception as e:   # report, and keep the eager figure
        log(f"graph capture failed ({type(e).__name__}: {e}); eager steps give the rate")
    ms = graph["wall_ms"] if graph is not None else run["wall_ms"]
    value = nnz / (ms / 1e3)
    avg = run["stage_avg"]
    per_block = block_ms(stack, avg)

    rooflines = stage_rooflines(spec, mb, stack, avg)
    # dominant single-kernel stage: the aggregate or sparse stage with the largest time
    dom_key = max(rooflines, key=lambda k: rooflines[k]["ms"])
    dom = rooflines[dom_key]
    dom_stage, dom_layer = dom_key.split("[")[0], int(dom_key.split("[")[1][:-1])
    kernel_name = {"aggregate": "k_gather_flat", "sparse": "k_transpose_pipe"}[dom_stage]
    # launch position of the dominant stage within a step's launches of its kernel: the
    # gather runs once per block, input side first; the transposed sum once per requested
    # source type, output side first
    if dom_stage == "aggregate":
        position = dom_layer
    else:
        position = 0
        for l in reversed(range(stack.L)):
            db = stack.blocks[l]
            n = sum(1 for t in range(db.num_types)
                    if db.grad_src_types >> t & 1 and db.n_src[t] > 0)
            if l == dom_layer:
                break
            position += n
    traffic = read_traffic(kernel_name, spec.name, position)
    mfma, mfma_bwd = mfma_stages(spec, mb, stack, avg)
    gather_ids = gather_by_ids(spec, mb, stack)

    # attainable streaming bandwidth of this machine: a plain 1 GiB fp32 copy (read + write)
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.neg(src, out=dst)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(5):
        torch.neg(src, out=dst)
    c1.record()
    torch.cuda.synchronize()
    copy_gbs = 2.0 * src.numel() * 4 * 5 / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del src, dst

    cpu = adagrad = skewed = configs = sampling = featureless = link_prediction = None
    if args.cpu_budget > 0 and not args.main_only:
        host = host_info()
        nt = oracle_threads()
        log(f"timing the CPU oracle on a sample of block 0 ({nt} threads, then 1)")
        res = {}
        for th in (nt, 1):
            eps, s_nnz, s_el, s_rows = cpu_baseline(spec, mb, tables, ids, weights,
                                                    args.cpu_budget, th)
            res[th] = {"value": eps, "unit": "edges/s", "cores": th, "kind": "oracle",
                       "sample": f"block 0 restricted to its first destination rows per type "
                                 f"({s_rows} rows, {s_nnz} edges, full segments), fp64 "
                                 f"forward + backward (weight grads, embedding-type input "
                                 f"grad), {th} thread(s), {s_el:.1f}s"}
        cpu = dict(res[nt])
        cpu["host"] = host
        cpu["one_thread"] = {k: res[1][k] for k in ("value", "cores", "sample")}

    # the sparse optimizer step of the learnable tables fused into block 0's transposed sum:
    # full training steps (plan, forward, backward, table update) after the others, since
    # they change the tables
    if not args.main_only:
        adagrad, skewed, configs, sampling, featureless, link_prediction = other_legs(
            args, spec, mb, tables, stack, dy, nnz, dev)

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "edges/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic",
        "config": {"workload": spec.name, "blocks_nnz": [b.nnz for b in mb.blocks],
                   "fanouts": list(spec.fanouts), "seeds": spec.n_seeds,
                   "dims": list(spec.dims), "relations": len(spec.rels),
                   "table_rows": list(spec.type_rows),
                   "learnable_tables": [spec.ntype_names[t] for t in range(len(spec.ntype_names))
                                        if spec.featureless[t]]},
        "step_launch": "hip_graph_replay" if graph is not None else "eager",
        "ms_per_step_eager": round(run["wall_ms"], 4),
        "step_ms_events": graph["step_stats"] if graph is not None else run["step_stats"],
        "step_ms_events_eager": run["step_stats"],
        "ms_per_block": per_block,
        "stage_ms": {f"{s}[{l}]": round(v, 4) for (s, l), v in sorted(avg.items(), key=lambda x: (x[0][1], x[0][0]))},
        "roofline": {"bound": "hbm", "kernel": kernel_name, "stage": dom_key,
                     "achieved": dom["GB/s"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": dom["frac"], "traffic": traffic,
                     "traffic_over_bytes": (round(traffic / dom["bytes"], 3)
                                            if traffic is not None else None),
                     "bytes": dom["bytes"], "impl_bytes": dom["impl_bytes"],
                     "launch_position": position},
        "hbm_kernels": rooflines,
        "aggregate[0]_rows_by_id_lookup": gather_ids,
        "copy_probe_GBs": round(copy_gbs, 1),
        "mfma_transforms": mfma,
        "mfma_backward": mfma_bwd,
        "train_step_sparse_adagrad": adagrad,
        "skewed": skewed,
        "configs": configs,
        "sampling": sampling,
        "featureless_features": featureless,
        "link_prediction": link_prediction,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    return 0

if __name__ == "__main__":
    sys.exit(main())
