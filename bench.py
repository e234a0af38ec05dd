"""Benchmark of the message-passing aggregation path on one MI355X.

Workload: a seeded Chung-Lu power-law graph with N = 2,449,029 nodes and
E = 123,718,280 edges (mean in-degree 50.5, expected top degree 17,000),
features N x 100 in fp32 and in bf16 (the bf16 copy is the RNE rounding of the
fp32 draws).  It stands in for a products-scale public graph; no dataset is
used.

One step = the whole hot path over that graph, inputs already in HBM:
  COO -> CSR (stable radix sort by destination + rowptr), the degree-binned
  plan, then sum, mean and max+argmax aggregation for fp32 features and again
  for bf16 features (fp32 accumulation; sums and means written fp32, bf16 max
  written bf16, exact).  The bf16 table (200-byte rows) is first copied into
  rows 256 bytes apart, once per step, so that every gathered row spans two
  cache lines; the fp32 rows (400 bytes) span four lines at any offset and
  are used as they are.

value = sum over the step's operations of their algorithmic bytes (each edge
gathers one full feature row; see algorithmic_bytes()) / step time, in GB/s.

Other modes (used to produce the committed summaries under profiles/):
  --summarize-stats DIR OUT        kernel-trace stats of a rocprofv3 run -> OUT
  --summarize-counters F W OUT     FETCH_SIZE (F) and WRITE_SIZE (W) runs -> OUT
  --summarize-step-counters F W OPS OUT   the same for every operation of a step
  --summarize-sq DIR OUT           shader counters (occupancy, VALU, waits) per kernel
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "SpMM effective HBM GB/s (% of peak) + edge·features/s, sum/mean/max"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
WORKLOAD = "chunglu-124M"
BACKWARD = "chunglu-124M-backward"
STACKED = "chunglu-124M-stacked"
SORT_TILE = 16384  # keys per tile of the library's radix passes (1024 threads x 16)
PROJECTION = "hetero-20M-projection"
READOUT = "readout-2.4M"
EXPLAIN = "chunglu-124M-explain"
DOMINANT = "spmm_main<float, 4, true, false, 1, false, 0, false>"  # fp32 sum, the largest launch of a step
# the dominant kernel's source: spmm.hip and the aggregation section of the
# internal header (file, first line marker or None, end marker or None)
DOMINANT_SRC = [("paper_2507_16991_amd/csrc/spmm.hip", None, None),
                ("paper_2507_16991_amd/csrc/mp_internal.hpp", "// ---- aggregation (spmm.hip)",
                 "// ---- backward (backward.hip)")]
COUNTER_SUMMARY = os.path.join(ROOT, "profiles", "spmm_main_f32_sum_chunglu124M_counters.txt")
CALIB_BYTES = 1 << 30  # plain copy used to scale the HBM counters
SORT_STATUS = []  # device status words of the sorts a step runs


# ---- algorithmic bytes ------------------------------------------------------------

def spmm_bytes(N, E, F, xb, reduce, out_b=4, max_b=4, rowptr_b=4, w=False):
    """Each edge reads its column index and gathers one feature row; every
    output row is written once."""
    b = (N + 1) * rowptr_b + 4 * E + E * F * xb + (4 * E if w else 0)
    if reduce & 3:
        b += N * F * out_b
    if reduce & 4:
        b += N * F * (max_b + 4)
    return b


def csr_bytes(N, E, rowptr_b=4, perm=False):
    """Read src and dst, write col (and perm) and rowptr."""
    return 8 * E + 4 * E + (4 * E if perm else 0) + (N + 1) * rowptr_b


def transpose_bytes(N_dst, N_src, E):
    """Read rowptr and col, write rowptrT, colT and posT."""
    return 4 * (N_dst + 1) + 4 * E + 4 * (N_src + 1) + 8 * E


def grad_x_bytes(N_dst, N_src, E, F, mode):
    """Transposed gather of the output gradient, one output row per source.
    Mean adds the scaled copy of the gradient.  Max reads the argmax table
    once and writes the win masks (ceil(F/32) words per edge), then gathers
    each edge's forward position and win-mask words, and only the routed
    gradient elements, one per destination row and feature."""
    b = 4 * (N_src + 1) + 4 * E + N_src * F * 4
    if mode == "mean":
        b += 4 * (N_dst + 1) + 2 * N_dst * F * 4
    if mode == "max":
        mask = E * ((F + 31) // 32) * 4
        return b + 4 * (N_dst + 1) + N_dst * F * 4 + 2 * mask + 4 * E + N_dst * F * 4
    return b + E * F * 4


def grad_w_bytes(N_dst, E, F):
    """One x row gathered per edge, the output gradient read once per row,
    one fp32 per edge written."""
    return 4 * (N_dst + 1) + 4 * E + E * F * 4 + N_dst * F * 4 + 4 * E


def multi_bytes(N, E, F, xb, names, rowptr_b=4, col=True):
    """One gather of every edge's row feeds all requested statistics; each
    output row is written once (max and min with their int32 positions)."""
    b = (N + 1) * rowptr_b + (4 * E if col else 0) + E * F * xb
    for n in names:
        b += N * F * (8 if n in ("max", "min") else 4)
    return b


def plan_bytes(N):
    """Read rowptr, write the class-sorted row list and the chunk offsets."""
    return 4 * (N + 1) + 4 * N + 4 * (N + 1)


def source_digest(parts):
    """SHA-1 of the listed source text: whole files, or the lines of a file
    from a start marker up to (not including) an end marker."""
    h = hashlib.sha1()
    for path, start, end in parts:
        with open(os.path.join(ROOT, path), "rb") as f:
            text = f.read()
        if start is not None:
            text = text[text.index(start.encode()):]
        if end is not None:
            text = text[:text.index(end.encode())]
        h.update(text)
    return h.hexdigest()


def read_traffic():
    """HBM bytes per launch of the dominant kernel from the committed counter
    summary, or None when it is absent or was taken on different source."""
    try:
        kv = {}
        for line in open(COUNTER_SUMMARY):
            if ":" in line:
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
        if kv.get("kernel_source_sha1") != source_digest(DOMINANT_SRC):
            return None
        return float(kv["hbm_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


# ---- benchmark ------------------------------------------------------------------------

def hetero_bytes(g, F):
    """Per destination type with incoming relations: combined CSR build (read
    src+dst, write col and rowptr) and the sum (rowptr, col, one bf16 row
    gathered per edge, fp32 out).  Built for all types in one pass, the same
    bytes (every type of the benchmark graph is a destination)."""
    b_csr = b_sum = ef = 0
    for t, n in enumerate(g.n_per_type):
        e = sum(g.rel_src[r].shape[0] for r in range(len(g.rel_src)) if g.rel_dst_type[r] == t)
        if e == 0:
            continue
        b_csr += csr_bytes(n, e)
        b_sum += spmm_bytes(n, e, F, 2, 1)
        ef += e * F
    return b_csr, b_sum, ef


class ColdEvents:
    """Events of one cold-cache step: before each operation a 1 GiB buffer is
    written (more than the 256 MB MALL and the 4 MB L2 of each XCD), so every
    operation starts with its inputs evicted from the caches; start[i] and
    end[i] bracket operation i alone."""

    def __init__(self, torch, n_ops, flush):
        self.start = [torch.cuda.Event(enable_timing=True) for _ in range(n_ops)]
        self.end = [torch.cuda.Event(enable_timing=True) for _ in range(n_ops)]
        self.flush = flush

    def times(self):
        return [a.elapsed_time(b) for a, b in zip(self.start, self.end)]


def make_mark(stream):
    """mark(evs, i): the boundary before operation i (i = n_ops: after the
    last).  evs is None (untimed), a list of n_ops + 1 events (warm: the
    operations back to back), or a ColdEvents (a cache flush before each)."""
    def mark(evs, i):
        if evs is None:
            return
        if isinstance(evs, ColdEvents):
            if i > 0:
                evs.end[i - 1].record(stream)
            if i < len(evs.start):
                evs.flush()
                evs.start[i].record(stream)
        else:
            evs[i].record(stream)
    return mark


def build_step(args, mp, torch, np, dev):
    """Generate the workload, upload it, and return (graph, step(evs), op list).

    Each op is (name, algorithmic bytes, edge*feature count); step(evs)
    records events evs[0..len(ops)] around the ops on the current stream."""
    import graphgen

    t0 = time.time()
    if args.workload == PROJECTION:
        return projection_step(args, mp, torch, np, dev)
    if args.workload in (BACKWARD, EXPLAIN):
        g = graphgen.workload(WORKLOAD, seed=args.seed, bf16=False)
    elif args.workload in (STACKED, READOUT):
        g = graphgen.workload(WORKLOAD, seed=args.seed)
    else:
        g = graphgen.workload(args.workload, seed=args.seed)
    print(f"[bench] generated {args.workload} in {time.time() - t0:.1f}s", file=sys.stderr,
          flush=True)
    stream = torch.cuda.current_stream()
    mark = make_mark(stream)

    if args.workload == "hetero-20M":
        F = g.F
        rels = [(g.rel_src_type[r], g.rel_dst_type[r], torch.from_numpy(g.rel_src[r]).to(dev),
                 torch.from_numpy(g.rel_dst[r]).to(dev)) for r in range(len(g.rel_src))]
        xs = [torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16) for x in g.x_bf16]
        b_csr, b_sum, ef = hetero_bytes(g, F)
        n_all = sum(g.n_per_type)
        e_all = sum(a.shape[0] for a in g.rel_src)
        ops = [("hetero_build", b_csr, 0), ("plan", plan_bytes(n_all), 0),
               ("hetero_sum_bf16", b_sum, ef)]
        state = {}
        # every destination type at once: one CSR over all nodes (global ids)
        # whose row slices are the per-type CSRs, one plan, one aggregation
        # into the per-type outputs stacked in type order
        out = torch.empty(n_all, F, dtype=torch.float32, device=dev)

        def step(evs=None):
            mark(evs, 0)
            state["csr"] = mp.hetero_build(g.n_per_type, rels, mp.MP_ALL_TYPES)
            mark(evs, 1)
            plan = mp.Plan(state["csr"][0], e_all, F, torch.bfloat16)
            mark(evs, 2)
            mp.hetero_spmm(g.n_per_type, xs, mp.MP_ALL_TYPES, state["csr"][0], state["csr"][1],
                           plan=plan, out=out)
            mark(evs, 3)
        g.n_dst, g.E = sum(g.n_per_type), sum(a.shape[0] for a in g.rel_src)
        return g, step, ops

    if args.workload == BACKWARD:
        return backward_step(g, mp, torch, np, dev, mark)
    if args.workload == EXPLAIN:
        return explain_step(g, mp, torch, np, dev, mark, args.seed)
    if args.workload == STACKED:
        return stacked_step(g, mp, torch, np, dev, mark)
    if args.workload == READOUT:
        return readout_step(g, mp, torch, np, dev, mark, args.seed)

    N, E, F = g.n_dst, g.E, g.F
    src = torch.from_numpy(g.src).to(dev)
    dst = torch.from_numpy(g.dst).to(dev)
    web = args.workload == "web-1.6B"
    it = mp.MP_I64 if web else mp.MP_I32
    rp_b = 8 if web else 4
    weighted = g.w is not None
    rowptr = torch.empty(N + 1, dtype=torch.int64 if web else torch.int32, device=dev)
    col = torch.empty(E, dtype=torch.int32, device=dev)
    perm = torch.empty(E, dtype=torch.int32, device=dev) if weighted else None
    w_coo = torch.from_numpy(g.w).to(dev) if weighted else None
    w_csr = torch.empty(E, dtype=torch.float32, device=dev) if weighted else None
    ws_csr = torch.empty(mp.mp_coo_to_csr_workspace(E, N, it, int(weighted)), dtype=torch.uint8,
                         device=dev)
    nplan = mp.mp_spmm_plan_size(N, E)
    xs = {}
    if g.x is not None:
        xs["f32"] = (torch.from_numpy(g.x).to(dev), mp.MP_F32, 4)
    if g.x_bf16 is not None and args.workload in (WORKLOAD, "web-1.6B"):
        xs["bf16"] = (torch.from_numpy(g.x_bf16.view(np.int16)).to(dev).view(torch.bfloat16),
                      mp.MP_BF16, 2)
    plan_buf = torch.empty(nplan, dtype=torch.uint8, device=dev)
    out = torch.empty(N, F, dtype=torch.float32, device=dev)
    mx = {k: torch.empty(N, F, dtype=torch.float32 if k == "f32" else torch.bfloat16,
                         device=dev) for k in xs}
    arg = torch.empty(N, F, dtype=torch.int32, device=dev)

    csr_b = csr_bytes(N, E, rowptr_b=rp_b, perm=weighted) + (8 * E if weighted else 0)
    ops = [("csr", csr_b, 0), ("plan", plan_bytes(N), 0)]
    if web:
        reds = [("sum+max", mp.MP_SUM | mp.MP_MAX, False)]
    elif args.workload == "powerlaw-1.2M":
        reds = [("mean", mp.MP_MEAN, False), ("wsum", mp.MP_SUM, True)]
    elif args.workload == "uniform-10k":
        reds = [("sum", mp.MP_SUM, False)]
    else:
        reds = [("sum", mp.MP_SUM, False), ("mean", mp.MP_MEAN, False), ("max", mp.MP_MAX, False)]
    # a feature table whose rows are not whole cache lines is first copied
    # into rows a whole number of lines apart (once per step, shared by the
    # table's aggregations): each gathered row then touches the fewest lines
    calls = []
    for k, (x, xd, xb) in xs.items():
        ld = mp.aligned_ld(F, x.dtype)
        if ld != F:
            xp = torch.empty(N, ld, dtype=x.dtype, device=dev)[:, :F]
            ops.append((f"layout_{k}", 2 * N * F * xb, 0))
            calls.append(("layout", k, x, xp, xd, ld))
            x = xp
        for rn, red, wt in reds:
            mb = 4 if k == "f32" else 2
            ops.append((f"{rn}_{k}", spmm_bytes(N, E, F, xb, red, max_b=mb, rowptr_b=rp_b, w=wt),
                        E * F))
            calls.append(("spmm", k, x, xd, red, wt, ld))

    # the gather ceilings of this workload: the CSR column stream over each
    # feature table, as the aggregations read it (table, row stride and
    # algorithmic row bytes)
    g.probe = {"col": col, "tables": {c[1]: (c[2], c[6] * xs[c[1]][2], F * xs[c[1]][2])
                                      for c in calls if c[0] == "spmm"}}
    if args.workload == WORKLOAD:
        # the radix passes' data movement: the first pass's order over dst
        # (its digit: the key's bits split evenly over the passes, the first
        # pass taking the narrower share)
        kb = max(1, (N - 1).bit_length())
        passes = -(-kb // 9)
        g.probe["scatter"] = (dst, kb // passes)
    plans = {}
    wss = {}

    sort_status = mp.new_status(dev)  # checked once after the timed steps
    SORT_STATUS.append(sort_status)

    def step(evs=None):
        mark(evs, 0)
        mp.mp_coo_to_csr(src, dst, E, N, rowptr, it, col, perm, w_coo, w_csr, ws_csr,
                         ws_csr.numel(), sort_status)
        mark(evs, 1)
        # one plan per CSR, shared by both feature dtypes
        k0 = next(iter(xs))
        if "h" in plans:
            mp.mp_spmm_plan_free(plans["h"])
        plans["h"] = mp.mp_spmm_plan_build(rowptr, it, N, E, F, xs[k0][1], plan_buf, nplan)
        mark(evs, 2)
        i = 2
        for c in calls:
            if c[0] == "layout":
                _, k, x, xp, xd, ld = c
                mp.mp_copy_rows(x, F, xp, ld, N, F, xd)
                i += 1
                mark(evs, i)
                continue
            _, k, x, xd, red, wt, ld = c
            h = plans["h"]
            nb = mp.mp_spmm_workspace(h, red)
            key = (k, red)
            if key not in wss or wss[key].numel() < nb:
                wss[key] = torch.empty(max(nb, 1), dtype=torch.uint8, device=dev)
            hs = bool(red & (mp.MP_SUM | mp.MP_MEAN))
            hm = bool(red & mp.MP_MAX)
            mp.mp_spmm(h, rowptr, it, col, w_csr if wt else None, x, xd, N, N, F, ld, red,
                       out if hs else None, mp.MP_F32, mx[k] if hm else None, xd,
                       arg if hm else None, wss[key], wss[key].numel())
            i += 1
            mark(evs, i)

    return g, step, ops


def backward_step(g, mp, torch, np, dev, mark):
    """Backward of the headline graph's aggregation: the transposed CSR with
    its plan, then dL/dx for sum, mean and max and dL/dw for sum, from a
    seeded fp32 output gradient.  The forward CSR and the forward argmax are
    built once before timing (they come from the forward pass)."""
    import graphgen

    N, E, F = g.n_dst, g.E, g.F
    it = mp.MP_I32
    src = torch.from_numpy(g.src).to(dev)
    dst = torch.from_numpy(g.dst).to(dev)
    rowptr, col, _, _ = mp.coo_to_csr(src, dst, N)
    del src, dst
    x = torch.from_numpy(g.x).to(dev)
    G = torch.from_numpy(graphgen.normal_f32(1, 11, N * F).reshape(N, F)).to(dev)
    _, _, argout = mp.spmm(rowptr, col, x, mp.MP_MAX, plan=mp.Plan(rowptr, E, F))
    rowptrT = torch.empty(N + 1, dtype=torch.int32, device=dev)
    colT = torch.empty(E, dtype=torch.int32, device=dev)
    posT = torch.empty(E, dtype=torch.int32, device=dev)
    ws_t = torch.empty(mp.mp_csr_transpose_workspace(E, N, it, 1), dtype=torch.uint8, device=dev)
    nplan = mp.mp_spmm_plan_size(N, E)
    plan_buf = torch.empty(nplan, dtype=torch.uint8, device=dev)
    gx = torch.empty(N, F, dtype=torch.float32, device=dev)
    gw = torch.empty(E, dtype=torch.float32, device=dev)
    ws_w = torch.empty(mp.mp_spmm_backward_w_workspace(E), dtype=torch.uint8, device=dev)
    ops = [("transpose", transpose_bytes(N, N, E), 0), ("plan", plan_bytes(N), 0)]
    for m in ("sum", "mean", "max"):
        ops.append((f"grad_x_{m}_f32", grad_x_bytes(N, N, E, F, m), E * F))
    ops.append(("grad_w_sum_f32", grad_w_bytes(N, E, F), E * F))
    plans, wss = {}, {}

    sort_status = mp.new_status(dev)  # checked once after the timed steps
    SORT_STATUS.append(sort_status)

    def step(evs=None):
        mark(evs, 0)
        mp.mp_csr_transpose(rowptr, it, col, N, N, E, rowptrT, it, colT, posT, None, None, ws_t,
                            ws_t.numel(), sort_status)
        mark(evs, 1)
        if "h" in plans:
            mp.mp_spmm_plan_free(plans["h"])
        plans["h"] = h = mp.mp_spmm_plan_build(rowptrT, it, N, E, F, mp.MP_F32, plan_buf, nplan)
        mark(evs, 2)
        i = 2
        for red in (mp.MP_SUM, mp.MP_MEAN, mp.MP_MAX):
            nb = mp.mp_spmm_backward_x_workspace(h, N, E, F, red)
            if red not in wss or wss[red].numel() < nb:
                wss[red] = torch.empty(max(nb, 1), dtype=torch.uint8, device=dev)
            mp.mp_spmm_backward_x(h, rowptrT, it, colT, posT, None, rowptr, it, argout, G,
                                  mp.MP_F32, N, N, E, F, red, gx, mp.MP_F32, wss[red],
                                  wss[red].numel())
            i += 1
            mark(evs, i)
        mp.mp_spmm_backward_w(rowptr, it, col, x, mp.MP_F32, G, mp.MP_F32, None, N, N, E, F,
                              mp.MP_SUM, gw, ws_w, ws_w.numel())
        mark(evs, i + 1)

    # the gather ceilings: G's rows in the transposed CSR's column order, as
    # the sum and mean gradients read them, and one 16-byte chunk of each (a
    # scattered read per edge: the access pattern of the max gradient's won
    # chunks and mask words)
    g.probe = {"col": colT, "tables": {"G": (G, F * 4, F * 4)}, "chunk16": (G, F * 4)}
    return g, step, ops


def explain_step(g, mp, torch, np, dev, mark, seed):
    """One explainer iteration on the headline graph in explanation mode:
    messages materialized in edge space (fp32, 49.5 GB), an edge mask applied
    by the callback, sum aggregation, then the backward pass: dL/dmsg, the
    mask gradient (COO order), the callback's input gradient, and dL/dx over
    the transposed CSR with forward positions as columns.  The CSR, its
    transpose and their plans are built once before timing (the cached
    EdgeIndex formats).  The edge mask (U(0.5, 1)) is held per edge of the
    destination-sorted edge list, i.e. in CSR order, as for an EdgeIndex
    sorted by destination (whose COO order is the CSR order); the output
    gradient is N(0,1)."""
    import graphgen

    N, E, F = g.n_dst, g.E, g.F
    it = mp.MP_I32
    src = torch.from_numpy(g.src).to(dev)
    dst = torch.from_numpy(g.dst).to(dev)
    rowptr, col, _, _ = mp.coo_to_csr(src, dst, N)
    del src, dst
    rowptrT, _, posT, _ = mp.csr_transpose(rowptr, col, N)
    x = torch.from_numpy(g.x).to(dev)
    mask = torch.from_numpy(graphgen.uniform_f32(seed, 9, E) * np.float32(0.25)
                            + np.float32(0.75)).to(dev)
    G = torch.from_numpy(graphgen.normal_f32(1, 11, N * F).reshape(N, F)).to(dev)
    plan = mp.Plan(rowptr, E, F)
    planT = mp.Plan(rowptrT, E, F)
    m_pre = torch.empty(E, F, dtype=torch.float32, device=dev)
    m = torch.empty(E, F, dtype=torch.float32, device=dev)  # masked messages, then dL/dm_pre
    dm = torch.empty(E, F, dtype=torch.float32, device=dev)
    out = torch.empty(N, F, dtype=torch.float32, device=dev)
    gx = torch.empty(N, F, dtype=torch.float32, device=dev)
    dmask = torch.empty(E, dtype=torch.float32, device=dev)
    ws_b = torch.empty(mp.mp_message_backward_workspace(E), dtype=torch.uint8, device=dev)
    ws_f = plan.workspace(mp.MP_SUM)
    ws_t = planT.workspace(mp.MP_SUM)
    torch.cuda.synchronize()
    EF4 = E * F * 4
    rp = 4 * (N + 1)
    ops = [("msg_gather_f32", 4 * E + 2 * EF4, 0),
           ("mask_callback", 4 * E + 2 * EF4, 0),
           ("msg_sum", rp + EF4 + N * F * 4, E * F),
           ("msg_backward_sum", rp + N * F * 4 + EF4, 0),
           ("mask_grad", 2 * EF4 + 4 * E, 0),
           ("msg_input_grad", 4 * E + 2 * EF4, 0),
           ("grad_x_sum", rp + 4 * E + EF4 + N * F * 4, E * F)]
    nb = lambda t: 0 if t is None else t.numel()
    # the input gradient's own gather: rows of the E-row message-gradient
    # table in transposed order (each row once, in a scattered order)
    g.probe = {"col": posT, "tables": {"msg": (m, F * 4, F * 4)}}

    def step(evs=None):
        mark(evs, 0)
        mp.mp_message_gather(col, None, x, mp.MP_F32, N, E, F, m_pre, mp.MP_F32)
        mark(evs, 1)
        mp.mp_message_scale(m_pre, m, E, F, mask, None, E)
        mark(evs, 2)
        mp.mp_message_aggregate(plan.handle, rowptr, it, m, mp.MP_F32, E, N, F, mp.MP_SUM, out,
                                mp.MP_F32, None, mp.MP_F32, None, ws_f, nb(ws_f))
        mark(evs, 3)
        mp.mp_message_backward(rowptr, it, None, G, mp.MP_F32, N, E, F, mp.MP_SUM, dm, ws_b,
                               ws_b.numel())
        mark(evs, 4)
        mp.mp_edge_dot(dm, mp.MP_F32, m_pre, mp.MP_F32, None, E, None, E, F, dmask)
        mark(evs, 5)
        mp.mp_message_scale(dm, m, E, F, mask, None, E)
        mark(evs, 6)
        mp.mp_spmm(planT.handle, rowptrT, it, posT, None, m, mp.MP_F32, E, N, F, F, mp.MP_SUM, gx,
                   mp.MP_F32, None, mp.MP_F32, None, ws_t, nb(ws_t))
        mark(evs, 7)

    return g, step, ops


PNA = ["mean", "min", "max", "std"]


def stacked_step(g, mp, torch, np, dev, mark):
    """The headline graph with a stacked aggregation (mean, min, max and std,
    the aggregator set of principal neighbourhood aggregation) from one gather,
    for fp32 and for bf16 features, after COO->CSR and the plan."""
    N, E, F = g.n_dst, g.E, g.F
    it = mp.MP_I32
    src = torch.from_numpy(g.src).to(dev)
    dst = torch.from_numpy(g.dst).to(dev)
    xs = {"f32": (torch.from_numpy(g.x).to(dev), mp.MP_F32, 4),
          "bf16": (torch.from_numpy(g.x_bf16.view(np.int16)).to(dev).view(torch.bfloat16),
                   mp.MP_BF16, 2)}
    rowptr = torch.empty(N + 1, dtype=torch.int32, device=dev)
    col = torch.empty(E, dtype=torch.int32, device=dev)
    ws_csr = torch.empty(mp.mp_coo_to_csr_workspace(E, N, it, 0), dtype=torch.uint8, device=dev)
    nplan = mp.mp_spmm_plan_size(N, E)
    plan_buf = torch.empty(nplan, dtype=torch.uint8, device=dev)
    outs = [(mp.AGGR[n], torch.empty(N, F, dtype=torch.float32, device=dev),
             torch.empty(N, F, dtype=torch.int32, device=dev) if n in ("max", "min") else None)
            for n in PNA]
    ops = [("csr", csr_bytes(N, E), 0), ("plan", plan_bytes(N), 0)]
    tables = []  # (key, x, dtype code, row stride, padded copy or None)
    for k, (x, xd, xb) in xs.items():
        ld = mp.aligned_ld(F, x.dtype)
        xp = torch.empty(N, ld, dtype=x.dtype, device=dev)[:, :F] if ld != F else None
        if xp is not None:
            ops.append((f"layout_{k}", 2 * N * F * xb, 0))
        ops.append((f"stacked_{k}", multi_bytes(N, E, F, xb, PNA), E * F))
        tables.append((k, x, xd, ld, xp))
    plans, wss = {}, {}

    sort_status = mp.new_status(dev)  # checked once after the timed steps
    SORT_STATUS.append(sort_status)

    def step(evs=None):
        mark(evs, 0)
        mp.mp_coo_to_csr(src, dst, E, N, rowptr, it, col, None, None, None, ws_csr,
                         ws_csr.numel(), sort_status)
        mark(evs, 1)
        if "h" in plans:
            mp.mp_spmm_plan_free(plans["h"])
        plans["h"] = h = mp.mp_spmm_plan_build(rowptr, it, N, E, F, mp.MP_F32, plan_buf, nplan)
        mark(evs, 2)
        nb = mp.mp_spmm_multi_workspace(h)
        if "ws" not in wss or wss["ws"].numel() < nb:
            wss["ws"] = torch.empty(max(nb, 1), dtype=torch.uint8, device=dev)
        i = 2
        for k, x, xd, ld, xp in tables:
            if xp is not None:
                mp.mp_copy_rows(x, F, xp, ld, N, F, xd)
                i += 1
                mark(evs, i)
                x = xp
            mp.mp_spmm_multi(h, rowptr, it, col, None, x, xd, N, N, F, ld, outs, wss["ws"],
                             wss["ws"].numel())
            i += 1
            mark(evs, i)

    return g, step, ops


def readout_step(g, mp, torch, np, dev, mark, seed):
    """A global readout: the headline graph's 2,449,029 node rows (F = 100,
    fp32 and bf16) split into 1,024 graphs of a seeded mini-batch, given as a
    sorted batch vector; ptr from the sorted-COO
    fast path, the plan, then sum, mean, max and std per graph from one pass.
    Graph sizes are proportional to seeded uniform draws in [1, 2 N / 1024]."""
    import graphgen

    N, F = g.n_src, g.F
    B = 1024
    u = graphgen.uniform_ints(seed, 13, B, 2 * N // B).astype(np.int64) + 1
    sizes = u * N // int(u.sum())  # proportional to the draws, summing to N
    sizes[-1] = N - int(sizes[:-1].sum())
    batch = torch.from_numpy(np.repeat(np.arange(B, dtype=np.int32), sizes)).to(dev)
    nodes = torch.arange(N, dtype=torch.int32, device=dev)
    ptr = torch.empty(B + 1, dtype=torch.int32, device=dev)
    col = torch.empty(N, dtype=torch.int32, device=dev)
    xs = {"f32": (torch.from_numpy(g.x).to(dev), mp.MP_F32, 4),
          "bf16": (torch.from_numpy(g.x_bf16.view(np.int16)).to(dev).view(torch.bfloat16),
                   mp.MP_BF16, 2)}
    nplan = mp.mp_spmm_plan_size(B, N)
    plan_buf = torch.empty(nplan, dtype=torch.uint8, device=dev)
    names = ["sum", "mean", "max", "std"]
    outs = [(mp.AGGR[n], torch.empty(B, F, dtype=torch.float32, device=dev),
             torch.empty(B, F, dtype=torch.int32, device=dev) if n == "max" else None)
            for n in names]
    ops = [("ptr", 4 * N + 4 * (B + 1), 0), ("plan", plan_bytes(B), 0)]
    for k, (_, _, xb) in xs.items():
        ops.append((f"readout_{k}", multi_bytes(B, N, F, xb, names, col=False), N * F))
    plans, wss = {}, {}

    def step(evs=None):
        mark(evs, 0)
        mp.mp_sorted_coo_to_csr(nodes, batch, N, B, ptr, mp.MP_I32, col, None, None, None)
        mark(evs, 1)
        if "h" in plans:
            mp.mp_spmm_plan_free(plans["h"])
        plans["h"] = h = mp.mp_spmm_plan_build(ptr, mp.MP_I32, B, N, F, mp.MP_F32, plan_buf,
                                               nplan)
        mark(evs, 2)
        nb = mp.mp_spmm_multi_workspace(h)
        if "ws" not in wss or wss["ws"].numel() < nb:
            wss["ws"] = torch.empty(max(nb, 1), dtype=torch.uint8, device=dev)
        i = 2
        for k, (x, xd, _) in xs.items():
            mp.mp_readout_multi(h, ptr, mp.MP_I32, x, xd, N, B, F, F, outs, wss["ws"],
                                wss["ws"].numel())
            i += 1
            mark(evs, i)

    from types import SimpleNamespace
    return SimpleNamespace(n_dst=B, n_src=N, E=N, F=F), step, ops


def projection_step(args, mp, torch, np, dev):
    """Typed projections {H_T W_T} of the typed graph's node tables (1.9M,
    736k, 8.7k rows; F = F' = 128; bf16 x, W and output gradient, N(0,1),
    W scaled by 1/sqrt(F)): forward (fp32 out), input gradient (fp32) and
    weight gradient (fp32), as one training step of the projection."""
    import graphgen
    from types import SimpleNamespace

    sizes = [1_900_000, 736_000, 8_700]
    F = Fo = 128
    T = len(sizes)
    seg = [0] + [int(v) for v in np.cumsum(sizes)]
    N = seg[-1]
    t0 = time.time()
    bf = lambda a: torch.from_numpy(graphgen.f32_to_bf16(a).view(np.int16)).to(dev).view(
        torch.bfloat16)
    x = bf(graphgen.normal_f32(args.seed, 3, N * F).reshape(N, F))
    W = bf((graphgen.normal_f32(args.seed, 5, T * F * Fo) / np.sqrt(F)).astype(np.float32)
           .reshape(T, F, Fo))
    dout = bf(graphgen.normal_f32(args.seed, 11, N * Fo).reshape(N, Fo))
    print(f"[bench] generated projection inputs in {time.time() - t0:.1f}s", file=sys.stderr,
          flush=True)
    out = torch.empty(N, Fo, dtype=torch.float32, device=dev)
    dx = torch.empty(N, F, dtype=torch.float32, device=dev)
    dW = torch.empty(T, F, Fo, dtype=torch.float32, device=dev)
    ws_f = torch.empty(mp.mp_segment_matmul_workspace(T, F, Fo), dtype=torch.uint8, device=dev)
    nb = mp.mp_segment_matmul_backward_workspace(seg, T, F, Fo)
    ws_b = torch.empty(nb, dtype=torch.uint8, device=dev)
    chunks = nb // (F * Fo * 4)
    wb = T * F * Fo * 2
    ops = [("proj_fwd", 2 * N * F + 2 * wb + 4 * N * Fo, 0),
           ("proj_dx", 2 * N * Fo + wb + 4 * N * F, 0),
           ("proj_dw", 2 * N * F + 2 * N * Fo + 2 * chunks * F * Fo * 4 + T * F * Fo * 4, 0)]
    flops = 2 * N * F * Fo

    mark = make_mark(torch.cuda.current_stream())

    def step(evs=None):
        mark(evs, 0)
        mp.mp_segment_matmul(seg, T, x, W, F, Fo, out, mp.MP_F32, ws_f, ws_f.numel())
        mark(evs, 1)
        mp.mp_segment_matmul_backward(seg, T, x, W, dout, F, Fo, dx, mp.MP_F32, None, None, 0)
        mark(evs, 2)
        mp.mp_segment_matmul_backward(seg, T, x, W, dout, F, Fo, None, mp.MP_F32, dW, ws_b,
                                      ws_b.numel())
        mark(evs, 3)

    return SimpleNamespace(n_dst=N, n_src=N, E=0, F=F, flops_per_op=flops), step, ops


OP_KERNELS = {
    "proj_fwd": "gmm_nt (bf16 MFMA 32x32x16, fp32 out)",
    "proj_dx": "gmm_nt (bf16 MFMA 32x32x16, fp32 out)",
    "proj_dw": "gmm_tn_partial + reduce_partials (bf16 MFMA 32x32x16)",
    "stacked_f32": "spmm_main, stats mode (mean, min, max, std from one gather)",
    "stacked_bf16": "spmm_main, stats mode (mean, min, max, std from one gather)",
    "readout_f32": "spmm_main, stats mode over consecutive node rows (readout)",
    "readout_bf16": "spmm_main, stats mode over consecutive node rows (readout)",
    "grad_x_sum_f32": "spmm_main (sum over the transposed CSR)",
    "grad_x_mean_f32": "spmm_main (sum over the transposed CSR of G/deg)",
    "grad_x_max_f32": "spmm_main, masked (argmax routing over the transposed CSR)",
    "grad_w_sum_f32": "spmm_grad_w (per-edge dot products)",
    "msg_gather_f32": "message_gather (edge-space gather of x rows)",
    "mask_callback": "message_scale (edge mask)",
    "msg_sum": "spmm_main over message rows",
    "msg_backward_sum": "message_backward (dL/dmsg)",
    "mask_grad": "spmm_grad_w as per-edge dot products",
    "msg_input_grad": "message_scale (callback input gradient)",
    "grad_x_sum": "spmm_main over the transposed CSR, message rows gathered by position",
}


def run(args):
    import numpy as np
    import torch

    import paper_2507_16991_amd as mp

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}); the multi-GPU "
              "path is a design, not a build", file=sys.stderr)
        sys.exit(2)
    mp.lib()  # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    g, step, ops = build_step(args, mp, torch, np, dev)
    N, E, F = g.n_dst, g.E, g.F
    names = [o[0] for o in ops]
    op_bytes = {o[0]: o[1] for o in ops}
    if args.dump_ops:
        with open(args.dump_ops, "w") as f:
            json.dump([{"name": o[0], "bytes": o[1]} for o in ops], f)
    step_bytes = sum(o[1] for o in ops)
    step_ef = sum(o[2] for o in ops)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if args.calibrate_copy:
        a = torch.empty(CALIB_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    # warm: K steps back to back, one event per operation boundary
    all_evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(ops) + 1)]
               for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        step(all_evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_step = wall * 1e3 / args.steps
    for st in SORT_STATUS:  # every sort of the timed steps completed
        mp.check_status(st, "device sort of a timed step")
    warm = {n: [evs[i].elapsed_time(evs[i + 1]) for evs in all_evs] for i, n in enumerate(names)}
    op_ms = {n: float(np.mean(v)) for n, v in warm.items()}

    # cold: every operation alone after a 1 GiB write (caches flushed)
    cold = {}
    if args.cold_reps > 0:
        flush_buf = torch.empty(1 << 28, dtype=torch.int32, device=dev)
        cev = [ColdEvents(torch, len(ops), lambda: flush_buf.fill_(7))
               for _ in range(args.cold_reps)]
        for c in cev:
            step(c)
        torch.cuda.synchronize()
        for st in SORT_STATUS:
            mp.check_status(st, "device sort of a cold step")
        times = [c.times() for c in cev]
        cold = {n: [t[i] for t in times] for i, n in enumerate(names)}
        del flush_buf

    def gbs(nbytes, ms):
        return round(nbytes / (ms * 1e-3) / 1e9, 1)

    breakdown = {}
    for n in names:
        w = warm[n]
        d = {"ms": round(op_ms[n], 4), "ms_median": round(float(np.median(w)), 4),
             "ms_min": round(float(np.min(w)), 4), "GB_per_s": gbs(op_bytes[n], op_ms[n])}
        if n in cold:
            cm = float(np.median(cold[n]))
            d.update({"cold_ms_median": round(cm, 4),
                      "cold_ms_min": round(float(np.min(cold[n])), 4),
                      "cold_GB_per_s": gbs(op_bytes[n], cm)})
        breakdown[n] = d
    for n in names:  # the sorts: edges (keys) per second
        if n in ("csr", "transpose", "hetero_build"):
            breakdown[n]["keys_per_s"] = round(E / (op_ms[n] * 1e-3), -6)
    if getattr(g, "flops_per_op", 0):
        for n in names:  # every projection op is 2 N F F' flops
            breakdown[n]["TFLOP_per_s"] = round(g.flops_per_op / (op_ms[n] * 1e-3) / 1e12, 1)
    ceil = measure_ceilings(g, mp, torch, np, dev) if args.ceilings and hasattr(g, "probe") \
        else None
    if ceil:
        for n in names:  # gradients over the transposed CSR against G's gather
            if "gather_G" in ceil and n in ("grad_x_sum_f32", "grad_x_mean_f32"):
                breakdown[n]["frac_of_gather_ceiling"] = round(
                    breakdown[n]["GB_per_s"] / ceil["gather_G"]["GB_per_s"], 4)
            if "gather_msg" in ceil and n == "grad_x_sum":
                breakdown[n]["frac_of_gather_ceiling"] = round(
                    breakdown[n]["GB_per_s"] / ceil["gather_msg"]["GB_per_s"], 4)
        for n in names:  # aggregations against the gather of their own table
            k = n.rsplit("_", 1)[-1]
            if f"gather_{k}" in ceil and n.split("_")[0] in ("sum", "mean", "max", "wsum",
                                                              "sum+max"):
                breakdown[n]["frac_of_gather_ceiling"] = round(
                    breakdown[n]["GB_per_s"] / ceil[f"gather_{k}"]["GB_per_s"], 4)
    value = step_bytes / (ms_step * 1e-3) / 1e9
    web = args.workload == "web-1.6B"
    headline = args.workload == WORKLOAD
    dom = max((o for o in ops if o[2] > 0 or args.workload in (PROJECTION, EXPLAIN)),
              key=lambda o: op_ms[o[0]])[0]
    dom_kernel = DOMINANT + ", fp32 sum" if headline else OP_KERNELS.get(dom, f"spmm_main ({dom})")
    if headline:
        dom = "sum_f32"
    dom_ms, dom_bytes = op_ms[dom], op_bytes[dom]
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    traffic = read_traffic() if headline else None
    descs = {
        WORKLOAD: (f"{WORKLOAD}: Chung-Lu power-law graph, N={N}, E={E}, F={F}, features fp32 "
                   f"and bf16 (N(0,1)), seed {args.seed}",
                   "COO->CSR + plan + {sum, mean, max+argmax} x {fp32, bf16 features}"),
        "web-1.6B": (f"web-1.6B: power-law in-degree (alpha 2.0), uniform sources, N={N}, E={E}, "
                     f"F={F}, bf16 features U(-1,1), int64 rowptr, seed {args.seed}",
                     "COO->CSR + plan + fused {sum fp32, max bf16 + argmax}"),
        "powerlaw-1.2M": (f"powerlaw-1.2M: Zipf-like in-degree (alpha 2.1), uniform sources, "
                          f"N={N}, E={E}, F={F}, fp32 N(0,1), GCN weights, seed {args.seed}",
                          "COO->CSR (+perm, weights to CSR order) + plan + mean + weighted sum"),
        "uniform-10k": (f"uniform-10k: uniform random graph, N={N}, E={E}, F={F}, fp32 U(-1,1), "
                        f"seed {args.seed}", "COO->CSR + plan + sum"),
        PROJECTION: (f"{PROJECTION}: typed projections of the node tables of hetero-20M "
                     f"(1.9M, 736k, 8.7k rows), F = F' = {F}, bf16 inputs, seed {args.seed}",
                     "segment matmul forward + input gradient + weight gradient"),
        STACKED: (f"{STACKED}: the Chung-Lu graph of {WORKLOAD} (N={N}, E={E}, F={F}, fp32 and "
                  f"bf16 N(0,1) features), seed {args.seed}",
                  "COO->CSR + plan + stacked {mean, min, max, std} x {fp32, bf16 features}"),
        READOUT: (f"{READOUT}: the {WORKLOAD} node rows (2449029 x {F}, fp32 and bf16) in "
                  f"1024 graphs of a sorted batch vector, seed {args.seed}",
                  "ptr from the sorted batch + plan + readout {sum, mean, max, std} x "
                  "{fp32, bf16}"),
        EXPLAIN: (f"{EXPLAIN}: the Chung-Lu graph of {WORKLOAD} (N={N}, E={E}, F={F}, fp32 "
                  f"x and output gradient N(0,1), edge mask U(0.5, 1) in CSR order), seed {args.seed}",
                  "materialized messages + edge-mask callback + sum + dL/dmsg + mask gradient "
                  "+ callback input gradient + dL/dx"),
        BACKWARD: (f"{BACKWARD}: the Chung-Lu graph of {WORKLOAD} (N={N}, E={E}, F={F}, fp32 "
                   f"x and output gradient N(0,1)), seed {args.seed}",
                   "CSR transpose + plan + dL/dx {sum, mean, max} + dL/dw sum"),
        "hetero-20M": (f"hetero-20M: 3 node types (1.9M, 736k, 8.7k), 4 relations (5.4M, 7.1M, "
                       f"7.1M, 1.0M edges), F={F} bf16, seed {args.seed}",
                       "all destination types at once: one combined CSR over all nodes + plan + "
                       "sum over relations (row slices = the per-type CSRs and outputs)"),
    }
    desc, stepdesc = descs[args.workload]
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": desc, "step": stepdesc, "accumulate": "fp32",
                   "rowptr": "int64" if web else "int32"},
        "edge_features_per_s": round(step_ef / (ms_step * 1e-3), 1),
        "percent_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "ops": breakdown,
        "roofline": {
            "bound": "hbm",
            "kernel": dom_kernel + (" (+ hub fix-up)" if dom_kernel.startswith("spmm_main") else ""),
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None if traffic is None else round(traffic / (dom_ms * 1e-3) / 1e9, 1),
            "traffic_note": "FETCH_SIZE + WRITE_SIZE per launch (copy-calibrated) over the "
                            "launch time: bytes leaving the L2, MALL hits included, so an "
                            "upper bound on HBM traffic",
            "traffic_bytes_per_launch": None if traffic is None else int(traffic),
            "algorithmic_bytes_per_launch": dom_bytes,
            "avg_launch_ms": round(dom_ms, 4),
        },
    }
    if ceil:
        result["ceilings"] = ceil
        k = dom.rsplit("_", 1)[-1]
        if f"gather_{k}" in ceil:
            mc = ceil[f"gather_{k}"]["GB_per_s"]
            result["roofline"]["measured_ceiling"] = {
                "GB_per_s": mc, "probe": ceil[f"gather_{k}"]["what"]}
            result["roofline"]["frac_of_measured_ceiling"] = round(achieved / mc, 4)
    if args.cpu_baseline and headline:
        result["cpu_baseline"] = cpu_baseline(g, N, E, F, step_bytes, args)
    print(json.dumps(result), flush=True)


def measure_ceilings(g, mp, torch, np, dev, reps=5):
    """What the device delivers for the aggregation's traffic, measured with
    the library's bandwidth probes on this workload's own buffers: a streaming
    read and a copy, and, per feature table, the row gather in CSR column
    order (every edge reads its column index and one row; no reduction, no
    output); on the headline graph also a radix pass's data movement (8-byte
    words scattered into the stable order of dst's first digit).  GB/s of
    algorithmic bytes (for the gather 4 + F*b per edge, for the scatter 16 per
    word), median of `reps` timed runs after one untimed."""
    col = g.probe["col"]
    E = int(col.numel())
    sink = torch.zeros(mp.MP_PROBE_SINK_WORDS, dtype=torch.int32, device=dev)
    big = torch.empty(1 << 28, dtype=torch.int32, device=dev)  # 1 GiB
    big2 = torch.empty_like(big)

    def timed(fn):
        ts = []
        for r in range(reps + 1):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts[1:]))

    res = {}
    for name, nbytes, fn in [("read", 1 << 30, lambda: mp.mp_probe_read(big, 1 << 30, sink)),
                             ("copy", 2 << 30, lambda: mp.mp_probe_copy(big, big2, 1 << 30))]:
        ms = timed(fn)
        res[name] = {"ms": round(ms, 4), "GB_per_s": round(nbytes / (ms * 1e-3) / 1e9, 1),
                     "what": "1 GiB streaming read" if name == "read" else
                     "1 GiB streaming copy (read + write)"}
    del big, big2
    for k, (x, stride, row) in g.probe["tables"].items():
        probe_row = (row + 15) // 16 * 16
        ms = timed(lambda: mp.mp_probe_gather(col, E, x, stride, probe_row, sink))
        res[f"gather_{k}"] = {
            "ms": round(ms, 4), "GB_per_s": round(E * (4 + row) / (ms * 1e-3) / 1e9, 1),
            "what": f"{E} rows of {row} B ({k} features, rows {stride} B apart) gathered in CSR "
                    f"column order, 16-byte loads"}
    if "scatter" in g.probe:
        # one radix pass's data movement over the packed (key, payload) words:
        # every word read in order and written to its place in the stable
        # order of dst's first digit, first in source order (a scatter that
        # does not stage), then with the words of each tile of SORT_TILE keys
        # taken in digit order (the order in which the staged pass writes, so
        # a wavefront writes consecutive places of one digit run)
        keys, bits = g.probe["scatter"]
        n = int(keys.numel())
        dig = (keys & ((1 << bits) - 1)).to(torch.int64)
        order = torch.argsort(dig, stable=True)
        dest = torch.empty(n, dtype=torch.int32, device=dev)
        dest[order] = torch.arange(n, dtype=torch.int32, device=dev)
        tile = torch.arange(n, dtype=torch.int64, device=dev) // SORT_TILE
        staged = torch.argsort(tile * (1 << bits) + dig, stable=True)
        dest_staged = dest[staged]
        del order, dig, tile, staged
        w_in = torch.zeros(n, dtype=torch.int64, device=dev)
        w_out = torch.empty_like(w_in)
        for name, d, how in (("scatter8", dest, "in source order"),
                             ("scatter8_staged", dest_staged,
                              f"each tile of {SORT_TILE} taken in digit order")):
            ms = timed(lambda: mp.mp_probe_scatter(w_in, d, n, 8, w_out))
            res[name] = {
                "ms": round(ms, 4), "GB_per_s": round(16 * n / (ms * 1e-3) / 1e9, 1),
                "what": f"{n} 8-byte words read in order ({how}) and written to their places "
                        f"in the stable order by the low {bits}-bit digit of dst: one packed "
                        f"radix pass's reads and writes, 16 B per key (the 4-byte "
                        f"destinations read besides)"}
        del dest, dest_staged, w_in, w_out
    if "chunk16" in g.probe:
        x, stride = g.probe["chunk16"]
        ms = timed(lambda: mp.mp_probe_gather(col, E, x, stride, 16, sink))
        res["chunk16"] = {
            "ms": round(ms, 4), "G_reads_per_s": round(E / (ms * 1e-3) / 1e9, 2),
            "what": f"{E} scattered 16-byte reads: the first chunk of each row (rows {stride} B "
                    f"apart) in CSR column order"}
    return res


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(g, N, E, F, step_bytes, args):
    """The CPU oracle on the same step: its COO->CSR on the whole graph, and
    its aggregation (sum, mean and max in one pass, fp32 and bf16 features)
    on all rows, or on a leading block of rows (--cpu-rows) whose time is then
    scaled by E / (edges in the block)."""
    import numpy as np

    import oracle

    threads = oracle.default_threads()
    t0 = time.perf_counter()
    rp, col, _, _ = oracle.coo_to_csr(g.src, g.dst, N)
    t_csr = time.perf_counter() - t0
    rows_n = N if args.cpu_rows <= 0 else min(N, args.cpu_rows)
    rows = np.arange(rows_n, dtype=np.int64)
    e_s = int(rp[rows_n] - rp[0])
    t0 = time.perf_counter()
    oracle.spmm(rp, col, x=g.x, rows=rows, nthreads=threads)
    oracle.spmm(rp, col, x_bf16=g.x_bf16, rows=rows, nthreads=threads)
    t_agg = time.perf_counter() - t0
    t_step = t_csr + t_agg * (E / max(e_s, 1))
    scaled = "" if rows_n == N else f", scaled by E/{e_s}"
    # the same aggregation on one thread, over a leading block of rows
    r1 = int(np.searchsorted(rp, E // 32))
    rows1 = np.arange(r1, dtype=np.int64)
    e1 = int(rp[r1])
    t0 = time.perf_counter()
    oracle.spmm(rp, col, x=g.x, rows=rows1, nthreads=1)
    oracle.spmm(rp, col, x_bf16=g.x_bf16, rows=rows1, nthreads=1)
    t_one = (time.perf_counter() - t0) * (E / max(e1, 1))
    t_step1 = t_csr + t_one
    return {
        "value": round(step_bytes / t_step / 1e9, 3),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "cpu_model": cpu_model(),
        "sample": f"oracle COO->CSR on all {E} edges (1 thread, {t_csr:.2f}s) + oracle "
                  f"aggregation (sum/mean/max in one pass, fp32 and bf16 features) on rows "
                  f"0..{rows_n - 1} ({e_s} edges, {t_agg:.2f}s, {threads} threads){scaled}; "
                  f"one full step {t_step:.1f}s",
        "one_thread": {
            "value": round(step_bytes / t_step1 / 1e9, 3),
            "unit": "GB/s",
            "sample": f"the same aggregation on 1 thread over rows 0..{r1 - 1} ({e1} edges), "
                      f"scaled by E/{e1} to {t_one:.1f}s; with the COO->CSR, one full step "
                      f"{t_step1:.1f}s"},
    }


# ---- rocprofv3 summaries -----------------------------------------------------------------

def _find(dirname, pattern):
    hits = glob.glob(os.path.join(dirname, "**", pattern), recursive=True)
    if not hits:
        raise SystemExit(f"no {pattern} under {dirname}")
    return hits[0]


def short_name(name):
    """Kernel name without namespaces, return type and parameter list."""
    name = name.replace("mp::(anonymous namespace)::", "").replace("void ", "")
    depth = 0
    for i, ch in enumerate(name):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return name[:i]
    return name


def summarize_stats(d, out, cmd):
    path = _find(d, "*kernel_stats.csv")
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    lines = [f"# rocprofv3 kernel stats ({os.path.basename(path)})", f"command: {cmd}", "",
             f"{'kernel':<70} {'calls':>6} {'avg_us':>10} {'total_ms':>10} {'pct':>6}"]
    for r in rows[:25]:
        name = short_name(r["Name"])[:70]
        lines.append(f"{name:<70} {r['Calls']:>6} {float(r['AverageNs']) / 1e3:>10.1f} "
                     f"{float(r['TotalDurationNs']) / 1e6:>10.2f} {float(r['Percentage']):>6.2f}")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter_rows(d):
    path = _find(d, "*counter_collection.csv")
    return list(csv.DictReader(open(path)))


def _is_calib(kernel_name):
    """torch's copy kernel (the --calibrate-copy run), not the library's own
    row copy."""
    k = kernel_name.lower()
    return ("copy" in k or "elementwise" in k) and not short_name(kernel_name).startswith("copy_rows")


def _per_dispatch(rows, counter):
    """{(dispatch id, kernel name): value} summed over the counter's instances."""
    acc = {}
    for r in rows:
        if r.get("Counter_Name") != counter:
            continue
        key = (r["Dispatch_Id"], r["Kernel_Name"])
        acc[key] = acc.get(key, 0.0) + float(r["Counter_Value"])
    return acc


def _segment_ops(dispatches):
    """Split one step's dispatches (in dispatch order) into its operations:
    everything before the first plan kernel is the COO->CSR, from there to
    the plan header the plan, a row copy is a layout operation, and each
    aggregation is [spmm_tiny] spmm_main [spmm_fixup].  Returns a list of
    (kind, [dispatch rows])."""
    segs = []
    phase = "csr"
    for d in dispatches:
        k = short_name(d["name"])
        if phase == "csr" and k.startswith("plan_classes"):
            phase = "plan"
        if phase in ("csr", "plan"):
            if not segs or segs[-1][0] != phase:
                segs.append((phase, []))
            segs[-1][1].append(d)
            if k.startswith("plan_header"):
                phase = "ops"
            continue
        if k.startswith("copy_rows"):
            segs.append(("layout", [d]))
        elif k.startswith("spmm_tiny"):
            segs.append(("agg", [d]))
        elif k.startswith("spmm_main"):
            if segs and segs[-1][0] == "agg" and \
                    short_name(segs[-1][1][-1]["name"]).startswith("spmm_tiny"):
                segs[-1][1].append(d)
            else:
                segs.append(("agg", [d]))
        elif k.startswith("spmm_fixup") and segs and segs[-1][0] == "agg":
            segs[-1][1].append(d)
        else:
            segs.append(("other", [d]))
    return segs


def summarize_step_counters(fetch_dir, write_dir, ops_path, out, cmd):
    """FETCH_SIZE and WRITE_SIZE of every operation of one step (two pmc runs
    of `bench.py --steps 1 --warmup 0 --dump-ops ops_path --calibrate-copy`),
    scaled by the copy calibration, against each operation's algorithmic
    bytes."""
    fr = _per_dispatch(_counter_rows(fetch_dir), "FETCH_SIZE")
    wr = _per_dispatch(_counter_rows(write_dir), "WRITE_SIZE")
    ops = json.load(open(ops_path))
    copy_f = [v for (i, k), v in fr.items() if _is_calib(k)]
    copy_w = [v for (i, k), v in wr.items() if _is_calib(k)]
    scale_f = CALIB_BYTES / (max(copy_f) * 1024.0) if copy_f else 1.0
    scale_w = CALIB_BYTES / (max(copy_w) * 1024.0) if copy_w else 1.0

    def step_dispatches(table):
        rows = sorted(((int(i), k, v) for (i, k), v in table.items()), key=lambda t: t[0])
        return [{"id": i, "name": k, "kib": v} for i, k, v in rows
                if not _is_calib(k)
                and "fill" not in k.lower()]

    fs, ws = _segment_ops(step_dispatches(fr)), _segment_ops(step_dispatches(wr))
    names = [o["name"] for o in ops]
    algo = {o["name"]: o["bytes"] for o in ops}
    lines = ["# HBM-side traffic of every operation of one step, from rocprofv3 counters",
             f"command_fetch: {cmd.format(ctr='FETCH_SIZE')}",
             f"command_write: {cmd.format(ctr='WRITE_SIZE')}",
             f"fetch_scale: {scale_f:.4f}  write_scale: {scale_w:.4f}  (copy of "
             f"{CALIB_BYTES} bytes: FETCH_SIZE and WRITE_SIZE scaled so it reads and writes "
             f"that many)",
             "FETCH_SIZE and WRITE_SIZE count L2 egress: the bytes the L2 requests from "
             "and writes to the fabric, MALL hits included, so fetch + write is an upper "
             "bound on HBM traffic, not a measured HBM rate.",
             "",
             f"{'operation':<14} {'fetch_GB':>10} {'write_GB':>10} {'total_GB':>10} "
             f"{'algo_GB':>10} {'ratio':>7}  kernels"]
    if len(fs) != len(names) or len(ws) != len(names):
        lines.append(f"(segmentation found {len(fs)} / {len(ws)} operations for {len(names)} "
                     f"named ones: {names})")
    for n, (kf, df), (kw, dw) in zip(names, fs, ws):
        f_b = sum(d["kib"] for d in df) * 1024.0 * scale_f
        w_b = sum(d["kib"] for d in dw) * 1024.0 * scale_w
        ks = ", ".join(sorted({short_name(d["name"]).split("<")[0] for d in df}))
        lines.append(f"{n:<14} {f_b / 1e9:>10.3f} {w_b / 1e9:>10.3f} {(f_b + w_b) / 1e9:>10.3f} "
                     f"{algo[n] / 1e9:>10.3f} {(f_b + w_b) / max(algo[n], 1):>7.3f}  {ks}")
        per = {}
        for d in df:
            per.setdefault(short_name(d["name"]).split("<")[0], [0.0, 0.0])[0] += d["kib"]
        for d in dw:
            per.setdefault(short_name(d["name"]).split("<")[0], [0.0, 0.0])[1] += d["kib"]
        if len(per) > 1:
            for k, (kf_, kw_) in sorted(per.items(), key=lambda t: -(t[1][0] + t[1][1])):
                lines.append(f"  {k:<24} {kf_ * 1024.0 * scale_f / 1e9:>10.3f} "
                             f"{kw_ * 1024.0 * scale_w / 1e9:>10.3f}")
    lines.append(f"kernel_source_sha1: {source_digest(DOMINANT_SRC)}")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


SQ_COUNTERS = ["SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_ACTIVE_INST_VALU",
               "SQ_INSTS_VALU", "SQ_INSTS_VMEM_RD", "SQ_INSTS_LDS", "SQ_BUSY_CYCLES",
               "GRBM_GUI_ACTIVE"]
CU_NUM = 256
XCD_NUM = 8
CLOCK_HZ = 2.4e9


def summarize_sq(d, out, cmd, kernels=None):
    """Per-kernel shader counters of one `rocprofv3 --pmc <SQ_COUNTERS>` run,
    averaged over the kernel's dispatches, with the ratios rocprofv3 itself
    defines for gfx950: occupancy = 400 * SQ_WAVE_CYCLES / GRBM_GUI_ACTIVE /
    CUs / 32 (percent of 32 wavefronts per CU), VALU busy = 100 *
    SQ_ACTIVE_INST_VALU / CUs / GRBM_GUI_ACTIVE; wait = SQ_WAIT_ANY /
    SQ_WAVE_CYCLES (the share of wavefront time spent waiting on memory,
    LDS or a barrier); and the VALU floor, SQ_INSTS_VALU / (CUs * clock),
    the time the kernel's vector instructions take at one wave64 instruction
    per CU per cycle.  rocprofv3's CSV holds GRBM_GUI_ACTIVE summed over the
    8 XCDs, while its formulas take one XCD's count (a maximum over them), so
    the count is divided by 8 here; clk = that count / the kernel's duration
    is the shader clock the kernel ran at."""
    rows = _counter_rows(d)
    per = {}  # short kernel name -> counter -> [values per dispatch]
    lds = {}  # short kernel name -> LDS bytes per workgroup
    for r in rows:
        name = short_name(r["Kernel_Name"])
        lds[name] = r.get("LDS_Block_Size", "?")
        c = r.get("Counter_Name")
        if c not in SQ_COUNTERS:
            continue
        key = (r["Dispatch_Id"], name)
        red = max if c == "GRBM_GUI_ACTIVE" else (lambda a, b: a + b)
        disp = per.setdefault(name, {}).setdefault(c, {})
        v = float(r["Counter_Value"])
        disp[key] = red(disp[key], v) if key in disp else v
    dur = {}
    try:
        for r in csv.DictReader(open(_find(d, "*kernel_stats.csv"))):
            dur[short_name(r["Name"])] = float(r["AverageNs"]) / 1e6
    except SystemExit:
        pass
    lines = ["# Shader counters per kernel (rocprofv3 --pmc, averaged over dispatches)",
             f"command: {cmd}",
             "G = GRBM_GUI_ACTIVE / 8 (the CSV sums it over the 8 XCDs); "
             "occ% = 400*SQ_WAVE_CYCLES/G/256/32 (share of 32 wavefronts per CU); "
             "valu% = 100*SQ_ACTIVE_INST_VALU/256/G; wait% = SQ_WAIT_ANY/SQ_WAVE_CYCLES; "
             "clk = G / ms; valu_floor_ms = SQ_INSTS_VALU/(256 CUs * 2.4 GHz); "
             "ms = kernel-trace average (counter collection serializes dispatches)",
             "",
             f"{'kernel':<64} {'calls':>5} {'ms':>8} {'lds_B':>6} {'clk_GHz':>7} "
             f"{'occ%':>6} {'valu%':>6} {'wait%':>6} {'valu/wave':>9} {'vmem/wave':>9} "
             f"{'lds/wave':>8} {'valu_floor_ms':>13}"]
    order = sorted(per, key=lambda n: -dur.get(n, 0.0))
    for name in order:
        if kernels and not any(k in name for k in kernels):
            continue
        c = {k: sum(v.values()) / max(len(v), 1) for k, v in per[name].items()}
        calls = max(len(v) for v in per[name].values())
        g = c.get("GRBM_GUI_ACTIVE", 0.0) / XCD_NUM
        wc = c.get("SQ_WAVE_CYCLES", 0.0)
        waves = max(c.get("SQ_WAVES", 0.0), 1.0)
        occ = 400.0 * wc / g / CU_NUM / 32 if g else float("nan")
        valu = 100.0 * c.get("SQ_ACTIVE_INST_VALU", 0.0) / CU_NUM / g if g else float("nan")
        wait = 100.0 * c.get("SQ_WAIT_ANY", 0.0) / wc if wc else float("nan")
        floor_ms = c.get("SQ_INSTS_VALU", 0.0) / (CU_NUM * CLOCK_HZ) * 1e3
        ms = dur.get(name)
        clk = g / (ms * 1e-3) / 1e9 if ms else float("nan")
        lines.append(f"{name[:64]:<64} {calls:>5} {'' if ms is None else f'{ms:.3f}':>8} "
                     f"{lds.get(name, '?'):>6} {clk:>7.2f} {occ:>6.1f} {valu:>6.1f} {wait:>6.1f} "
                     f"{c.get('SQ_INSTS_VALU', 0.0) / waves:>9.0f} "
                     f"{c.get('SQ_INSTS_VMEM_RD', 0.0) / waves:>9.0f} "
                     f"{c.get('SQ_INSTS_LDS', 0.0) / waves:>8.0f} {floor_ms:>13.3f}")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_counters(fetch_dir, write_dir, out, cmd):
    fr = _per_dispatch(_counter_rows(fetch_dir), "FETCH_SIZE")
    wr = _per_dispatch(_counter_rows(write_dir), "WRITE_SIZE")

    def pick(table, needle):
        vals = [v for (i, k), v in table.items() if needle in k]
        return vals

    # calibration: the plain copy of CALIB_BYTES (reads and writes that many)
    copy_f = [v for (i, k), v in fr.items() if _is_calib(k)]
    copy_w = [v for (i, k), v in wr.items() if _is_calib(k)]
    cf = max(copy_f) if copy_f else None
    cw = max(copy_w) if copy_w else None
    scale_f = CALIB_BYTES / (cf * 1024.0) if cf else 1.0
    scale_w = CALIB_BYTES / (cw * 1024.0) if cw else 1.0
    dom_f = pick(fr, DOMINANT)
    dom_w = pick(wr, DOMINANT)
    if not dom_f or not dom_w:
        raise SystemExit("dominant kernel not found in the counter runs")
    f_b = sum(dom_f) / len(dom_f) * 1024.0 * scale_f
    w_b = sum(dom_w) / len(dom_w) * 1024.0 * scale_w
    lines = [
        "# HBM traffic of the dominant kernel from rocprofv3 counters",
        f"command_fetch: {cmd.format(ctr='FETCH_SIZE')}",
        f"command_write: {cmd.format(ctr='WRITE_SIZE')}",
        f"kernel: {DOMINANT}",
        f"launches: {len(dom_f)}",
        f"fetch_kib_per_launch_raw: {sum(dom_f) / len(dom_f):.1f}",
        f"write_kib_per_launch_raw: {sum(dom_w) / len(dom_w):.1f}",
        f"copy_calibration_bytes: {CALIB_BYTES}",
        f"copy_fetch_kib_raw: {cf}",
        f"copy_write_kib_raw: {cw}",
        f"fetch_scale: {scale_f:.4f}",
        f"write_scale: {scale_w:.4f}",
        f"hbm_fetch_bytes_per_launch: {f_b:.0f}",
        f"hbm_write_bytes_per_launch: {w_b:.0f}",
        f"hbm_bytes_per_launch: {f_b + w_b:.0f}",
        f"kernel_source_sha1: {source_digest(DOMINANT_SRC)}",
    ]
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--workload", default=WORKLOAD,
                    choices=[WORKLOAD, BACKWARD, STACKED, READOUT, PROJECTION, EXPLAIN, "web-1.6B",
                             "powerlaw-1.2M", "uniform-10k", "hetero-20M"],
                    help="benchmark workload (the default is the metric's configuration)")
    ap.add_argument("--cpu-rows", type=int, default=0,
                    help="rows of the CPU-oracle aggregation sample (0: all rows)")
    ap.add_argument("--no-cpu-baseline", dest="cpu_baseline", action="store_false")
    ap.add_argument("--cold-reps", type=int, default=3,
                    help="cold-cache steps (each operation alone after a 1 GiB write)")
    ap.add_argument("--no-ceilings", dest="ceilings", action="store_false",
                    help="skip the bandwidth probes (read, copy, row gather)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run one plain 1 GiB copy after warm-up (counter scaling)")
    ap.add_argument("--summarize-stats", nargs=2, metavar=("DIR", "OUT"))
    ap.add_argument("--summarize-counters", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "OUT"))
    ap.add_argument("--summarize-sq", nargs=2, metavar=("DIR", "OUT"),
                    help="per-kernel shader counters of a `rocprofv3 --pmc` run of SQ_COUNTERS")
    ap.add_argument("--summarize-step-counters", nargs=4,
                    metavar=("FETCH_DIR", "WRITE_DIR", "OPS_JSON", "OUT"))
    ap.add_argument("--dump-ops", metavar="PATH",
                    help="write the step's operations (name, algorithmic bytes) as JSON")
    ap.add_argument("--cmd", default="", help="command line recorded in a summary ({ctr} is "
                    "replaced by the counter name in counter summaries)")
    args = ap.parse_args()
    if args.summarize_sq:
        summarize_sq(*args.summarize_sq, args.cmd)
        return
    if args.summarize_stats:
        summarize_stats(*args.summarize_stats, args.cmd)
        return
    if args.summarize_counters:
        summarize_counters(*args.summarize_counters, args.cmd)
        return
    if args.summarize_step_counters:
        summarize_step_counters(*args.summarize_step_counters, args.cmd)
        return
    run(args)


if __name__ == "__main__":
    main()
