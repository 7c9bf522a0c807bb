#!/usr/bin/env python3
"""Benchmark of the VarioPath demand -> plan -> pack hot path on one MI355X.

One step = one AlltoAllv invocation of the 256-rank DeepSeek-V3-like MoE
dispatch (4096 tokens/rank, hidden 7168 bf16, 256 experts top-8, 26 hot
experts holding half of the per-draw mass, hot set redrawn per matrix):

  vp_demand   all 256 ranks' routing -> the 256 x 256 byte-demand matrix
              (+ rank 0's (expert, token) order and offsets)
  vp_control_words  the sparse expert-parallel control word of every pair
  vp_plan     Alg. 2 on that matrix against the node-circulant catalog
  vp_pack     rank 0's token rows into channel-ordered send slices

all enqueued on one stream with no host synchronisation, inputs resident in
HBM.  Steps cycle over `--matrices` distinct demand matrices and two send
buffers.  Unless --no-batch, vp_plan_batch then plans D with D^T, and 16 to
256 matrices, in one launch each ("plan_batch": launch time and us per
matrix; the headline plan time stays the one-matrix latency).  Unless
--no-receive, the dispatch unpack and the combine pack / unpack of the first
matrix are timed ("receive").  Unless --no-sweep, the other four workloads (N = 8, 16, 64 and the
16-rank Ulysses case) follow with six timed steps each, under "per_config";
unless --no-extra, the planner then runs on the uniform, skew and head/context
demands with the full and the nearest-path catalog (the peer/path ablation),
under "extra_demands".
Prints one JSON line.  `value` is the pack's throughput in GB/s
(send bytes + distinct source bytes + index bytes, over the time of the
whole vp_pack call); the planner's microseconds per matrix, the step time
and the roofline of the dominant copy kernel ride along.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

METRIC = "pack HBM GB/s (% of peak) + vp_plan µs per N×N demand matrix, N=8..256"
PEAK_HBM_GBS = 8000.0
HERE = os.path.dirname(os.path.abspath(__file__))
TRAFFIC_FILE = os.path.join(HERE, "profiles", "pack_traffic.json")
KERNEL_NAME = {"moe": "scatter_rows_kernel (vp_pack_gather, token rows)",
               "heads": "pack_heads_kernel (vp_pack_heads: schedule checks and copy in one kernel)"}


def host_cpu():
    """Model name of the host CPU and the threads this process may run on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, len(os.sched_getaffinity(0))


def pack_source_sha() -> str:
    """Hash of pack.hip's code with comments and blank lines left out: the
    committed HBM-traffic profile applies while the code it measured is
    unchanged."""
    import re
    with open(os.path.join(HERE, "paper_2609_34340_amd", "csrc", "pack.hip")) as f:
        text = f.read()
    code = [ln.rstrip() for ln in re.sub(r"//[^\n]*", "", text).split("\n")]
    return hashlib.sha256("\n".join(ln for ln in code if ln.strip()).encode()).hexdigest()[:16]


def rank0_accounting(w, routing0: np.ndarray):
    """Bytes a pack of rank 0 must move: the send bytes, the distinct source
    rows, and the rows it indexes (for the GB/s accounting only)."""
    eloc = w.experts // w.n_ranks
    remote = (routing0 // eloc) != 0
    rows = int(remote.sum())
    distinct = int(remote.any(axis=1).sum())
    return rows * w.row_bytes, distinct * w.row_bytes, rows


def cpu_baseline(w, routing_np, tokens_np):
    """The oracle, single-threaded, on one matrix: demand of every rank, the
    plan, and rank 0's pack."""
    import oracle
    cat = oracle.Catalog(w.topo)
    t0 = time.perf_counter()
    dem = [oracle.demand(routing_np[i], w.n_ranks, w.experts, i, w.row_bytes) for i in range(w.n_ranks)]
    t1 = time.perf_counter()
    D = np.stack([d["row"] for d in dem])
    s = cat.plan(D, w.row_bytes)
    t2 = time.perf_counter()
    send, _ = oracle.pack_rows(tokens_np, w.row_bytes, dem[0]["sorted_tok"], dem[0]["dest_off"], 0, s)
    t3 = time.perf_counter()
    S, U, rows = rank0_accounting(w, routing_np[0])
    slices = int((s["bytes"][:, 0] > 0).sum())
    pack_bytes = S + U + 4 * rows + 16 * slices
    model, threads = host_cpu()
    return dict(value=round(pack_bytes / (t3 - t2) / 1e9, 3), unit="GB/s", cores=1, kind="oracle",
                cpu_model=model, host_threads_visible=threads,
                sample="one %d x %d matrix of the workload: demand of all %d ranks, one plan (K=%d), "
                       "rank-0 pack of %.1f MB" % (w.n_ranks, w.n_ranks, w.n_ranks, s["K"], send.size / 1e6),
                demand_s=round(t1 - t0, 3), plan_us_per_matrix=round((t2 - t1) * 1e6, 1),
                pack_s=round(t3 - t2, 4))


def cpu_baseline_heads(w, act_np):
    """The oracle, single-threaded, on the Ulysses workload: every rank's
    head-demand row, one plan, and rank 0's head pack."""
    import oracle
    import vpgen
    cat = oracle.Catalog(w.topo)
    hl = vpgen.head_split(w.heads, w.n_ranks)
    t0 = time.perf_counter()
    D = np.stack([oracle.demand_heads(w.tokens, hl, w.row_bytes, i) for i in range(w.n_ranks)])
    t1 = time.perf_counter()
    s = cat.plan(D, w.row_bytes)
    t2 = time.perf_counter()
    send, _ = oracle.pack_heads(act_np, w.token_stride, hl, w.row_bytes, 0, s)
    t3 = time.perf_counter()
    slices = int((s["bytes"][:, 0] > 0).sum())
    pack_bytes = 2 * send.size + 16 * slices
    model, threads = host_cpu()
    return dict(value=round(pack_bytes / (t3 - t2) / 1e9, 3), unit="GB/s", cores=1, kind="oracle",
                cpu_model=model, host_threads_visible=threads,
                sample="the %d x %d head-demand matrix: demand of all %d ranks, one plan (K=%d), rank-0 head "
                       "pack of %.1f MB" % (w.n_ranks, w.n_ranks, w.n_ranks, s["K"], send.size / 1e6),
                demand_s=round(t1 - t0, 4), plan_us_per_matrix=round((t2 - t1) * 1e6, 1),
                pack_s=round(t3 - t2, 4))


def measure(w, steps, warmup, M, dev, graph=False):
    """Time `steps` demand -> plan -> pack steps of workload `w` on one stream
    (after `warmup` untimed ones), cycling over M matrices and two send
    buffers.  Returns the per-stage event times and the per-matrix facts."""
    import torch
    import vpgen
    import paper_2609_34340_amd as vp

    if w.mode == "moe":
        routing_np = [vpgen.routing_all(w, m) for m in range(M)]
        routing = [torch.from_numpy(r).to(dev) for r in routing_np]
        tokens_np = vpgen.tokens_bf16(w, 0)
        acct = [rank0_accounting(w, r[0]) for r in routing_np]
        pipe = vp.Pipeline(w.topo, "moe", w.row_bytes, n_experts=w.experts, tokens=w.tokens, top_k=w.top_k)
        head_lo = None
    else:
        hl = vpgen.head_split(w.heads, w.n_ranks)
        head_lo = torch.from_numpy(hl).to(dev)
        tokens_np = vpgen.tokens_bf16(w, 0)
        S = int(w.tokens * (hl[-1] - (hl[1] - hl[0])) * w.row_bytes)
        acct = [(S, S, S // w.row_bytes)]
        routing_np, routing = None, [None]
        M = 1
        pipe = vp.Pipeline(w.topo, "heads", w.row_bytes, tokens=w.tokens, token_stride=w.token_stride)
    tokens = torch.from_numpy(tokens_np).to(dev)
    sends = [pipe.send, torch.empty_like(pipe.send)]
    E = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731

    def run(step, ev=None):
        m = step % M
        if ev is not None:
            ev[0].record()
        pipe.demand_stage(routing[m], head_lo)
        if ev is not None:
            ev[1].record()
        pipe.words_stage()
        if ev is not None:
            ev[2].record()
        pipe.plan_stage()
        if ev is not None:
            ev[3].record()
        # rows: the pack's two halves, so that the copy kernel has events of
        # its own; heads: the one-kernel pack (no separate prepare)
        if w.mode == "moe":
            pipe.pack_prepare_stage(tokens, head_lo)
        if ev is not None:
            ev[4].record()
        if w.mode == "moe":
            pipe.pack_gather_stage(tokens, sends[step % 2])
        else:
            pipe.pack_stage(tokens, head_lo, sends[step % 2])
        if ev is not None:
            ev[5].record()

    for s in range(warmup):
        run(s)
    torch.cuda.synchronize()
    if vp.read_status(pipe.status) != 0:
        raise SystemExit("device error during warmup: %d" % vp.read_status(pipe.status))

    evs = [[E() for _ in range(6)] for _ in range(steps)]
    start, end = E(), E()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record()
    for s in range(steps):
        run(s, evs[s])
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if vp.read_status(pipe.status) != 0:
        raise SystemExit("device error in the timed region: %d" % vp.read_status(pipe.status))
    r = dict(total_ms=start.elapsed_time(end), wall=wall,
             demand_ms=np.array([e[0].elapsed_time(e[1]) for e in evs]),
             words_ms=np.array([e[1].elapsed_time(e[2]) for e in evs]),
             plan_ms=np.array([e[2].elapsed_time(e[3]) for e in evs]),
             prep_ms=np.array([e[3].elapsed_time(e[4]) for e in evs]),
             copy_ms=np.array([e[4].elapsed_time(e[5]) for e in evs]))
    r["pack_ms"] = r["prep_ms"] + r["copy_ms"]

    # the copy kernel on its own: 50 launches captured in a HIP graph and
    # replayed between two events, so that neither the host's launch cost nor
    # the per-step events are in the figure (the last matrix's schedule).
    # Rows: the two halves of the pack, the scatter after one prepare (a copy
    # may be repeated after a prepare); heads: the one-kernel pack.  No stage
    # records a memset.  The send buffer after the replays must equal the
    # eager result.
    def graph_ms(fn, reps=50):
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        with torch.cuda.graph(g):
            for _ in range(reps):
                fn()
        g.replay()
        a, b = E(), E()
        a.record()
        g.replay()
        b.record()
        torch.cuda.synchronize()
        del g
        return a.elapsed_time(b) / reps

    if graph:
        sends[0].zero_()
        pipe.pack_stage(tokens, head_lo, sends[0])
        torch.cuda.synchronize()
        eager = sends[0].clone()
        sends[0].zero_()
        if w.mode == "moe":
            r["prep_graph_ms"] = graph_ms(lambda: pipe.pack_prepare_stage(tokens, head_lo))
            r["copy_graph_ms"] = graph_ms(lambda: pipe.pack_gather_stage(tokens, sends[0]))
        else:
            r["copy_graph_ms"] = graph_ms(lambda: pipe.pack_stage(tokens, head_lo, sends[0]))
        torch.cuda.synchronize()
        if vp.read_status(pipe.status) != 0 or not torch.equal(sends[0], eager):
            raise SystemExit("the graph-replayed pack differs from the eager one")
        del eager

        # the whole step (demand, control words, plan, one-call pack) of the
        # first matrix captured once and replayed `steps` times between two
        # events: the step time without the host's launch gaps; the send
        # buffer after the replays must equal the eager step's
        def whole():
            pipe.demand_stage(routing[0], head_lo)
            pipe.words_stage()
            pipe.plan_stage()
            pipe.pack_stage(tokens, head_lo, sends[0])

        sends[0].zero_()
        whole()
        torch.cuda.synchronize()
        eager = sends[0].clone()
        sends[0].zero_()
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            whole()
        torch.cuda.current_stream().wait_stream(side)
        with torch.cuda.graph(g):
            whole()
        g.replay()
        a, b = E(), E()
        a.record()
        for _ in range(steps):
            g.replay()
        b.record()
        torch.cuda.synchronize()
        r["step_graph_ms"] = a.elapsed_time(b) / steps
        if vp.read_status(pipe.status) != 0 or not torch.equal(sends[0], eager):
            raise SystemExit("the graph-replayed step differs from the eager one")
        del g, eager

    # one rank's own row (R = 1: its routing, counts, demand row and sort),
    # the unit each rank runs in deployment; mean of 20 calls, HIP events
    if w.mode == "moe":
        r1 = routing[0][:1].contiguous()
        ws1 = torch.zeros(max(vp.demand_workspace_bytes(1, w.tokens, w.top_k, w.experts), 1), dtype=torch.uint8,
                          device=dev)
        o1 = vp.demand(r1, w.n_ranks, w.experts, w.row_bytes, sort_row=0, ws=ws1)
        a, b = E(), E()
        a.record()
        for _ in range(20):
            vp.demand(r1, w.n_ranks, w.experts, w.row_bytes, sort_row=0, ws=ws1, out=o1, status=o1["status"])
        b.record()
        torch.cuda.synchronize()
        if vp.read_status(o1["status"]) != 0:
            raise SystemExit("device error in the one-rank demand")
        r["demand_r1_ms"] = a.elapsed_time(b) / 20
        del r1, ws1, o1

    # schedule facts per matrix (untimed): K, slices, modeled completion time
    Ks, slices, That = [], [], []
    for m in range(M):
        pipe.demand_stage(routing[m], head_lo)
        pipe.plan_stage()
        torch.cuda.synchronize()
        h = vp.schedule_to_host(pipe.sched)
        Ks.append(h["K"])
        slices.append(int((h["bytes"][:, pipe.self_rank] > 0).sum()))
        num, den = pipe.cat.modeled_time(h["K"], h["inst"], h["bytes"], pipe.params.lambda_ns)
        That.append(num / den / 1e6)
    step_m = [s % M for s in range(steps)]
    S_b = np.array([acct[m][0] for m in step_m], dtype=np.float64)
    U_b = np.array([acct[m][1] for m in step_m], dtype=np.float64)
    rows = np.array([acct[m][2] for m in step_m], dtype=np.float64)
    sl = np.array([slices[m] for m in step_m], dtype=np.float64)
    r["pack_bytes"] = S_b + U_b + 4 * rows + 16 * sl
    r["gather_bytes"] = S_b + U_b
    r["send_bytes"] = S_b
    r["K"] = np.array([Ks[m] for m in step_m], dtype=np.float64)
    r["That_ms"] = np.array([That[m] for m in step_m])
    r["M"] = M
    r["routing_np"], r["tokens_np"] = routing_np, tokens_np
    del pipe, sends, tokens
    torch.cuda.empty_cache()
    return r


def receive_section(w, routing_np, dev, reps=10):
    """Receive side and combine of the first matrix, timed with HIP events
    (mean of `reps` calls): the dispatch unpack at the busiest receiving rank
    r (its received rows into the expert-major output), the combine pack at r
    (those rows back, in the order of the schedule planned on D^T) and the
    combine unpack at rank 0 (its returned rows into (token, slot) order).
    Buffers hold arbitrary bytes: only sizes and the schedules matter to the
    copies.  GB/s counts every row read once and written once."""
    import torch
    import paper_2609_34340_amd as vp
    N, rb = w.n_ranks, w.row_bytes
    sb = vp.slot_bytes(rb)
    cat = vp.Catalog(w.topo)
    cat.upload()
    p = vp.plan_params(N, rb)
    st = vp.new_status(dev)
    dem = vp.demand(torch.from_numpy(routing_np).to(dev), N, w.experts, rb, sort_row=0, status=st)
    D = dem["demand"]
    disp = vp.plan(cat, D, p, status=st, out=vp.alloc_schedule(N, p.k_max, dev, layout=True))
    comb = vp.plan(cat, vp.demand_transpose(D), p, status=st, out=vp.alloc_schedule(N, p.k_max, dev, layout=True))
    torch.cuda.synchronize()
    Dh = D.cpu().numpy()
    r = int(Dh.sum(axis=0).argmax())
    rows_r = int(Dh[:, r].sum()) // rb
    counts = dem["counts"]
    eloc = w.experts // N
    out_rows = int(counts[:, r * eloc:(r + 1) * eloc].sum().item())
    recv = torch.empty(rows_r * sb, dtype=torch.uint8, device=dev)
    outb = torch.empty(max(out_rows, 1) * sb, dtype=torch.uint8, device=dev)
    send = torch.empty(rows_r * rb, dtype=torch.uint8, device=dev)
    step_off = torch.empty(p.k_max + 1, dtype=torch.int64, device=dev)
    rows_0 = int(Dh[0].sum()) // rb
    recv0 = torch.empty(rows_0 * sb, dtype=torch.uint8, device=dev)
    combined = torch.empty(w.tokens * w.top_k * sb, dtype=torch.uint8, device=dev)
    ws = torch.empty(vp.unpack_workspace_bytes(max(rows_r, rows_0, out_rows)), dtype=torch.uint8, device=dev)

    def timed(fn):
        fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / reps

    res = {"receiver": r, "rows": rows_r, "row_bytes": rb}
    us = timed(lambda: vp.unpack_rows(recv, rb, counts, r, disp, outb, st, ws=ws))
    res["unpack_rows"] = {"us": round(us, 2), "GBps": round(2 * rows_r * rb / us / 1e3, 1)}
    us = timed(lambda: vp.pack_combine(outb, rb, counts, r, comb, send, step_off, st, ws=ws))
    res["pack_combine"] = {"us": round(us, 2), "GBps": round(2 * rows_r * rb / us / 1e3, 1)}
    us = timed(lambda: vp.unpack_combine(recv0, rb, w.tokens, w.top_k, dem["sorted_tok"], dem["sorted_slot"],
                                         dem["dest_off"], 0, comb, combined, st, ws=ws))
    res["unpack_combine"] = {"us": round(us, 2), "GBps": round(2 * rows_0 * rb / us / 1e3, 1), "rank": 0,
                             "rows": rows_0}
    if vp.read_status(st) != 0:
        raise SystemExit("device error on the receive side: %d" % vp.read_status(st))
    del recv, outb, send, recv0, combined, ws
    torch.cuda.empty_cache()
    return res


def batch_section(w, routing_list, dev, sizes=(2, 16, 64, 256)):
    """vp_plan_batch: B matrices planned side by side (one workgroup each).
    B = 2 is a layer's dispatch matrix D and its combine matrix D^T; larger
    batches cycle over the workload's distinct matrices.  Reports the launch
    time and microseconds per matrix (HIP events, mean of 3 launches after
    one warm launch)."""
    import torch
    import paper_2609_34340_amd as vp
    cat = vp.Catalog(w.topo)
    cat.upload()
    p = vp.plan_params(w.n_ranks, w.row_bytes)
    mats = []
    for R in routing_list:
        d = vp.demand(torch.from_numpy(R).to(dev), w.n_ranks, w.experts, w.row_bytes, sort_row=-1)
        mats.append(d["demand"])
    out = {"distinct_matrices": len(mats)}
    for B in sizes:
        if B == 2:
            D = torch.stack([mats[0], mats[0].t().contiguous()])
        else:
            D = torch.stack([mats[b % len(mats)] for b in range(B)])
        sched = vp.alloc_schedule_batch(B, w.n_ranks, p.k_max, dev)
        st = torch.zeros(B, dtype=torch.int32, device=dev)
        ws = torch.empty(vp.plan_batch_workspace_bytes(cat, p, B), dtype=torch.uint8, device=dev)
        vp.plan_batch(cat, D, p, status=st, out=sched, ws=ws)
        a, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(3):
            vp.plan_batch(cat, D, p, status=st, out=sched, ws=ws)
        b_.record()
        torch.cuda.synchronize()
        if (st != 0).any():
            raise SystemExit("device error in the batched plan: %s" % st.cpu().numpy())
        ms = a.elapsed_time(b_) / 3
        key = "dispatch_and_combine" if B == 2 else "B%d" % B
        out[key] = {"batch": B, "launch_ms": round(ms, 3), "us_per_matrix": round(ms * 1e3 / B, 1)}
        del D, sched, ws
    torch.cuda.empty_cache()
    return out


def extra_demand(vp, case, matrix, dev):
    """int64 [N, N] demand of an extra case on the GPU: given matrices are
    uploaded; a head/context layout runs vp_demand_heads per all-to-all group
    and places each group's block on the diagonal."""
    import torch
    import vpgen
    if case.kind == "uniform":
        return torch.from_numpy(vpgen.uniform_demand(case)).to(dev)
    if case.kind == "zipf_pairs":
        return torch.from_numpy(vpgen.zipf_pair_demand(case, matrix)).to(dev)
    N = case.topo.n_ranks
    T, hl = vpgen.hc_layout(case)
    hl_d = torch.from_numpy(hl).to(dev)
    D = torch.zeros((N, N), dtype=torch.int64, device=dev)
    for grp in vpgen.hc_groups(case):
        lo, hi = int(grp[0]), int(grp[-1]) + 1
        D[lo:hi, lo:hi] = vp.demand_heads(T, hl_d, case.unit, first_rank=0, R=case.H)
    return D


def extra_section(dev, reps=3):
    """Planner on the uniform, skew (pairwise Zipf) and head/context demands,
    with the full catalog and with the nearest-path catalog of the peer/path
    ablation (Sec. 6.3, Table 3: demand-aware peers, fixed nearest path).
    Per case: plan us per matrix (HIP events, mean of `reps` runs per
    matrix), K and the modeled completion time T of Eq. (2); the ablation
    ratios put T of the nearest-path plan and of the fixed cyclic rotation
    (vp_rotation_time, nearest or per-stage best paths, shared links split
    equally) over T of the full plan, averaged over the case's matrices."""
    import torch
    import vpgen
    import paper_2609_34340_amd as vp
    cats, out = {}, {}
    for name, case in vpgen.EXTRA.items():
        n_mat = 5 if case.kind == "zipf_pairs" else 1
        res = {"N": case.topo.n_ranks}
        Ts = {}
        for variant in ("full", "nearest"):
            key = (case.topo, variant)
            if key not in cats:
                c = vp.Catalog(case.topo)
                if variant == "nearest":
                    c = c.restrict(vp.RESTRICT_NEAREST_PATH)
                c.upload()
                cats[key] = c
            cat = cats[key]
            p = vp.plan_params(cat.N, case.unit)
            sched = vp.alloc_schedule(cat.N, p.k_max, dev)
            st = vp.new_status(dev)
            ws = torch.empty(vp.plan_workspace_bytes(cat, p), dtype=torch.uint8, device=dev)
            Ks, That, us = [], [], []
            for m in range(n_mat):
                D = extra_demand(vp, case, m, dev)
                if variant == "full":
                    Dh = D.cpu().numpy()
                    for rule, key in [(vp.ROTATION_NEAREST_PATH, "rot_nearest"), (vp.ROTATION_DYNAMIC_PATH, "rot_dynamic")]:
                        num, den = cat.rotation_time(Dh, rule)
                        Ts.setdefault(key, []).append(num / den / 1e6)
                vp.plan(cat, D, p, status=st, out=sched, ws=ws)   # warm
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                for _ in range(reps):
                    vp.plan(cat, D, p, status=st, out=sched, ws=ws)
                b.record()
                torch.cuda.synchronize()
                if vp.read_status(st) != 0:
                    raise SystemExit("device error planning %s (%s): %d" % (name, variant, vp.read_status(st)))
                us.append(a.elapsed_time(b) * 1e3 / reps)
                h = vp.schedule_to_host(sched)
                num, den = cat.modeled_time(h["K"], h["inst"], h["bytes"], p.lambda_ns)
                Ks.append(h["K"])
                That.append(num / den / 1e6)
            Ts[variant] = That
            res[variant] = {"plan_us_per_matrix": round(float(np.mean(us)), 1), "activations_K": round(float(np.mean(Ks)), 1),
                            "modeled_T_ms": round(float(np.mean(That)), 4), "families": cat.n_families}
        full = np.array(Ts["full"])
        res["nearest_over_full_T"] = round(float(np.mean(np.array(Ts["nearest"]) / full)), 4)
        # Table 3 layout: completion time over the demand-aware, dynamic-path plan's
        res["ablation"] = {"fixed_peers_nearest_path": round(float(np.mean(np.array(Ts["rot_nearest"]) / full)), 4),
                           "fixed_peers_dynamic_path": round(float(np.mean(np.array(Ts["rot_dynamic"]) / full)), 4),
                           "demand_aware_nearest_path": res["nearest_over_full_T"],
                           "demand_aware_dynamic_path": 1.0}
        res["matrices"] = n_mat
        out[name] = res
    return out


def summary(w, r):
    value = float(r["pack_bytes"].sum() / (r["pack_ms"].sum() * 1e-3) / 1e9)
    plan_us = float(r["plan_ms"].mean() * 1e3)
    return {"N": w.n_ranks, "plan_us_per_matrix": round(plan_us, 1),
            "plan_us_per_activation": round(plan_us / float(r["K"].mean()), 3),
            "activations_K": int(round(r["K"].mean())),
            "modeled_T_ms": round(float(r["That_ms"].mean()), 3),
            "plan_over_modeled_T": round(plan_us / (1e3 * float(r["That_ms"].mean())), 5),
            "demand_us": round(float(r["demand_ms"].mean() * 1e3), 1),
            "demand_one_rank_us": round(float(r["demand_r1_ms"] * 1e3), 1) if "demand_r1_ms" in r else None,
            "control_words_us": round(float(r["words_ms"].mean() * 1e3), 1) if w.mode == "moe" else None,
            "pack_us": round(float(r["pack_ms"].mean() * 1e3), 1),
            "pack_GBps": round(value, 2), "pack_pct_of_peak": round(100 * value / PEAK_HBM_GBS, 2),
            "pack_bytes_MB": round(float(r["pack_bytes"].mean()) / 1e6, 2),
            # median over the timed steps, and the logical rate 2S/t (every send
            # byte read and written once; cache-served duplicate rows can make
            # it exceed what HBM carried)
            "pack_us_median": round(float(np.median(r["pack_ms"]) * 1e3), 1),
            "pack_logical_2S_GBps": round(float(2 * r["send_bytes"].sum() / (r["pack_ms"].sum() * 1e-3) / 1e9), 2),
            # the copy kernel alone, 50 launches from a replayed HIP graph:
            # algorithmic bytes over its time (rows: the scatter half, after
            # a prepare of prepare_us_graph; heads: the one-kernel pack)
            "copy_kernel": KERNEL_NAME[w.mode],
            "copy_us_graph": round(float(r["copy_graph_ms"] * 1e3), 2) if "copy_graph_ms" in r else None,
            "copy_frac_graph": round(float(r["gather_bytes"][-1] / (r["copy_graph_ms"] * 1e-3) / 1e9)
                                           / PEAK_HBM_GBS, 4) if "copy_graph_ms" in r else None,
            "prepare_us_graph": round(float(r["prep_graph_ms"] * 1e3), 2) if "prep_graph_ms" in r else None,
            # the whole step replayed from one HIP graph (--graph)
            "ms_per_step_graph": round(float(r["step_graph_ms"]), 4) if "step_graph_ms" in r else None,
            # the same kernel inside the timed steps (events around it: for
            # short kernels the events' own cost is a visible share)
            "copy_us_in_steps": round(float(r["copy_ms"].mean() * 1e3), 2),
            "copy_frac_in_steps": round(float(r["gather_bytes"].sum() / (r["copy_ms"].sum() * 1e-3) / 1e9)
                                        / PEAK_HBM_GBS, 4)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=5, help="workload configuration 1..5")
    ap.add_argument("--matrices", type=int, default=4, help="distinct demand matrices cycled")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the short runs of the other configurations (plan time at every N)")
    ap.add_argument("--no-batch", action="store_true", help="skip the batched-planner timings")
    ap.add_argument("--no-receive", action="store_true", help="skip the receive-side and combine timings")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the planner on the extra demands and the nearest-path ablation")
    ap.add_argument("--graph", action="store_true",
                    help="also time the copy kernel by 50 launches replayed from a HIP graph (reported beside "
                         "the timed steps' figure) and the whole step replayed from one graph "
                         "(ms_per_step_graph); leave it off for profiler runs of the default command")
    ap.add_argument("--calibrate-copy", type=int, default=0,
                    help="after the timed region, run one plain device copy of this many MiB")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the hot path is the per-rank demand -> plan -> "
              "pack work, which runs on a single MI355X; run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    import vpgen

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = vpgen.config(args.config)
    dev = torch.device("cuda:0")
    M = max(1, min(args.matrices, args.steps))
    print("[bench] %s: %d matrices, %d warmup + %d timed steps" % (w.name, M, args.warmup, args.steps),
          file=sys.stderr, flush=True)
    r = measure(w, args.steps, args.warmup, M, dev, graph=args.graph)
    head = summary(w, r)
    # the copy kernel's algorithmic bytes over its time between HIP events
    # around it in the timed steps (with --graph, its graph-replayed time is
    # reported beside it)
    achieved = float(r["gather_bytes"].sum() / (r["copy_ms"].sum() * 1e-3) / 1e9)

    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        if t.get("kernel_source_sha") == pack_source_sha() and w.name in t.get("workloads", {}):
            traffic = t["workloads"][w.name].get("bytes_per_launch")

    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        a = torch.empty(n, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()

    out = {
        "metric": METRIC,
        "value": head["pack_GBps"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["total_ms"] / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": "C%d %s: N=%d ranks (%d nodes x 2 sockets x 2 PCIe switches x 2 GPUs), "
                               "%s, tokens/rank=%d, unit=%d B" % (
                                   w.cid, w.name, w.n_ranks, w.topo.n_nodes,
                                   ("%d experts top-%d" % (w.experts, w.top_k)) if w.mode == "moe"
                                   else "Ulysses %d heads x %d" % (w.heads, w.head_dim),
                                   w.tokens, w.row_bytes),
                   "matrices": r["M"], "self_rank": 0},
        "pct_of_peak": head["pack_pct_of_peak"],
        "plan_us_per_matrix": head["plan_us_per_matrix"],
        "plan_us_per_activation": head["plan_us_per_activation"],
        "demand_us": head["demand_us"],
        "demand_one_rank_us": head["demand_one_rank_us"],
        "control_words_us": head["control_words_us"],
        "pack_us": head["pack_us"],
        "pack_us_median": head["pack_us_median"],
        "pack_logical_2S_GBps": head["pack_logical_2S_GBps"],
        "activations_K": head["activations_K"],
        "modeled_T_ms": head["modeled_T_ms"],
        "plan_over_modeled_T": head["plan_over_modeled_T"],
        "wall_s": round(r["wall"], 3),
        "roofline": {"bound": "hbm", "kernel": KERNEL_NAME[w.mode],
                     "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": int(r["gather_bytes"].mean()),
                     "avg_launch_us": head["copy_us_in_steps"],
                     "timing": "HIP events around the kernel in the timed steps, on its stream",
                     "avg_launch_us_graph": head["copy_us_graph"],
                     "frac_graph": head["copy_frac_graph"]},
        "prepare_us_graph": head["prepare_us_graph"],
        "ms_per_step_graph": head["ms_per_step_graph"],
    }
    if w.mode == "moe" and not args.no_receive:
        print("[bench] receive side and combine", file=sys.stderr, flush=True)
        out["receive"] = receive_section(w, r["routing_np"][0], dev)
    if w.mode == "moe" and not args.no_batch:
        print("[bench] batched planning", file=sys.stderr, flush=True)
        out["plan_batch"] = batch_section(w, r["routing_np"], dev)
    if not args.no_sweep:
        # the other configurations, briefly: the planner at every N and each pack
        per = {}
        for cid in range(1, 6):
            if cid == args.config:
                continue
            wc = vpgen.config(cid)
            print("[bench] sweep C%d %s" % (cid, wc.name), file=sys.stderr, flush=True)
            per["C%d" % cid] = summary(wc, measure(wc, 6, 2, 2, dev, graph=args.graph))
        out["per_config"] = per
    if not args.no_extra:
        print("[bench] extra demands and nearest-path ablation", file=sys.stderr, flush=True)
        out["extra_demands"] = extra_section(dev)
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on one matrix", file=sys.stderr, flush=True)
        if w.mode == "moe":
            out["cpu_baseline"] = cpu_baseline(w, r["routing_np"][0], r["tokens_np"])
        else:
            out["cpu_baseline"] = cpu_baseline_heads(w, r["tokens_np"])
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
