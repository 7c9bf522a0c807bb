"""Where one planner iteration's time goes, phase by phase.

A copy of the library built with -DVP_PHASE_STAMPS (thread 0 of the
planner's workgroup stores the cycle counter at every phase boundary of
every iteration) plans one matrix of each given workload (the demand built
by vp_demand on the GPU); the mean cycles of each phase over the iterations
between the first and the last are printed:

    python -m paper_2609_34340_amd.phase_stamps --build      # on the CPU: libvp_stamps.so
    python -m paper_2609_34340_amd.phase_stamps 1 4 2 3 5    # on the GPU

The product library is not touched.
"""
from __future__ import annotations

import ctypes
import os
import sys

import numpy as np

PHASES = ["scoring (wave 0)", "scoring barrier", "argmax", "gather + draws", "AA (wave 0 runs)",
          "AA barrier", "evaluate", "update", "loop top"]
# (name, from column, to column) of the points stamped inside the phases
SUB = [("gather: thread 0's items", 3, 9), ("gather: start draws after them", 9, 10),
       ("gather: barrier", 10, 4), ("evaluate: best start read", 6, 11), ("evaluate: the rest", 11, 7),
       ("update: reads (lists, binding, credits)", 7, 12), ("update: schedule and layout stores", 12, 13),
       ("update: residual, aggregates, totals", 13, 14), ("update: barrier", 14, 8)]


HERE = os.path.dirname(os.path.abspath(__file__))
STAMPED = os.path.join(HERE, "libvp_stamps.so")


def build_stamped():
    from . import build as vpbuild
    return vpbuild.build(verbose=True, lib=STAMPED, build_dir=os.path.join(HERE, "_build_stamps"),
                         extra=["-DVP_PHASE_STAMPS"])


def main(configs):
    import torch

    import paper_2609_34340_amd as vp
    sys.path.insert(0, os.path.dirname(HERE))
    import vpgen

    if not os.path.exists(STAMPED):
        raise SystemExit("build the stamped copy first: python -m paper_2609_34340_amd.phase_stamps --build")
    vp.LIB_PATH = STAMPED
    lib = vp.lib()
    lib.vp_phase_stamps_read.argtypes = [ctypes.c_void_p]
    for c in configs:
        w = vpgen.config(c)
        cat = vp.Catalog(w.topo)
        cat.upload()
        N = w.n_ranks
        if w.mode == "moe":
            D = vp.demand(torch.from_numpy(vpgen.routing_all(w, 0)).cuda(), N, w.experts, w.row_bytes,
                          sort_row=-1)["demand"]
        else:
            hl = torch.from_numpy(vpgen.head_split(w.heads, N)).cuda()
            D = vp.demand_heads(w.tokens, hl, w.row_bytes, first_rank=0, R=N)
        p = vp.plan_params(N, w.row_bytes)
        out = vp.plan(cat, D, p, out=vp.alloc_schedule(N, p.k_max, "cuda", layout=True))
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        vp.plan(cat, D, p, out=out)
        e1.record()
        torch.cuda.synchronize()
        assert vp.read_status(out["status"]) == 0
        buf = (ctypes.c_ulonglong * (4096 * 16))()
        assert lib.vp_phase_stamps_read(buf) == 0
        T = np.frombuffer(buf, dtype=np.uint64).reshape(4096, 16).astype(np.int64)
        K = int(out["K"].item())
        A, nxt = T[1:K - 1, :9], T[2:K, 0]
        per_iter = float(np.mean(nxt - A[:, 0]))
        print("C%d %s: N=%d, plan %.1f us (stamped copy), K=%d, %.0f cycles per iteration" % (
            c, w.name, N, e0.elapsed_time(e1) * 1e3, K, per_iter), flush=True)
        cols = [A[:, i + 1] - A[:, i] for i in range(8)] + [nxt - A[:, 8]]
        for name, d in zip(PHASES, cols):
            print("   %-18s %7.0f cycles  %5.1f %%" % (name, np.mean(d), 100 * np.mean(d) / per_iter), flush=True)
        # points inside the phases (thread 0's view)
        B = T[1:K - 1]
        for name, a, b in SUB:
            print("      %-34s %7.0f cycles" % (name, float(np.mean(B[:, b] - B[:, a]))), flush=True)


if __name__ == "__main__":
    if sys.argv[1:] == ["--build"]:
        build_stamped()
    else:
        main([int(x) for x in sys.argv[1:]] or [1, 4, 2, 3, 5])
