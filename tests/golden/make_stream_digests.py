#!/usr/bin/env python3
"""Write stream_digests.json: the oracle's demand, schedule and rank-0 pack
digests for every checked matrix of the 64-rank and 256-rank demand streams.

Only the oracle and the seeded input generators are called.  Runs one worker
process per matrix batch (about 3 minutes on 8 cores).

    python tests/golden/make_stream_digests.py [--jobs 8]
    python tests/golden/make_stream_digests.py --all-256 [--jobs 8]   # every matrix of the 256-rank stream
    python tests/golden/make_stream_digests.py --sys-256              # matrix 0 of it on SYS nodes (about a minute)
    python tests/golden/make_stream_digests.py --ranks-1024           # 1,024 ranks (about 12 minutes)
"""
from __future__ import annotations

import argparse
import json
import multiprocessing as mp
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

import numpy as np  # noqa: E402

import stream_digest as sd  # noqa: E402

_tok = {}


def oracle_job(args):
    import oracle
    import vpgen
    cid, m = args
    w = vpgen.config(cid)
    if cid not in _tok:
        _tok[cid] = (vpgen.tokens_bf16(w, 0), oracle.Catalog(w.topo))
    tok, cat = _tok[cid]
    R = vpgen.routing_all(w, m)
    dem = [oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes) for i in range(w.n_ranks)]
    D = np.stack([d["row"] for d in dem])
    s = cat.plan(D, w.row_bytes)
    send, off = oracle.pack_rows(tok, w.row_bytes, dem[0]["sorted_tok"], dem[0]["dest_off"], 0, s)
    return dict(matrix=m, K=int(s["K"]), tau=int(s["tau"]), demand=sd.demand_digest(D),
                schedule=sd.schedule_digest(s), send_bytes=int(send.size),
                send=sd.send_digest(sd.send_sample(send), send.size), step_off=sd.step_off_digest(off))


def sys256():
    """The oracle's demand and schedule digests for the first matrix of the
    256-rank workload on nodes with cross-socket peer to peer."""
    import dataclasses
    import oracle
    import vpgen
    w = vpgen.config(5)
    topo = dataclasses.replace(w.topo, flags=1)
    R = vpgen.routing_all(w, 0)
    D = np.stack([oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes)["row"] for i in range(w.n_ranks)])
    t0 = time.time()
    s = oracle.Catalog(topo).plan(D, w.row_bytes)
    print("SYS 256 ranks: K=%d in %.0f s" % (s["K"], time.time() - t0), flush=True)
    out = dict(workload=w.name, topology="%s, SYS peer to peer" % (topo.as_tuple(),), matrix=0, K=int(s["K"]),
               tau=int(s["tau"]), demand=sd.demand_digest(D), schedule=sd.schedule_digest(s))
    with open(sd.GOLDEN_SYS256, "w") as f:
        json.dump(out, f, indent=0)
        f.write("\n")
    print("wrote", sd.GOLDEN_SYS256)


def ranks1024():
    """The oracle's schedule digest for the hot-destination demand on 1,024
    ranks (128 nodes), k_max = 32N."""
    import oracle
    import vpgen
    topo = vpgen.Topology(128)
    N, unit = topo.n_ranks, 4096
    D = vpgen.hot_destinations_demand(N, unit, 1024)
    t0 = time.time()
    s = oracle.Catalog(topo).plan(D, unit, k_max=32 * N)
    print("1024 ranks: K=%d in %.0f s" % (s["K"], time.time() - t0), flush=True)
    out = dict(topology="%s" % (topo.as_tuple(),), unit=unit, k_max=32 * N, K=int(s["K"]), tau=int(s["tau"]),
               demand=sd.demand_digest(D), schedule=sd.schedule_digest(s))
    with open(sd.GOLDEN_1024, "w") as f:
        json.dump(out, f, indent=0)
        f.write("\n")
    print("wrote", sd.GOLDEN_1024)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=8)
    ap.add_argument("--all-256", action="store_true",
                    help="digest all 1000 matrices of the 256-rank stream into %s" % os.path.basename(sd.GOLDEN_ALL5))
    ap.add_argument("--sys-256", action="store_true",
                    help="digest matrix 0 of the 256-rank workload on SYS nodes into %s" %
                         os.path.basename(sd.GOLDEN_SYS256))
    ap.add_argument("--ranks-1024", action="store_true",
                    help="digest the 1,024-rank plan into %s" % os.path.basename(sd.GOLDEN_1024))
    args = ap.parse_args()
    import oracle
    import vpgen
    oracle.build()
    if args.sys_256:
        sys256()
        return
    if args.ranks_1024:
        ranks1024()
        return
    out = {"sample_stride": sd.SAMPLE_STRIDE, "streams": {}}
    ctx = mp.get_context("spawn")
    streams = {5: list(range(1000))} if args.all_256 else sd.STREAMS
    target = sd.GOLDEN_ALL5 if args.all_256 else sd.GOLDEN
    for cid, mats in streams.items():
        t0 = time.time()
        with ctx.Pool(args.jobs) as pool:
            rows = pool.map(oracle_job, [(cid, m) for m in mats], chunksize=1)
        out["streams"][str(cid)] = {"workload": vpgen.config(cid).name, "matrices": rows}
        print("C%d: %d matrices in %.0f s" % (cid, len(rows), time.time() - t0), flush=True)
    with open(target, "w") as f:
        json.dump(out, f, indent=0)
        f.write("\n")
    print("wrote", target)


if __name__ == "__main__":
    main()
