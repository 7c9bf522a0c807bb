"""vp_plan_batch: several matrices planned side by side, one workgroup
each, must give every matrix the schedule the oracle gives it (through the
stored stream digests, element by element for a dispatch matrix D and its
combine matrix D^T, and for batches of random matrices with their buffer
layout); a bad matrix fails alone."""
import json
import sys

import numpy as np
import pytest
import torch

import oracle
import stream_digest as sd
import vpgen

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def vp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_34340_amd as vp
    vp.lib()
    return vp


def host(s, b):
    K = int(s["K"][b].item())
    return dict(K=K, family=s["family"][b, :K].cpu().numpy(), dst=s["dst"][b, :K].cpu().numpy(),
                inst=s["inst"][b, :K].cpu().numpy(), bytes=s["bytes"][b, :K].cpu().numpy(),
                tau=int(s["tau"][b].item()))


def test_batch_of_the_64_rank_stream(vp):
    """Eight matrices of the 64-rank stream in one launch: each hashes to the
    oracle's digest of that matrix."""
    w = vpgen.config(3)
    with open(sd.GOLDEN) as f:
        ref = {r["matrix"]: r for r in json.load(f)["streams"]["3"]["matrices"]}
    mats = [0, 1, 2, 3, 17, 42, 77, 99]
    log("batch of %d C3 matrices" % len(mats))
    cat = vp.Catalog(w.topo)
    cat.upload()
    Ds = []
    for m in mats:
        R = vpgen.routing_all(w, m)
        d = vp.demand(torch.from_numpy(R).cuda(), w.n_ranks, w.experts, w.row_bytes, sort_row=-1)
        Ds.append(d["demand"])
    D = torch.stack(Ds)
    p = vp.plan_params(w.n_ranks, w.row_bytes)
    s = vp.plan_batch(cat, D, p)
    torch.cuda.synchronize()
    assert (s["status"] == 0).all()
    for b, m in enumerate(mats):
        assert sd.demand_digest(D[b].cpu().numpy()) == ref[m]["demand"]
        h = host(s, b)
        assert h["K"] == ref[m]["K"] and h["tau"] == ref[m]["tau"]
        assert sd.schedule_digest(h) == ref[m]["schedule"], "matrix %d" % m


@pytest.mark.parametrize("cid", [2, 5])
def test_dispatch_and_combine_in_one_launch(vp, cid):
    """D and D^T planned together, with the buffer layout, equal the oracle's
    plans and the single-matrix call's layout."""
    w = vpgen.config(cid)
    log("batch D and D^T C%d" % cid)
    R = vpgen.routing_all(w, 0)
    Dn = np.stack([oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes)["row"] for i in range(w.n_ranks)])
    D = torch.from_numpy(np.stack([Dn, np.ascontiguousarray(Dn.T)])).cuda()
    cat = vp.Catalog(w.topo)
    cat.upload()
    p = vp.plan_params(w.n_ranks, w.row_bytes)
    s = vp.plan_batch(cat, D, p, out=vp.alloc_schedule_batch(2, w.n_ranks, p.k_max, layout=True))
    one = vp.plan(cat, D[1].contiguous(), p, out=vp.alloc_schedule(w.n_ranks, p.k_max, layout=True))
    torch.cuda.synchronize()
    assert (s["status"] == 0).all() and int(one["status"].item()) == 0
    ocat = oracle.Catalog(w.topo)
    for b, M in enumerate((Dn, Dn.T)):
        o = ocat.plan(np.ascontiguousarray(M), w.row_bytes)
        h = host(s, b)
        assert h["K"] == o["K"] and h["tau"] == o["tau"]
        for key in ("family", "dst", "inst", "bytes"):
            assert np.array_equal(h[key], o[key]), key
    K = int(one["K"].item())
    for key in ("dst", "bytes", "send_off", "stream_off", "recv_src"):
        assert torch.equal(s[key][1, :K], one[key][:K]), key
    zero = vp.plan(cat, D[0].contiguous(), p, out=vp.alloc_schedule(w.n_ranks, p.k_max, layout=True))
    torch.cuda.synchronize()
    K0 = int(zero["K"].item())
    for key in ("dst", "bytes", "send_off", "stream_off", "recv_src"):
        assert torch.equal(s[key][0, :K0], zero[key][:K0]), key


def test_bad_matrix_fails_alone(vp):
    w = vpgen.config(1)
    R = vpgen.routing_all(w, 0)
    Dn = np.stack([oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes)["row"] for i in range(w.n_ranks)])
    bad = Dn.copy()
    bad[2, 5] = -w.row_bytes
    D = torch.from_numpy(np.stack([Dn, bad, Dn])).cuda()
    cat = vp.Catalog(w.topo)
    cat.upload()
    p = vp.plan_params(w.n_ranks, w.row_bytes)
    s = vp.plan_batch(cat, D, p)
    torch.cuda.synchronize()
    st = s["status"].cpu().numpy()
    assert st[0] == 0 and st[2] == 0 and st[1] == vp.INVALID_DEMAND
    o = oracle.Catalog(w.topo).plan(Dn, w.row_bytes)
    for b in (0, 2):
        h = host(s, b)
        assert h["K"] == o["K"] and np.array_equal(h["dst"], o["dst"]) and np.array_equal(h["bytes"], o["bytes"])


def test_pipelines_on_concurrent_streams(vp):
    """The library keeps no state between calls on a device (every call's
    state is in its own arguments and workspaces): two whole steps of
    different workloads (the 8-rank and 64-rank MoE dispatches), each on its
    own stream and enqueued interleaved so that their kernels can overlap,
    give each workload the demand, schedule and send buffer it gets alone."""
    cases = []
    for cid in (1, 3):
        w = vpgen.config(cid)
        pipe = vp.Pipeline(w.topo, "moe", w.row_bytes, n_experts=w.experts, tokens=w.tokens, top_k=w.top_k)
        R = torch.from_numpy(vpgen.routing_all(w, 0)).cuda()
        tok = torch.from_numpy(vpgen.tokens_bf16(w, 0)).cuda()
        cases.append((cid, pipe, R, tok))
    alone = []
    for cid, pipe, R, tok in cases:
        log("step alone C%d" % cid)
        send = pipe.step(routing=R, tokens=tok)
        torch.cuda.synchronize()
        assert vp.read_status(pipe.status) == 0
        K = int(pipe.sched["K"].item())
        alone.append(dict(K=K, demand=pipe.dem["demand"].clone(), dst=pipe.sched["dst"][:K].clone(),
                          bytes=pipe.sched["bytes"][:K].clone(), step_off=pipe.step_off[:K + 1].clone(),
                          send=send[:int(pipe.step_off[K].item())].clone()))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for rep in range(2):
        log("steps on two streams, round %d" % rep)
        for (cid, pipe, R, tok), st in zip(cases, streams):
            pipe.send.zero_()
            pipe.dem["demand"].fill_(-1)
            pipe.sched["dst"].fill_(-1)
        torch.cuda.synchronize()
        # stage by stage, alternating between the streams
        for stage in ("demand", "words", "plan", "pack"):
            for (cid, pipe, R, tok), st in zip(cases, streams):
                s = st
                if stage == "demand":
                    pipe.demand_stage(R, None, stream=s)
                elif stage == "words":
                    pipe.words_stage(stream=s)
                elif stage == "plan":
                    pipe.plan_stage(stream=s)
                else:
                    pipe.pack_stage(tok, None, stream=s)
        torch.cuda.synchronize()
        for (cid, pipe, R, tok), ref in zip(cases, alone):
            assert vp.read_status(pipe.status) == 0, cid
            K = int(pipe.sched["K"].item())
            assert K == ref["K"], cid
            assert torch.equal(pipe.dem["demand"], ref["demand"]), cid
            assert torch.equal(pipe.sched["dst"][:K], ref["dst"]), cid
            assert torch.equal(pipe.sched["bytes"][:K], ref["bytes"]), cid
            assert torch.equal(pipe.step_off[:K + 1], ref["step_off"]), cid
            assert torch.equal(pipe.send[:ref["send"].numel()], ref["send"]), cid


@pytest.mark.parametrize("topo", [vpgen.Topology(2, 2, 2, 2), vpgen.Topology(2, 1, 2, 2, 2),
                                  vpgen.Topology(2, 2, 2, 2, 1, 32, 25, 1), vpgen.Topology(3, 1, 2, 3)])
def test_batch_of_random_demands(vp, topo):
    """Twelve random matrices of mixed density and scale (an all-zero one
    among them) in one launch, with the buffer layout: every matrix's
    schedule, step offsets and receive view equal what the oracle's
    schedule gives, element by element."""
    N, unit, B = topo.n_ranks, 4096, 12
    rng = np.random.default_rng(N + topo.flags + 7 * topo.nics_per_switch)
    Ds = []
    for b in range(B):
        dens, scale = [(0.05, 3), (0.3, 20), (1.0, 50), (0.6, 1)][b % 4]
        D = rng.integers(0, scale + 1, (N, N)) * (rng.random((N, N)) < dens)
        np.fill_diagonal(D, 0)
        Ds.append((D * unit).astype(np.int64))
    Ds[5][:] = 0
    log("batch of random demands topo %s" % (topo.as_tuple(),))
    cat = vp.Catalog(topo)
    cat.upload()
    oc = oracle.Catalog(topo)
    p = vp.plan_params(N, unit, k_max=64 * N)
    out = vp.alloc_schedule_batch(B, N, p.k_max, layout=True)
    s = vp.plan_batch(cat, torch.from_numpy(np.stack(Ds)).cuda(), p, out=out)
    torch.cuda.synchronize()
    assert (s["status"].cpu().numpy() == 0).all()
    for b in range(B):
        o = oc.plan(Ds[b], unit, k_max=64 * N)
        g = host(s, b)
        assert (g["K"], g["tau"]) == (o["K"], o["tau"]), b
        for key in ("family", "dst", "inst", "bytes"):
            assert np.array_equal(g[key], o[key]), (b, key)
        K = o["K"]
        if K:
            # send offsets: running sums of each rank's lanes; stream offsets: bytes
            # of the same pair before the step; receive view: the inverse of dst
            nb, dst = o["bytes"], o["dst"]
            want_so = np.cumsum(nb, axis=0) - nb
            assert np.array_equal(s["send_off"][b, :K].cpu().numpy(), want_so), b
            co = np.zeros((K, N), np.int64)
            seen = np.zeros((N, N), np.int64)
            for k in range(K):
                co[k] = seen[np.arange(N), dst[k]]
                seen[np.arange(N), dst[k]] += nb[k]
            assert np.array_equal(s["stream_off"][b, :K].cpu().numpy(), co), b
            rs = np.zeros((K, N), np.int32)
            rs[np.arange(K)[:, None], dst] = np.arange(N, dtype=np.int32)[None, :]
            assert np.array_equal(s["recv_src"][b, :K].cpu().numpy(), rs), b
