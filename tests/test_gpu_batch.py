"""vp_plan_batch: several matrices planned side by side, one workgroup
each, must give every matrix the schedule the oracle gives it (through the
stored stream digests, and element by element for a dispatch matrix D and
its combine matrix D^T); a bad matrix fails alone."""
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
