"""GPU planner on the extra demands (uniform AlltoAll, skew AlltoAllv at
s = 0.4 / 0.6 / 0.8, Wan2.1-like head/context layouts) with the full catalog
and with the nearest-path catalog of the peer/path ablation, against the
oracle, bit-exact; the head/context demand itself comes from vp_demand_heads
per all-to-all group."""
import os
import sys

import numpy as np
import pytest
import torch

import extra_cases
import oracle
import vpgen

pytestmark = pytest.mark.gpu
_cat = {}


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def vp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_34340_amd as vp
    vp.lib()
    return vp


def catalogs(vp, topo, nearest):
    key = (topo.as_tuple(), nearest)
    if key not in _cat:
        c = vp.Catalog(topo)
        if nearest:
            c = c.restrict(vp.RESTRICT_NEAREST_PATH)
        c.upload()
        _cat[key] = (c, oracle.Catalog(topo, nearest=nearest))
    return _cat[key]


def check(vp, case, nearest, matrix):
    gc, oc = catalogs(vp, case.topo, nearest)
    D_dev = extra_cases.gpu_demand(vp, case, matrix)
    D = extra_cases.oracle_demand(case, matrix)
    torch.cuda.synchronize()
    assert np.array_equal(D_dev.cpu().numpy(), D), "demand differs"
    p = vp.plan_params(gc.N, case.unit)
    st = vp.new_status()
    s = vp.plan(gc, D_dev, p, status=st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    g = vp.schedule_to_host(s)
    o = oc.plan(D, case.unit)
    assert g["K"] == o["K"] and g["tau"] == o["tau"]
    for key in ("family", "dst", "inst", "bytes"):
        assert np.array_equal(g[key], o[key]), key


@pytest.mark.parametrize("nearest", [False, True])
@pytest.mark.parametrize("name", extra_cases.NAMES)
def test_extra_plan_parity(vp, name, nearest):
    case = vpgen.extra(name)
    mats = range(extra_cases.ZIPF_MATRICES) if name.startswith("zipf-pairs-16-s0.6") else [0]
    for m in mats:
        log("extra plan parity %s nearest=%s matrix %d" % (name, nearest, m))
        check(vp, case, nearest, m)


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_sys_topology_plan_parity(vp, cid):
    """MoE demand on nodes with cross-socket peer to peer (SYS paths)."""
    import dataclasses
    w = vpgen.config(cid)
    topo = dataclasses.replace(w.topo, flags=vp.TOPO_SYS_P2P)
    log("SYS topology plan parity C%d" % cid)
    R = vpgen.routing_all(w, 0, 2048)
    D = np.stack([oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes)["row"] for i in range(w.n_ranks)])
    gc, oc = catalogs(vp, topo, False)
    p = vp.plan_params(gc.N, w.row_bytes)
    st = vp.new_status()
    s = vp.plan(gc, torch.from_numpy(D).cuda(), p, status=st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    g = vp.schedule_to_host(s)
    o = oc.plan(D, w.row_bytes)
    assert g["K"] == o["K"] and g["tau"] == o["tau"]
    for key in ("family", "dst", "inst", "bytes"):
        assert np.array_equal(g[key], o[key]), key
    # some lane takes a SYS path
    assert (gc.instances()["cls"][g["inst"]] == vp.PATH_SYS).any()


def test_sys_topology_256_ranks_plan_parity(vp):
    """256 ranks with SYS paths (60,104 families): the GPU schedule equals the
    oracle's through the digests tests/golden/make_stream_digests.py --sys-256
    stored (the oracle takes about a minute there), and is a valid
    decomposition (every activation feasible, sums to D, progressing)."""
    import dataclasses
    import json
    from oracle.checks import TopoModel, schedule_valid
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import stream_digest as sd
    with open(sd.GOLDEN_SYS256) as f:
        ref = json.load(f)
    w = vpgen.config(5)
    topo = dataclasses.replace(w.topo, flags=vp.TOPO_SYS_P2P)
    log("SYS topology 256 ranks")
    R = vpgen.routing_all(w, 0)
    D = np.stack([oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes)["row"] for i in range(w.n_ranks)])
    assert sd.demand_digest(D) == ref["demand"]
    gc = vp.Catalog(topo)
    gc.upload()
    p = vp.plan_params(gc.N, w.row_bytes)
    st = vp.new_status()
    s = vp.plan(gc, torch.from_numpy(D).cuda(), p, status=st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    g = vp.schedule_to_host(s)
    assert (g["K"], g["tau"]) == (ref["K"], ref["tau"])
    assert sd.schedule_digest(g) == ref["schedule"]
    schedule_valid(TopoModel(topo), D, g, gc.instances()["cls"])
    assert (g["bytes"].sum(axis=1) > 0).all()


def test_plan_state_beyond_lds_is_refused_on_host(vp):
    """Two nodes of two sockets x two switches x three GPUs with cross-socket
    peer to peer give 2,185 shapes and 2,744 families, whose planner tables do
    not fit in one workgroup's LDS: vp_plan refuses the catalog on the host
    with VP_ERR_UNSUPPORTED and enqueues nothing (the outputs keep their
    sentinel), and a plan on a catalog that fits still runs afterwards."""
    topo = vpgen.Topology(2, 2, 2, 3, 1, 32, 12, vp.TOPO_SYS_P2P)
    gc = vp.Catalog(topo)
    gc.upload()
    N = gc.N
    D = torch.full((N, N), 4096, dtype=torch.int64, device="cuda")
    D.fill_diagonal_(0)
    p = vp.plan_params(N, 4096)
    st = vp.new_status()
    out = vp.alloc_schedule(N, p.k_max)
    out["K"].fill_(-7)
    with pytest.raises(vp.VPError) as e:
        vp.plan(gc, D, p, status=st, out=out)
    assert e.value.status == vp.UNSUPPORTED
    assert "LDS" in str(e.value)
    torch.cuda.synchronize()
    assert int(out["K"].item()) == -7 and vp.read_status(st) == 0
    # a catalog that fits: the same nodes without SYS paths
    small = vp.Catalog(vpgen.Topology(2, 2, 2, 3, 1, 32, 12, 0))
    small.upload()
    s = vp.plan(small, D, vp.plan_params(N, 4096), status=st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    g = vp.schedule_to_host(s)
    assert g["K"] >= 1 and int(g["bytes"].sum()) == int(D.sum().item())
