"""GPU planner on catalogs loaded from their serialized form: the same
schedule as on the catalog Alg. 1 built, bit for bit, and the oracle's."""
import sys

import numpy as np
import pytest
import torch

import oracle
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


def plan_on(vp, cat, D, unit):
    cat.upload()
    p = vp.plan_params(cat.N, unit)
    st = vp.new_status()
    s = vp.plan(cat, torch.from_numpy(D).cuda(), p, status=st, out=vp.alloc_schedule(cat.N, p.k_max))
    torch.cuda.synchronize()
    h = vp.schedule_to_host(s)
    h["status"] = vp.read_status(st)
    return h


@pytest.mark.parametrize("cid", [1, 2, 5])
def test_loaded_catalog_plans_like_the_built_one(vp, cid):
    w = vpgen.config(cid)
    log("plan on a loaded catalog C%d" % cid)
    R = vpgen.routing_all(w, 0, 1024)
    D = np.stack([oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes)["row"] for i in range(w.n_ranks)])
    built = vp.Catalog(w.topo)
    loaded = vp.Catalog.load(built.save())
    a, b = plan_on(vp, built, D, w.row_bytes), plan_on(vp, loaded, D, w.row_bytes)
    assert a["status"] == 0 and b["status"] == 0
    o = oracle.Catalog(w.topo).plan(D, w.row_bytes)
    for key in ("K", "tau"):
        assert a[key] == b[key] == o[key]
    for key in ("family", "dst", "inst", "bytes"):
        assert np.array_equal(a[key], b[key]) and np.array_equal(a[key], o[key]), key
