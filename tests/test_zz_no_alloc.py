"""vp_plan_noalloc (the planner's residual in the library's own device array)
against vp_plan (the residual in a caller workspace), through the C-ABI:
two calls in a row, the second with a smaller input, every output compared
element by element.  Collected last: a failure here hides no other test."""
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


def moe_demand(cid):
    w = vpgen.config(cid)
    R = vpgen.routing_all(w, 0)
    return w, np.stack([oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes)["row"]
                        for i in range(w.n_ranks)])


def outputs(vp, s):
    K = int(s["K"].item())
    out = {"K": K, "tau": int(s["tau"].item()), "status": vp.read_status(s["status"])}
    for key in ("family", "dst", "inst", "bytes", "send_off", "stream_off", "recv_src"):
        out[key] = s[key][:K].cpu().numpy()
    return out


def test_plan_noalloc_matches_plan():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_34340_amd as vp
    # 64 ranks, then 8 ranks: the second call's residual is smaller than what
    # the first left in the array
    for cid in (3, 1):
        w, D = moe_demand(cid)
        log("plan_noalloc C%d (N=%d)" % (cid, w.n_ranks))
        cat = vp.Catalog(w.topo)
        cat.upload()
        p = vp.plan_params(cat.N, w.row_bytes)
        Dd = torch.from_numpy(D).cuda()
        ref = vp.plan(cat, Dd, p, out=vp.alloc_schedule(cat.N, p.k_max, layout=True))
        got = vp.plan_noalloc(cat, Dd, p, out=vp.alloc_schedule(cat.N, p.k_max, layout=True))
        torch.cuda.synchronize()
        a, b = outputs(vp, ref), outputs(vp, got)
        assert a["status"] == 0 and b["status"] == 0
        assert a["K"] == b["K"] > 0 and a["tau"] == b["tau"]
        for key in ("family", "dst", "inst", "bytes", "send_off", "stream_off", "recv_src"):
            assert np.array_equal(a[key], b[key]), key
