"""Host-side checks of the HIP library (no GPU needed): the C-ABI exports every
function include/vp.h declares, the host catalog builder (an independent
slot-by-slot enumeration) equals the oracle's Alg. 1 catalog in canonical
order, host-side argument errors are reported, and the modeled time helper
matches the oracle."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import vpgen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vp.h")


@pytest.fixture(scope="module")
def vp():
    import paper_2609_34340_amd as vp
    if not os.path.exists(vp.LIB_PATH):
        from paper_2609_34340_amd import build
        build.build()
    return vp


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\*\s]+?\b(vp_\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_symbol(vp):
    names = declared_functions()
    assert len(names) >= 18
    L = ctypes.CDLL(vp.LIB_PATH)
    missing = [n for n in names if not hasattr(L, n)]
    assert not missing, missing


@pytest.mark.parametrize("topo", [vpgen.tiny_topology(), vpgen.config(1).topo, vpgen.config(2).topo,
                                  vpgen.config(3).topo, vpgen.config(5).topo,
                                  vpgen.Topology(3, 1, 2, 3), vpgen.Topology(2, 2, 1, 4),
                                  vpgen.Topology(1, 1, 1, 4), vpgen.Topology(4, 1, 3, 2, 1, 32, 50)])
def test_catalog_equals_oracle(vp, topo):
    ours = vp.Catalog(topo)
    ref = oracle.Catalog(topo)
    assert (ours.N, ours.G, ours.g, ours.Q, ours.n_nodes) == (ref.N, ref.G, ref.g, ref.Q, ref.n_nodes)
    assert ours.n_shapes == ref.n_shapes and ours.n_families == ref.n_families
    a, b = ours.instances(), ref.table()
    for key, rkey in [("cls", "cls"), ("src", "src"), ("dst", "dst"), ("copy", "copy"), ("bw", "bw")]:
        assert np.array_equal(a[key], b[rkey]), key
    sa, sb = ours.shapes(), ref.shapes()
    for key in ("k", "fam_begin", "fam_end", "L", "R"):
        assert np.array_equal(sa[key], sb[key]), key
    fa, fb = ours.families(), ref.families()
    for key in ("shape", "k", "ids"):
        assert np.array_equal(fa[key], fb[key]), key


def test_unsupported_topologies_are_rejected(vp):
    for topo in [vpgen.Topology(1, gpus_per_switch=1), vpgen.Topology(1, gpus_per_switch=5),
                 vpgen.Topology(1, nics_per_switch=0), vpgen.Topology(300),
                 vpgen.Topology(1, sockets_per_node=3, switches_per_socket=3)]:
        with pytest.raises(vp.VPError):
            vp.Catalog(topo)


def test_modeled_time_matches_oracle(vp):
    w = vpgen.config(2)
    R = vpgen.routing_all(w, 0, tokens=512)
    D = np.stack([oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes)["row"] for i in range(w.n_ranks)])
    ref = oracle.Catalog(w.topo)
    s = ref.plan(D, w.row_bytes)
    ours = vp.Catalog(w.topo)
    assert ours.modeled_time(s["K"], s["inst"], s["bytes"]) == ref.modeled_time(s)


def test_plan_params_defaults(vp):
    p = vp.plan_params(256, 14336)
    assert (p.k_target, p.lambda_ns, p.unit_bytes, p.n_start, p.i_aa, p.seed, p.k_max) == \
        (512, 10_000, 14336, 4, 8, 0, 2048)


def test_workspace_queries(vp):
    assert vp.demand_workspace_bytes(4096, 8, 256) >= 256 * 4 * 16
    assert vp.pack_workspace_bytes(2048, 468_729_856, 14336) >= 8 * (468_729_856 // 14336)
    # rows: a copy counter and top-k send-unit slots per token
    assert vp.pack_workspace_bytes(2048, 468_729_856, 14336, 4096, 8) >= 4096 * 4 * 9
    assert vp.pack_workspace_bytes(2048, 468_729_856, 14336, -1, 8) == 0
