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
                                  vpgen.Topology(1, 1, 1, 4), vpgen.Topology(4, 1, 3, 2, 1, 32, 50),
                                  # several NICs per switch
                                  vpgen.Topology(1, 1, 2, 2, 2), vpgen.Topology(1, 2, 1, 2, 2),
                                  vpgen.Topology(1, 1, 2, 3, 2), vpgen.Topology(2, 1, 2, 2, 2),
                                  vpgen.Topology(3, 1, 2, 2, 3), vpgen.Topology(1, nics_per_switch=2)])
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
                 vpgen.Topology(1, sockets_per_node=3, switches_per_socket=3),
                 vpgen.Topology(1, nics_per_switch=5),
                 # 2Q + 2Qm resource bits above 64 / more than 256 node-local instances
                 vpgen.Topology(1, 2, 4, 2, 4), vpgen.Topology(1, 2, 4, 2, 2)]:
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
    # partial histograms of every row (int32 per part and expert), chunk
    # counts of the sorted row
    assert vp.demand_workspace_bytes(256, 4096, 8, 256) >= 256 * 4 * 8 * 4
    assert vp.demand_workspace_bytes(1, 4096, 8, 256) < vp.demand_workspace_bytes(256, 4096, 8, 256)
    assert vp.demand_workspace_bytes(0, 4096, 8, 256) == 0
    # heads: a 40-byte descriptor and a 4-byte first unit per step, whatever
    # the send buffer's size
    assert vp.pack_workspace_bytes(2048, 468_729_856, 14336) >= 2048 * 44
    assert vp.pack_workspace_bytes(2048, 468_729_856, 14336) == vp.pack_workspace_bytes(2048, 1 << 40, 256)
    # rows: one 8-byte send-unit entry per (token, routing slot)
    assert vp.pack_workspace_bytes(2048, 468_729_856, 14336, 4096, 8) >= 2048 * 44 + 4096 * 8 * 8
    assert vp.pack_workspace_bytes(2048, 468_729_856, 14336, -1, 8) == 0


# ------------------------------------------------------- serialized catalog

def fnv1a64(b: bytes) -> int:
    h = 0xcbf29ce484222325
    for x in b:
        h = ((h ^ x) * 0x100000001b3) & 0xFFFFFFFFFFFFFFFF
    return h


def reseal(body: bytes) -> bytes:
    return body + fnv1a64(body).to_bytes(8, "little")


HEAD = 8 + 6 * 4 + 2 * 8 + 3 * 4


def assert_same_catalog(a, b):
    assert (a.N, a.G, a.g, a.Q, a.n_nodes, a.n_shapes, a.n_families, a.n_instances) == \
        (b.N, b.G, b.g, b.Q, b.n_nodes, b.n_shapes, b.n_families, b.n_instances)
    for x, y in [(a.instances(), b.instances()), (a.shapes(), b.shapes()), (a.families(), b.families())]:
        for key in x:
            assert np.array_equal(x[key], y[key]), key


@pytest.mark.parametrize("topo", [vpgen.tiny_topology(), vpgen.config(1).topo, vpgen.config(2).topo,
                                  vpgen.config(5).topo, vpgen.Topology(3, 1, 2, 3), vpgen.Topology(2, 2, 1, 4),
                                  vpgen.Topology(1, 1, 2, 2, 2), vpgen.Topology(2, 1, 2, 2, 2)])
def test_catalog_save_load_round_trip(vp, topo):
    c = vp.Catalog(topo)
    p = c.save()
    # header, one byte per node-local instance id of every local family
    # (shift-0 ones, then the NIC-carrying ones shared by every shift), hash
    F0 = int((c.families()["k"] == 0).sum())
    F1 = (c.n_families - F0) // (c.n_nodes - 1) if c.n_nodes > 1 else 0
    assert len(p) == HEAD + (F0 + F1) * c.Q * c.g + 8
    assert p[:8] == b"VPCATLG1" and fnv1a64(p[:-8]) == int.from_bytes(p[-8:], "little")
    d = vp.Catalog.load(p)
    assert_same_catalog(c, d)
    assert d.save() == p


def test_catalog_payload_sizes(vp):
    """One byte per node-local instance id: 152 shift-0 families for one
    8-GPU node, 152 + 352 node-local families for every multi-node size."""
    for cid, F in [(1, 152), (2, 504), (3, 504), (5, 504)]:
        c = vp.Catalog(vpgen.config(cid).topo)
        assert len(c.save()) == HEAD + F * 8 + 8


def test_catalog_load_rejects_damaged_payloads(vp):
    p = vp.Catalog(vpgen.config(2).topo).save()
    body = p[:-8]
    QG = 8
    bad = {
        "magic": reseal(b"XPCATLG1" + body[8:]),
        "hash": body + bytes(8),
        "truncated": reseal(body[:-QG]),
        # a family with a repeated instance id (not strictly ascending)
        "repeat": reseal(body[:HEAD] + bytes([body[HEAD]]) * 2 + body[HEAD + 2:]),
        # two families swapped: no longer in canonical order
        "order": reseal(body[:HEAD] + body[HEAD + QG:HEAD + 2 * QG] + body[HEAD:HEAD + QG] + body[HEAD + 2 * QG:]),
        # an instance id past the table
        "id": reseal(body[:HEAD + QG - 1] + bytes([250]) + body[HEAD + QG:]),
        # gpus_per_switch 5
        "topology": reseal(body[:20] + (5).to_bytes(4, "little") + body[24:]),
    }
    for name, q in bad.items():
        with pytest.raises(vp.VPError):
            vp.Catalog.load(q)
        assert name


def test_catalog_load_accepts_a_restricted_subset(vp):
    """Dropping whole families keeps a valid (restricted) catalog."""
    c = vp.Catalog(vpgen.config(1).topo)
    p = c.save()
    body = bytearray(p[:-8])
    F0 = int.from_bytes(body[HEAD - 12:HEAD - 8], "little")
    keep = [f for f in range(F0) if f % 3 != 1]
    fams = b"".join(bytes(body[HEAD + f * 8:HEAD + (f + 1) * 8]) for f in keep)
    body[HEAD - 12:HEAD - 8] = len(keep).to_bytes(4, "little")
    d = vp.Catalog.load(reseal(bytes(body[:HEAD]) + fams))
    assert d.n_families == len(keep)
    ids = c.families()["ids"]
    assert np.array_equal(d.families()["ids"], ids[keep])


@pytest.mark.parametrize("topo", [vpgen.tiny_topology(), vpgen.config(1).topo, vpgen.config(2).topo,
                                  vpgen.config(5).topo, vpgen.Topology(3, 1, 2, 3), vpgen.Topology(2, 2, 1, 4)])
def test_nearest_path_restriction_equals_oracle(vp, topo):
    ours = vp.Catalog(topo).restrict(vp.RESTRICT_NEAREST_PATH)
    ref = oracle.Catalog(topo, nearest=True)
    assert (ours.n_shapes, ours.n_families) == (ref.n_shapes, ref.n_families)
    sa, sb = ours.shapes(), ref.shapes()
    for key in ("k", "fam_begin", "fam_end", "L", "R"):
        assert np.array_equal(sa[key], sb[key]), key
    fa, fb = ours.families(), ref.families()
    for key in ("shape", "k", "ids"):
        assert np.array_equal(fa[key], fb[key]), key
    # a restricted catalog survives its own serialized form
    assert vp.Catalog.load(ours.save()).n_families == ours.n_families
    with pytest.raises(vp.VPError):
        vp.Catalog(topo).restrict(7)


@pytest.mark.parametrize("name", ["uniform-16", "zipf-pairs-16-s0.6", "wan21-H4C2", "wan21-H8C2"])
def test_rotation_time_equals_oracle(vp, name):
    import extra_cases
    case = vpgen.extra(name)
    D = extra_cases.oracle_demand(case, 1)
    cat = vp.Catalog(case.topo)
    for rule, near in [(vp.ROTATION_NEAREST_PATH, True), (vp.ROTATION_DYNAMIC_PATH, False)]:
        assert cat.rotation_time(D, rule) == oracle.rotation_time(case.topo, D, near)


def test_rotation_time_limits(vp):
    cat = vp.Catalog(vpgen.config(3).topo)   # 64 ranks: too many path choices in one stage
    D = np.ones((64, 64), np.int64) * 4096
    np.fill_diagonal(D, 0)
    with pytest.raises(vp.VPError):
        cat.rotation_time(D, vp.ROTATION_DYNAMIC_PATH)
    cat.rotation_time(D, vp.ROTATION_NEAREST_PATH)
    with pytest.raises(vp.VPError):
        cat.rotation_time(-D, vp.ROTATION_NEAREST_PATH)


SYS_TOPOS = [vpgen.Topology(1, 2, 1, 2, flags=1), vpgen.Topology(1, flags=1), vpgen.Topology(2, flags=1),
             vpgen.Topology(32, flags=1), vpgen.Topology(2, 4, 1, 2, flags=1), vpgen.Topology(3, 2, 2, 3, flags=1)]


@pytest.mark.parametrize("nearest", [False, True])
@pytest.mark.parametrize("topo", SYS_TOPOS)
def test_sys_catalog_equals_oracle(vp, topo, nearest):
    ours = vp.Catalog(topo)
    if nearest:
        ours = ours.restrict(vp.RESTRICT_NEAREST_PATH)
    ref = oracle.Catalog(topo, nearest=nearest)
    a, b = ours.instances(), ref.table()
    for key in ("cls", "src", "dst", "copy", "bw"):
        assert np.array_equal(a[key], b[key]), key
    sa, sb = ours.shapes(), ref.shapes()
    for key in ("k", "fam_begin", "fam_end", "L", "R"):
        assert np.array_equal(sa[key], sb[key]), key
    fa, fb = ours.families(), ref.families()
    for key in ("shape", "k", "ids"):
        assert np.array_equal(fa[key], fb[key]), key
    assert vp.Catalog.load(ours.save()).n_families == ours.n_families


def test_sys_flag_limits(vp):
    with pytest.raises(vp.VPError):
        vp.Catalog(vpgen.Topology(1, 8, 1, 2, flags=1))   # more than 4 sockets
    with pytest.raises(vp.VPError):
        vp.Catalog(vpgen.Topology(1, flags=2))            # unknown flag


@pytest.mark.parametrize("topo", [vpgen.Topology(1, 2, 1, 2, flags=1), vpgen.Topology(2, flags=1)])
def test_sys_rotation_time_equals_oracle(vp, topo):
    rng = np.random.default_rng(5)
    N = topo.n_ranks
    D = rng.integers(0, 64, (N, N)).astype(np.int64) * 4096
    np.fill_diagonal(D, 0)
    cat = vp.Catalog(topo)
    for rule, near in [(vp.ROTATION_NEAREST_PATH, True), (vp.ROTATION_DYNAMIC_PATH, False)]:
        assert cat.rotation_time(D, rule) == oracle.rotation_time(topo, D, near)


def test_plan_noalloc_refuses_more_than_256_ranks(vp):
    """The library-owned residual holds 256 ranks: a 1,024-rank catalog is
    refused on the host before any device call (no GPU needed)."""
    import ctypes as C
    cat = vp.Catalog(vpgen.Topology(128))
    p = vp.plan_params(cat.N, 4096)
    st = vp.lib().vp_plan_noalloc(cat.handle, None, C.byref(p), None, None, None, None, None, None, None, None,
                                  None, None, None)
    assert st == vp.UNSUPPORTED
    assert b"256" in vp.lib().vp_last_error()


def test_catalog_load_rejects_a_family_under_other_nic_names(vp):
    """With two NICs per switch a payload may name each family only by its
    renaming class's representative: the same family with the two NICs of a
    switch swapped is refused even though it is feasible and in order."""
    topo = vpgen.Topology(1, 1, 2, 2, 2)
    c = vp.Catalog(topo)
    inst = c.instances()
    body = bytearray(c.save()[:-8])
    QG = 4
    F0 = int.from_bytes(body[HEAD - 12:HEAD - 8], "little")
    swapped = None
    for f in range(F0):
        ids = list(body[HEAD + f * QG:HEAD + (f + 1) * QG])
        if not any(inst["cls"][i] == vp.PATH_NIC for i in ids):
            continue
        # swap the source NICs of switch 0 (copy = x * 2 + y)
        new = []
        for i in ids:
            if inst["cls"][i] == vp.PATH_NIC and inst["src"][i] == 0:
                cp = int(inst["copy"][i]) ^ 2
                j = [k for k in range(len(inst["cls"])) if inst["cls"][k] == vp.PATH_NIC and
                     inst["src"][k] == inst["src"][i] and inst["dst"][k] == inst["dst"][i] and inst["copy"][k] == cp][0]
                new.append(j)
            else:
                new.append(i)
        if sorted(new) != ids:
            swapped = sorted(new)
            break
    assert swapped is not None
    # replace the whole catalog by that one renamed family
    body[HEAD - 12:HEAD - 8] = (1).to_bytes(4, "little")
    with pytest.raises(vp.VPError) as e:
        vp.Catalog.load(reseal(bytes(body[:HEAD]) + bytes(swapped)))
    assert "NIC" in str(e.value)


def test_catalog_of_a_node_too_large_for_the_search_is_refused(vp):
    """One node of two sockets with four switches of two GPUs each has more
    candidate channel sets than the catalog search holds before pruning
    (2^22): the build returns VP_ERR_UNSUPPORTED with a message instead of
    growing without bound."""
    import ctypes as C
    h = C.c_void_p()
    st = vp.lib().vp_build_catalog(C.byref(vp.topology(vpgen.Topology(1, 2, 4, 2))), C.byref(h))
    assert st == vp.UNSUPPORTED
    assert b"2^22" in vp.lib().vp_last_error()


def test_threaded_catalog_build_is_deterministic(vp):
    """The pruning rules run on several host threads for large searches
    (two nodes of four switches with two NICs each: 750,644 channel sets for
    the NIC-carrying patterns); two builds give the same catalog byte for
    byte, and one 4,096-set-or-larger search agrees with the oracle in
    test_catalog_equals_oracle."""
    topo = vpgen.Topology(2, 2, 2, 2, 2)
    a, b = vp.Catalog(topo).save(), vp.Catalog(topo).save()
    assert a == b
    assert vp.Catalog.load(a).n_families == 64932
