"""Pins of the oracle's catalog (Alg. 1, PrunePaths, PruneFamilies, the
node-circulant reduction) against independent checks: the balance and
compatibility definitions Eq. (3)-(4), rank-level brute force of Eq. (1) on
tiny topologies, symmetry closure, and hand-derived counts."""
import collections
import itertools
import json
import os

import numpy as np
import pytest

import oracle
import vpgen
from oracle.checks import PIX, PXB, NIC, TopoModel, brute_force_channels, instantiate

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def two_node_one_socket():
    return vpgen.Topology(2, sockets_per_node=1, switches_per_socket=2, gpus_per_switch=2)


def cluster_families(cat):
    return [cat.cluster_family(f) for f in range(cat.n_families)]


def fam_key(fam):
    return tuple(sorted(zip(fam["cls"].tolist(), fam["a"].tolist(), fam["d"].tolist())))


def test_golden_counts():
    """Hand-derived counts; the tiny topology also matches the first row of
    the catalog-scale table (3 shapes, 6 families) as a consistency check."""
    with open(os.path.join(GOLDEN, "catalog_counts.json")) as f:
        gold = json.load(f)
    for row in gold["rows"]:
        t = row["topology"]
        topo = vpgen.Topology(t["n_nodes"], t["sockets"], t["switches"], t["g"])
        cat = oracle.Catalog(topo, full=row.get("full", False))
        assert cat.n_families == row["families"], row
        if "shapes" in row:
            assert cat.n_shapes == row["shapes"], row


@pytest.mark.parametrize("topo", [vpgen.tiny_topology(), vpgen.config(1).topo,
                                  vpgen.config(2).topo, vpgen.config(3).topo])
def test_shapes_and_families_satisfy_eq3_eq4(topo):
    cat = oracle.Catalog(topo)
    tm = TopoModel(topo)
    sh = cat.shapes()
    fams = cat.families()
    G, g, Q = tm.G, tm.g, tm.Q
    covered = np.zeros((G, G), bool)
    for j in range(cat.n_shapes):
        # materialise the G x G shape from its node blocks
        M = np.zeros((G, G), np.int64)
        k = int(sh["k"][j])
        for n in range(tm.nn):
            M[n * Q:(n + 1) * Q, n * Q:(n + 1) * Q] += sh["L"][j]
            m = (n + k) % tm.nn
            M[n * Q:(n + 1) * Q, m * Q:(m + 1) * Q] += sh["R"][j]
        assert (M.sum(1) == g).all() and (M.sum(0) == g).all(), "Eq. (3)"
        assert sh["fam_end"][j] > sh["fam_begin"][j]
        covered |= M > 0
        for f in range(sh["fam_begin"][j], sh["fam_end"][j]):
            assert fams["shape"][f] == j
            cf = cat.cluster_family(f)
            cnt = np.zeros((G, G), np.int64)
            used = set()
            for c, a, d in zip(cf["cls"], cf["a"], cf["d"]):
                assert c in tm.unpruned_classes(a, d)
                cnt[a, d] += 1
                for r in tm.shared(c, a, d):
                    assert r not in used, "Eq. (4) resource reuse"
                    used.add(r)
            assert (cnt == M).all(), "Eq. (4) shape consistency"
    assert covered.all(), "some group pair is covered by no shape"


def test_brute_force_tiny_topology_equals_catalog():
    topo = vpgen.tiny_topology()
    tm = TopoModel(topo)
    cat = oracle.Catalog(topo)
    inst = set()
    for f in cluster_families(cat):
        inst |= instantiate(tm, f)
    assert inst == brute_force_channels(tm)


def test_brute_force_one_node_equals_catalog():
    """All 14,833 derangements of 8 ranks with every unpruned path vector,
    filtered by Eq. (1), are exactly the instantiations of the 152 families."""
    topo = vpgen.config(1).topo
    tm = TopoModel(topo)
    cat = oracle.Catalog(topo)
    inst = set()
    for f in cluster_families(cat):
        got = instantiate(tm, f)
        assert got, "family with no valid endpoint binding"
        assert not (got & inst), "two families instantiate the same channel"
        inst |= got
    assert inst == brute_force_channels(tm)


def test_circulant_subset_of_full_catalog():
    topo = two_node_one_socket()
    full = oracle.Catalog(topo, full=True)
    circ = oracle.Catalog(topo)
    fk = {fam_key(f) for f in cluster_families(full)}
    ck = [fam_key(f) for f in cluster_families(circ)]
    assert len(set(ck)) == len(ck)
    assert set(ck) <= fk
    # full catalog is also exactly the brute-force channel set of its topology
    tm = TopoModel(topo)
    inst = set()
    for f in cluster_families(full):
        inst |= instantiate(tm, f)
    assert inst == brute_force_channels(tm)


def test_prune_paths_removes_exactly_nic_loopback():
    topo = vpgen.config(2).topo
    cat = oracle.Catalog(topo)
    tab = cat.table()
    fams = cat.families()
    loop = {i for i in range(cat.n_table) if tab["cls"][i] == NIC and tab["src"][i] == tab["dst"][i]}
    used0 = set(fams["ids"][fams["k"] == 0].reshape(-1).tolist())
    used1 = set(fams["ids"][fams["k"] == 1].reshape(-1).tolist())
    assert not (loop & used0), "an intra-node NIC loopback survived PrunePaths"
    assert used0 | loop == set(range(cat.n_table)), "a non-dominated instance is never used"
    assert loop <= used1, "remote NIC lanes between equal slots must stay"


def test_prune_families_leaves_no_duplicate_or_dominated_family():
    topo = vpgen.config(1).topo
    cat = oracle.Catalog(topo)
    tm = TopoModel(topo)
    sh = cat.shapes()
    for j in range(cat.n_shapes):
        members = [cat.cluster_family(f) for f in range(sh["fam_begin"][j], sh["fam_end"][j])]
        keys = [fam_key(f) for f in members]
        assert len(set(keys)) == len(keys)
        for f1, f2 in itertools.permutations(members, 2):
            # dominance: per group pair, identical footprints with no lower rate
            by1, by2 = collections.Counter(), collections.Counter()
            for c, a, d in zip(f1["cls"], f1["a"], f1["d"]):
                by1[(a, d, tm.shared(c, a, d))] += 1
            for c, a, d in zip(f2["cls"], f2["a"], f2["d"]):
                by2[(a, d, tm.shared(c, a, d))] += 1
            # identical footprint multisets imply equal rates in this model,
            # so dominance can only hold between equal families
            assert by1 != by2


def slot_perm_group():
    """Automorphisms of one node: swap the two switches of a socket, swap sockets."""
    gens = [(1, 0, 2, 3), (0, 1, 3, 2), (2, 3, 0, 1)]
    group = {(0, 1, 2, 3)}
    frontier = list(group)
    while frontier:
        p = frontier.pop()
        for s in gens:
            q = tuple(s[p[i]] for i in range(4))
            if q not in group:
                group.add(q)
                frontier.append(q)
    return sorted(group)


def test_symmetry_closure_one_node():
    cat = oracle.Catalog(vpgen.config(1).topo)
    fams = {fam_key(f) for f in cluster_families(cat)}
    perms = slot_perm_group()
    assert len(perms) == 8
    for p in perms:
        for key in fams:
            img = tuple(sorted((c, p[a], p[d]) for c, a, d in key))
            assert img in fams


def test_symmetry_closure_circulant():
    topo = vpgen.config(3).topo     # 8 nodes
    cat = oracle.Catalog(topo)
    tm = TopoModel(topo)
    Q, nn = tm.Q, tm.nn
    fams = {fam_key(f) for f in cluster_families(cat)}

    def node_map(key, fn):
        return tuple(sorted((c, fn(a // Q) * Q + a % Q, fn(d // Q) * Q + d % Q) for c, a, d in key))

    for key in list(fams)[::7]:
        assert node_map(key, lambda n: (n + 3) % nn) in fams       # node shift
        assert node_map(key, lambda n: (-n) % nn) in fams          # reflection k -> -k
        for p in slot_perm_group():
            img = tuple(sorted((c, (a // Q) * Q + p[a % Q], (d // Q) * Q + p[d % Q])
                               for c, a, d in key))
            assert img in fams


@pytest.mark.parametrize("cid,families", [(1, 152), (2, 504), (3, 2616), (5, 11064)])
def test_config_family_counts(cid, families):
    cat = oracle.Catalog(vpgen.config(cid).topo)
    assert cat.n_families == families
    fams = cat.families()
    # every k != 0 shift holds the same 352 NIC-carrying local patterns
    for k in range(1, cat.n_nodes):
        assert (fams["k"] == k).sum() == 352


def test_node_block_aggregates_give_the_same_shape_scores():
    """P9: for node-circulant shapes, sum_ad Dhat_ad M_ad equals
    sum A (.) L + sum B_k (.) R with A = sum_n diagonal node blocks of Dhat and
    B_k = sum_n node blocks (n, n + k): the form a factorised scorer may use."""
    topo = vpgen.config(3).topo
    cat = oracle.Catalog(topo)
    tm = TopoModel(topo)
    sh = cat.shapes()
    Q, nn, G = tm.Q, tm.nn, tm.G
    rng = np.random.default_rng(3)
    Dhat = rng.integers(0, 10**9, (G, G)).astype(np.int64)
    blocks = Dhat.reshape(nn, Q, nn, Q).transpose(0, 2, 1, 3)
    A = sum(blocks[n, n] for n in range(nn))
    B = [sum(blocks[n, (n + k) % nn] for n in range(nn)) for k in range(nn)]
    for j in range(cat.n_shapes):
        k = int(sh["k"][j])
        M = np.zeros((G, G), np.int64)
        for n in range(nn):
            M[n * Q:(n + 1) * Q, n * Q:(n + 1) * Q] += sh["L"][j]
            m = (n + k) % nn
            M[n * Q:(n + 1) * Q, m * Q:(m + 1) * Q] += sh["R"][j]
        direct = int((Dhat * M).sum())
        fact = int((A * sh["L"][j]).sum() + (B[k] * sh["R"][j]).sum())
        assert direct == fact


def test_splitmix64_matches_published_outputs():
    with open(os.path.join(GOLDEN, "splitmix64_seed0.json")) as f:
        gold = json.load(f)
    got = oracle.splitmix_stream(3, state=0)
    assert [int(x) for x in got] == [int(h, 16) for h in gold["outputs_hex"]]
    # keyed streams differ in every key field
    base = (0, 5, 7, 1, 3, 0)
    ref = oracle.splitmix_stream(4, key=base)
    for i in range(6):
        k2 = list(base)
        k2[i] += 1
        assert not np.array_equal(oracle.splitmix_stream(4, key=k2), ref)


# ------------------------------------------ "fixed nearest path" catalogs

def test_nearest_path_tiny_topology_hand_count():
    """One socket, two switches of two GPUs: of the 6 families (3 shapes),
    the all-PIX family and the one-PXB-each-way family keep nearest paths;
    the other three cross lanes need a NIC between the two switches."""
    cat = oracle.Catalog(vpgen.tiny_topology(), nearest=True)
    assert (cat.n_shapes, cat.n_families) == (2, 2)


@pytest.mark.parametrize("topo,full", [(vpgen.tiny_topology(), False), (vpgen.config(1).topo, False),
                                       (None, True)])
def test_brute_force_nearest_paths_equal_restricted_catalog(topo, full):
    """Every feasible channel whose lanes all take their pair's nearest path
    (rank-level brute force) is exactly the instantiations of the restricted
    catalog's families."""
    topo = topo or two_node_one_socket()
    tm = TopoModel(topo)
    cat = oracle.Catalog(topo, full=full, nearest=True)
    inst = set()
    for f in cluster_families(cat):
        got = instantiate(tm, f)
        assert got and not (got & inst)
        inst |= got
    assert inst == brute_force_channels(tm, nearest=True)


@pytest.mark.parametrize("cid", [2, 3, 5])
def test_nearest_path_catalog_is_the_filtered_catalog(cid):
    """Multi-node: the restricted catalog is the circulant catalog minus the
    families with a NIC lane between two switches of one socket, in the same
    order."""
    topo = vpgen.config(cid).topo
    tm = TopoModel(topo)
    full, near = oracle.Catalog(topo), oracle.Catalog(topo, nearest=True)
    keep = []
    for f in range(full.n_families):
        fam = full.cluster_family(f)
        ok = all(int(c) == tm.nearest_class(int(a), int(d)) for c, a, d in zip(fam["cls"], fam["a"], fam["d"]))
        if ok:
            keep.append(fam_key(fam))
    assert [fam_key(near.cluster_family(f)) for f in range(near.n_families)] == keep


# ------------------------------------------ cross-socket peer to peer (SYS)

def two_socket_node(sys_p2p):
    return vpgen.Topology(1, sockets_per_node=2, switches_per_socket=1, gpus_per_switch=2,
                          flags=oracle.TOPO_SYS_P2P if sys_p2p else 0)


def test_sys_hand_counts():
    """Two sockets of one switch with two GPUs each.  Without peer to peer
    the only cross path is the NIC, usable once each way: all-PIX, and one
    PIX plus one NIC lane per switch (2 families, 2 shapes).  With SYS the
    pair has two disjoint paths ({UP, X, DN} and {TX, RX}), as PXB and NIC
    inside one socket: 6 families in 3 shapes, 2 of them on nearest paths."""
    assert (oracle.Catalog(two_socket_node(False)).n_shapes, oracle.Catalog(two_socket_node(False)).n_families) == (2, 2)
    c = oracle.Catalog(two_socket_node(True))
    assert (c.n_shapes, c.n_families) == (3, 6)
    assert oracle.Catalog(two_socket_node(True), nearest=True).n_families == 2


@pytest.mark.parametrize("nearest", [False, True])
@pytest.mark.parametrize("topo", [two_socket_node(True), vpgen.Topology(1, flags=1)])
def test_brute_force_sys_equals_catalog(topo, nearest):
    """Rank-level brute force with SYS paths (every derangement, every path
    vector, Eq. (1) with the socket links) equals the catalog's
    instantiations, with and without the nearest-path restriction."""
    tm = TopoModel(topo)
    cat = oracle.Catalog(topo, nearest=nearest)
    inst = set()
    for f in cluster_families(cat):
        got = instantiate(tm, f)
        assert got and not (got & inst)
        inst |= got
    assert inst == brute_force_channels(tm, nearest=nearest)


def test_sys_circulant_subset_of_full_catalog():
    topo = vpgen.Topology(2, sockets_per_node=2, switches_per_socket=1, gpus_per_switch=2, flags=1)
    full = oracle.Catalog(topo, full=True)
    circ = oracle.Catalog(topo)
    assert {fam_key(f) for f in cluster_families(circ)} <= {fam_key(f) for f in cluster_families(full)}
    tm = TopoModel(topo)
    inst = set()
    for f in cluster_families(full):
        inst |= instantiate(tm, f)
    assert inst == brute_force_channels(tm)


# ------------------------------------------------ several NICs per switch

def multi_nic(n_nodes=1, sockets=1, switches=2, g=2, m=2):
    return vpgen.Topology(n_nodes, sockets, switches, g, nics_per_switch=m)


def labels_of(cat, f):
    """Cluster view of family f and the path label of each instance: the
    source and destination NIC of its NIC lanes (from the instance's copy)."""
    cf = cat.cluster_family(f)
    copy = cat.table()["copy"]
    m = cat.topo.nics_per_switch
    labs = [(NIC, int(copy[i]) // m, int(copy[i]) % m) if c == NIC else (int(c), -1, -1)
            for c, i in zip(cf["cls"], cf["id"])]
    return cf, labs


def test_multi_nic_hand_counts():
    """Two NICs per switch, counted by hand with Burnside's lemma over the
    renamings of each switch's two NICs.  One socket with two switches of two
    GPUs: all-PIX (1 family); one lane each way plus a PIX lane per switch
    (PXB or one of four NIC pairs each way: 25 choices, 7 classes); two lanes
    each way (PXB plus a NIC pair, or two NIC lanes on disjoint NICs: 6
    choices each way, 36 in all, 10 classes): 3 shapes, 18 families.  Two
    sockets of one switch each (NIC paths only across): 1 + 4 + 2 = 7."""
    a = oracle.Catalog(multi_nic())
    assert (a.n_shapes, a.n_families) == (3, 18)
    b = oracle.Catalog(multi_nic(sockets=2, switches=1))
    assert (b.n_shapes, b.n_families) == (3, 7)


@pytest.mark.parametrize("topo", [multi_nic(), multi_nic(sockets=2, switches=1), multi_nic(g=3)],
                         ids=["one-socket", "two-sockets", "three-gpus"])
def test_brute_force_multi_nic_equals_catalog_up_to_renaming(topo):
    """Every channel that brute force finds over derangements and labelled
    path vectors (Eq. (1)), renamed to its smallest form, is an instantiation
    of exactly one catalog family renamed the same way."""
    from oracle.checks import brute_force_labeled, canonical_labeled, instantiate_labeled
    tm = TopoModel(topo)
    cat = oracle.Catalog(topo)
    seen = set()
    for f in range(cat.n_families):
        cf, labs = labels_of(cat, f)
        got = {canonical_labeled(tm, ch) for ch in instantiate_labeled(tm, cf, labs)}
        assert got, "family with no valid endpoint binding"
        assert not (got & seen), "two families differ only by NIC names"
        seen |= got
    assert seen == {canonical_labeled(tm, ch) for ch in brute_force_labeled(tm)}


def test_multi_nic_families_satisfy_eq3_eq4():
    """The 8-GPU node with two NICs per switch: every family is balanced and
    uses no labelled resource twice."""
    from oracle.checks import shared_labeled
    topo = vpgen.Topology(1, nics_per_switch=2)
    cat = oracle.Catalog(topo)
    tm = TopoModel(topo)
    for f in range(0, cat.n_families, 37):
        cf, labs = labels_of(cat, f)
        outd, ind, used = collections.Counter(cf["a"].tolist()), collections.Counter(cf["d"].tolist()), set()
        assert all(v == tm.g for v in outd.values()) and all(v == tm.g for v in ind.values())
        for lab, a, d in zip(labs, cf["a"], cf["d"]):
            for r in shared_labeled(tm, lab, int(a), int(d)):
                assert r not in used
                used.add(r)
