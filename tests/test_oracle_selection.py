"""Pins of the planner's selection steps (Sec. 4.2), each checked from outside
the oracle's own code:

- Step 1, Eq. (5)-(6): replaying a schedule, the shape of every activation is
  the first shape in canonical order that maximises sum D-hat * M over the
  residual before that step, recomputed here with numpy (with ties
  present in the replayed inputs).
- Steps 2-3, Eq. (9)-(10): on every bucket with several families, each
  candidate's lane volumes are min(cap, residual) (Eq. (9)), its logged
  slowest lane is a lane of largest x / bw, and the family kept is the first
  in canonical order with the largest utility, all in exact fractions; the
  inputs include winners that are not first, utility ties, and candidates
  whose largest-volume lane is not their slowest.
- MultiStartAA's starts (readings R14, R15): start bindings worked out by
  hand on the tiny topology (the forced top-credit triple, its ties, a
  repair around the protected instance); the keyed SplitMix64 composition
  and the Fisher-Yates shuffles restated from their published definitions.
- Eq. (2): the oracle's modeled completion time equals the independent
  checker's on every workload's schedule.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import vpgen
from oracle.checks import TopoModel, modeled_time

_cats = {}


def catalog(topo):
    key = topo.as_tuple()
    if key not in _cats:
        _cats[key] = oracle.Catalog(topo)
    return _cats[key]


def dense_shapes(cat):
    """J x G x G lane counts: a shape (k, L, R) puts L on every node's
    diagonal block and R on the block from node n to node n + k."""
    sh = cat.shapes()
    if cat.full:
        return sh["L"].astype(np.int64)
    Q, nn = cat.Q, cat.n_nodes
    M = np.zeros((cat.n_shapes, cat.G, cat.G), np.int64)
    for m in range(cat.n_shapes):
        k = int(sh["k"][m])
        for n in range(nn):
            M[m, n * Q:(n + 1) * Q, n * Q:(n + 1) * Q] += sh["L"][m]
            n2 = (n + k) % nn
            if k:
                M[m, n * Q:(n + 1) * Q, n2 * Q:(n2 + 1) * Q] += sh["R"][m]
    return M


def workload_demand(cid):
    w = vpgen.config(cid)
    N = w.n_ranks
    if w.mode == "heads":
        hl = vpgen.head_split(w.heads, N)
        return w, np.stack([oracle.demand_heads(w.tokens, hl, w.row_bytes, i) for i in range(N)])
    R = vpgen.routing_all(w, 0)
    return w, np.stack([oracle.demand(R[i], N, w.experts, i, w.row_bytes)["row"] for i in range(N)])


def sparse_demand(rng, N, unit, density):
    D = (rng.random((N, N)) < density) * rng.integers(1, 9, (N, N)) * unit * 16
    D = D.astype(np.int64)
    np.fill_diagonal(D, 0)
    return D


# ------------------------------------------------------------ Step 1

def replay_shapes(cat, D, s):
    """Assert every activation's shape is the lowest-index Eq. (6) argmax
    on the residual before it; return the number of steps with a tie."""
    N, G, g = cat.N, cat.G, cat.g
    M = dense_shapes(cat).reshape(cat.n_shapes, -1)
    fam_shape = cat.families()["shape"]
    rem = np.array(D, dtype=np.int64)
    rows = np.arange(N)
    ties = 0
    for k in range(s["K"]):
        Dhat = rem.reshape(G, g, G, g).sum(axis=(1, 3))
        sc = M @ Dhat.reshape(-1)
        best = sc.max()
        assert best > 0
        want = int(np.flatnonzero(sc == best)[0])
        assert int(fam_shape[s["family"][k]]) == want, "step %d: shape %d, Eq. (6) argmax %d" % (
            k, fam_shape[s["family"][k]], want)
        ties += int((sc == best).sum() > 1)
        rem[rows, s["dst"][k]] -= s["bytes"][k]
    assert (rem == 0).all()
    return ties


@pytest.mark.parametrize("cid", [1, 2, 3, 4])
def test_shape_choice_on_the_workloads(cid):
    w, D = workload_demand(cid)
    cat = catalog(w.topo)
    replay_shapes(cat, D, cat.plan(D, w.row_bytes))


def test_shape_choice_with_ties():
    """Sparse demands leave many group pairs empty, so several shapes share
    the best score: the first in canonical order must win."""
    rng = np.random.default_rng(61)
    ties = 0
    for topo in (vpgen.tiny_topology(), vpgen.config(1).topo, vpgen.config(2).topo):
        cat = catalog(topo)
        for _ in range(6):
            D = sparse_demand(rng, cat.N, 4096, 0.15)
            if D.sum() == 0:
                continue
            ties += replay_shapes(cat, D, cat.plan(D, 4096))
    assert ties > 20


# ------------------------------------------------------------ Steps 2-3

def quantum(cat, D, unit):
    """tau as the plan reports it for D (one iteration planned)."""
    return cat.plan(D, unit, k_max=1, check=False)["tau"]


def check_bucket(cat, D, unit, m, lam, iteration=0):
    """Check the family choice on shape m; returns coverage flags (winner
    not first, utility tie, a candidate whose largest-volume lane is not its
    slowest)."""
    tab = cat.table()
    tau = quantum(cat, D, unit)
    cands, chosen = cat.shape_candidates(D, unit, m, iteration=iteration, lambda_ns=lam)
    fb, fe = cat.shapes()["fam_begin"][m], cat.shapes()["fam_end"][m]
    assert [c["family"] for c in cands] == list(range(fb, fe))
    U = []
    lane_differs = False
    for c in cands:
        bw = tab["bw"][cat.cluster_family(c["family"])["id"]].astype(np.int64)
        cap = np.maximum(unit, (tau * bw) // unit * unit)
        x = np.minimum(cap, D[c["src"], c["dst"]])
        assert np.array_equal(c["x"], x), "volumes are not Eq. (9)"
        S = int(x.sum())
        assert c["S"] == S
        slow = max(Fraction(int(a), int(b)) for a, b in zip(x, bw))
        if S:
            assert Fraction(c["xm"], c["bm"]) == slow, "logged slowest lane is not a max of x / bw"
        U.append(Fraction(0) if S == 0 else Fraction(S) / (lam + slow))
        big = int(np.argmax(x))   # the lane of largest volume, whatever its rate
        lane_differs |= S > 0 and Fraction(int(x[big]), int(bw[big])) < slow
    best = max(U)
    want = fb + U.index(best)
    assert chosen == want, "kept family %d, Eq. (10) argmax %d" % (chosen, want)
    return (U.index(best) != 0, U.count(best) > 1, lane_differs)


@pytest.mark.parametrize("name", ["C1", "C2", "C1sys"])
def test_family_choice_on_every_multi_family_bucket(name):
    topo = {"C1": vpgen.config(1).topo, "C2": vpgen.config(2).topo,
            "C1sys": vpgen.Topology(1, flags=oracle.TOPO_SYS_P2P)}[name]
    cat = catalog(topo)
    sh = cat.shapes()
    multi = [m for m in range(cat.n_shapes) if sh["fam_end"][m] - sh["fam_begin"][m] > 1]
    assert multi
    rng = np.random.default_rng(7)
    unit = 4096
    cover = np.zeros(3, np.int64)
    # six scales of the same kind of demand: the quantum, and with it how the
    # PCIe and NIC caps round to whole units, differs from trial to trial
    for trial in range(6):
        dense = rng.integers(0, 12, (cat.N, cat.N)) * unit * (1 + 4 * trial)
        D = np.where(rng.random((cat.N, cat.N)) < 0.5, dense, 0).astype(np.int64)
        np.fill_diagonal(D, 0)
        lam = [0, 10_000, 1_000_000, 10_000, 0, 100_000][trial]
        for m in multi[:60]:
            cover += np.array(check_bucket(cat, D, unit, m, lam, iteration=trial))
    # the inputs exercise what the choice depends on
    assert cover[0] > 0, "no bucket whose best family is not its first"
    assert cover[1] > 0, "no utility tie between families"
    assert cover[2] > 0, "no candidate whose largest lane is not its slowest"


# ------------------------------------------------------------ starts

def tiny_d(entries):
    D = np.zeros((4, 4), np.int64)
    for (i, j), v in entries.items():
        D[i, j] = v
    return D


# The tiny topology (one socket, two switches of two GPUs): group 0 = ranks
# {0, 1}, group 1 = ranks {2, 3}.  Family 1 holds node-local instances
# {0, 2, 4, 5}: t0 = PIX in switch 0, t1 = PIX in switch 1, t2 = PXB 0 -> 1,
# t3 = PXB 1 -> 0.  Family order gives group 0 the out-list [t0, t2] and the
# in-list [t0, t3], group 1 the out-list [t1, t3] and the in-list [t1, t2],
# so the canonical binding (m-th out-instance of group a takes source
# a*g + m, m-th in-instance of group d takes destination d*g + m) is
#   t0: 0 -> 0, t1: 2 -> 2, t2: 1 -> 3, t3: 3 -> 1.
# With unit 1 and K_target 1 every quantum is 1 ns here (L_max <= 32), so
# the PCIe caps are 32 bytes and every credit below equals its entry.
# Family 2 is the same with t3 = NIC 1 -> 0 (instance 8, cap 25 bytes).
START0_CASES = {
    # top triple (t0, 0, 1) = 5: t0 takes destination 1 from t3 (t3 -> 0);
    # repair: t1 is bound 2 -> 2, its group's first other in-instance t2
    # (not the protected t0) trades destinations: t1 -> 3, t2 -> 2
    "forced_intra": (1, {(0, 1): 5, (2, 3): 4, (1, 3): 3, (3, 0): 2}, [0, 2, 1, 3], [1, 3, 2, 0]),
    # (0, 1) and (1, 0) tie at 5: the smaller triple (t0, 0, 1) wins (the
    # other would bind t0 1 -> 0 and give sources [1, 2, 0, 3])
    "tie_to_smallest": (1, {(0, 1): 5, (1, 0): 5, (1, 3): 2}, [0, 2, 1, 3], [1, 3, 2, 0]),
    # top triple (t3, 3, 1) = 7 is already bound; t0 is bound 0 -> 0 and its
    # group's only other in-instance is the protected t3, so t0 trades
    # sources with t2 (t0: 1 -> 0, t2: 0 -> 3); then t1 2 -> 2 trades
    # destinations with t2 (t1 -> 3, t2 -> 2)
    "repair_around_protected": (1, {(3, 1): 7, (0, 1): 1}, [1, 2, 0, 3], [0, 3, 2, 1]),
    # no positive credit: canonical binding, both PIX lanes repaired by
    # destination trades with t3 and t2
    "no_credit": (1, {}, [0, 2, 1, 3], [1, 3, 2, 0]),
    # family 2, top triple (t3, 2, 0) = min(30, 25) = 25 beats (t0, 0, 1) =
    # 24: t3 takes source 2 from t1 (t1: 3 -> 2) and destination 0 from t0
    # (t0: 0 -> 1); nothing left to repair
    "forced_nic_both_sides": (2, {(2, 0): 30, (0, 1): 24}, [0, 3, 1, 2], [1, 2, 3, 0]),
}


@pytest.mark.parametrize("case", sorted(START0_CASES))
def test_canonical_start_by_hand(case):
    cat = catalog(vpgen.tiny_topology())
    assert list(cat.families()["ids"][1]) == [0, 2, 4, 5] and list(cat.families()["ids"][2]) == [0, 2, 4, 8]
    f, entries, src, dst = START0_CASES[case]
    s, d = cat.start_binding(tiny_d(entries), 1, f, 0, k_target=1)
    assert list(s) == src and list(d) == dst


MASK = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15


def mix64(z):
    """SplitMix64's output function (Steele, Lea, Flood, OOPSLA 2014)."""
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK
    return z ^ (z >> 31)


def keyed_state(seed, fields):
    """Reading R15: the key absorbs each field as key <- mix(key + gamma) xor field."""
    key = seed
    for v in fields:
        key = mix64((key + GAMMA) & MASK) ^ v
    return key


def draws(state, n):
    out = []
    for _ in range(n):
        state = (state + GAMMA) & MASK
        out.append(mix64(state))
    return out


@pytest.mark.parametrize("key", [(0, 0, 0, 1, 0, 0), (0, 7, 3, 2, 5, 1), (12345, 999, 11063, 3, 127, 1),
                                 (MASK, 1, 2, 3, 4, 0)])
def test_keyed_stream_restated(key):
    want = draws(keyed_state(key[0], key[1:]), 8)
    got = [int(v) for v in oracle.splitmix_stream(8, key=key)]
    assert got == want


def shuffled_start(cat, f, start, iteration, seed):
    """Reading R15 restated: per group and side, Fisher-Yates (m = g-1 .. 1,
    j = draw mod (m + 1), swap) over the group's g ranks, assigned to its
    out-list (side 0) or in-list (side 1) in family order."""
    cf = cat.cluster_family(f)
    g, G = cat.g, cat.G
    n = len(cf["a"])
    src, dst = [0] * n, [0] * n
    for side in (0, 1):
        for x in range(G):
            state = keyed_state(seed, (iteration, f, start, x, side))
            perm = list(range(g))
            for m in range(g - 1, 0, -1):
                state = (state + GAMMA) & MASK
                j = mix64(state) % (m + 1)
                perm[m], perm[j] = perm[j], perm[m]
            members = [t for t in range(n) if (cf["a"] if side == 0 else cf["d"])[t] == x]
            for m, t in enumerate(members):
                (src if side == 0 else dst)[t] = x * g + perm[m]
    return src, dst


@pytest.mark.parametrize("iteration,seed", [(0, 0), (5, 0), (17, 99), (3, 2 ** 63 + 5)])
def test_shuffled_starts_restated(iteration, seed):
    """Family 0 of the tiny topology has no lane inside a switch, so no repair
    applies and the start is the raw shuffle."""
    cat = catalog(vpgen.tiny_topology())
    D = tiny_d({(0, 2): 3, (2, 1): 4})
    for start in (1, 2, 3):
        s, d = cat.start_binding(D, 1, 0, start, iteration=iteration, seed=seed)
        want = shuffled_start(cat, 0, start, iteration, seed)
        assert (list(s), list(d)) == want


def test_shuffled_starts_repaired_only_where_needed():
    """On the 8-GPU node every shuffled start is self-transfer free, and a
    shuffle that binds no rank to itself is kept exactly as drawn."""
    cat = catalog(vpgen.config(1).topo)
    rng = np.random.default_rng(3)
    D = rng.integers(0, 5, (8, 8)).astype(np.int64) * 4096
    np.fill_diagonal(D, 0)
    kept = repaired = 0
    for f in range(0, cat.n_families, 3):
        for start in (1, 2, 3):
            s, d = cat.start_binding(D, 4096, f, start, iteration=f, seed=1)
            assert not (np.asarray(s) == np.asarray(d)).any()
            rs, rd = shuffled_start(cat, f, start, f, 1)
            if all(a != b for a, b in zip(rs, rd)):
                assert (list(s), list(d)) == (rs, rd)
                kept += 1
            else:
                repaired += 1
    assert kept > 0 and repaired > 0


# ------------------------------------------------------------ Eq. (2)

@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_modeled_time_matches_the_checker(cid):
    w, D = workload_demand(cid)
    cat = catalog(w.topo)
    s = cat.plan(D, w.row_bytes)
    num, den = cat.modeled_time(s)
    want = modeled_time(TopoModel(w.topo), s, cat.table()["cls"], oracle.DEFAULT_LAMBDA_NS)
    assert Fraction(num, den) == want
