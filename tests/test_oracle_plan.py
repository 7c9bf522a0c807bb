"""Pins of the oracle's scheduler (Alg. 2): schedule validity and the
feasibility of every activation (Sec. 3), monotone AA (Sec. 4.2 Step 2),
progress per iteration, local optimality of every AA result checked with
scipy's assignment solver, the exact utility order against Fraction,
closed-form special cases and an exhaustive minimum-makespan search."""
import itertools
from fractions import Fraction

import numpy as np
import pytest
from scipy.optimize import linear_sum_assignment

import oracle
import vpgen
from oracle.checks import (NIC, PIX, PXB, TopoModel, exhaustive_makespan, modeled_time,
                           schedule_valid, schedule_valid_np, utility)

_cat_cache = {}


def catalog(topo):
    key = topo.as_tuple()
    if key not in _cat_cache:
        _cat_cache[key] = oracle.Catalog(topo)
    return _cat_cache[key]


def demand_for(cid, matrix=0):
    w = vpgen.config(cid)
    N = w.n_ranks
    if w.mode == "heads":
        hl = vpgen.head_split(w.heads, N)
        return np.stack([oracle.demand_heads(w.tokens, hl, w.row_bytes, i) for i in range(N)])
    R = vpgen.routing_all(w, matrix)
    return np.stack([oracle.demand(R[i], N, w.experts, i, w.row_bytes)["row"] for i in range(N)])


def cls_table(cat):
    return cat.table()["cls"]


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_schedule_valid_and_progressing(cid):
    """P1-P3: X(E_k) sum to D, every activation feasible under Eq. (1), every
    activation serves bytes, K within K_max."""
    w = vpgen.config(cid)
    cat = catalog(w.topo)
    tm = TopoModel(w.topo)
    D = demand_for(cid)
    s = cat.plan(D, w.row_bytes)
    schedule_valid(tm, D, s, cls_table(cat))
    assert 0 < s["K"] <= 8 * w.n_ranks
    served = s["bytes"].sum(axis=1)
    assert (served > 0).all(), "an iteration made no progress"
    assert (s["bytes"] % w.row_bytes == 0).all()
    # family ids point into the chosen shape's bucket and lanes use its instances
    fams = cat.families()
    for k in range(s["K"]):
        f = s["family"][k]
        assert sorted(np.unique(s["inst"][k])) == sorted(np.unique(fams["ids"][f]))


def test_plan_deterministic():
    """P16: two runs are identical."""
    w = vpgen.config(2)
    cat = catalog(w.topo)
    D = demand_for(2)
    a, b = cat.plan(D, w.row_bytes), cat.plan(D, w.row_bytes)
    for key in ("K", "family", "dst", "inst", "bytes", "tau"):
        assert np.array_equal(a[key], b[key])


def test_tau_from_k_target():
    """tau = ceil(L_max / (bw_max * K_target)) with L_max the largest row or column sum."""
    w = vpgen.config(2)
    D = demand_for(2)
    s = catalog(w.topo).plan(D, w.row_bytes, k_target=32)
    Lmax = max(D.sum(0).max(), D.sum(1).max())
    assert s["tau"] == -(-int(Lmax) // (32 * 32))


def test_aa_never_decreases_binding_score():
    """P4: F_B after every AA half-sweep is non-decreasing (trace of all starts)."""
    w = vpgen.config(1)
    cat = catalog(w.topo)
    D = demand_for(1)
    s = cat.plan(D, w.row_bytes, trace_cap=200_000)
    tr = s["trace"]
    assert len(tr) > 0
    for key, grp in itertools.groupby(tr.tolist(), key=lambda e: (e[0], e[1], e[2])):
        vals = [e[4] for e in grp]
        assert all(b >= a for a, b in zip(vals, vals[1:])), key


def credits_table(D_rem, tau, unit, bw):
    cap = max(unit, (tau * bw) // unit * unit)
    return np.minimum(D_rem, cap)


@pytest.mark.parametrize("cid", [1, 2])
def test_every_aa_result_is_locally_optimal(cid):
    """Each emitted binding is a fixed point of both AA halves: for every group,
    no reassignment of its ranks to its instances (scipy's assignment solver,
    self pairs forbidden) has a higher credit sum than the chosen one."""
    w = vpgen.config(cid)
    cat = catalog(w.topo)
    tm = TopoModel(w.topo)
    D = demand_for(cid)
    s = cat.plan(D, w.row_bytes, i_aa=10_000)
    bw_of = cat.table()["bw"]
    N, g = tm.N, tm.g
    D_rem = D.copy()
    for k in range(s["K"]):
        pi = s["dst"][k]
        bw = bw_of[s["inst"][k]]
        for side in (0, 1):
            for grp in range(tm.G):
                ranks = list(range(grp * g, grp * g + g))
                if side == 0:
                    lanes = ranks                                   # out-lanes of grp
                else:
                    lanes = [i for i in range(N) if pi[i] // g == grp]   # in-lanes of grp
                W = np.full((g, g), -10**18, dtype=np.float64)
                cur = 0
                for m, i in enumerate(lanes):
                    cur += min(D_rem[i, pi[i]], max(w.row_bytes, s["tau"] * bw[i] // w.row_bytes * w.row_bytes))
                    for c, r in enumerate(ranks):
                        src, dst = (r, pi[i]) if side == 0 else (i, r)
                        if src != dst:
                            W[m, c] = credits_table(D_rem[src, dst], s["tau"], w.row_bytes, bw[i])
                rows, cols = linear_sum_assignment(W, maximize=True)
                best = W[rows, cols].sum()
                assert best == cur, (k, side, grp)
        D_rem[np.arange(N), pi] -= s["bytes"][k]
    assert (D_rem == 0).all()


def test_exact_utility_order_matches_fractions():
    """P11: the planner's cross-multiplied comparison of Eq. (10) agrees with
    exact rationals, including near ties and ties."""
    rng = np.random.default_rng(1)
    rates = [32, 25, 7, 64]
    cases = []
    for _ in range(3000):
        S1, S2 = (int(v) for v in rng.integers(0, 10**9, 2))
        x1, x2 = (int(v) for v in rng.integers(1, 10**8, 2))
        b1, b2 = rng.choice(rates, 2)
        lam = int(rng.choice([0, 1, 10_000, 10**7]))
        cases.append((S1, x1, int(b1), S2, x2, int(b2), lam))
    # exact ties and near ties
    cases += [(640, 64, 32, 500, 50, 25, 10_000), (800, 64, 32, 800, 50, 25, 0),
              (10**12, 10**8, 32, 10**12 + 1, 10**8, 32, 5), (0, 0, 32, 1, 1, 25, 0)]
    for S1, x1, b1, S2, x2, b2, lam in cases:
        if S1 > 0:
            x1 = max(x1, 1)
        u1 = utility(S1, [(x1, b1)], lam)
        u2 = utility(S2, [(x2, b2)], lam)
        assert oracle.utility_greater(S1, x1, b1, S2, x2, b2, lam) == (u1 > u2)


def test_empty_demand_gives_empty_schedule():
    topo = vpgen.config(1).topo
    s = catalog(topo).plan(np.zeros((8, 8), np.int64), 4096)
    assert s["K"] == 0


def test_single_pair_uses_fastest_path_in_one_activation():
    """P12: one non-zero entry between two switches of one socket, drained in a
    single quantum (K_target = 1), goes over PXB (32 B/ns beats NIC's 25), and
    T = lambda + D/32 is optimal."""
    topo = vpgen.config(1).topo
    cat = catalog(topo)
    tm = TopoModel(topo)
    unit = 4096
    D = np.zeros((8, 8), np.int64)
    D[0, 3] = 24 * unit          # rank 0 (switch 0) -> rank 3 (switch 1), same socket
    s = cat.plan(D, unit, k_target=1)
    assert s["K"] == 1
    ct = cls_table(cat)
    assert ct[s["inst"][0][0]] == PXB and s["dst"][0][0] == 3
    T = modeled_time(tm, s, ct, 10_000)
    assert T == 10_000 + Fraction(24 * unit, 32)


def test_channel_shaped_demand_takes_one_activation():
    """P12: a demand equal to one feasible channel's pattern with entries at
    most one quantum's capacity is served by exactly one activation."""
    topo = vpgen.tiny_topology()
    cat = catalog(topo)
    unit = 4096
    D = np.zeros((4, 4), np.int64)
    for i, j in [(0, 1), (1, 0), (2, 3), (3, 2)]:      # all PIX lanes
        D[i, j] = 8 * unit
    s = cat.plan(D, unit, k_target=1)
    assert s["K"] == 1


def tiny_demands():
    rng = np.random.default_rng(7)
    pairs = [(i, j) for i in range(4) for j in range(4) if i != j]
    out = []
    for _ in range(6):
        D = np.zeros((4, 4), np.int64)
        for p in rng.choice(len(pairs), 3, replace=False):
            i, j = pairs[p]
            D[i, j] = int(rng.integers(1, 3))
        out.append(D)
    return out


@pytest.mark.parametrize("lam", [200, 10_000])
def test_exhaustive_optimum_bounds_the_planner(lam):
    """P13: on the tiny topology the exhaustive minimum T* (Dijkstra over
    residual demands, every feasible channel, every integer lane volume) is
    never above the planner's T; the single-pair case meets it exactly."""
    topo = vpgen.tiny_topology()
    cat = catalog(topo)
    tm = TopoModel(topo)
    ct = cls_table(cat)
    unit = 4096
    ratios = []
    for Du in tiny_demands():
        s = cat.plan(Du * unit, unit, lambda_ns=lam)
        T = modeled_time(tm, s, ct, lam)
        Tstar = exhaustive_makespan(tm, Du, unit, lam)
        assert T >= Tstar
        ratios.append(float(Tstar / T))
    one = np.zeros((4, 4), np.int64)
    one[0, 2] = 2
    s = cat.plan(one * unit, unit, lambda_ns=lam, k_target=1)
    assert modeled_time(tm, s, ct, lam) == exhaustive_makespan(tm, one, unit, lam)
    assert min(ratios) > 0


def test_uniform_single_switch_closed_form():
    """P14: one switch of 4 GPUs (every lane PIX), D = c (J - I) units:
    T* = (N - 1)(lambda + c unit / bw), attained by the N-1 cyclic shifts.  The
    exhaustive solver must reproduce it and the planner may not beat it."""
    topo = vpgen.Topology(1, sockets_per_node=1, switches_per_socket=1, gpus_per_switch=4)
    cat = catalog(topo)
    tm = TopoModel(topo)
    unit, lam, c = 4096, 500, 1
    Du = c * (np.ones((4, 4), np.int64) - np.eye(4, dtype=np.int64))
    closed = 3 * (lam + Fraction(c * unit, 32))
    assert exhaustive_makespan(tm, Du, unit, lam) == closed
    s = cat.plan(Du * unit, unit, lambda_ns=lam, k_target=1)
    T = modeled_time(tm, s, cls_table(cat), lam)
    assert T >= closed
    assert T == closed      # one quantum per pair: the planner finds the three shifts


def test_invalid_demands_are_rejected():
    topo = vpgen.config(1).topo
    cat = catalog(topo)
    D = np.zeros((8, 8), np.int64)
    D[1, 1] = 4096
    assert cat.plan(D, 4096, check=False)["status"] == oracle.INVALID_DEMAND
    D[1, 1] = 0
    D[1, 2] = 100
    assert cat.plan(D, 4096, check=False)["status"] == oracle.INVALID_DEMAND
    D[1, 2] = -4096
    assert cat.plan(D, 4096, check=False)["status"] == oracle.INVALID_DEMAND


def test_capacity_limit_is_reported():
    w = vpgen.config(1)
    cat = catalog(w.topo)
    D = demand_for(1)
    s = cat.plan(D, w.row_bytes, k_max=3, check=False)
    assert s["status"] == oracle.CAPACITY and s["K"] == 3


def _both_validators(tm, D, dst, cls, nb):
    """(lane checker verdict, vectorised checker verdict): True when valid."""
    res = []
    sched = {"K": dst.shape[0], "dst": dst, "inst": cls, "bytes": nb}
    for f in (lambda: schedule_valid(tm, D, sched, np.arange(4)),
              lambda: schedule_valid_np(tm, D, dst, cls, nb)):
        try:
            f()
            res.append(True)
        except AssertionError:
            res.append(False)
    return tuple(res)


@pytest.mark.parametrize("cid", [1, 2, 4])
def test_vectorised_validity_agrees_with_the_lane_checker(cid):
    """The vectorised validity check used at 1,024 ranks accepts what the
    per-lane checker accepts and rejects the same planted faults: a lane
    class foreign to its group pair, two NIC lanes out of one switch in one
    step (Eq. (1)), a rank that sends to itself, a byte moved between pairs."""
    w = vpgen.config(cid)
    cat = catalog(w.topo)
    tm = TopoModel(w.topo)
    D = demand_for(cid)
    s = cat.plan(D, w.row_bytes)
    dst, nb = s["dst"].copy(), s["bytes"].copy()
    cls = cls_table(cat)[s["inst"]].astype(np.int64)
    assert _both_validators(tm, D, dst, cls, nb) == (True, True)
    g = w.topo.gpus_per_switch
    rows = np.arange(w.n_ranks)
    # a lane inside one switch labelled NIC
    k, i = np.argwhere(cls == PIX)[0]
    c2 = cls.copy()
    c2[k, i] = NIC
    assert _both_validators(tm, D, dst, c2, nb) == (False, False)
    # two lanes leaving one switch for other switches, both on the NIC
    for k in range(s["K"]):
        out = np.flatnonzero(dst[k] // g != rows // g)
        grp = out // g
        dup = [x for x in out if (grp == x // g).sum() >= 2]
        if len(dup) >= 2:
            c3 = cls.copy()
            c3[k, dup[:2]] = NIC
            pair_ok = all(tm.classes(int(x) // g, int(dst[k, x]) // g).count(NIC) for x in dup[:2])
            if pair_ok:
                assert _both_validators(tm, D, dst, c3, nb) == (False, False)
                break
    else:
        pytest.fail("no step with two lanes leaving one switch")
    # rank 0 and rank j = pi(0) swap destinations: rank j now sends to itself
    d4 = dst.copy()
    j = int(dst[0, 0])
    d4[0, 0], d4[0, j] = dst[0, j], j
    assert _both_validators(tm, D, d4, cls, nb) == (False, False)
    # one byte moved from one lane to another
    n5 = nb.copy()
    k, i = np.argwhere(n5 > 0)[0]
    n5[k, i] -= 1
    n5[k, (i + 1) % w.n_ranks] += 1
    assert _both_validators(tm, D, dst, cls, n5) == (False, False)


# ------------------------------------ extra demands and restricted catalogs

import extra_cases  # noqa: E402


@pytest.mark.parametrize("nearest", [False, True])
@pytest.mark.parametrize("name", extra_cases.NAMES)
def test_extra_demands_plan_valid(name, nearest):
    """P1-P3 on the uniform, skew and head/context demands, with the full and
    the nearest-path catalogs; with the latter every lane takes its pair's
    nearest path."""
    case = vpgen.extra(name)
    tm = TopoModel(case.topo)
    cat = oracle.Catalog(case.topo, nearest=nearest)
    D = extra_cases.oracle_demand(case, 0)
    s = cat.plan(D, case.unit)
    schedule_valid(tm, D, s, cat.table()["cls"])
    assert 0 < s["K"] <= 8 * case.topo.n_ranks
    assert (s["bytes"].sum(axis=1) > 0).all()
    if nearest:
        cls = cat.table()["cls"]
        g = case.topo.gpus_per_switch
        for k in range(s["K"]):
            for i in range(case.topo.n_ranks):
                assert cls[s["inst"][k][i]] == tm.nearest_class(i // g, s["dst"][k][i] // g)


def test_head_context_demand_is_block_diagonal():
    """Wan2.1 H4C2: ranks exchange only inside their group of four; each
    pair moves 9450 tokens x 10 heads x 256 B."""
    case = vpgen.extra("wan21-H4C2")
    D = extra_cases.oracle_demand(case)
    want = np.zeros((8, 8), np.int64)
    for b in (0, 4):
        want[b:b + 4, b:b + 4] = 9450 * 10 * 256
    np.fill_diagonal(want, 0)
    assert np.array_equal(D, want)
