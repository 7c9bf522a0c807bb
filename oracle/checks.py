"""Independent Python checkers that pin the oracle.

TEST INFRASTRUCTURE ONLY.  Nothing here calls the C++ oracle's internals:
each checker restates a property the paper fixes (channel feasibility
Eq. (1), balance Eq. (3), family compatibility Eq. (4), schedule validity,
the modeled completion time Eq. (2)) from an independent model of the
topology written directly in Python, or computes a reference result by
brute force on tiny inputs.

Topology model (restated independently): rank = ((node*S + socket)*W +
switch)*g + local; a rank group is one switch.  Directed shared resources:
UP/DN of each switch's root-complex link, TX/RX of each switch's NIC.  Paths:
PIX (same switch, no shared resource), PXB (same socket, different switch:
UP(src switch), DN(dst switch)), NIC (TX(src switch), RX(dst switch)) and,
when the topology enables cross-socket peer to peer, SYS (other socket of the
same node: UP(src switch), the directed link between the two sockets,
DN(dst switch)).  The endpoint GPU<->switch links are added as ("GU", rank) /
("GD", rank) when a cluster-level footprint is needed.
"""
from __future__ import annotations

import heapq
import itertools
from fractions import Fraction
from typing import Dict, List, Tuple

import numpy as np

PIX, PXB, NIC, SYS = 0, 1, 2, 3


class TopoModel:
    def __init__(self, topo):
        self.nn = topo.n_nodes
        self.S = topo.sockets_per_node
        self.W = topo.switches_per_socket
        self.g = topo.gpus_per_switch
        self.Q = self.S * self.W
        self.G = self.nn * self.Q
        self.N = self.G * self.g
        self.pcie = topo.pcie_bytes_per_ns
        self.nic = topo.nic_bytes_per_ns
        self.sys = bool(getattr(topo, "flags", 0) & 1)
        self.m = getattr(topo, "nics_per_switch", 1)   # NICs per switch, every GPU of it reaches each

    def group(self, rank: int) -> int:
        return rank // self.g

    def node(self, group: int) -> int:
        return group // self.Q

    def socket(self, group: int) -> int:
        return (group % self.Q) // self.W

    def classes(self, a: int, d: int) -> List[int]:
        """Path classes between group a and group d, before dominance pruning."""
        out = []
        if a == d:
            out.append(PIX)
        elif self.node(a) == self.node(d) and self.socket(a) == self.socket(d):
            out.append(PXB)
        elif self.node(a) == self.node(d) and self.sys:
            out.append(SYS)
        out.append(NIC)
        return out

    def unpruned_classes(self, a: int, d: int) -> List[int]:
        """Classes that survive dominance: NIC inside one switch is dominated by PIX."""
        return [c for c in self.classes(a, d) if not (a == d and c == NIC)]

    def nearest_class(self, a: int, d: int) -> int:
        """The one path a pair keeps under "fixed nearest path": the switch
        itself, else the socket's root complex, else the NICs."""
        return self.classes(a, d)[0]

    def rate(self, cls: int) -> int:
        return min(self.pcie, self.nic) if cls == NIC else self.pcie

    def shared(self, cls: int, a: int, d: int) -> Tuple:
        if cls == PIX:
            return ()
        if cls == PXB:
            return (("UP", a), ("DN", d))
        if cls == SYS:
            return (("UP", a), ("X", self.node(a), self.socket(a), self.socket(d)), ("DN", d))
        return (("TX", a), ("RX", d))

    def footprint(self, cls: int, i: int, j: int) -> Tuple:
        """Cluster-level footprint including the endpoint GPU<->switch links."""
        a, d = self.group(i), self.group(j)
        return self.shared(cls, a, d) + (("GU", i), ("GD", j))


def channel_feasible(tm: TopoModel, pi: List[int], cls: List[int]) -> bool:
    """Eq. (1) over shared resources plus the endpoint links (no repeats)."""
    seen = set()
    for i, (j, c) in enumerate(zip(pi, cls)):
        if j == i:
            return False
        for r in tm.footprint(c, i, j):
            if r in seen:
                return False
            seen.add(r)
    return True


def brute_force_channels(tm: TopoModel, nearest: bool = False) -> set:
    """Every feasible rank-level channel (pi, path classes) using unpruned
    paths, or with nearest=True only each pair's nearest path."""
    N = tm.N
    out = set()
    for pi in itertools.permutations(range(N)):
        if any(pi[i] == i for i in range(N)):
            continue
        if nearest:
            options = [[tm.nearest_class(tm.group(i), tm.group(pi[i]))] for i in range(N)]
        else:
            options = [tm.unpruned_classes(tm.group(i), tm.group(pi[i])) for i in range(N)]
        # incremental resource check per lane
        def rec(i, used, cls):
            if i == N:
                out.add((pi, tuple(cls)))
                return
            for c in options[i]:
                fp = tm.shared(c, tm.group(i), tm.group(pi[i]))
                if any(r in used for r in fp):
                    continue
                rec(i + 1, used | set(fp), cls + [c])
        rec(0, frozenset(), [])
    return out


def instantiate(tm: TopoModel, fam: Dict[str, np.ndarray]) -> set:
    """All endpoint bindings of one cluster-level family (self pairs excluded)."""
    g, G = tm.g, tm.G
    n = len(fam["cls"])
    outs = [[t for t in range(n) if fam["a"][t] == x] for x in range(G)]
    ins = [[t for t in range(n) if fam["d"][t] == x] for x in range(G)]
    perms = list(itertools.permutations(range(g)))
    res = set()
    for sp in itertools.product(perms, repeat=G):
        src = [0] * n
        for x in range(G):
            for m, t in enumerate(outs[x]):
                src[t] = x * g + sp[x][m]
        for dp in itertools.product(perms, repeat=G):
            dst = [0] * n
            for x in range(G):
                for m, t in enumerate(ins[x]):
                    dst[t] = x * g + dp[x][m]
            if any(src[t] == dst[t] for t in range(n)):
                continue
            pi = [0] * tm.N
            cl = [0] * tm.N
            for t in range(n):
                pi[src[t]] = dst[t]
                cl[src[t]] = int(fam["cls"][t])
            res.add((tuple(pi), tuple(cl)))
    return res


# ----------------------------------------------- several NICs per switch
#
# With m NICs per switch a NIC path is labelled by the NIC it leaves through
# and the NIC it arrives at: footprint TX of (source group, x) and RX of
# (destination group, y).  A path label is (class, x, y), x = y = -1 for the
# other classes.  Renaming the NICs of a group (a permutation per group,
# applied to the source NIC of lanes leaving it and to the destination NIC
# of lanes entering it) maps valid channels to valid channels.

def path_labels(tm: TopoModel, a: int, d: int) -> List[Tuple[int, int, int]]:
    out = []
    for c in tm.unpruned_classes(a, d):
        if c == NIC:
            out += [(NIC, x, y) for x in range(tm.m) for y in range(tm.m)]
        else:
            out.append((c, -1, -1))
    return out


def shared_labeled(tm: TopoModel, lab, a: int, d: int) -> Tuple:
    c, x, y = lab
    if c == NIC:
        return (("TX", a, x), ("RX", d, y))
    return tm.shared(c, a, d)


def brute_force_labeled(tm: TopoModel) -> set:
    """Every feasible rank-level channel (pi, path label per rank) by brute
    force over derangements and labelled path vectors (Eq. (1))."""
    N = tm.N
    out = set()
    for pi in itertools.permutations(range(N)):
        if any(pi[i] == i for i in range(N)):
            continue
        options = [path_labels(tm, tm.group(i), tm.group(pi[i])) for i in range(N)]

        def rec(i, used, labs):
            if i == N:
                out.add((pi, tuple(labs)))
                return
            for lab in options[i]:
                fp = shared_labeled(tm, lab, tm.group(i), tm.group(pi[i]))
                if any(r in used for r in fp):
                    continue
                rec(i + 1, used | set(fp), labs + [lab])
        rec(0, frozenset(), [])
    return out


def canonical_labeled(tm: TopoModel, ch) -> Tuple:
    """The smallest renaming of a labelled channel over all per-group NIC
    permutations."""
    pi, labs = ch
    best = None
    perms = list(itertools.permutations(range(tm.m)))
    for sig in itertools.product(perms, repeat=tm.G):
        img = []
        for i, (c, x, y) in enumerate(labs):
            if c == NIC:
                img.append((c, sig[tm.group(i)][x], sig[tm.group(pi[i])][y]))
            else:
                img.append((c, x, y))
        img = (pi, tuple(img))
        if best is None or img < best:
            best = img
    return best


def instantiate_labeled(tm: TopoModel, fam: Dict[str, np.ndarray], labels) -> set:
    """All endpoint bindings of one cluster-level family whose instance t has
    path label labels[t] (self pairs excluded): (pi, label per rank)."""
    g, G = tm.g, tm.G
    n = len(fam["cls"])
    outs = [[t for t in range(n) if fam["a"][t] == x] for x in range(G)]
    ins = [[t for t in range(n) if fam["d"][t] == x] for x in range(G)]
    perms = list(itertools.permutations(range(g)))
    res = set()
    for sp in itertools.product(perms, repeat=G):
        src = [0] * n
        for x in range(G):
            for m, t in enumerate(outs[x]):
                src[t] = x * g + sp[x][m]
        for dp in itertools.product(perms, repeat=G):
            dst = [0] * n
            for x in range(G):
                for m, t in enumerate(ins[x]):
                    dst[t] = x * g + dp[x][m]
            if any(src[t] == dst[t] for t in range(n)):
                continue
            pi = [0] * tm.N
            lab = [None] * tm.N
            for t in range(n):
                pi[src[t]] = dst[t]
                lab[src[t]] = labels[t]
            res.add((tuple(pi), tuple(lab)))
    return res


def schedule_valid(tm: TopoModel, D: np.ndarray, sched, cls_of_id) -> None:
    """Raise AssertionError unless the schedule is valid (Sec. 3 'Schedule validity')."""
    N = tm.N
    X = np.zeros((N, N), dtype=np.int64)
    for k in range(sched["K"]):
        pi = [int(x) for x in sched["dst"][k]]
        cls = [int(cls_of_id[int(x)]) for x in sched["inst"][k]]
        assert sorted(pi) == list(range(N)), "not a permutation"
        for i in range(N):
            assert cls[i] in tm.unpruned_classes(tm.group(i), tm.group(pi[i])), \
                "lane class does not match its group pair"
        assert channel_feasible(tm, pi, cls), "activation violates Eq. (1)"
        x = np.asarray(sched["bytes"][k], dtype=np.int64)
        assert (x >= 0).all()
        X[np.arange(N), pi] += x
    assert (X == D).all(), "activations do not reconstruct D"


def schedule_valid_np(tm: TopoModel, D: np.ndarray, dst: np.ndarray, cls: np.ndarray, nbytes: np.ndarray,
                      chunk: int = 256) -> None:
    """The checks of schedule_valid, vectorised for large schedules: every
    step is a derangement, every lane's path class is one its group pair
    has (before dominance pruning, NIC inside a switch excluded), no two
    lanes of a step share a modeled resource (Eq. (1); the endpoint links are
    distinct in any permutation), volumes are non-negative and the steps sum
    to D.  dst, cls, nbytes: [K, N] destination, path class, bytes."""
    dst = np.asarray(dst, np.int64)
    cls = np.asarray(cls, np.int64)
    nb = np.asarray(nbytes, np.int64)
    K, N = dst.shape
    assert N == tm.N
    rows = np.arange(N)
    assert (np.sort(dst, axis=1) == rows[None, :]).all(), "not a permutation"
    assert not (dst == rows[None, :]).any(), "a rank sends to itself"
    assert (nb >= 0).all()
    a = np.broadcast_to(rows // tm.g, (K, N))
    d = dst // tm.g
    same_group = a == d
    same_node = a // tm.Q == d // tm.Q
    sa, sd = (a % tm.Q) // tm.W, (d % tm.Q) // tm.W
    same_socket = same_node & (sa == sd)
    ok = np.where(same_group, cls == PIX,
                  np.where(same_socket, (cls == PXB) | (cls == NIC),
                           np.where(same_node & tm.sys, (cls == SYS) | (cls == NIC), cls == NIC)))
    assert ok.all(), "lane class does not match its group pair"
    G = tm.G
    xid = (a // tm.Q * tm.S + sa) * tm.S + sd
    res = np.full((K, N, 3), -1, np.int64)
    pxb_like = (cls == PXB) | (cls == SYS)
    res[..., 0] = np.where(pxb_like, a, np.where(cls == NIC, 2 * G + a, -1))
    res[..., 1] = np.where(pxb_like, G + d, np.where(cls == NIC, 3 * G + d, -1))
    res[..., 2] = np.where(cls == SYS, 4 * G + xid, -1)
    # unused slots get distinct negative ids so that they never collide
    filler = -1 - np.arange(N * 3, dtype=np.int64).reshape(N, 3)
    res = np.where(res < 0, filler[None], res).reshape(K, N * 3)
    for k0 in range(0, K, chunk):
        r = np.sort(res[k0:k0 + chunk], axis=1)
        assert not (r[:, 1:] == r[:, :-1]).any(), "activation violates Eq. (1)"
    X = np.zeros((N, N), np.int64)
    np.add.at(X, (np.broadcast_to(rows, (K, N)), dst), nb)
    assert (X == np.asarray(D, np.int64)).all(), "activations do not reconstruct D"


def modeled_time(tm: TopoModel, sched, cls_of_id, lam: int) -> Fraction:
    """Eq. (2) with exact rationals."""
    total = Fraction(0)
    for k in range(sched["K"]):
        worst = Fraction(0)
        for i in range(tm.N):
            x = int(sched["bytes"][k][i])
            b = tm.rate(int(cls_of_id[int(sched["inst"][k][i])]))
            worst = max(worst, Fraction(x, b))
        total += lam + worst
    return total


def utility(S: int, lanes: List[Tuple[int, int]], lam: int) -> Fraction:
    """Eq. (10): S / (lambda + max_i x_i / b_i); zero when S = 0."""
    if S == 0:
        return Fraction(0)
    return Fraction(S) / (lam + max(Fraction(x, b) for x, b in lanes))


def exhaustive_makespan(tm: TopoModel, D_units: np.ndarray, unit: int, lam: int) -> Fraction:
    """Minimum modeled completion time over all valid schedules (tiny inputs).

    Dijkstra over residual-demand states; an edge is one feasible rank-level
    channel with any integer lane volumes (0..residual, in units) costing
    lambda + max_i x_i / bw_i.  Zero-volume activations are never useful.
    """
    N = tm.N
    chans = sorted(brute_force_channels(tm))
    start = tuple(int(v) for v in D_units.reshape(-1))
    best = {start: Fraction(0)}
    heap = [(Fraction(0), start)]
    while heap:
        cost, st = heapq.heappop(heap)
        if best.get(st, None) != cost:
            continue
        if not any(st):
            return cost
        R = np.array(st, dtype=np.int64).reshape(N, N)
        seen_moves = set()
        for pi, cl in chans:
            lanes = [(i, pi[i], cl[i]) for i in range(N) if R[i, pi[i]] > 0]
            if not lanes:
                continue
            ranges = [range(0, int(R[i, j]) + 1) for i, j, _ in lanes]
            for xs in itertools.product(*ranges):
                if not any(xs):
                    continue
                key = tuple(sorted((i, j, c, x) for (i, j, c), x in zip(lanes, xs) if x))
                if key in seen_moves:
                    continue
                seen_moves.add(key)
                dur = max(Fraction(x * unit, tm.rate(c)) for (i, j, c), x in zip(lanes, xs) if x)
                nst = list(st)
                for (i, j, c), x in zip(lanes, xs):
                    nst[i * N + j] -= x
                nst = tuple(nst)
                nc = cost + lam + dur
                if nc < best.get(nst, None) if nst in best else True:
                    best[nst] = nc
                    heapq.heappush(heap, (nc, nst))
    raise RuntimeError("unreachable")
