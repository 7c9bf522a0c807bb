"""Pins of the oracle's fixed-rotation model (Sec. 6.3 peer/path ablation,
Table 3 "fixed peer rotation"): hand-worked stage times with shared links,
the contention-free single-switch closed form, and the order of the two path
rules."""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import vpgen

LAM = oracle.DEFAULT_LAMBDA_NS


def T(topo, D, nearest, lam=LAM):
    n, d = oracle.rotation_time(topo, D, nearest, lam)
    return Fraction(n, d)


def test_tiny_topology_uniform_by_hand():
    """Ranks 0,1 on switch 0 and 2,3 on switch 1 of one socket, c bytes per
    pair.  Shifts 1 and 3: two PIX lanes and one cross lane each way, no
    sharing: c/32.  Shift 2: two lanes each way between the switches; on
    nearest paths both take the same uplink and downlink (rate 16 each): c/16;
    with a path choice one goes through the NICs (25): c/25."""
    c = 3 << 20
    D = np.full((4, 4), c, np.int64)
    np.fill_diagonal(D, 0)
    topo = vpgen.tiny_topology()
    assert T(topo, D, True) == 3 * LAM + Fraction(c, 32) + Fraction(c, 16) + Fraction(c, 32)
    assert T(topo, D, False) == 3 * LAM + Fraction(c, 32) + Fraction(c, 25) + Fraction(c, 32)


def test_single_switch_closed_form():
    """One switch of four GPUs: every lane is PIX, nothing is shared:
    (N - 1)(lambda + c / 32), the uniform optimum as well."""
    topo = vpgen.Topology(1, 1, 1, 4)
    c = 1 << 22
    D = np.full((4, 4), c, np.int64)
    np.fill_diagonal(D, 0)
    for near in (True, False):
        assert T(topo, D, near) == 3 * (LAM + Fraction(c, 32))


def test_empty_stages_are_skipped():
    topo = vpgen.tiny_topology()
    D = np.zeros((4, 4), np.int64)
    D[0, 2] = 64 << 10           # only shift 2 carries bytes: one PXB lane
    assert T(topo, D, True) == LAM + Fraction(64 << 10, 32)
    assert T(topo, np.zeros((4, 4), np.int64), False) == 0


def test_cross_socket_lanes_share_the_nic():
    """Ranks 0,1 (switch 0, socket 0) to ranks 4,5 (switch 2, socket 1) in one
    stage: both lanes need switch 0's NIC: 25 / 2 each."""
    topo = vpgen.config(1).topo
    D = np.zeros((8, 8), np.int64)
    D[0, 4] = D[1, 5] = 1 << 20
    for near in (True, False):
        assert T(topo, D, near) == LAM + Fraction(2 << 20, 25)


@pytest.mark.parametrize("cid", [1, 2])
def test_dynamic_paths_never_slower(cid):
    w = vpgen.config(cid)
    R = vpgen.routing_all(w, 0, 256)
    D = np.stack([oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes)["row"] for i in range(w.n_ranks)])
    assert T(w.topo, D, False) <= T(w.topo, D, True)


def test_sys_rotation_by_hand():
    """Two sockets, one switch of two GPUs each, c bytes per pair.  Shift 2
    sends both GPUs of a switch to the other socket: on nearest (SYS) paths
    the two lanes share the uplink, the socket link and the downlink (16 each:
    c/16); with a path choice one lane takes the NICs (25): c/25.  Shifts 1
    and 3 have one cross lane each way: c/32."""
    topo = vpgen.Topology(1, 2, 1, 2, flags=oracle.TOPO_SYS_P2P)
    c = 5 << 20
    D = np.full((4, 4), c, np.int64)
    np.fill_diagonal(D, 0)
    assert T(topo, D, True) == 3 * LAM + Fraction(c, 32) * 2 + Fraction(c, 16)
    assert T(topo, D, False) == 3 * LAM + Fraction(c, 32) * 2 + Fraction(c, 25)
    # without peer to peer every cross lane is a NIC lane: shift 2 shares
    # the NIC (12.5 each), shifts 1 and 3 have one NIC lane each way (25)
    topo0 = vpgen.Topology(1, 2, 1, 2)
    assert T(topo0, D, False) == 3 * LAM + Fraction(c, 25) * 2 + Fraction(2 * c, 25)
