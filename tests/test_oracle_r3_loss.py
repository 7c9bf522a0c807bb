"""What the node-circulant catalog (reading R3) costs against the full Alg. 1
catalog (Sec. 4.1), on topologies small enough for both: the oracle plans the
same demands with each and the modeled completion time T-hat (Eq. (2)) is
compared.  The full catalog holds every feasible family, the circulant one
only families that repeat one node-local pattern in every node, so the
circulant plan can be slower; the planner is a heuristic, so it is not slower
on every matrix.  The test prints the ratios and bounds their mean."""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import vpgen

UNIT = 4096


def demands(N, kind, rng, n):
    out = []
    while len(out) < n:
        if kind == "uniform":
            D = np.full((N, N), 16, np.int64)
        elif kind == "dense":
            D = rng.integers(0, 40, (N, N))
        elif kind == "sparse":
            D = rng.integers(0, 40, (N, N)) * (rng.random((N, N)) < 0.3)
        else:   # two hot destinations
            D = rng.integers(0, 4, (N, N))
            D[:, rng.choice(N, 2, replace=False)] += rng.integers(20, 60, (N, 2))
        D = D.astype(np.int64) * UNIT
        np.fill_diagonal(D, 0)
        if D.sum():
            out.append(D)
    return out


@pytest.mark.parametrize("shape", [(2, 1, 2, 2), (2, 2, 1, 2), (3, 1, 2, 2)])
def test_circulant_catalog_cost_in_modeled_time(shape):
    topo = vpgen.Topology(*shape)
    full, circ = oracle.Catalog(topo, full=True), oracle.Catalog(topo)
    assert circ.n_families < full.n_families
    N = topo.n_ranks
    rng = np.random.default_rng(3)
    all_r = []
    for kind in ("uniform", "dense", "sparse", "hot"):
        r = []
        for D in demands(N, kind, rng, 4):
            tf = Fraction(*full.modeled_time(full.plan(D, UNIT, k_max=64 * N)))
            tc = Fraction(*circ.modeled_time(circ.plan(D, UNIT, k_max=64 * N)))
            r.append(float(tc / tf))
        print("%s %-8s circulant/full T-hat: mean %.3f, %.3f-%.3f (families %d of %d)"
              % (shape, kind, np.mean(r), min(r), max(r), circ.n_families, full.n_families))
        all_r += r
    # the circulant plan stays within a quarter of the full one on average
    assert 0.9 < np.mean(all_r) < 1.25
