"""The stored stream digests agree with the oracle as it stands: the demand
and schedule digests of the first and last matrix of the 64-rank stream and of
the first matrix of the 256-rank stream (also on SYS nodes) are recomputed
here (the full streams and the send-buffer digests are rebuilt by
golden/make_stream_digests.py)."""
import json

import numpy as np
import pytest

import oracle
import stream_digest as sd
import vpgen


@pytest.fixture(scope="module")
def golden():
    with open(sd.GOLDEN) as f:
        return json.load(f)


def test_streams_cover_the_checked_matrices(golden):
    for cid, mats in sd.STREAMS.items():
        rows = golden["streams"][str(cid)]["matrices"]
        assert [r["matrix"] for r in rows] == mats
        assert golden["streams"][str(cid)]["workload"] == vpgen.config(cid).name
        # the plan drains every matrix in at least N - 1 steps and within K_max = 8N
        N = vpgen.config(cid).n_ranks
        assert all(N - 1 <= r["K"] <= 8 * N for r in rows)


@pytest.mark.parametrize("cid,m", [(3, 0), (3, 99), (5, 0)])
def test_stream_digest_matches_oracle(golden, cid, m):
    w = vpgen.config(cid)
    ref = {r["matrix"]: r for r in golden["streams"][str(cid)]["matrices"]}[m]
    R = vpgen.routing_all(w, m)
    D = np.stack([oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes)["row"] for i in range(w.n_ranks)])
    assert sd.demand_digest(D) == ref["demand"]
    s = oracle.Catalog(w.topo).plan(D, w.row_bytes)
    assert s["K"] == ref["K"] and s["tau"] == ref["tau"]
    assert sd.schedule_digest(s) == ref["schedule"]
    assert int(s["bytes"][:, 0].sum()) == ref["send_bytes"]


def test_full_256_stream_digests_agree_with_the_subset(golden):
    """The digests of all 1000 matrices of the 256-rank stream (written by
    the same script from the oracle) repeat the subset's digests exactly."""
    import os
    if not os.path.exists(sd.GOLDEN_ALL5):
        pytest.skip("no full-stream digests")
    with open(sd.GOLDEN_ALL5) as f:
        full = {r["matrix"]: r for r in json.load(f)["streams"]["5"]["matrices"]}
    assert sorted(full) == list(range(1000))
    for r in golden["streams"]["5"]["matrices"]:
        assert full[r["matrix"]] == r


def test_sys256_digest_matches_oracle():
    """The stored digest of the 256-rank workload on SYS nodes (the GPU
    parity reference of tests/test_gpu_extra.py) is the oracle's plan as it
    stands (about a minute on one core)."""
    import dataclasses
    with open(sd.GOLDEN_SYS256) as f:
        ref = json.load(f)
    w = vpgen.config(5)
    topo = dataclasses.replace(w.topo, flags=1)
    R = vpgen.routing_all(w, ref["matrix"])
    D = np.stack([oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes)["row"] for i in range(w.n_ranks)])
    assert sd.demand_digest(D) == ref["demand"]
    s = oracle.Catalog(topo).plan(D, w.row_bytes)
    assert (s["K"], s["tau"]) == (ref["K"], ref["tau"])
    assert sd.schedule_digest(s) == ref["schedule"]


def test_ranks1024_digest_is_for_the_generated_demand():
    """The stored 1,024-rank digest (the GPU parity reference of
    tests/test_gpu_parity.py; the oracle's plan takes about ten minutes, so
    only the script recomputes it) names the demand vpgen generates, and a K
    any valid schedule of it can have."""
    with open(sd.GOLDEN_1024) as f:
        ref = json.load(f)
    N = 1024
    D = vpgen.hot_destinations_demand(N, ref["unit"], 1024)
    assert sd.demand_digest(D) == ref["demand"]
    assert ref["k_max"] == 32 * N and N - 1 <= ref["K"] <= ref["k_max"]
