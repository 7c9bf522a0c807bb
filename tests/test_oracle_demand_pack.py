"""Pins of the oracle's demand build and send-buffer pack against numpy
library routines: bincount for the histogram, cumsum for the offsets, a
stable argsort for the (expert, token) order, and fancy-index / strided
gathers for the pack (Sec. 3 model setup; Sec. 5 buffer layout)."""
import numpy as np
import pytest

import oracle
import vpgen


@pytest.mark.parametrize("cid,tokens", [(1, None), (2, 2048), (3, 1024), (5, 1024)])
def test_demand_matches_numpy(cid, tokens):
    w = vpgen.config(cid)
    N, E = w.n_ranks, w.experts
    eloc = E // N
    for rank in (0, N - 1):
        r = vpgen.routing(w, rank, 0, tokens)
        T, k = r.shape
        out = oracle.demand(r, N, E, rank, w.row_bytes)
        counts = np.bincount(r.ravel(), minlength=E)
        assert (out["counts"] == counts).all()
        per_rank = counts.reshape(N, eloc).sum(1)
        row = per_rank * w.row_bytes
        row[rank] = 0
        assert (out["row"] == row).all()
        assert out["row"].sum() == w.row_bytes * (T * k - per_rank[rank])
        flat = np.argsort(r.ravel(), kind="stable")
        assert (out["sorted_tok"] == flat // k).all()
        assert (out["sorted_slot"] == flat % k).all()
        # every assignment appears exactly once, with the expert it was routed to
        assert (r[out["sorted_tok"], out["sorted_slot"]] == np.sort(r.ravel(), kind="stable")).all()
        assert (out["dest_off"] == np.concatenate([[0], np.cumsum(per_rank)])).all()


def test_demand_rejects_bad_expert_id():
    r = np.zeros((4, 2), np.int32)
    r[2, 1] = 32
    with pytest.raises(oracle.OracleError):
        oracle.demand(r, 8, 32, 0, 4096)


def test_heads_demand_closed_form():
    w = vpgen.config(4)
    hl = vpgen.head_split(w.heads, w.n_ranks)
    for rank in (0, 9):
        row = oracle.demand_heads(w.tokens, hl, w.row_bytes, rank)
        ref = w.tokens * np.diff(hl) * 256
        ref[rank] = 0
        assert (row == ref).all()
        assert set(np.unique(ref[ref > 0])) <= {1 << 20, 3 << 19}


def numpy_rows_pack(tokens, row_bytes, order, dest_off, self_rank, sched):
    """Reference: streams by fancy indexing, slices taken in step order."""
    rows = tokens.reshape(tokens.shape[0], -1).view(np.uint8).reshape(tokens.shape[0], row_bytes)
    streams = {j: rows[order[dest_off[j]:dest_off[j + 1]]].reshape(-1)
               for j in range(len(dest_off) - 1)}
    cursor = {j: 0 for j in streams}
    parts, per_dst = [], {j: [] for j in streams}
    for k in range(sched["K"]):
        x = int(sched["bytes"][k][self_rank])
        if x == 0:
            continue
        j = int(sched["dst"][k][self_rank])
        sl = streams[j][cursor[j]:cursor[j] + x]
        cursor[j] += x
        parts.append(sl)
        per_dst[j].append(sl)
    return (np.concatenate(parts) if parts else np.zeros(0, np.uint8)), streams, per_dst


@pytest.mark.parametrize("cid,tokens", [(1, None), (2, 1024)])
def test_pack_rows_matches_numpy_gather(cid, tokens):
    w = vpgen.config(cid)
    N = w.n_ranks
    R = vpgen.routing_all(w, 0, tokens)
    dem = [oracle.demand(R[i], N, w.experts, i, w.row_bytes) for i in range(N)]
    D = np.stack([d["row"] for d in dem])
    cat = oracle.Catalog(w.topo)
    s = cat.plan(D, w.row_bytes)
    self_rank = 0
    tok = vpgen.tokens_bf16(w, self_rank, tokens)
    send, step_off = oracle.pack_rows(tok, w.row_bytes, dem[0]["sorted_tok"], dem[0]["dest_off"],
                                      self_rank, s)
    ref, streams, per_dst = numpy_rows_pack(tok, w.row_bytes, dem[0]["sorted_tok"],
                                            dem[0]["dest_off"], self_rank, s)
    assert send.size == D[self_rank].sum() == ref.size
    assert (send == ref).all()
    for j in range(N):
        if j != self_rank:
            assert (np.concatenate(per_dst[j]) == streams[j]).all(), "slices do not rebuild stream"
    # step offsets: prefix sums of this rank's lane volumes
    x = s["bytes"][:, self_rank]
    assert (step_off == np.concatenate([[0], np.cumsum(x)])).all()


def test_pack_heads_matches_numpy_strided_slice():
    w = vpgen.config(4)
    N = w.n_ranks
    hl = vpgen.head_split(w.heads, N)
    D = np.stack([oracle.demand_heads(w.tokens, hl, w.row_bytes, i) for i in range(N)])
    cat = oracle.Catalog(w.topo)
    s = cat.plan(D, w.row_bytes)
    for self_rank in (0, 12):
        act = vpgen.tokens_bf16(w, self_rank)
        send, _ = oracle.pack_heads(act, w.token_stride, hl, w.row_bytes, self_rank, s)
        a8 = act.view(np.uint8).reshape(w.tokens, w.heads, w.row_bytes)
        streams = {j: a8[:, hl[j]:hl[j + 1], :].reshape(-1) for j in range(N)}
        cursor = {j: 0 for j in range(N)}
        parts = []
        for k in range(s["K"]):
            x = int(s["bytes"][k][self_rank])
            if x:
                j = int(s["dst"][k][self_rank])
                parts.append(streams[j][cursor[j]:cursor[j] + x])
                cursor[j] += x
        ref = np.concatenate(parts)
        assert send.size == D[self_rank].sum() and (send == ref).all()
        assert all(cursor[j] == streams[j].size for j in range(N) if j != self_rank)
