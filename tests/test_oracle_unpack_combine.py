"""Pins of the oracle's receive side and combine direction (Sec. 5 buffer
layout and 128-byte receive slots; the return AlltoAllv of expert
parallelism, planned on the transposed demand).  Every rank of a small
cluster packs, a transfer emulation moves the slices, and the checks are
independent of the oracle's index arithmetic: the expert-major output is
rebuilt with numpy from the routing alone, and a dispatch followed by a
combine with identity experts must hand every token its own row back in
every slot routed off-rank."""
import numpy as np
import pytest

import oracle
import vpgen


def cluster(cid, tokens):
    w = vpgen.config(cid)
    N = w.n_ranks
    R = vpgen.routing_all(w, 0, tokens)
    dem = [oracle.demand(R[i], N, w.experts, i, w.row_bytes) for i in range(N)]
    D = np.stack([d["row"] for d in dem])
    tok = [vpgen.tokens_bf16(w, i, tokens) for i in range(N)]
    counts = np.stack([d["counts"] for d in dem])
    return w, R, dem, D, tok, counts


def dispatch(w, dem, D, tok):
    N = w.n_ranks
    s = oracle.Catalog(w.topo).plan(D, w.row_bytes)
    sends, offs = [], []
    for i in range(N):
        send, off = oracle.pack_rows(tok[i], w.row_bytes, dem[i]["sorted_tok"], dem[i]["dest_off"], i, s)
        sends.append(send)
        offs.append(off)
    return s, sends, offs


@pytest.mark.parametrize("cid,tokens", [(1, 256), (2, 128)])
def test_layout_tiles_every_stream_and_receive_buffer(cid, tokens):
    w, R, dem, D, tok, counts = cluster(cid, tokens)
    N = w.n_ranks
    s = oracle.Catalog(w.topo).plan(D, w.row_bytes)
    lay = oracle.layout(s, N)
    K = s["K"]
    for i in range(N):
        # send offsets: slices of rank i back to back in step order
        x = s["bytes"][:, i]
        assert (lay["send_off"][:, i] == np.concatenate([[0], np.cumsum(x)[:-1]])).all()
    for r in range(N):
        # slices addressed to r tile [0, column sum) without gap or overlap
        spans = sorted((lay["recv_off"][k, i], s["bytes"][k, i]) for k in range(K) for i in range(N)
                       if s["dst"][k, i] == r and s["bytes"][k, i])
        pos = 0
        for o, x in spans:
            assert o == pos
            pos += x
        assert pos == D[:, r].sum()
    for i in range(N):
        for j in range(N):
            # the last slice of every stream ends at the pair's demand
            ks = [k for k in range(K) if s["dst"][k, i] == j and s["bytes"][k, i]]
            if ks:
                assert lay["stream_off"][ks[-1], i] + s["bytes"][ks[-1], i] == D[i, j]


@pytest.mark.parametrize("cid,tokens", [(1, 256), (2, 128)])
def test_unpack_builds_the_expert_major_output(cid, tokens):
    w, R, dem, D, tok, counts = cluster(cid, tokens)
    N, E = w.n_ranks, w.experts
    eloc = E // N
    rb, sb = w.row_bytes, oracle.slot_bytes(w.row_bytes)
    assert sb % 128 == 0
    s, sends, offs = dispatch(w, dem, D, tok)
    for r in range(N):
        recv = oracle.receive(r, N, s, rb, sends, offs)
        out = oracle.unpack_rows(recv, r, N, s, rb, counts)
        # numpy: local expert m's rows from every source in (source, token) order
        rows = out.reshape(-1, sb)[:, :rb]
        o = 0
        for m in range(eloc):
            e = r * eloc + m
            for i in range(N):
                t = np.nonzero((R[i] == e).any(axis=1))[0]
                if i != r:   # rows a rank keeps are not transferred
                    assert (rows[o:o + t.size] == tok[i].view(np.uint8).reshape(-1, rb)[t]).all()
                o += t.size
        assert o == oracle.expert_rows(counts, r, N)


@pytest.mark.parametrize("cid,tokens", [(1, 256), (2, 128)])
def test_dispatch_then_combine_returns_every_row(cid, tokens):
    """Identity experts: the combine, planned on the transposed demand, brings
    each token's row back to every routing slot whose expert is off-rank."""
    w, R, dem, D, tok, counts = cluster(cid, tokens)
    N, E, k = w.n_ranks, w.experts, w.top_k
    eloc = E // N
    rb, sb = w.row_bytes, oracle.slot_bytes(w.row_bytes)
    T = tok[0].shape[0]
    s, sends, offs = dispatch(w, dem, D, tok)
    outs = [oracle.unpack_rows(oracle.receive(r, N, s, rb, sends, offs), r, N, s, rb, counts) for r in range(N)]
    sc = oracle.Catalog(w.topo).plan(np.ascontiguousarray(D.T), rb)
    csends, coffs = [], []
    for r in range(N):
        send, off = oracle.pack_combine(outs[r], r, N, sc, rb, counts)
        assert send.size == max(int(D[:, r].sum()), 1)
        csends.append(send)
        coffs.append(off)
    for i in range(N):
        recv = oracle.receive(i, N, sc, rb, csends, coffs)
        comb = oracle.unpack_combine(recv, i, N, sc, rb, T, k, dem[i]["sorted_tok"], dem[i]["sorted_slot"],
                                     dem[i]["dest_off"]).reshape(T, k, sb)[:, :, :rb]
        remote = (R[i] // eloc) != i
        want = np.broadcast_to(tok[i].view(np.uint8).reshape(T, 1, rb), (T, k, rb))
        assert (comb[remote] == want[remote]).all()
        assert (comb[~remote] == 0).all()
