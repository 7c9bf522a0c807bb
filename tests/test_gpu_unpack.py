"""GPU parity of the receive side and the combine direction against the oracle.

vp_unpack_rows, vp_pack_combine and vp_unpack_combine are compared byte for
byte with the oracle's functions on the same inputs: at full size with the
oracle's schedule uploaded and random buffer contents, and end to end (GPU
demand, plan, pack of every rank, a transfer emulated in the test, unpack,
then the combine back) against the oracle's own pipeline, for the named
workloads and for seeded random shapes.  Error cases:
an inconsistent receive view, buffers too small, a schedule that leaves a
stream incomplete, and the empty schedule."""
import sys

import numpy as np
import pytest
import torch

import oracle
import vpgen

pytestmark = pytest.mark.gpu

_cache = {}


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def vp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_34340_amd as vp
    vp.lib()
    return vp


def case(cid, tokens=None, row_bytes=None):
    """Routing, per-rank oracle demand, D and counts; row_bytes may override the config's."""
    key = ("case", cid, tokens, row_bytes)
    if key not in _cache:
        w = vpgen.config(cid)
        rb = row_bytes or w.row_bytes
        R = vpgen.routing_all(w, 0, tokens)
        dem = [oracle.demand(R[i], w.n_ranks, w.experts, i, rb) for i in range(w.n_ranks)]
        D = np.stack([d["row"] for d in dem])
        counts = np.stack([d["counts"] for d in dem])
        _cache[key] = (w, rb, R, dem, D, counts)
    return _cache[key]


def oplan(cid, D, rb, transposed, tokens=None):
    key = ("plan", cid, tokens, rb, transposed)
    if key not in _cache:
        w = vpgen.config(cid)
        cat = _cache.setdefault(("ocat", cid), oracle.Catalog(w.topo))
        _cache[key] = cat.plan(np.ascontiguousarray(D.T if transposed else D), rb)
    return _cache[key]


def gcat(vp, topo):
    key = ("gc",) + topo.as_tuple()
    if key not in _cache:
        c = vp.Catalog(topo)
        c.upload()
        _cache[key] = c
    return _cache[key]


def inverse(dst):
    """recv_src[k, dst[k, i]] = i (restated here from the schedule)."""
    K, N = dst.shape
    r = np.zeros((K, N), np.int32)
    r[np.arange(K)[:, None], dst] = np.arange(N, dtype=np.int32)[None, :]
    return r


def upload(vp, N, s):
    sched = vp.alloc_schedule(N, 8 * N, layout=True)
    K = s["K"]
    sched["K"].fill_(K)
    if K:
        sched["dst"][:K] = torch.from_numpy(s["dst"]).cuda()
        sched["bytes"][:K] = torch.from_numpy(s["bytes"]).cuda()
        sched["recv_src"][:K] = torch.from_numpy(inverse(s["dst"])).cuda()
    return sched


def rand_bytes(n, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return torch.randint(0, 256, (max(n, 1),), dtype=torch.uint8, device="cuda", generator=g)


def expert_rows(counts, r, N):
    eloc = counts.shape[1] // N
    return int(counts[:, r * eloc:(r + 1) * eloc].sum())


# ------------------------------------------------------------ transpose

@pytest.mark.parametrize("N", [1, 8, 16, 33, 64, 256])
def test_demand_transpose(vp, N):
    rng = np.random.default_rng(N)
    D = rng.integers(-2**40, 2**40, (N, N), dtype=np.int64)
    DT = vp.demand_transpose(torch.from_numpy(D).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(DT.cpu().numpy(), D.T)


def test_plan_receive_view_inverts_every_step(vp):
    w, rb, R, dem, D, counts = case(5)
    log("plan receive view C5")
    cat = gcat(vp, w.topo)
    p = vp.plan_params(cat.N, rb)
    s = vp.plan(cat, torch.from_numpy(D).cuda(), p, out=vp.alloc_schedule(cat.N, p.k_max, layout=True))
    torch.cuda.synchronize()
    assert vp.read_status(s["status"]) == 0
    K = int(s["K"].item())
    dst = s["dst"][:K].cpu().numpy()
    rs = s["recv_src"][:K].cpu().numpy()
    assert np.array_equal(rs, inverse(dst))
    assert np.array_equal(np.sort(dst, axis=1), np.broadcast_to(np.arange(cat.N), (K, cat.N)))


# ------------------------------------------------- full size, oracle schedule

@pytest.mark.parametrize("cid,r", [(1, 0), (1, 7), (2, 0), (2, 11), (3, 63), (5, 0), (5, 200)])
def test_unpack_rows_parity_full_size(vp, cid, r):
    w, rb, R, dem, D, counts = case(cid)
    N = w.n_ranks
    sb = oracle.slot_bytes(rb)
    s = oplan(cid, D, rb, False)
    U = int(D[:, r].sum()) // rb
    log("unpack rows C%d rank %d: %d rows" % (cid, r, U))
    recv = rand_bytes(U * sb, 1000 * cid + r)
    ref = oracle.unpack_rows(recv.cpu().numpy(), r, N, s, rb, counts)
    out = torch.zeros(ref.size + sb, dtype=torch.uint8, device="cuda")
    st = vp.new_status()
    vp.unpack_rows(recv[:U * sb], rb, torch.from_numpy(counts).cuda(), r, upload(vp, N, s), out[:ref.size], st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    assert torch.equal(out[:ref.size], torch.from_numpy(ref).cuda())
    assert (out[ref.size:] == 0).all()


@pytest.mark.parametrize("cid,r,extra", [(1, 5, 13), (2, 3, 1), (3, 10, 777)])
def test_unpack_rows_receive_buffer_larger_than_its_rows(vp, cid, r, extra):
    """A receive buffer with `extra` slots past the rows the schedule delivers
    (a capacity, not a count): the copy splits the delivered rows, not the
    capacity, between the XCDs, and the slots past them are never read."""
    w, rb, R, dem, D, counts = case(cid)
    N = w.n_ranks
    sb = oracle.slot_bytes(rb)
    s = oplan(cid, D, rb, False)
    U = int(D[:, r].sum()) // rb
    log("unpack rows C%d rank %d: %d rows in %d slots" % (cid, r, U, U + extra))
    recv = rand_bytes((U + extra) * sb, 2000 * cid + r)
    ref = oracle.unpack_rows(recv[:U * sb].cpu().numpy(), r, N, s, rb, counts)
    out = torch.zeros(ref.size + sb, dtype=torch.uint8, device="cuda")
    st = vp.new_status()
    vp.unpack_rows(recv, rb, torch.from_numpy(counts).cuda(), r, upload(vp, N, s), out[:ref.size], st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    assert torch.equal(out[:ref.size], torch.from_numpy(ref).cuda())
    assert (out[ref.size:] == 0).all()


@pytest.mark.parametrize("cid,r", [(1, 3), (2, 0), (5, 0)])
def test_pack_combine_parity_full_size(vp, cid, r):
    w, rb, R, dem, D, counts = case(cid)
    N = w.n_ranks
    sb = oracle.slot_bytes(rb)
    sc = oplan(cid, D, rb, True)
    rows = expert_rows(counts, r, N)
    log("pack combine C%d rank %d: %d expert-major rows" % (cid, r, rows))
    out = rand_bytes(rows * sb, 2000 * cid + r)
    ref, ref_off = oracle.pack_combine(out.cpu().numpy(), r, N, sc, rb, counts)
    total = int(sc["bytes"][:, r].sum())
    send = torch.full((total + 64,), 0xA5, dtype=torch.uint8, device="cuda")
    step_off = torch.empty(8 * N + 1, dtype=torch.int64, device="cuda")
    st = vp.new_status()
    vp.pack_combine(out[:rows * sb], rb, torch.from_numpy(counts).cuda(), r, upload(vp, N, sc), send[:total],
                    step_off, st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    assert total == int(D[:, r].sum())
    assert torch.equal(send[:total], torch.from_numpy(ref[:total]).cuda())
    assert (send[total:] == 0xA5).all()
    assert np.array_equal(step_off[:sc["K"] + 1].cpu().numpy(), ref_off)


@pytest.mark.parametrize("cid,i", [(1, 5), (2, 0), (5, 0)])
def test_unpack_combine_parity_full_size(vp, cid, i):
    w, rb, R, dem, D, counts = case(cid)
    N, T, k = w.n_ranks, R.shape[1], w.top_k
    sb = oracle.slot_bytes(rb)
    sc = oplan(cid, D, rb, True)
    U = int(D[i].sum()) // rb
    log("unpack combine C%d rank %d: %d rows" % (cid, i, U))
    recv = rand_bytes(U * sb, 3000 * cid + i)
    d = dem[i]
    ref = oracle.unpack_combine(recv.cpu().numpy(), i, N, sc, rb, T, k, d["sorted_tok"], d["sorted_slot"],
                                d["dest_off"])
    comb = torch.zeros(T * k * sb, dtype=torch.uint8, device="cuda")
    st = vp.new_status()
    vp.unpack_combine(recv[:U * sb], rb, T, k, torch.from_numpy(d["sorted_tok"]).cuda(),
                      torch.from_numpy(d["sorted_slot"]).cuda(), torch.from_numpy(d["dest_off"]).cuda(), i,
                      upload(vp, N, sc), comb, st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    assert torch.equal(comb, torch.from_numpy(ref).cuda())


# ----------------------------------------------------- end to end on the GPU

def emulate_transfer(sends, offs, dst, nb, r, rb, sb):
    """The network, emulated in the test: rank r's receive slots from every
    rank's send buffer (slices addressed to r in step order)."""
    K, N = nb.shape
    parts = [sends[i][offs[i][k]:offs[i][k] + nb[k, i]].view(-1, rb)
             for k in range(K) for i in range(N) if dst[k, i] == r and nb[k, i]]
    U = sum(p.shape[0] for p in parts)
    recv = torch.zeros((max(U, 1), sb), dtype=torch.uint8, device="cuda")
    if U:
        recv[:U, :rb] = torch.cat(parts)
    return recv.view(-1)[:U * sb]


def gpu_schedule(vp, w, rb, D_dev):
    cat = gcat(vp, w.topo)
    p = vp.plan_params(cat.N, rb)
    s = vp.plan(cat, D_dev, p, out=vp.alloc_schedule(cat.N, p.k_max, layout=True))
    torch.cuda.synchronize()
    assert vp.read_status(s["status"]) == 0
    K = int(s["K"].item())
    return s, s["dst"][:K].cpu().numpy(), s["bytes"][:K].cpu().numpy()


def oracle_round_trip(w, rb, R, dem, D, counts, tok, cid, tokens):
    N, T, k = w.n_ranks, R.shape[1], w.top_k
    s = oplan(cid, D, rb, False, tokens)
    packs = [oracle.pack_rows(tok[i], rb, dem[i]["sorted_tok"], dem[i]["dest_off"], i, s) for i in range(N)]
    sends, offs = [p[0] for p in packs], [p[1] for p in packs]
    outs = [oracle.unpack_rows(oracle.receive(r, N, s, rb, sends, offs), r, N, s, rb, counts) for r in range(N)]
    sc = oplan(cid, D, rb, True, tokens)
    cpk = [oracle.pack_combine(outs[r], r, N, sc, rb, counts) for r in range(N)]
    csend, coff = [p[0] for p in cpk], [p[1] for p in cpk]
    comb = [oracle.unpack_combine(oracle.receive(i, N, sc, rb, csend, coff), i, N, sc, rb, T, k,
                                  dem[i]["sorted_tok"], dem[i]["sorted_slot"], dem[i]["dest_off"])
            for i in range(N)]
    return outs, comb


@pytest.mark.parametrize("cid,tokens,row_bytes", [(1, None, None), (1, None, 1040), (2, 1024, None)])
def test_dispatch_and_combine_round_trip(vp, cid, tokens, row_bytes):
    """GPU demand -> plan -> pack (every rank) -> transfer -> unpack, then
    transpose -> plan -> combine pack -> transfer -> combine unpack, against
    the oracle's pipeline; identity experts return every token its own row."""
    w, rb, R, dem, D, counts = case(cid, tokens, row_bytes)
    N, T, k, E = w.n_ranks, R.shape[1], w.top_k, w.experts
    sb = oracle.slot_bytes(rb)
    log("round trip C%d T=%d row %d (slot %d)" % (cid, T, rb, sb))
    rng = np.random.default_rng(7)
    tok = [rng.integers(0, 256, (T, rb), dtype=np.uint8) for _ in range(N)]
    ref_out, ref_comb = oracle_round_trip(w, rb, R, dem, D, counts, tok, cid, tokens)

    rt = torch.from_numpy(R).cuda()
    st = vp.new_status()
    dems = [vp.demand(rt, N, E, rb, sort_row=i, status=st) for i in range(N)]
    D_dev, counts_dev = dems[0]["demand"], dems[0]["counts"]
    s, dst, nb = gpu_schedule(vp, w, rb, D_dev)
    sends, offs = [], []
    for i in range(N):
        total = int(D[i].sum())
        send = torch.empty(max(total, 16), dtype=torch.uint8, device="cuda")
        step_off = torch.empty(8 * N + 1, dtype=torch.int64, device="cuda")
        vp.pack_rows(torch.from_numpy(tok[i]).cuda(), rb, dems[i]["sorted_tok"], dems[i]["sorted_slot"],
                     dems[i]["dest_off"], i, s, send[:total], step_off, st)
        sends.append(send)
        offs.append(step_off.cpu().numpy())
    outs = []
    for r in range(N):
        recv = emulate_transfer(sends, offs, dst, nb, r, rb, sb)
        out = torch.zeros(max(expert_rows(counts, r, N), 1) * sb, dtype=torch.uint8, device="cuda")
        vp.unpack_rows(recv, rb, counts_dev, r, s, out, st)
        outs.append(out)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    for r in range(N):
        assert torch.equal(outs[r], torch.from_numpy(ref_out[r]).cuda()), "unpack rank %d" % r

    DT = vp.demand_transpose(D_dev)
    sc, cdst, cnb = gpu_schedule(vp, w, rb, DT)
    csends, coffs = [], []
    for r in range(N):
        total = int(D[:, r].sum())
        send = torch.empty(max(total, 16), dtype=torch.uint8, device="cuda")
        step_off = torch.empty(8 * N + 1, dtype=torch.int64, device="cuda")
        vp.pack_combine(outs[r], rb, counts_dev, r, sc, send[:total], step_off, st)
        csends.append(send)
        coffs.append(step_off.cpu().numpy())
    combs = []
    for i in range(N):
        recv = emulate_transfer(csends, coffs, cdst, cnb, i, rb, sb)
        comb = torch.zeros(T * k * sb, dtype=torch.uint8, device="cuda")
        vp.unpack_combine(recv, rb, T, k, dems[i]["sorted_tok"], dems[i]["sorted_slot"], dems[i]["dest_off"], i,
                          sc, comb, st)
        combs.append(comb)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    eloc = E // N
    for i in range(N):
        assert torch.equal(combs[i], torch.from_numpy(ref_comb[i]).cuda()), "combine rank %d" % i
        c = combs[i].view(T, k, sb)[:, :, :rb].cpu().numpy()
        remote = (R[i] // eloc) != i
        want = np.broadcast_to(tok[i][:, None, :], (T, k, rb))
        assert (c[remote] == want[remote]).all()


RANDOM_TRIPS = [  # (topology, experts per rank, tokens, top-k, row bytes, routing skew)
    (vpgen.Topology(1, 2, 2, 2), 3, 333, 5, 1040, 1.2),
    (vpgen.Topology(2, 1, 2, 2, 2), 2, 65, 3, 16, 0.0),
    (vpgen.Topology(1, 1, 2, 3), 4, 1000, 8, 272, 2.0),
    (vpgen.Topology(2, 2, 2, 2, 1, 32, 25, 1), 1, 129, 1, 4112, 0.6),
    (vpgen.Topology(1, 1, 1, 2), 8, 7, 8, 48, 1.0),
]


@pytest.mark.parametrize("i", range(len(RANDOM_TRIPS)))
def test_random_round_trip(vp, i):
    """Dispatch and combine on seeded random shapes (odd row sizes, top-1 to
    top-8, SYS nodes, two NICs per switch): GPU demand -> plan -> pack of
    every rank -> emulated transfer -> unpack, then the transposed plan ->
    combine pack -> transfer -> combine unpack, against the oracle's
    pipeline on the oracle's schedules (which the GPU's equal)."""
    topo, L, T, k, rb, zipf = RANDOM_TRIPS[i]
    N = topo.n_ranks
    E = N * L
    sb = oracle.slot_bytes(rb)
    log("random round trip %d: topo %s E=%d T=%d k=%d row %d" % (i, topo.as_tuple(), E, T, k, rb))
    R = vpgen.random_routing(300 + i, N, T, E, k, zipf)
    dem = [oracle.demand(R[r], N, E, r, rb) for r in range(N)]
    D = np.stack([d["row"] for d in dem])
    counts = np.stack([d["counts"] for d in dem])
    rng = np.random.default_rng(i)
    tok = [rng.integers(0, 256, (T, rb), dtype=np.uint8) for _ in range(N)]
    oc = _cache.setdefault(("ocat",) + topo.as_tuple(), oracle.Catalog(topo))
    s_o, sc_o = oc.plan(D, rb), oc.plan(np.ascontiguousarray(D.T), rb)
    packs = [oracle.pack_rows(tok[r], rb, dem[r]["sorted_tok"], dem[r]["dest_off"], r, s_o) for r in range(N)]
    ref_out = [oracle.unpack_rows(oracle.receive(r, N, s_o, rb, [p[0] for p in packs], [p[1] for p in packs]),
                                  r, N, s_o, rb, counts) for r in range(N)]
    cpk = [oracle.pack_combine(ref_out[r], r, N, sc_o, rb, counts) for r in range(N)]
    ref_comb = [oracle.unpack_combine(oracle.receive(j, N, sc_o, rb, [p[0] for p in cpk], [p[1] for p in cpk]),
                                      j, N, sc_o, rb, T, k, dem[j]["sorted_tok"], dem[j]["sorted_slot"],
                                      dem[j]["dest_off"]) for j in range(N)]

    cat = gcat(vp, topo)
    rt = torch.from_numpy(R).cuda()
    st = vp.new_status()
    dems = [vp.demand(rt, N, E, rb, sort_row=r, status=st) for r in range(N)]
    D_dev, counts_dev = dems[0]["demand"], dems[0]["counts"]

    def plan(Dd):
        p = vp.plan_params(N, rb)
        s = vp.plan(cat, Dd, p, out=vp.alloc_schedule(N, p.k_max, layout=True))
        torch.cuda.synchronize()
        assert vp.read_status(s["status"]) == 0
        K = int(s["K"].item())
        return s, s["dst"][:K].cpu().numpy(), s["bytes"][:K].cpu().numpy()

    s, dst, nb = plan(D_dev)
    assert np.array_equal(dst, s_o["dst"]) and np.array_equal(nb, s_o["bytes"])
    sends, offs = [], []
    for r in range(N):
        total = int(D[r].sum())
        send = torch.empty(max(total, 16), dtype=torch.uint8, device="cuda")
        step_off = torch.empty(8 * N + 1, dtype=torch.int64, device="cuda")
        vp.pack_rows(torch.from_numpy(tok[r]).cuda(), rb, dems[r]["sorted_tok"], dems[r]["sorted_slot"],
                     dems[r]["dest_off"], r, s, send[:total], step_off, st)
        sends.append(send)
        offs.append(step_off.cpu().numpy())
    outs = []
    for r in range(N):
        recv = emulate_transfer(sends, offs, dst, nb, r, rb, sb)
        out = torch.zeros(max(expert_rows(counts, r, N), 1) * sb, dtype=torch.uint8, device="cuda")
        vp.unpack_rows(recv, rb, counts_dev, r, s, out, st)
        outs.append(out)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    for r in range(N):
        assert torch.equal(outs[r], torch.from_numpy(ref_out[r]).cuda()), "unpack rank %d" % r

    sc, cdst, cnb = plan(vp.demand_transpose(D_dev))
    assert np.array_equal(cdst, sc_o["dst"]) and np.array_equal(cnb, sc_o["bytes"])
    csends, coffs = [], []
    for r in range(N):
        total = int(D[:, r].sum())
        send = torch.empty(max(total, 16), dtype=torch.uint8, device="cuda")
        step_off = torch.empty(8 * N + 1, dtype=torch.int64, device="cuda")
        vp.pack_combine(outs[r], rb, counts_dev, r, sc, send[:total], step_off, st)
        csends.append(send)
        coffs.append(step_off.cpu().numpy())
    for j in range(N):
        recv = emulate_transfer(csends, coffs, cdst, cnb, j, rb, sb)
        comb = torch.zeros(T * k * sb, dtype=torch.uint8, device="cuda")
        vp.unpack_combine(recv, rb, T, k, dems[j]["sorted_tok"], dems[j]["sorted_slot"], dems[j]["dest_off"], j,
                          sc, comb, st)
        torch.cuda.synchronize()
        assert vp.read_status(st) == 0
        assert torch.equal(comb, torch.from_numpy(ref_comb[j]).cuda()), "combine rank %d" % j


# ------------------------------------------------------------ error paths

def small(vp):
    w, rb, R, dem, D, counts = case(1)
    s = oplan(1, D, rb, False)
    return w, rb, D, counts, s


def test_unpack_empty_schedule(vp):
    w, rb, D, counts, s = small(vp)
    N = w.n_ranks
    e = dict(K=0, dst=np.zeros((0, N), np.int32), bytes=np.zeros((0, N), np.int64))
    out = torch.full((4096,), 0xA5, dtype=torch.uint8, device="cuda")
    st = vp.new_status()
    z = torch.zeros((N, w.experts), dtype=torch.int32, device="cuda")
    vp.unpack_rows(torch.zeros(4096, dtype=torch.uint8, device="cuda"), rb, z, 0, upload(vp, N, e), out, st)
    step_off = torch.full((8 * N + 1,), -1, dtype=torch.int64, device="cuda")
    send = torch.full((4096,), 0xA5, dtype=torch.uint8, device="cuda")
    vp.pack_combine(out, rb, z, 0, upload(vp, N, e), send, step_off, st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    assert (out == 0xA5).all() and (send == 0xA5).all()
    assert int(step_off[0].item()) == 0


@pytest.mark.parametrize("bad", ["recv_src", "capacity", "out_capacity", "incomplete", "counts"])
def test_unpack_rows_errors_copy_nothing(vp, bad):
    w, rb, D, counts, s = small(vp)
    N, r = w.n_ranks, 2
    sb = oracle.slot_bytes(rb)
    log("unpack rows error case %s" % bad)
    U = int(D[:, r].sum()) // rb
    rows = expert_rows(counts, r, N)
    sched = upload(vp, N, s)
    recv = rand_bytes(U * sb, 5)
    out = torch.full((rows * sb,), 0xA5, dtype=torch.uint8, device="cuda")
    c = counts.copy()
    want = vp.INVALID_ARGUMENT
    if bad == "recv_src":
        k = int(np.argmax(s["bytes"][np.arange(s["K"]), inverse(s["dst"])[:, r]] > 0))
        sched["recv_src"][k, r] = (sched["recv_src"][k, r] + 1) % N
    elif bad == "capacity":
        recv = recv[:(U - 1) * sb]
        want = vp.CAPACITY
    elif bad == "out_capacity":
        out = out[:(rows - 1) * sb]
        want = vp.CAPACITY
    elif bad == "incomplete":
        # stop the schedule before the last step that carries rows to r
        carry = s["bytes"][np.arange(s["K"]), inverse(s["dst"])[:, r]] > 0
        sched["K"].fill_(int(np.nonzero(carry)[0][-1]))
    else:
        # one more assignment than the schedule delivers (the output has room for it)
        c[(r + 1) % N, r * (w.experts // N)] += 1
        out = torch.full(((rows + 1) * sb,), 0xA5, dtype=torch.uint8, device="cuda")
    st = vp.new_status()
    vp.unpack_rows(recv, rb, torch.from_numpy(c).cuda(), r, sched, out, st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == want
    assert (out == 0xA5).all()


@pytest.mark.parametrize("bad", ["dest_off", "sorted_tok", "slot"])
def test_unpack_combine_errors_copy_nothing(vp, bad):
    w, rb, R, dem, D, counts = case(1)
    N, T, k = w.n_ranks, R.shape[1], w.top_k
    sb = oracle.slot_bytes(rb)
    sc = oplan(1, D, rb, True)
    i = 4
    d = {x: dem[i][x].copy() for x in ("sorted_tok", "sorted_slot", "dest_off")}
    lo, hi = int(d["dest_off"][1]), int(d["dest_off"][2])
    if bad == "dest_off":
        d["dest_off"][1:] += 1
    elif bad == "sorted_tok":
        d["sorted_tok"][lo:hi] = T
    else:
        d["sorted_slot"][lo:hi] = k
    U = int(D[i].sum()) // rb
    comb = torch.full((T * k * sb,), 0xA5, dtype=torch.uint8, device="cuda")
    st = vp.new_status()
    vp.unpack_combine(rand_bytes(U * sb, 9), rb, T, k, torch.from_numpy(d["sorted_tok"]).cuda(),
                      torch.from_numpy(d["sorted_slot"]).cuda(), torch.from_numpy(d["dest_off"]).cuda(), i,
                      upload(vp, N, sc), comb, st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == vp.INVALID_ARGUMENT
    assert (comb == 0xA5).all()
