"""The whole path on seeded random shapes against the oracle, bit-exact.

Token rows (MoE dispatch):

Each case draws a topology (2 to 64 ranks, SYS nodes and two NICs per switch
among them), experts per rank, tokens (ragged around the demand kernels'
tiles), top-k, routing skew, row size and self rank; then checks the GPU
demand of every rank (rows, expert counts, the self rank's (expert, token)
order, routing slots and destination offsets, Sec. 3 model setup), the GPU
plan with its buffer layout (Alg. 2; K, tau, family, destination, instance
and bytes of every step) and the self rank's pack (Sec. 5 buffer layout) with
the planner's layout and with the plain schedule: send bytes, nothing written
past them, step offsets.  Head blocks (head/context re-layout): the same for
random uneven head splits, head sizes, tokens and row padding."""
import sys

import numpy as np
import pytest
import torch

import oracle
import vpgen

pytestmark = pytest.mark.gpu
_cat = {}

TOPOS = [vpgen.Topology(1, 2, 2, 2), vpgen.Topology(2, 2, 2, 2), vpgen.Topology(8, 2, 2, 2),
         vpgen.Topology(1, 1, 2, 3), vpgen.Topology(3, 1, 2, 2), vpgen.Topology(2, 2, 1, 4),
         vpgen.Topology(1, 1, 1, 2), vpgen.Topology(2, 2, 2, 2, 1, 32, 50), vpgen.Topology(2, 1, 2, 2, 2),
         vpgen.Topology(3, 2, 2, 2, 1, 32, 25, 1)]
N_CASES = 40


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def vp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_34340_amd as vp
    vp.lib()
    return vp


def case_params(i):
    """Shape of case i (a pure function of i)."""
    r = np.random.default_rng(1000 + i)
    topo = TOPOS[i % len(TOPOS)]
    N = topo.n_ranks
    L = int(r.choice([1, 2, 3, 4, 8, 16]))
    while N * L > 4096:
        L //= 2
    E = N * L
    k = int(r.integers(1, min(8, E) + 1))
    T = int(r.choice([1, 2, 63, 64, 65, 511, 1000, 2048, 3001]))
    while N * T * k > 2_000_000 and T > 1:
        T //= 2
    row = 16 * int(r.choice([1, 2, 7, 65, 256, 900, 1024, 2049]))
    zipf = float(r.choice([0.0, 0.6, 1.2, 2.0]))
    self_rank = int(r.integers(N))
    return topo, E, T, k, row, zipf, self_rank


def catalogs(vp, topo):
    key = topo.as_tuple()
    if key not in _cat:
        c = vp.Catalog(topo)
        c.upload()
        _cat[key] = (c, oracle.Catalog(topo))
    return _cat[key]


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_path_parity(vp, i):
    topo, E, T, k, row, zipf, self_rank = case_params(i)
    N = topo.n_ranks
    log("random path case %d: topo %s E=%d T=%d k=%d row=%d zipf=%.1f self=%d" %
        (i, topo.as_tuple(), E, T, k, row, zipf, self_rank))
    gc, oc = catalogs(vp, topo)
    R = vpgen.random_routing(i, N, T, E, k, zipf)
    dem = [oracle.demand(R[r], N, E, r, row) for r in range(N)]
    D = np.stack([d["row"] for d in dem])
    od = dem[self_rank]

    gd = vp.demand(torch.from_numpy(R).cuda(), N, E, row, sort_row=self_rank)
    torch.cuda.synchronize()
    assert vp.read_status(gd["status"]) == 0
    assert np.array_equal(gd["demand"].cpu().numpy(), D)
    assert np.array_equal(gd["counts"].cpu().numpy(), np.stack([d["counts"] for d in dem]))
    assert np.array_equal(gd["sorted_tok"][:T * k].cpu().numpy(), od["sorted_tok"])
    assert np.array_equal(gd["sorted_slot"][:T * k].cpu().numpy(), od["sorted_slot"])
    assert np.array_equal(gd["dest_off"].cpu().numpy(), od["dest_off"])

    p = vp.plan_params(N, row, k_max=64 * N)   # skewed random routing can need more than 8N steps
    st = vp.new_status()
    s = vp.plan(gc, gd["demand"], p, status=st, out=vp.alloc_schedule(N, p.k_max, layout=True))
    torch.cuda.synchronize()
    o = oc.plan(D, row, k_max=64 * N)
    assert vp.read_status(st) == 0 == o["status"]
    h = vp.schedule_to_host(s)
    assert (h["K"], h["tau"]) == (o["K"], o["tau"])
    for key in ("family", "dst", "inst", "bytes"):
        assert np.array_equal(np.asarray(h[key]), np.asarray(o[key])), key

    tok = np.random.default_rng(i).integers(0, 256, (T, row), dtype=np.uint8)
    ref, ref_off = oracle.pack_rows(tok, row, od["sorted_tok"], od["dest_off"], self_rank, o)
    K = o["K"]
    rows = max(K, 1)
    plain = {"K": s["K"], "dst": s["dst"][:rows], "bytes": s["bytes"][:rows]}
    for name, sched in (("layout", s), ("plain", plain)):
        cap = ref.size + 64
        send = torch.full((cap,), 0xA5, dtype=torch.uint8, device="cuda")
        step_off = torch.empty(p.k_max + 1, dtype=torch.int64, device="cuda")
        pst = vp.new_status()
        vp.pack_rows(torch.from_numpy(tok).cuda(), row, gd["sorted_tok"], gd["sorted_slot"], gd["dest_off"],
                     self_rank, sched, send, step_off, pst)
        torch.cuda.synchronize()
        assert vp.read_status(pst) == 0, name
        assert torch.equal(send[:ref.size].cpu(), torch.from_numpy(ref)), name
        assert (send[ref.size:] == 0xA5).all(), name + ": wrote past the packed bytes"
        assert np.array_equal(step_off[:K + 1].cpu().numpy(), ref_off), name


N_HEADS_CASES = 20


def heads_params(i):
    """Shape of head/context case i: heads split unevenly (some ranks may own
    none), head size, tokens, row padding and self rank."""
    r = np.random.default_rng(5000 + i)
    topo = TOPOS[(3 * i + 1) % len(TOPOS)]
    N = topo.n_ranks
    H = int(r.integers(N, 4 * N + 1))
    cuts = np.sort(r.integers(0, H + 1, N - 1))
    hl = np.concatenate([[0], cuts, [H]]).astype(np.int64)
    head_bytes = 16 * int(r.choice([1, 3, 8, 16, 17, 64]))
    T = int(r.choice([1, 7, 64, 333, 1024]))
    pad = 16 * int(r.choice([0, 0, 1, 5]))
    self_rank = int(r.integers(N))
    return topo, hl, head_bytes, T, H * head_bytes + pad, self_rank


@pytest.mark.parametrize("i", range(N_HEADS_CASES))
def test_random_heads_path_parity(vp, i):
    """Sec. 6.2 head/context re-layout on seeded random splits: the GPU demand
    of every rank, the plan with its layout, and the self rank's head pack
    (one-kernel pack with the layout, prepare and gather without) against
    the oracle."""
    topo, hl, hb, T, stride, self_rank = heads_params(i)
    N = topo.n_ranks
    log("random heads case %d: topo %s heads %d bytes %d T=%d stride %d self=%d" %
        (i, topo.as_tuple(), int(hl[-1]), hb, T, stride, self_rank))
    gc, oc = catalogs(vp, topo)
    D = np.stack([oracle.demand_heads(T, hl, hb, r) for r in range(N)])
    hl_d = torch.from_numpy(hl).cuda()
    gD = vp.demand_heads(T, hl_d, hb, first_rank=0, R=N)
    torch.cuda.synchronize()
    assert np.array_equal(gD.cpu().numpy(), D)

    p = vp.plan_params(N, hb)
    st = vp.new_status()
    s = vp.plan(gc, gD, p, status=st, out=vp.alloc_schedule(N, p.k_max, layout=True))
    torch.cuda.synchronize()
    o = oc.plan(D, hb)
    assert vp.read_status(st) == 0 == o["status"]
    h = vp.schedule_to_host(s)
    assert (h["K"], h["tau"]) == (o["K"], o["tau"])
    for key in ("family", "dst", "inst", "bytes"):
        assert np.array_equal(np.asarray(h[key]), np.asarray(o[key])), key

    act = np.random.default_rng(i).integers(0, 256, (T, stride), dtype=np.uint8)
    ref, ref_off = oracle.pack_heads(act, stride, hl, hb, self_rank, o)
    K = o["K"]
    plain = {"K": s["K"], "dst": s["dst"][:max(K, 1)], "bytes": s["bytes"][:max(K, 1)]}
    for name, sched in (("layout", s), ("plain", plain)):
        send = torch.full((ref.size + 64,), 0xA5, dtype=torch.uint8, device="cuda")
        step_off = torch.empty(p.k_max + 1, dtype=torch.int64, device="cuda")
        pst = vp.new_status()
        vp.pack_heads(torch.from_numpy(act).cuda(), stride, hl_d, hb, self_rank, sched, send, step_off, pst)
        torch.cuda.synchronize()
        assert vp.read_status(pst) == 0, name
        assert torch.equal(send[:ref.size].cpu(), torch.from_numpy(ref)), name
        assert (send[ref.size:] == 0xA5).all(), name + ": wrote past the packed bytes"
        assert np.array_equal(step_off[:K + 1].cpu().numpy(), ref_off), name


@pytest.mark.parametrize("k", [64, 65, 255])
def test_many_slots_path_parity(vp, k):
    """Top-k at and beyond one wavefront's worth of routing slots, up to the
    largest k the demand takes (255): the sort's slot bytes, and the scatter's
    path that keeps routing order for more than 64 slots, against the
    oracle."""
    topo = vpgen.Topology(1, 2, 2, 2)
    N, E, T, row = 8, 512, 37, 272
    self_rank = 3
    log("many slots k=%d" % k)
    gc, oc = catalogs(vp, topo)
    R = vpgen.random_routing(100 + k, N, T, E, k, 0.8)
    dem = [oracle.demand(R[r], N, E, r, row) for r in range(N)]
    D = np.stack([d["row"] for d in dem])
    od = dem[self_rank]
    gd = vp.demand(torch.from_numpy(R).cuda(), N, E, row, sort_row=self_rank)
    p = vp.plan_params(N, row)
    st = vp.new_status()
    s = vp.plan(gc, gd["demand"], p, status=st, out=vp.alloc_schedule(N, p.k_max, layout=True))
    torch.cuda.synchronize()
    assert vp.read_status(gd["status"]) == 0 == vp.read_status(st)
    assert np.array_equal(gd["demand"].cpu().numpy(), D)
    assert np.array_equal(gd["sorted_tok"][:T * k].cpu().numpy(), od["sorted_tok"])
    assert np.array_equal(gd["sorted_slot"][:T * k].cpu().numpy(), od["sorted_slot"])
    o = oc.plan(D, row)
    h = vp.schedule_to_host(s)
    assert (h["K"], h["tau"]) == (o["K"], o["tau"])
    for key in ("family", "dst", "inst", "bytes"):
        assert np.array_equal(np.asarray(h[key]), np.asarray(o[key])), key
    tok = np.random.default_rng(k).integers(0, 256, (T, row), dtype=np.uint8)
    ref, ref_off = oracle.pack_rows(tok, row, od["sorted_tok"], od["dest_off"], self_rank, o)
    send = torch.full((ref.size + 64,), 0xA5, dtype=torch.uint8, device="cuda")
    step_off = torch.empty(p.k_max + 1, dtype=torch.int64, device="cuda")
    pst = vp.new_status()
    vp.pack_rows(torch.from_numpy(tok).cuda(), row, gd["sorted_tok"], gd["sorted_slot"], gd["dest_off"],
                 self_rank, s, send, step_off, pst)
    torch.cuda.synchronize()
    assert vp.read_status(pst) == 0
    assert torch.equal(send[:ref.size].cpu(), torch.from_numpy(ref))
    assert (send[ref.size:] == 0xA5).all()
    assert np.array_equal(step_off[:o["K"] + 1].cpu().numpy(), ref_off)


def test_pack_at_1024_ranks(vp):
    """The largest rank count the library takes: demand of all 1,024 ranks
    (one expert each, top-8 over 256 tokens) against the oracle, a GPU plan
    checked for validity (sums to D, every step a derangement sharing no
    modeled resource, Eq. (1); its exactness at this size is pinned by the
    1,024-rank digest test), and rank 777's pack with the planner's layout
    against the oracle's pack of that same schedule."""
    from oracle.checks import TopoModel, schedule_valid_np
    topo = vpgen.Topology(128)
    N, E, T, k, row, self_rank = 1024, 1024, 256, 8, 1024, 777
    log("pack at 1024 ranks")
    R = vpgen.random_routing(1024, N, T, E, k, 0.5)
    dem = [oracle.demand(R[r], N, E, r, row) for r in range(N)]
    D = np.stack([d["row"] for d in dem])
    od = dem[self_rank]
    gc, _ = catalogs_gpu_only(vp, topo)
    gd = vp.demand(torch.from_numpy(R).cuda(), N, E, row, sort_row=self_rank)
    p = vp.plan_params(N, row, k_max=16 * N)
    st = vp.new_status()
    s = vp.plan(gc, gd["demand"], p, status=st, out=vp.alloc_schedule(N, p.k_max, layout=True))
    torch.cuda.synchronize()
    assert vp.read_status(gd["status"]) == 0 == vp.read_status(st)
    assert np.array_equal(gd["demand"].cpu().numpy(), D)
    assert np.array_equal(gd["sorted_tok"][:T * k].cpu().numpy(), od["sorted_tok"])
    assert np.array_equal(gd["dest_off"].cpu().numpy(), od["dest_off"])
    h = vp.schedule_to_host(s)
    K = h["K"]
    log("1024 ranks: K = %d" % K)
    rows = np.arange(N)
    X = np.zeros((N, N), np.int64)
    np.add.at(X, (np.broadcast_to(rows, (K, N)), h["dst"]), h["bytes"])
    assert np.array_equal(X, D)
    schedule_valid_np(TopoModel(topo), D, h["dst"], gc.instances()["cls"][h["inst"]], h["bytes"])
    tok = np.random.default_rng(777).integers(0, 256, (T, row), dtype=np.uint8)
    ref, ref_off = oracle.pack_rows(tok, row, od["sorted_tok"], od["dest_off"], self_rank, h)
    send = torch.full((ref.size + 64,), 0xA5, dtype=torch.uint8, device="cuda")
    step_off = torch.empty(p.k_max + 1, dtype=torch.int64, device="cuda")
    pst = vp.new_status()
    vp.pack_rows(torch.from_numpy(tok).cuda(), row, gd["sorted_tok"], gd["sorted_slot"], gd["dest_off"],
                 self_rank, s, send, step_off, pst)
    torch.cuda.synchronize()
    assert vp.read_status(pst) == 0
    assert torch.equal(send[:ref.size].cpu(), torch.from_numpy(ref))
    assert (send[ref.size:] == 0xA5).all()
    assert np.array_equal(step_off[:K + 1].cpu().numpy(), ref_off)


def catalogs_gpu_only(vp, topo):
    """The library's catalog alone (the oracle's is not needed, and takes
    long to enumerate at 128 nodes)."""
    key = ("gpu",) + topo.as_tuple()
    if key not in _cat:
        c = vp.Catalog(topo)
        c.upload()
        _cat[key] = (c, None)
    return _cat[key]


def test_heads_pack_at_1024_ranks(vp):
    """Head/context re-layout on 1,024 ranks (an uneven split of 2,500 heads
    of 64 B, some ranks owning none): demand against the oracle, a validated
    GPU plan, and rank 5's head pack (the prepare-and-gather pair: more steps
    than the one-kernel pack takes) against the oracle's pack of that
    schedule."""
    from oracle.checks import TopoModel, schedule_valid_np
    topo = vpgen.Topology(128)
    N, H, hb, T, self_rank = 1024, 2500, 64, 48, 5
    r = np.random.default_rng(2500)
    hl = np.concatenate([[0], np.sort(r.integers(0, H + 1, N - 1)), [H]]).astype(np.int64)
    stride = H * hb + 32
    log("heads pack at 1024 ranks")
    D = np.stack([oracle.demand_heads(T, hl, hb, i) for i in range(N)])
    gc, _ = catalogs_gpu_only(vp, topo)
    hl_d = torch.from_numpy(hl).cuda()
    gD = vp.demand_heads(T, hl_d, hb, first_rank=0, R=N)
    p = vp.plan_params(N, hb)
    st = vp.new_status()
    s = vp.plan(gc, gD, p, status=st, out=vp.alloc_schedule(N, p.k_max, layout=True))
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    assert np.array_equal(gD.cpu().numpy(), D)
    h = vp.schedule_to_host(s)
    K = h["K"]
    log("1024 ranks heads: K = %d" % K)
    rows = np.arange(N)
    X = np.zeros((N, N), np.int64)
    np.add.at(X, (np.broadcast_to(rows, (K, N)), h["dst"]), h["bytes"])
    assert np.array_equal(X, D)
    schedule_valid_np(TopoModel(topo), D, h["dst"], gc.instances()["cls"][h["inst"]], h["bytes"])
    act = np.random.default_rng(5).integers(0, 256, (T, stride), dtype=np.uint8)
    ref, ref_off = oracle.pack_heads(act, stride, hl, hb, self_rank, h)
    send = torch.full((ref.size + 64,), 0xA5, dtype=torch.uint8, device="cuda")
    step_off = torch.empty(p.k_max + 1, dtype=torch.int64, device="cuda")
    pst = vp.new_status()
    vp.pack_heads(torch.from_numpy(act).cuda(), stride, hl_d, hb, self_rank, s, send, step_off, pst)
    torch.cuda.synchronize()
    assert vp.read_status(pst) == 0
    assert torch.equal(send[:ref.size].cpu(), torch.from_numpy(ref))
    assert (send[ref.size:] == 0xA5).all()
    assert np.array_equal(step_off[:K + 1].cpu().numpy(), ref_off)
