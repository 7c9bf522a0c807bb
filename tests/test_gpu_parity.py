"""GPU parity: the HIP library against the CPU oracle, bit-exact.

Every comparison is element by element on the same seeded inputs: demand
counts, rows, the (expert, token) order and offsets; the whole schedule (K,
family, destination, instance and bytes of every lane, tau); and the packed
send buffer with its step offsets.  The five workload configurations run at
full size; extra cases cover ragged and empty inputs, other topologies, other
planner parameters and the device-side error paths."""
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


def ocat(topo):
    key = ("oc",) + topo.as_tuple()
    if key not in _cache:
        _cache[key] = oracle.Catalog(topo)
    return _cache[key]


def gcat(vp, topo):
    key = ("gc",) + topo.as_tuple()
    if key not in _cache:
        c = vp.Catalog(topo)
        c.upload()
        _cache[key] = c
    return _cache[key]


def moe_case(cid, matrix=0, tokens=None):
    key = ("moe", cid, matrix, tokens)
    if key not in _cache:
        w = vpgen.config(cid)
        R = vpgen.routing_all(w, matrix, tokens)
        dem = [oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes) for i in range(w.n_ranks)]
        D = np.stack([d["row"] for d in dem])
        _cache[key] = (w, R, dem, D)
    return _cache[key]


def oracle_plan(cid, D, matrix=0, tokens=None, **kw):
    key = ("plan", cid, matrix, tokens, tuple(sorted(kw.items())))
    if key not in _cache:
        w = vpgen.config(cid)
        _cache[key] = ocat(w.topo).plan(D, w.row_bytes, **kw)
    return _cache[key]


def heads_case():
    w = vpgen.config(4)
    hl = vpgen.head_split(w.heads, w.n_ranks)
    D = np.stack([oracle.demand_heads(w.tokens, hl, w.row_bytes, i) for i in range(w.n_ranks)])
    return w, hl, D


def assert_schedule_equal(g, o):
    assert g["K"] == o["K"], (g["K"], o["K"])
    assert g["tau"] == o["tau"]
    for key in ("family", "dst", "inst", "bytes"):
        a, b = np.asarray(g[key]), np.asarray(o[key])
        if not np.array_equal(a, b):
            bad = np.argwhere(a != b)[:5]
            raise AssertionError("%s differs at %s: gpu %s oracle %s" % (
                key, bad.tolist(), [a[tuple(x)] for x in bad], [b[tuple(x)] for x in bad]))


def gpu_plan(vp, topo, D, unit, layout=False, **kw):
    cat = gcat(vp, topo)
    p = vp.plan_params(cat.N, unit, **kw)
    st = vp.new_status()
    out = vp.alloc_schedule(cat.N, p.k_max, layout=layout)
    s = vp.plan(cat, torch.from_numpy(np.ascontiguousarray(D)).cuda(), p, status=st, out=out)
    torch.cuda.synchronize()
    h = vp.schedule_to_host(s)
    h["status"] = vp.read_status(st)
    if layout:
        K = h["K"]
        h["send_off"] = s["send_off"][:K].cpu().numpy()
        h["stream_off"] = s["stream_off"][:K].cpu().numpy()
    return h


def layout_np(dst, nbytes):
    """Sec. 5 buffer layout restated from a schedule: bytes each rank sent
    before step k, and bytes it sent to step k's destination before step k."""
    K, N = nbytes.shape
    send_off = np.zeros((K, N), np.int64)
    stream_off = np.zeros((K, N), np.int64)
    sent = np.zeros(N, np.int64)
    to = np.zeros((N, N), np.int64)
    rows = np.arange(N)
    for k in range(K):
        send_off[k] = sent
        stream_off[k] = to[rows, dst[k]]
        sent += nbytes[k]
        to[rows, dst[k]] += nbytes[k]
    return send_off, stream_off


# ---------------------------------------------------------------- demand

@pytest.mark.parametrize("cid", [1, 2, 3, 5])
def test_demand_parity_full_size(vp, cid):
    w, R, dem, D = moe_case(cid)
    log("demand parity C%d: N=%d T=%d k=%d E=%d" % (cid, w.n_ranks, w.tokens, w.top_k, w.experts))
    rt = torch.from_numpy(R).cuda()
    for sort_row in (0, w.n_ranks - 1):
        out = vp.demand(rt, w.n_ranks, w.experts, w.row_bytes, first_rank=0, sort_row=sort_row)
        torch.cuda.synchronize()
        assert vp.read_status(out["status"]) == 0
        assert np.array_equal(out["demand"].cpu().numpy(), D)
        assert np.array_equal(out["counts"].cpu().numpy(), np.stack([d["counts"] for d in dem]))
        assert np.array_equal(out["sorted_tok"].cpu().numpy(), dem[sort_row]["sorted_tok"])
        assert np.array_equal(out["sorted_slot"].cpu().numpy(), dem[sort_row]["sorted_slot"])
        assert np.array_equal(out["dest_off"].cpu().numpy(), dem[sort_row]["dest_off"])


@pytest.mark.parametrize("T,k,E,N,first", [(1000, 3, 24, 8, 5), (2049, 8, 256, 64, 0), (1, 1, 8, 8, 7),
                                            (4097, 2, 4096, 16, 3), (20011, 8, 256, 64, 2)])
def test_demand_ragged(vp, T, k, E, N, first):
    log("demand ragged T=%d k=%d E=%d N=%d" % (T, k, E, N))
    rng = np.random.default_rng(T + E)
    R = np.stack([np.stack([rng.choice(E, k, replace=False) for _ in range(T)]) for _ in range(2)]).astype(np.int32)
    out = vp.demand(torch.from_numpy(R).cuda(), N, E, 4096, first_rank=first if first + 2 <= N else N - 2,
                    sort_row=1)
    torch.cuda.synchronize()
    fr = first if first + 2 <= N else N - 2
    assert vp.read_status(out["status"]) == 0
    for r in range(2):
        ref = oracle.demand(R[r], N, E, fr + r, 4096)
        assert np.array_equal(out["demand"][r].cpu().numpy(), ref["row"])
        assert np.array_equal(out["counts"][r].cpu().numpy(), ref["counts"])
    ref = oracle.demand(R[1], N, E, fr + 1, 4096)
    assert np.array_equal(out["sorted_tok"].cpu().numpy()[:T * k], ref["sorted_tok"])
    assert np.array_equal(out["sorted_slot"].cpu().numpy()[:T * k], ref["sorted_slot"])
    assert np.array_equal(out["dest_off"].cpu().numpy(), ref["dest_off"])


def test_demand_reused_workspace_and_single_rank(vp):
    """One workspace, zero-filled once, serves calls of every shape in turn
    (nothing in it needs clearing between calls): all rows of the 64-rank workload,
    then one rank's own row (R = 1, the deployed unit) at each end of the
    rank range, then the 8-rank workload, then all 64 rows again; each call
    element-wise against the oracle."""
    ws = torch.zeros(vp.demand_workspace_bytes(64, 16384, 8, 256), dtype=torch.uint8, device="cuda")
    w3, R3, dem3, D3 = moe_case(3)
    w1, R1, dem1, D1 = moe_case(1)
    calls = [(w3, R3, dem3, 0, 64, 5), (w3, R3, dem3, 0, 1, 0), (w3, R3, dem3, 63, 1, 0), (w1, R1, dem1, 0, 8, 7),
             (w3, R3, dem3, 0, 64, 63)]
    for w, R, dem, first, nrows, sort_row in calls:
        log("demand reuse: N=%d first=%d R=%d sort_row=%d" % (w.n_ranks, first, nrows, sort_row))
        out = vp.demand(torch.from_numpy(np.ascontiguousarray(R[first:first + nrows])).cuda(), w.n_ranks,
                        w.experts, w.row_bytes, first_rank=first, sort_row=sort_row, ws=ws)
        torch.cuda.synchronize()
        assert vp.read_status(out["status"]) == 0
        for r in range(nrows):
            assert np.array_equal(out["demand"][r].cpu().numpy(), dem[first + r]["row"])
            assert np.array_equal(out["counts"][r].cpu().numpy(), dem[first + r]["counts"])
        ref = dem[first + sort_row]
        assert np.array_equal(out["sorted_tok"].cpu().numpy(), ref["sorted_tok"])
        assert np.array_equal(out["sorted_slot"].cpu().numpy(), ref["sorted_slot"])
        assert np.array_equal(out["dest_off"].cpu().numpy(), ref["dest_off"])


@pytest.mark.parametrize("cid,rank,tokens", [(1, 0, None), (1, 7, None), (5, 0, None), (5, 255, None), (5, 100, 1000),
                                             (5, 3, 4097), (5, 9, 4095)])
def test_demand_one_rank(vp, cid, rank, tokens):
    """One rank's own row (R = 1, the deployed unit) with its sort: rows of up
    to 32,768 ids take the one-launch path, longer ones the two-pass path
    (4,097 tokens of top-8); ragged lengths; every output element-wise
    against the oracle."""
    w = vpgen.config(cid)
    R = vpgen.routing(w, rank, 0, tokens)
    log("demand one rank C%d rank %d T=%d" % (cid, rank, R.shape[0]))
    ref = oracle.demand(R, w.n_ranks, w.experts, rank, w.row_bytes)
    out = vp.demand(torch.from_numpy(np.ascontiguousarray(R[None])).cuda(), w.n_ranks, w.experts, w.row_bytes,
                    first_rank=rank, sort_row=0)
    torch.cuda.synchronize()
    assert vp.read_status(out["status"]) == 0
    assert np.array_equal(out["demand"][0].cpu().numpy(), ref["row"])
    assert np.array_equal(out["counts"][0].cpu().numpy(), ref["counts"])
    n = R.size
    assert np.array_equal(out["sorted_tok"][:n].cpu().numpy(), ref["sorted_tok"])
    assert np.array_equal(out["sorted_slot"][:n].cpu().numpy(), ref["sorted_slot"])
    assert np.array_equal(out["dest_off"].cpu().numpy(), ref["dest_off"])


def test_demand_one_rank_bad_id(vp):
    """A bad id in a one-launch row is reported; the others are still counted."""
    w = vpgen.config(1)
    R = vpgen.routing(w, 0, 0, 100).copy()
    R[7, 1] = w.experts
    out = vp.demand(torch.from_numpy(R[None]).cuda(), w.n_ranks, w.experts, w.row_bytes, sort_row=0)
    torch.cuda.synchronize()
    assert vp.read_status(out["status"]) == vp.INVALID_ARGUMENT
    good = R[R < w.experts]
    assert int(out["counts"][0].sum().item()) == good.size


def test_demand_empty_and_bad_ids(vp):
    log("demand empty / bad ids")
    R = torch.zeros((1, 0, 2), dtype=torch.int32, device="cuda")
    out = vp.demand(R, 8, 32, 4096)
    torch.cuda.synchronize()
    assert vp.read_status(out["status"]) == 0
    assert (out["demand"] == 0).all() and (out["dest_off"] == 0).all()
    bad = torch.zeros((1, 16, 2), dtype=torch.int32, device="cuda")
    bad[0, 3, 1] = 32
    out = vp.demand(bad, 8, 32, 4096)
    torch.cuda.synchronize()
    assert vp.read_status(out["status"]) == vp.INVALID_ARGUMENT
    bad[0, 3, 1] = -1
    out = vp.demand(bad, 8, 32, 4096)
    torch.cuda.synchronize()
    assert vp.read_status(out["status"]) == vp.INVALID_ARGUMENT


def test_demand_heads_parity(vp):
    w, hl, D = heads_case()
    log("heads demand parity")
    st = vp.new_status()
    out = vp.demand_heads(w.tokens, torch.from_numpy(hl).cuda(), w.row_bytes, 0, w.n_ranks, status=st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    assert np.array_equal(out.cpu().numpy(), D)


# ------------------------------------------------------------------ plan

@pytest.mark.parametrize("cid", [1, 2, 4, 3, 5])
def test_plan_parity_full_size(vp, cid):
    if cid == 4:
        w, _, D = heads_case()
    else:
        w, _, _, D = moe_case(cid)
    log("plan parity C%d (N=%d)" % (cid, w.n_ranks))
    g = gpu_plan(vp, w.topo, D, w.row_bytes, layout=cid in (2, 5))
    assert g["status"] == 0
    o = oracle_plan(cid, D)
    assert_schedule_equal(g, o)
    if cid in (2, 5):
        so, co = layout_np(o["dst"], o["bytes"])
        assert np.array_equal(g["send_off"], so)
        assert np.array_equal(g["stream_off"], co)


def test_plan_parity_second_matrix_of_streams(vp):
    for cid in (3, 5):
        w, _, _, D = moe_case(cid, matrix=1)
        log("plan parity C%d matrix 1" % cid)
        g = gpu_plan(vp, w.topo, D, w.row_bytes)
        assert g["status"] == 0
        assert_schedule_equal(g, oracle_plan(cid, D, matrix=1))


def random_demand(rng, N, unit, density, scale):
    D = rng.integers(0, scale + 1, (N, N)) * (rng.random((N, N)) < density)
    np.fill_diagonal(D, 0)
    return (D * unit).astype(np.int64)


@pytest.mark.parametrize("topo", [vpgen.tiny_topology(), vpgen.config(1).topo, vpgen.config(2).topo,
                                  vpgen.Topology(3, 1, 2, 3), vpgen.Topology(2, 2, 1, 4),
                                  vpgen.Topology(1, 1, 1, 4), vpgen.Topology(4, 1, 3, 2, 1, 32, 50),
                                  # several NICs per switch (two NIC lanes may join one slot pair)
                                  vpgen.Topology(1, 1, 2, 2, 2), vpgen.Topology(1, 2, 1, 2, 2),
                                  vpgen.Topology(2, 1, 2, 2, 2), vpgen.Topology(3, 1, 2, 2, 3),
                                  vpgen.Topology(1, 1, 2, 3, 2)])
def test_plan_parity_random_demands(vp, topo):
    rng = np.random.default_rng(topo.n_ranks)
    oc = ocat(topo)
    unit = 4096
    for case, (density, scale, kw) in enumerate([
            (0.3, 5, {}), (1.0, 50, {}), (0.05, 3, {}), (1.0, 7, dict(lambda_ns=0)),
            (0.6, 20, dict(n_start=1)), (0.6, 20, dict(n_start=7, seed=12345)),
            (0.6, 20, dict(i_aa=0)), (0.6, 20, dict(k_target=topo.n_ranks))]):
        D = random_demand(rng, topo.n_ranks, unit, density, scale)
        kw = dict(kw, k_max=64 * topo.n_ranks)   # dense random demands can need more than 8N steps
        log("plan random topo N=%d case %d %s" % (topo.n_ranks, case, kw))
        g = gpu_plan(vp, topo, D, unit, **kw)
        o = oc.plan(D, unit, **kw)
        assert g["status"] == o["status"] == 0
        assert_schedule_equal(g, o)


def test_plan_empty_demand(vp):
    log("plan empty")
    topo = vpgen.config(1).topo
    g = gpu_plan(vp, topo, np.zeros((8, 8), np.int64), 4096)
    assert g["status"] == 0 and g["K"] == 0


def test_plan_device_errors(vp):
    topo = vpgen.config(1).topo
    log("plan errors")
    D = np.zeros((8, 8), np.int64)
    D[2, 2] = 4096
    assert gpu_plan(vp, topo, D, 4096)["status"] == vp.INVALID_DEMAND
    D[2, 2] = 0
    D[1, 5] = 4097
    assert gpu_plan(vp, topo, D, 4096)["status"] == vp.INVALID_DEMAND
    D[1, 5] = -4096
    assert gpu_plan(vp, topo, D, 4096)["status"] == vp.INVALID_DEMAND
    w, _, _, D1 = moe_case(1)
    g = gpu_plan(vp, topo, D1, w.row_bytes, k_max=3)
    o = ocat(topo).plan(D1, w.row_bytes, k_max=3, check=False)
    assert g["status"] == vp.CAPACITY == o["status"]
    assert_schedule_equal(g, o)


@pytest.mark.parametrize("case", ["entry_2p62_block", "entry_2p42", "cap_2p31_bytes", "cap_2p27_units",
                                  "total_2p42_bytes", "total_2p28_units", "invalid_first"])
def test_plan_device_limits(vp, case):
    """Each device-side refusal of the planner on a small 8-rank input: the
    kernel reports a status, emits nothing and returns.  Expected statuses
    follow from the documented limits by hand: tau = ceil(L_max / (32 *
    k_target)) and cap = tau * 32 at the PCIe rate."""
    topo = vpgen.config(1).topo
    log("plan device limit %s" % case)
    D = np.zeros((8, 8), np.int64)
    unit, kt, want = 1 << 20, 4096, vp.UNSUPPORTED
    if case == "entry_2p62_block":
        # every row, column and total sum of this block wraps to 0 in int64
        D[0:4, 4:8] = 1 << 62
    elif case == "entry_2p42":
        D[0, 1] = 1 << 42
    elif case == "cap_2p31_bytes":
        D[0, 1], kt = 1 << 31, 1          # tau = 2^26 ns, cap = 2^31 B
    elif case == "cap_2p27_units":
        D[0, 1], kt, unit = 1 << 30, 1, 8  # cap = 2^30 B = 2^27 units
    elif case == "total_2p42_bytes":
        D[0, 1] = D[2, 3] = 1 << 41        # caps 2^29 B, 2^22 units in all
    elif case == "total_2p28_units":
        D[0, 1] = D[2, 3] = 1 << 31
        unit = 16                          # 2^28 units; caps 2^19 B
    else:
        D[0, 1] = 1 << 42
        D[2, 2] = unit                     # an invalid entry wins over a limit
        want = vp.INVALID_DEMAND
    g = gpu_plan(vp, topo, D, unit, k_target=kt)
    assert g["status"] == want and g["K"] == 0


def test_plan_rejects_schedule_too_large_for_32_bit_offsets(vp):
    """k_max * N * 8 >= 2^32 is refused on the host before anything is
    enqueued (the planner addresses a matrix's schedule with 32-bit byte
    offsets); the buffers passed are small and never touched."""
    topo = vpgen.config(1).topo
    log("plan k_max limit")
    cat = gcat(vp, topo)
    p = vp.plan_params(cat.N, 4096, k_max=(1 << 29) // cat.N)
    out = vp.alloc_schedule(cat.N, 1, layout=True)
    D = torch.zeros((cat.N, cat.N), dtype=torch.int64, device="cuda")
    with pytest.raises(vp.VPError) as e:
        vp.plan(cat, D, p, out=out)
    assert e.value.status == vp.UNSUPPORTED and "k_max" in str(e.value)
    torch.cuda.synchronize()


def test_plan_deterministic(vp):
    w, _, _, D = moe_case(2)
    log("plan determinism")
    a = gpu_plan(vp, w.topo, D, w.row_bytes)
    b = gpu_plan(vp, w.topo, D, w.row_bytes)
    assert_schedule_equal(a, b)


# ------------------------------------------------------------------ pack

def upload_schedule(vp, N, sched_np, layout=False):
    """Device schedule buffers holding sched_np (and its buffer layout)."""
    sched = vp.alloc_schedule(N, 8 * N, layout=layout)
    K = sched_np["K"]
    sched["K"].fill_(K)
    if K:
        sched["dst"][:K] = torch.from_numpy(sched_np["dst"]).cuda()
        sched["bytes"][:K] = torch.from_numpy(sched_np["bytes"]).cuda()
        if layout:
            so, co = layout_np(sched_np["dst"], sched_np["bytes"])
            sched["send_off"][:K] = torch.from_numpy(so).cuda()
            sched["stream_off"][:K] = torch.from_numpy(co).cuda()
    return sched


def gpu_pack_rows(vp, w, R, sched_np, self_rank, tokens_np, cap_extra=0, cap=None, layout=False):
    rt = torch.from_numpy(R).cuda()
    dem = vp.demand(rt, w.n_ranks, w.experts, w.row_bytes, sort_row=self_rank)
    sched = upload_schedule(vp, w.n_ranks, sched_np, layout)
    K = sched_np["K"]
    total = int(sched_np["bytes"][:, self_rank].sum()) if K else 0
    cap = total + cap_extra if cap is None else cap
    send = torch.full((max(cap, 16),), 0xA5, dtype=torch.uint8, device="cuda")
    step_off = torch.empty(8 * w.n_ranks + 1, dtype=torch.int64, device="cuda")
    st = dem["status"]
    tok = torch.from_numpy(tokens_np).cuda()
    vp.pack_rows(tok, w.row_bytes, dem["sorted_tok"], dem["sorted_slot"], dem["dest_off"], self_rank, sched,
                 send[:cap] if cap else send[:0], step_off, st)
    torch.cuda.synchronize()
    return send, step_off, vp.read_status(st), total


@pytest.mark.parametrize("layout", [False, True])
@pytest.mark.parametrize("cid,self_rank", [(1, 0), (1, 5), (2, 0), (2, 9), (3, 0), (5, 0)])
def test_pack_rows_parity_full_size(vp, cid, self_rank, layout):
    w, R, dem, D = moe_case(cid)
    log("pack rows parity C%d rank %d layout %s" % (cid, self_rank, layout))
    s = oracle_plan(cid, D)
    tok = vpgen.tokens_bf16(w, self_rank)
    ref, ref_off = oracle.pack_rows(tok, w.row_bytes, dem[self_rank]["sorted_tok"],
                                    dem[self_rank]["dest_off"], self_rank, s)
    send, step_off, st, total = gpu_pack_rows(vp, w, R, s, self_rank, tok, cap_extra=64, layout=layout)
    assert st == 0
    assert total == ref.size
    assert torch.equal(send[:total], torch.from_numpy(ref).cuda())
    assert (send[total:total + 64] == 0xA5).all(), "wrote past the packed bytes"
    assert np.array_equal(step_off[:s["K"] + 1].cpu().numpy(), ref_off)


@pytest.mark.parametrize("row_bytes,cid", [(16, 1), (1040, 1), (4112, 2), (12304, 1), (36880, 1), (65536, 1)])
def test_pack_rows_parity_row_sizes(vp, row_bytes, cid):
    """Rows of one vector, ragged last passes, several rows per workgroup
    (top-2 and top-8), and rows past the in-register limit of the scatter,
    which are copied in chunks."""
    w = vpgen.config(cid)
    T = 512
    R = vpgen.routing_all(w, 0, T)
    log("pack rows parity C%d T=%d row %d" % (cid, T, row_bytes))
    dem = [oracle.demand(R[i], w.n_ranks, w.experts, i, row_bytes) for i in range(w.n_ranks)]
    D = np.stack([d["row"] for d in dem])
    s = ocat(w.topo).plan(D, row_bytes)
    tok = np.random.default_rng(row_bytes).integers(0, 256, (T, row_bytes), dtype=np.uint8)
    ref, ref_off = oracle.pack_rows(tok, row_bytes, dem[0]["sorted_tok"], dem[0]["dest_off"], 0, s)
    rt = torch.from_numpy(R).cuda()
    d = vp.demand(rt, w.n_ranks, w.experts, row_bytes, sort_row=0)
    sched = upload_schedule(vp, w.n_ranks, s, False)
    send = torch.full((ref.size + 64,), 0xA5, dtype=torch.uint8, device="cuda")
    step_off = torch.empty(8 * w.n_ranks + 1, dtype=torch.int64, device="cuda")
    vp.pack_rows(torch.from_numpy(tok).cuda(), row_bytes, d["sorted_tok"], d["sorted_slot"], d["dest_off"], 0,
                 sched, send[:ref.size], step_off, d["status"])
    torch.cuda.synchronize()
    assert vp.read_status(d["status"]) == 0
    assert torch.equal(send[:ref.size], torch.from_numpy(ref).cuda())
    assert (send[ref.size:] == 0xA5).all(), "wrote past the packed bytes"
    assert np.array_equal(step_off[:s["K"] + 1].cpu().numpy(), ref_off)


@pytest.mark.parametrize("layout", [False, True])
def test_pack_rows_capacity_error_writes_nothing(vp, layout):
    w, R, dem, D = moe_case(1)
    log("pack capacity error, layout %s" % layout)
    s = oracle_plan(1, D)
    tok = vpgen.tokens_bf16(w, 0)
    total = int(s["bytes"][:, 0].sum())
    send, _, st, _ = gpu_pack_rows(vp, w, R, s, 0, tok, cap=total - w.row_bytes, layout=layout)
    assert st == vp.CAPACITY
    assert (send == 0xA5).all()


@pytest.mark.parametrize("layout", [False, True])
def test_pack_rows_empty_schedule(vp, layout):
    w, R, dem, D = moe_case(1)
    log("pack rows, empty schedule, layout %s" % layout)
    s = dict(K=0, dst=np.zeros((0, w.n_ranks), np.int32), bytes=np.zeros((0, w.n_ranks), np.int64))
    send, step_off, st, total = gpu_pack_rows(vp, w, R, s, 0, vpgen.tokens_bf16(w, 0), cap_extra=64,
                                              layout=layout)
    assert st == 0 and total == 0
    assert int(step_off[0].item()) == 0
    assert (send == 0xA5).all()


@pytest.mark.parametrize("layout", [False, True])
@pytest.mark.parametrize("bad", ["token_id", "slot"])
def test_pack_rows_bad_token_list_writes_nothing(vp, bad, layout):
    """A token id or a routing slot out of range is reported and leaves the
    send buffer untouched."""
    w, R, dem, D = moe_case(1)
    log("pack rows, bad token list (%s)" % bad)
    s = oracle_plan(1, D)
    rt = torch.from_numpy(R).cuda()
    d = vp.demand(rt, w.n_ranks, w.experts, w.row_bytes, sort_row=0)
    lo, hi = int(d["dest_off"][1].item()), int(d["dest_off"][2].item())
    assert hi - lo > w.top_k
    if bad == "token_id":
        d["sorted_tok"][lo:hi] = w.tokens
    else:
        d["sorted_slot"][lo:hi] = w.top_k
    sched = upload_schedule(vp, w.n_ranks, s, layout)
    total = int(s["bytes"][:, 0].sum())
    send = torch.full((total,), 0xA5, dtype=torch.uint8, device="cuda")
    step_off = torch.empty(8 * w.n_ranks + 1, dtype=torch.int64, device="cuda")
    vp.pack_rows(torch.from_numpy(vpgen.tokens_bf16(w, 0)).cuda(), w.row_bytes, d["sorted_tok"],
                 d["sorted_slot"], d["dest_off"], 0, sched, send, step_off, d["status"])
    torch.cuda.synchronize()
    assert vp.read_status(d["status"]) == vp.INVALID_ARGUMENT
    assert (send == 0xA5).all()


def test_pipeline_reuse_across_matrices(vp):
    """One Pipeline, several matrices in a row: every call starts from its
    own inputs (the per-token copy lists are rebuilt each time)."""
    w = vpgen.config(2)
    pipe = vp.Pipeline(w.topo, "moe", w.row_bytes, n_experts=w.experts, tokens=w.tokens, top_k=w.top_k)
    tok = vpgen.tokens_bf16(w, 0)
    tok_d = torch.from_numpy(tok).cuda()
    for m in (1, 2, 1):
        log("pipeline reuse C2 matrix %d" % m)
        R = vpgen.routing_all(w, m)
        send = pipe.step(routing=torch.from_numpy(R).cuda(), tokens=tok_d)
        torch.cuda.synchronize()
        assert vp.read_status(pipe.status) == 0
        dem = [oracle.demand(R[i], w.n_ranks, w.experts, i, w.row_bytes) for i in range(w.n_ranks)]
        D = np.stack([x["row"] for x in dem])
        s = oracle.Catalog(w.topo).plan(D, w.row_bytes)
        ref, _ = oracle.pack_rows(tok, w.row_bytes, dem[0]["sorted_tok"], dem[0]["dest_off"], 0, s)
        assert torch.equal(send[:ref.size], torch.from_numpy(ref).cuda())


@pytest.mark.parametrize("layout", [False, True])
@pytest.mark.parametrize("self_rank", [0, 7, 12, 15])
def test_pack_heads_parity(vp, self_rank, layout):
    w, hl, D = heads_case()
    log("pack heads parity rank %d layout %s" % (self_rank, layout))
    s = oracle_plan(4, D)
    act = vpgen.tokens_bf16(w, self_rank)
    ref, ref_off = oracle.pack_heads(act, w.token_stride, hl, w.row_bytes, self_rank, s)
    sched = upload_schedule(vp, w.n_ranks, s, layout)
    K = s["K"]
    send = torch.full((ref.size + 32,), 0xA5, dtype=torch.uint8, device="cuda")
    step_off = torch.empty(8 * w.n_ranks + 1, dtype=torch.int64, device="cuda")
    st = vp.new_status()
    vp.pack_heads(torch.from_numpy(act).cuda(), w.token_stride, torch.from_numpy(hl).cuda(), w.row_bytes,
                  self_rank, sched, send[:ref.size], step_off, st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    assert torch.equal(send[:ref.size], torch.from_numpy(ref).cuda())
    assert (send[ref.size:] == 0xA5).all()
    assert np.array_equal(step_off[:K + 1].cpu().numpy(), ref_off)


# (N, self rank, head bytes, heads per rank, tokens, steps, largest slice in
# units, spare send capacity in units, row padding in bytes)
HEADS_SHAPES = [
    (4, 1, 16, [1, 2, 5, 3], 777, 600, 4, 0, 0),
    (3, 0, 48, [2, 2, 3], 513, 60, 200, 7, 48),
    (5, 4, 4096, [1, 3, 2, 1, 2], 100, 40, 30, 0, 0),
    (6, 2, 272, [2, 1, 1, 3, 2, 2], 1000, 120, 500, 1000, 16),
    (2, 1, 256, [3, 1], 4096, 9, 4096, 20000, 0),
]


def random_heads_schedule(rng, N, self_rank, T, hl, K, max_units, unit):
    """A schedule whose lane for self_rank sends, step by step, the next
    slice of a random destination's head stream (a quarter of the steps
    idle, streams partly covered when the steps run out); the other lanes
    are a fixed derangement with no bytes, which the pack never reads."""
    left = T * np.diff(hl)
    left[self_rank] = 0
    dst = np.empty((K, N), np.int32)
    nb = np.zeros((K, N), np.int64)
    rows = np.arange(N)
    for k in range(K):
        dst[k] = (rows + 1 + k % (N - 1)) % N
        open_ = np.flatnonzero(left > 0)
        if open_.size == 0 or rng.random() < 0.25:
            continue
        j = int(rng.choice(open_))
        x = int(rng.integers(1, min(left[j], max_units) + 1))
        dst[k, self_rank] = j
        nb[k, self_rank] = x * unit
        left[j] -= x
    return {"K": K, "dst": dst, "bytes": nb}


@pytest.mark.parametrize("layout", [False, True])
@pytest.mark.parametrize("shape", range(len(HEADS_SHAPES)))
def test_pack_heads_shapes(vp, shape, layout):
    """The heads pack on random schedules over other shapes than the
    Ulysses workload: 16-byte heads with more than 256 steps of a few units
    each (the gather's two-level step search, ranges that meet many steps),
    48- and 272-byte heads (unit vectors not a power of two), 4 KiB heads,
    a destination with one head, padded token rows, send buffers much
    larger than the total, and a few long steps over a two-rank stream."""
    N, self_rank, unit, per, T, K, max_units, spare, pad = HEADS_SHAPES[shape]
    log("pack heads shape %d layout %s" % (shape, layout))
    rng = np.random.default_rng(100 + shape)
    hl = np.concatenate([[0], np.cumsum(per)]).astype(np.int64)
    stride = int(hl[-1]) * unit + pad
    act = rng.integers(0, 256, T * stride, dtype=np.uint8)
    s = random_heads_schedule(rng, N, self_rank, T, hl, K, max_units, unit)
    ref, ref_off = oracle.pack_heads(act, stride, hl, unit, self_rank, s)
    k_max = K + 3
    sched = vp.alloc_schedule(N, k_max, layout=layout)
    sched["K"].fill_(K)
    sched["dst"][:K] = torch.from_numpy(s["dst"]).cuda()
    sched["bytes"][:K] = torch.from_numpy(s["bytes"]).cuda()
    if layout:
        so, co = layout_np(s["dst"], s["bytes"])
        sched["send_off"][:K] = torch.from_numpy(so).cuda()
        sched["stream_off"][:K] = torch.from_numpy(co).cuda()
    cap = ref.size + spare * unit
    send = torch.full((cap + 64,), 0xA5, dtype=torch.uint8, device="cuda")
    step_off = torch.empty(k_max + 1, dtype=torch.int64, device="cuda")
    st = vp.new_status()
    vp.pack_heads(torch.from_numpy(act).cuda(), stride, torch.from_numpy(hl).cuda(), unit, self_rank, sched,
                  send[:cap], step_off, st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    assert torch.equal(send[:ref.size], torch.from_numpy(ref).cuda())
    assert (send[ref.size:] == 0xA5).all()
    assert np.array_equal(step_off[:K + 1].cpu().numpy(), ref_off)


@pytest.mark.parametrize("layout", [False, True])
@pytest.mark.parametrize("case", ["capacity", "k", "heads", "self", "status"])
def test_pack_heads_errors_write_nothing(vp, case, layout):
    """Malformed calls of the heads pack set dev_status and write nothing to
    the send buffer, on the one-kernel path (the planner's layout) and the
    slice-kernel path: a send buffer one head short (VP_ERR_CAPACITY), K
    above k_max, a destination whose heads run past the token row, a lane of
    this rank that sends to itself, and an error already in dev_status
    (kept, nothing copied)."""
    w, hl, D = heads_case()
    log("pack heads error %s layout %s" % (case, layout))
    s_np = oracle_plan(4, D)
    ref, _ = oracle.pack_heads(vpgen.tokens_bf16(w, 0), w.token_stride, hl, w.row_bytes, 0, s_np)
    sched = upload_schedule(vp, w.n_ranks, s_np, layout)
    K = s_np["K"]
    cap = ref.size
    hl_bad = hl.copy()
    st = vp.new_status()
    want = vp.INVALID_ARGUMENT
    if case == "capacity":
        cap = ref.size - w.row_bytes
        want = vp.CAPACITY
    elif case == "k":
        sched["K"].fill_(8 * w.n_ranks + 1)
    elif case == "heads":
        hl_bad[-1] += 1   # the last destination's heads end past the row
    elif case == "self":
        k = int(np.flatnonzero(s_np["bytes"][:, 0] > 0)[0])
        sched["dst"][k, 0] = 0
    else:
        st.fill_(vp.NO_PROGRESS)
        want = vp.NO_PROGRESS
    send = torch.full((cap + 64,), 0xA5, dtype=torch.uint8, device="cuda")
    step_off = torch.empty(8 * w.n_ranks + 1, dtype=torch.int64, device="cuda")
    vp.pack_heads(torch.from_numpy(vpgen.tokens_bf16(w, 0)).cuda(), w.token_stride, torch.from_numpy(hl_bad).cuda(),
                  w.row_bytes, 0, sched, send[:cap], step_off, st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == want
    assert (send == 0xA5).all()
    assert K > 0


@pytest.mark.parametrize("where", ["first", "middle", "last"])
def test_pack_rejects_a_layout_that_does_not_tile(vp, where):
    """A send-offset layout that leaves a gap (here one unit) is refused by
    both packs before anything is copied: the rows pack on the 8-rank
    workload and the heads pack on the Ulysses workload, the latter on a
    workspace that a valid call filled just before."""
    log("pack gapped layout %s" % where)
    # rows
    w, R, dem, D = moe_case(1)
    s = oracle_plan(1, D)
    carrying = np.flatnonzero(s["bytes"][:, 0] > 0)
    k = {"first": 0, "middle": int(carrying[len(carrying) // 2]), "last": int(carrying[-1])}[where]
    rt = torch.from_numpy(R).cuda()
    gd = vp.demand(rt, w.n_ranks, w.experts, w.row_bytes, sort_row=0)
    sched = upload_schedule(vp, w.n_ranks, s, layout=True)
    sched["send_off"][k:, 0] += w.row_bytes
    total = int(s["bytes"][:, 0].sum())
    send = torch.full((total + 2 * w.row_bytes,), 0xA5, dtype=torch.uint8, device="cuda")
    step_off = torch.empty(8 * w.n_ranks + 1, dtype=torch.int64, device="cuda")
    st = gd["status"]
    vp.pack_rows(torch.from_numpy(vpgen.tokens_bf16(w, 0)).cuda(), w.row_bytes, gd["sorted_tok"],
                 gd["sorted_slot"], gd["dest_off"], 0, sched, send, step_off, st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == vp.INVALID_ARGUMENT
    assert (send == 0xA5).all()
    # heads: one valid call, then the gapped layout on the same workspace
    w, hl, D = heads_case()
    s = oracle_plan(4, D)
    act = torch.from_numpy(vpgen.tokens_bf16(w, 0)).cuda()
    hl_d = torch.from_numpy(hl).cuda()
    ref, _ = oracle.pack_heads(vpgen.tokens_bf16(w, 0), w.token_stride, hl, w.row_bytes, 0, s)
    sched = upload_schedule(vp, w.n_ranks, s, layout=True)
    cap = ref.size + 2 * w.row_bytes
    send = torch.full((cap,), 0xA5, dtype=torch.uint8, device="cuda")
    step_off = torch.empty(8 * w.n_ranks + 1, dtype=torch.int64, device="cuda")
    ws = torch.zeros(vp.pack_workspace_bytes(8 * w.n_ranks, cap, w.row_bytes), dtype=torch.uint8, device="cuda")
    st = vp.new_status()
    vp.pack_heads(act, w.token_stride, hl_d, w.row_bytes, 0, sched, send, step_off, st, ws=ws)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0 and torch.equal(send[:ref.size], torch.from_numpy(ref).cuda())
    carrying = np.flatnonzero(s["bytes"][:, 0] > 0)
    k = {"first": 0, "middle": int(carrying[len(carrying) // 2]), "last": int(carrying[-1])}[where]
    sched["send_off"][k:, 0] += w.row_bytes
    send.fill_(0xA5)
    vp.pack_heads(act, w.token_stride, hl_d, w.row_bytes, 0, sched, send, step_off, st, ws=ws)
    torch.cuda.synchronize()
    assert vp.read_status(st) == vp.INVALID_ARGUMENT
    assert (send == 0xA5).all()


# -------------------------------------------------------------- pipeline

@pytest.mark.parametrize("cid", [1, 4, 5])
def test_pipeline_matches_oracle(vp, cid):
    """The whole hot path as the benchmark runs it (one stream, no host sync
    between demand, plan and pack) against the oracle, end to end."""
    log("pipeline C%d" % cid)
    if cid == 4:
        w, hl, D = heads_case()
        pipe = vp.Pipeline(w.topo, "heads", w.row_bytes, tokens=w.tokens, token_stride=w.token_stride)
        act = vpgen.tokens_bf16(w, 0)
        send = pipe.step(tokens=torch.from_numpy(act).cuda(), head_lo=torch.from_numpy(hl).cuda())
        torch.cuda.synchronize()
        s = oracle_plan(4, D)
        ref, _ = oracle.pack_heads(act, w.token_stride, hl, w.row_bytes, 0, s)
    else:
        w, R, dem, D = moe_case(cid)
        pipe = vp.Pipeline(w.topo, "moe", w.row_bytes, n_experts=w.experts, tokens=w.tokens, top_k=w.top_k)
        tok = vpgen.tokens_bf16(w, 0)
        send = pipe.step(routing=torch.from_numpy(R).cuda(), tokens=torch.from_numpy(tok).cuda())
        torch.cuda.synchronize()
        s = oracle_plan(cid, D)
        ref, _ = oracle.pack_rows(tok, w.row_bytes, dem[0]["sorted_tok"], dem[0]["dest_off"], 0, s)
    assert vp.read_status(pipe.status) == 0
    assert np.array_equal(pipe.dem["demand"].cpu().numpy(), D)
    assert_schedule_equal(vp.schedule_to_host(pipe.sched), s)
    assert torch.equal(send[:ref.size], torch.from_numpy(ref).cuda())


@pytest.mark.parametrize("cid", [1, 4])
def test_pack_two_halves_match_one_call(vp, cid):
    """vp_pack_prepare_* followed by vp_pack_gather gives the send buffer and
    step offsets of the one-call pack on the pipeline's schedule; for heads
    the two halves are a different kernel pair than the one-kernel pack."""
    log("pack halves C%d" % cid)
    if cid == 4:
        w, hl, D = heads_case()
        pipe = vp.Pipeline(w.topo, "heads", w.row_bytes, tokens=w.tokens, token_stride=w.token_stride)
        tok = torch.from_numpy(vpgen.tokens_bf16(w, 0)).cuda()
        head_lo = torch.from_numpy(hl).cuda()
        one = pipe.step(tokens=tok, head_lo=head_lo).clone()
    else:
        w, R, dem, D = moe_case(cid)
        pipe = vp.Pipeline(w.topo, "moe", w.row_bytes, n_experts=w.experts, tokens=w.tokens, top_k=w.top_k)
        tok = torch.from_numpy(vpgen.tokens_bf16(w, 0)).cuda()
        head_lo = None
        one = pipe.step(routing=torch.from_numpy(R).cuda(), tokens=tok).clone()
    torch.cuda.synchronize()
    assert vp.read_status(pipe.status) == 0
    K = int(pipe.sched["K"].item())
    off_one = pipe.step_off[:K + 1].clone()
    two = torch.full_like(one, 0x5A)
    pipe.step_off.fill_(-1)
    pipe.pack_prepare_stage(tok, head_lo)
    pipe.pack_gather_stage(tok, two)
    torch.cuda.synchronize()
    assert vp.read_status(pipe.status) == 0
    total = int(off_one[K].item())
    assert total > 0
    assert torch.equal(pipe.step_off[:K + 1], off_one)
    assert torch.equal(two[:total], one[:total])


@pytest.mark.parametrize("cid", [1, 4])
def test_pack_replayed_from_a_hip_graph(vp, cid):
    """The pack records no memset, so a caller may capture it in a HIP graph:
    the one-call pack (rows: prepare and scatter; heads: the one-kernel pack)
    captured once and replayed three times, with an eager plan of another
    matrix and a host synchronisation between replays, gives the eager send
    buffer and step offsets after every replay."""
    log("pack graph C%d" % cid)
    if cid == 4:
        w, hl, D = heads_case()
        pipe = vp.Pipeline(w.topo, "heads", w.row_bytes, tokens=w.tokens, token_stride=w.token_stride)
        tok = torch.from_numpy(vpgen.tokens_bf16(w, 0)).cuda()
        head_lo = torch.from_numpy(hl).cuda()
        pipe.step(tokens=tok, head_lo=head_lo)
        other = torch.from_numpy(np.ascontiguousarray(D.T)).cuda()
    else:
        w, R, dem, D = moe_case(cid)
        pipe = vp.Pipeline(w.topo, "moe", w.row_bytes, n_experts=w.experts, tokens=w.tokens, top_k=w.top_k)
        tok = torch.from_numpy(vpgen.tokens_bf16(w, 0)).cuda()
        head_lo = None
        pipe.step(routing=torch.from_numpy(R).cuda(), tokens=tok)
        other = torch.from_numpy(np.ascontiguousarray(D.T)).cuda()
    torch.cuda.synchronize()
    assert vp.read_status(pipe.status) == 0
    K = int(pipe.sched["K"].item())
    total = int(pipe.step_off[K].item())
    eager = pipe.send[:total].clone()
    off = pipe.step_off[:K + 1].clone()
    send = torch.zeros_like(pipe.send)
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        pipe.pack_stage(tok, head_lo, send)
    torch.cuda.current_stream().wait_stream(side)
    with torch.cuda.graph(g):
        pipe.pack_stage(tok, head_lo, send)
    sched_other = vp.alloc_schedule(pipe.N, pipe.params.k_max, layout=True)
    for rep in range(3):
        send.zero_()
        pipe.step_off.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert vp.read_status(pipe.status) == 0
        assert torch.equal(send[:total], eager), rep
        assert torch.equal(pipe.step_off[:K + 1], off), rep
        # unrelated eager work between replays: a plan of another matrix
        vp.plan(pipe.cat, other, pipe.params, out=sched_other)
        torch.cuda.synchronize()


@pytest.mark.parametrize("cid", [1, 4])
def test_whole_step_replayed_from_a_hip_graph(vp, cid):
    """No call of the hot path records a memset, allocates or synchronises
    with the host, so a whole step -- demand (and control words), plan, pack
    -- can be captured in one HIP graph.  Replayed three times, with every
    output cleared before each replay and an eager plan of another matrix and
    a host synchronisation after it, each replay gives the eager step's
    demand matrix, schedule, buffer layout, step offsets and send buffer."""
    log("whole step graph C%d" % cid)
    if cid == 4:
        w, hl, D = heads_case()
        pipe = vp.Pipeline(w.topo, "heads", w.row_bytes, tokens=w.tokens, token_stride=w.token_stride)
        kw = dict(tokens=torch.from_numpy(vpgen.tokens_bf16(w, 0)).cuda(), head_lo=torch.from_numpy(hl).cuda())
    else:
        w, R, dem, D = moe_case(cid)
        pipe = vp.Pipeline(w.topo, "moe", w.row_bytes, n_experts=w.experts, tokens=w.tokens, top_k=w.top_k)
        kw = dict(routing=torch.from_numpy(R).cuda(), tokens=torch.from_numpy(vpgen.tokens_bf16(w, 0)).cuda())
    send = torch.zeros_like(pipe.send)
    pipe.step(send=send, **kw)
    torch.cuda.synchronize()
    assert vp.read_status(pipe.status) == 0
    K = int(pipe.sched["K"].item())
    total = int(pipe.step_off[K].item())
    outs = dict(demand=pipe.dem["demand"], K=pipe.sched["K"], family=pipe.sched["family"], dst=pipe.sched["dst"],
                bytes=pipe.sched["bytes"], send_off=pipe.sched["send_off"], stream_off=pipe.sched["stream_off"],
                step_off=pipe.step_off)
    eager = {k: v.clone() for k, v in outs.items()}
    eager_send = send[:total].clone()
    assert K > 0 and total > 0
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        pipe.step(send=send, **kw)
    torch.cuda.current_stream().wait_stream(side)
    with torch.cuda.graph(g):
        pipe.step(send=send, **kw)
    other = torch.from_numpy(np.ascontiguousarray(D.T)).cuda()
    sched_other = vp.alloc_schedule(pipe.N, pipe.params.k_max, layout=True)
    for rep in range(3):
        send.zero_()
        for v in outs.values():
            v.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert vp.read_status(pipe.status) == 0, rep
        for k, v in outs.items():
            # rows up to K are the schedule; the rest is not written
            a, b = (v[:K + 1], eager[k][:K + 1]) if k == "step_off" else (
                (v[:K], eager[k][:K]) if k in ("family", "dst", "bytes", "send_off", "stream_off") else (v, eager[k]))
            assert torch.equal(a, b), (rep, k)
        assert torch.equal(send[:total], eager_send), rep
        vp.plan(pipe.cat, other, pipe.params, out=sched_other)
        torch.cuda.synchronize()


def test_plan_largest_topology_parity(vp):
    """1,024 ranks (128 nodes), the planner's largest shape, under a MoE-like
    skew (light traffic between every pair plus a global hot tenth of the
    destinations, vpgen.hot_destinations_demand): the schedule hashes to the
    oracle's (stored by tests/golden/make_stream_digests.py --ranks-1024; the
    oracle takes about ten minutes there), and has the properties any valid
    schedule has -- the activations sum to D exactly, every step is a
    derangement whose lanes use path classes of their group pairs and share
    no modeled resource (Eq. (1)), every step serves bytes, and K stays
    within k_max (raised to 32N)."""
    import json
    import stream_digest as sd
    topo = vpgen.Topology(128)
    N = topo.n_ranks
    unit = 4096
    D = vpgen.hot_destinations_demand(N, unit, 1024)
    log("plan on 1024 ranks")
    # every pair carries bytes: the caller gives room beyond the default 8N
    g = gpu_plan(vp, topo, D, unit, k_max=32 * N)
    assert g["status"] == 0
    K = g["K"]
    log("1024 ranks: K = %d" % K)
    assert N - 1 <= K <= 32 * N
    dst, nb, inst = g["dst"], g["bytes"], g["inst"]
    rows = np.arange(N)
    for k in range(K):
        assert np.array_equal(np.sort(dst[k]), rows) and not (dst[k] == rows).any()
    X = np.zeros((N, N), np.int64)
    np.add.at(X, (np.broadcast_to(rows, (K, N)), dst), nb)
    assert np.array_equal(X, D)
    assert (nb.sum(axis=1) > 0).all()
    with open(sd.GOLDEN_1024) as f:
        ref = json.load(f)
    assert sd.demand_digest(D) == ref["demand"]
    assert (K, g["tau"]) == (ref["K"], ref["tau"])
    assert sd.schedule_digest(g) == ref["schedule"]
    cls = gcat(vp, topo).instances()["cls"][inst]
    # every step's lanes are resource-disjoint (Eq. (1)) on the topology model
    from oracle.checks import TopoModel, schedule_valid_np
    schedule_valid_np(TopoModel(topo), D, dst, cls, nb)
    gs, gd = rows[None, :] // topo.gpus_per_switch, dst // topo.gpus_per_switch
    Q = topo.sockets_per_node * topo.switches_per_socket
    same_switch = gs == gd
    same_socket = (gs // Q == gd // Q) & ((gs % Q) // topo.switches_per_socket == (gd % Q) // topo.switches_per_socket)
    assert (cls[same_switch] == vp.PATH_PIX).all()
    assert np.isin(cls[same_socket & ~same_switch], [vp.PATH_PXB, vp.PATH_NIC]).all()
    assert (cls[~same_socket] == vp.PATH_NIC).all()
