"""GPU parity over whole demand streams.

Every matrix of the 64-rank stream (100 matrices, expert permutation redrawn
per matrix) and of the 256-rank stream (1000 matrices, hot set redrawn per
matrix) runs through demand -> plan -> pack on the GPU; the demand matrix,
the whole schedule, rank 0's step offsets and a strided sample of its send
buffer must hash to the digests the oracle wrote (golden/stream_digests.json
and golden/stream_digests_256_all.json, made by golden/make_stream_digests.py).
Routing for the next matrices is generated in worker processes while the GPU
works."""
import json
import multiprocessing as mp
import sys
import time

import numpy as np
import pytest
import torch

import stream_digest as sd
import vpgen

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def golden():
    with open(sd.GOLDEN) as f:
        g = json.load(f)
    assert g["sample_stride"] == sd.SAMPLE_STRIDE
    return g


def check_stream(cid, rows):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_34340_amd as vp
    w = vpgen.config(cid)
    log("stream parity C%d: %d matrices (N=%d)" % (cid, len(rows), w.n_ranks))
    pipe = vp.Pipeline(w.topo, "moe", w.row_bytes, n_experts=w.experts, tokens=w.tokens, top_k=w.top_k)
    tok = torch.from_numpy(vpgen.tokens_bf16(w, 0)).cuda()
    ctx = mp.get_context("spawn")
    t0 = time.time()
    bad = []
    with ctx.Pool(sd.pool_size()) as pool:
        for n, (m, R) in enumerate(pool.imap(sd.routing_job, [(cid, r["matrix"]) for r in rows])):
            ref = rows[n]
            assert ref["matrix"] == m
            send = pipe.step(routing=torch.from_numpy(R).cuda(), tokens=tok)
            torch.cuda.synchronize()
            assert vp.read_status(pipe.status) == 0, "device error %d at matrix %d" % (
                vp.read_status(pipe.status), m)
            h = vp.schedule_to_host(pipe.sched)
            K = h["K"]
            length = int(pipe.step_off[K].item())
            got = dict(K=K, tau=h["tau"], demand=sd.demand_digest(pipe.dem["demand"].cpu().numpy()),
                       schedule=sd.schedule_digest(h), send_bytes=length,
                       send=sd.send_digest(send[:length:sd.SAMPLE_STRIDE].cpu().numpy(), length),
                       step_off=sd.step_off_digest(pipe.step_off[:K + 1].cpu().numpy()))
            diff = [k for k in got if got[k] != ref[k]]
            if diff:
                bad.append((m, diff))
            if n % 10 == 9:
                log("  C%d: %d matrices checked, %d differ (%.0f s)" % (cid, n + 1, len(bad), time.time() - t0))
    assert not bad, "matrices differing from the oracle: %s" % bad[:10]


@pytest.mark.parametrize("cid", [3])
def test_stream_parity(golden, cid):
    rows = golden["streams"][str(cid)]["matrices"]
    assert [r["matrix"] for r in rows] == sd.STREAMS[cid]
    check_stream(cid, rows)


def test_stream_parity_all_256():
    """All 1000 matrices of the 256-rank stream (about a minute on one GPU)."""
    with open(sd.GOLDEN_ALL5) as f:
        g = json.load(f)
    rows = g["streams"]["5"]["matrices"]
    assert [r["matrix"] for r in rows] == list(range(1000))
    check_stream(5, rows)
