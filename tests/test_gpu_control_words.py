"""GPU parity of the sparse expert-parallel control words (Sec. 5) and of
their decode at the receiver, against the oracle, bit-exact."""
import sys

import numpy as np
import pytest
import torch

import oracle
import vpgen

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def vp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_34340_amd as vp
    vp.lib()
    return vp


def words_np(t):
    return t.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("cid", [1, 2, 3, 5])
def test_control_words_parity_full_size(vp, cid):
    w = vpgen.config(cid)
    N, E = w.n_ranks, w.experts
    log("control words parity C%d (N=%d, L=%d)" % (cid, N, E // N))
    R = vpgen.routing_all(w, 0)
    d = vp.demand(torch.from_numpy(R).cuda(), N, E, w.row_bytes, sort_row=-1)
    words = vp.control_words(d["counts"], N, status=d["status"])
    torch.cuda.synchronize()
    assert vp.read_status(d["status"]) == 0
    counts = d["counts"].cpu().numpy()
    ref = np.stack([oracle.control_words(counts[i], N, i) for i in range(N)])
    assert np.array_equal(words_np(words), ref)
    # a pair has a word exactly when it has demand
    assert np.array_equal(words_np(words) != 0, d["demand"].cpu().numpy() != 0)


def test_control_words_row_subset_and_errors(vp):
    """Rows first_rank.. of a larger cluster; a count past the 32 - L bits and
    a negative count are reported; L > 31 is refused on the host."""
    rng = np.random.default_rng(3)
    N, E = 16, 128
    counts = rng.integers(0, 3, (5, E)).astype(np.int32)
    counts[:, ::7] = 0
    c = torch.from_numpy(counts).cuda()
    st = vp.new_status()
    words = vp.control_words(c, N, first_rank=9, status=st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    ref = np.stack([oracle.control_words(counts[i], N, 9 + i) for i in range(5)])
    assert np.array_equal(words_np(words), ref)

    big = counts.copy()
    big[2, 3 * 8 + 7] = 1 << 24          # L = 8: 24 count bits, designated expert 7 of rank 3
    st = vp.new_status()
    vp.control_words(torch.from_numpy(big).cuda(), N, first_rank=0, status=st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == vp.CAPACITY
    neg = counts.copy()
    neg[1, 40] = -1
    st = vp.new_status()
    vp.control_words(torch.from_numpy(neg).cuda(), N, first_rank=0, status=st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == vp.INVALID_ARGUMENT
    with pytest.raises(vp.VPError):
        vp.control_words(torch.zeros((1, 64), dtype=torch.int32, device="cuda"), 2)


@pytest.mark.parametrize("cid", [1, 2, 5])
def test_receive_counts_parity(vp, cid):
    """Each receiver decodes its column of the words with per-expert signals
    (junk where the decode must not read) and gets the oracle's counts."""
    w = vpgen.config(cid)
    N, E = w.n_ranks, w.experts
    L = E // N
    log("receive counts parity C%d" % cid)
    R = vpgen.routing_all(w, 0, 1024)
    d = vp.demand(torch.from_numpy(R).cuda(), N, E, w.row_bytes, sort_row=-1)
    words = vp.control_words(d["counts"], N, status=d["status"])
    counts = d["counts"].cpu().numpy()
    wn = np.stack([oracle.control_words(counts[i], N, i) for i in range(N)])
    rng = np.random.default_rng(cid)
    for r in sorted({0, 1, N // 2, N - 1}):
        block = counts[:, r * L:(r + 1) * L]
        signal = np.where(block > 0, block, rng.integers(1, 1000, block.shape)).astype(np.int32)
        signal[r] = rng.integers(1, 1000, L)
        ref = oracle.receive_counts(wn[:, r], signal, L)
        got = vp.receive_counts(words, N, torch.from_numpy(signal).cuda(), L, offset=r)
        torch.cuda.synchronize()
        assert np.array_equal(got.cpu().numpy(), ref), "receiver %d" % r
        # the gathered-vector form (stride 1)
        col = words[:, r].contiguous()
        got1 = vp.receive_counts(col, 1, torch.from_numpy(signal).cuda(), L)
        torch.cuda.synchronize()
        assert np.array_equal(got1.cpu().numpy(), ref)
    assert vp.read_status(d["status"]) == 0


@pytest.mark.parametrize("N,L,seed", [(3, 1, 0), (8, 2, 1), (7, 5, 2), (16, 16, 3), (5, 31, 4), (64, 4, 5)])
def test_control_words_random(vp, N, L, seed):
    """Random sparse counts for 1 to 31 local experts per rank, counts up to
    the largest the 32 - L count bits hold: the words of every source, and
    every receiver's decode of its column, against the oracle."""
    rng = np.random.default_rng(seed)
    E = N * L
    limit = (1 << (32 - L)) - 1
    counts = rng.integers(0, min(limit, 1 << 20) + 1, (N, E)).astype(np.int64)
    counts[rng.random((N, E)) < 0.5] = 0
    hot = rng.random((N, E)) < 0.05
    counts[hot] = limit                                # the largest count a word carries
    counts = counts.astype(np.int32)
    log("control words random N=%d L=%d" % (N, L))
    c = torch.from_numpy(counts).cuda()
    st = vp.new_status()
    words = vp.control_words(c, N, status=st)
    torch.cuda.synchronize()
    assert vp.read_status(st) == 0
    ref = np.stack([oracle.control_words(counts[i], N, i) for i in range(N)])
    assert np.array_equal(words_np(words), ref)
    for r in range(N):
        block = counts[:, r * L:(r + 1) * L]
        signal = np.where(block > 0, block, rng.integers(1, 1000, block.shape)).astype(np.int32)
        want = oracle.receive_counts(ref[:, r], signal, L)
        got = vp.receive_counts(words, N, torch.from_numpy(signal).cuda(), L, offset=r)
        torch.cuda.synchronize()
        assert np.array_equal(got.cpu().numpy(), want), "receiver %d" % r
        exp = block.copy()
        exp[r] = 0                                     # no words to itself
        assert np.array_equal(want, exp)
