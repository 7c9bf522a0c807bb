"""Pins of the oracle's sparse expert-parallel control words (Sec. 5,
efficient sparse data movement for expert parallelism).

- hand-worked words (tests/golden/control_words.json), including a count
  that overflows the 32 - L count bits;
- a pair gets a word exactly when its demand entry is nonzero;
- the bitmap's bits are the destination's experts with a nonzero count
  (np.nonzero), and the count field is the count of the highest of them;
- the receiver's decode (bitmap skips, the word's count for the designated
  expert, signals for the rest) rebuilds the counts block of every
  destination, whatever the signals hold where they are not read.
"""
import json
import os

import numpy as np
import pytest

import oracle
import vpgen

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "control_words.json")


def load():
    with open(GOLDEN) as f:
        return json.load(f)


@pytest.mark.parametrize("i", range(4))
def test_hand_worked_words(i):
    c = load()["cases"][i]
    w = oracle.control_words(np.array(c["counts"], np.int32), c["N"], c["self"])
    assert w.tolist() == c["words"], c["derivation"]


def test_count_overflow_is_a_capacity_error():
    c = load()["overflow"]
    with pytest.raises(oracle.OracleError) as e:
        oracle.control_words(np.array(c["counts"], np.int32), c["N"], c["self"])
    assert e.value.status == oracle.CAPACITY
    ok = list(c["counts"])
    ok[-1] -= 1   # 2^24 - 1 rows fit
    w = oracle.control_words(np.array(ok, np.int32), c["N"], c["self"])
    assert int(w[1]) >> 8 == (1 << 24) - 1


def test_too_many_local_experts_is_unsupported():
    with pytest.raises(oracle.OracleError) as e:
        oracle.control_words(np.zeros(64, np.int32), 2, 0)
    assert e.value.status == oracle.UNSUPPORTED


@pytest.mark.parametrize("cid", [1, 2, 3, 5])
def test_words_follow_the_counts(cid):
    w = vpgen.config(cid)
    N, E = w.n_ranks, w.experts
    L = E // N
    for r in (0, N - 1):
        R = vpgen.routing(w, r, 0, 1024)
        d = oracle.demand(R, N, E, r, w.row_bytes)
        words = oracle.control_words(d["counts"], N, r)
        assert np.array_equal(words != 0, d["row"] != 0)
        blocks = d["counts"].reshape(N, L)
        for j in range(N):
            if j == r:
                continue
            active = np.nonzero(blocks[j])[0]
            bitmap = int(words[j]) & ((1 << L) - 1)
            assert [l for l in range(L) if bitmap >> l & 1] == active.tolist()
            if active.size:
                assert int(words[j]) >> L == int(blocks[j][active[-1]])


@pytest.mark.parametrize("cid", [1, 2, 5])
def test_receiver_rebuilds_the_counts(cid):
    w = vpgen.config(cid)
    N, E = w.n_ranks, w.experts
    L = E // N
    counts = np.stack([oracle.demand(vpgen.routing(w, i, 0, 512), N, E, i, w.row_bytes)["counts"]
                       for i in range(N)])
    words = np.stack([oracle.control_words(counts[i], N, i) for i in range(N)])
    rng = np.random.default_rng(cid)
    for r in (0, N // 2, N - 1):
        block = counts[:, r * L:(r + 1) * L].copy()
        block[r] = 0                       # nothing travels to oneself
        # signals carry the counts of the active experts; the others hold junk
        signal = np.where(block > 0, block, rng.integers(1, 1000, block.shape)).astype(np.int32)
        got = oracle.receive_counts(words[:, r], signal, L)
        assert np.array_equal(got, block)
