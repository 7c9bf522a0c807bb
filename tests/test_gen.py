"""Checks on the seeded synthetic inputs (no method arithmetic involved)."""
import numpy as np
import pytest
import torch

import vpgen


def test_configs_match_workload_shapes():
    c = vpgen.CONFIGS
    assert [c[i].n_ranks for i in range(1, 6)] == [8, 16, 64, 16, 256]
    assert [c[i].row_bytes for i in range(1, 6)] == [4096, 4096, 8192, 256, 14336]
    assert c[4].token_stride == 10240
    assert c[5].experts == 256 and c[5].top_k == 8 and c[5].hidden == 7168


@pytest.mark.parametrize("cid", [1, 2, 3, 5])
def test_routing_rows_are_distinct_and_in_range(cid):
    w = vpgen.config(cid)
    r = vpgen.routing(w, 3, matrix=0, tokens=512)
    assert r.shape == (512, w.top_k) and r.dtype == np.int32
    assert r.min() >= 0 and r.max() < w.experts
    s = np.sort(r, axis=1)
    assert (np.diff(s, axis=1) > 0).all(), "top-k draws repeat an expert"


def test_routing_is_deterministic_and_rank_seeded():
    w = vpgen.config(2)
    a = vpgen.routing(w, 1, 0, tokens=256)
    b = vpgen.routing(w, 1, 0, tokens=256)
    c = vpgen.routing(w, 2, 0, tokens=256)
    assert (a == b).all() and not (a == c).all()


def test_zipf_first_draw_frequencies():
    # the first draw of every token follows p(e) exactly
    w = vpgen.config(2)
    p = vpgen.expert_weights(w)
    r = vpgen.routing(w, 0, tokens=200_000)
    f = np.bincount(r[:, 0], minlength=w.experts) / r.shape[0]
    assert np.abs(f - p).max() < 5 * np.sqrt(p.max() / r.shape[0])
    # the most popular expert has weight 1 / H(128, 1.2)
    H = (np.arange(1, 129) ** -1.2).sum()
    assert abs(p.max() - 1 / H) < 1e-12


def test_permutation_redrawn_per_matrix():
    w = vpgen.config(3)
    assert not np.allclose(vpgen.expert_weights(w, 0), vpgen.expert_weights(w, 1))
    w2 = vpgen.config(2)
    assert np.allclose(vpgen.expert_weights(w2, 0), vpgen.expert_weights(w2, 7))


def test_hot_set_mass():
    w = vpgen.config(5)
    p = vpgen.expert_weights(w, 0)
    hot = np.argsort(-p)[:26]
    assert abs(p[hot].sum() - 0.5) < 1e-12 and len(np.unique(p)) == 2
    r = vpgen.routing(w, 0, 0, tokens=20_000)
    share = np.isin(r, hot).mean()
    # without replacement the realised hot share sits a little under 50 %
    assert 0.40 < share < 0.5


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(10_000).astype(np.float32)
    x[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -0.0, 65504.0]   # ties and specials
    ours = vpgen.bf16_from_f32(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (ours == ref).all()


def test_head_split():
    hl = vpgen.head_split(40, 16)
    counts = np.diff(hl)
    assert hl[0] == 0 and hl[-1] == 40
    assert (counts[:8] == 2).all() and (counts[8:] == 3).all()


def test_random_routing_shapes_and_law():
    R = vpgen.random_routing(5, 3, 4000, 24, 4, 1.0)
    assert R.shape == (3, 4000, 4) and R.dtype == np.int32
    assert R.min() >= 0 and R.max() < 24
    assert all(len(set(row)) == 4 for row in R.reshape(-1, 4))          # distinct per token
    assert np.array_equal(R, vpgen.random_routing(5, 3, 4000, 24, 4, 1.0))
    assert not np.array_equal(R[0], R[1])                                # ranks draw apart
    # first draws follow rank^-1 over the shared permutation: the most
    # popular expert is drawn about 1 / H_24 of the time
    first = np.bincount(R[:, :, 0].ravel(), minlength=24) / R[:, :, 0].size
    h = (1.0 / np.arange(1, 25)).sum()
    assert abs(first.max() - 1.0 / h) < 0.02
    u = vpgen.random_routing(1, 1, 20000, 8, 1, 0.0)                     # zipf 0: uniform
    assert np.abs(np.bincount(u.ravel(), minlength=8) / 20000 - 0.125).max() < 0.01
