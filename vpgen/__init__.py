"""Seeded synthetic inputs for the demand -> plan -> pack path.

This module is shared by the oracle side and the HIP side as a source of
*inputs only*.  It contains no arithmetic of the scheduling method: no demand
counting, no catalog, no planning, no packing.  It produces

* topology parameters (node / socket / switch / GPU counts and link rates),
* token -> expert routing tables (top-k without replacement under a stated
  expert-popularity law),
* bf16 token rows and Ulysses-style head splits,
* demand matrices given directly for AlltoAll / skew AlltoAllv cases and the
  head/context layouts of a Wan2.1-like sequence-parallel model,

for the five workload configurations C1..C5 that stand in for the paper's
workloads (random top-k MoE routing over 256 experts with k = 8 and hidden
7168, Qwen3-30B-A3B-like prefill, and Wan2.1-like 40-head sequence
parallelism; Sec. 6 "Workloads", "Large-scale experiment", Sec. 6.2).

Seeding: numpy PCG64 keyed by ``SeedSequence([0, config, matrix, rank])``
for per-rank draws and ``SeedSequence([0, config, matrix])`` for per-matrix
draws (expert permutation, hot set).
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

__all__ = [
    "Topology", "Workload", "CONFIGS", "config", "tiny_topology",
    "routing", "routing_all", "tokens_bf16", "head_split", "bf16_from_f32",
    "expert_weights", "DemandCase", "EXTRA", "extra", "uniform_demand", "zipf_pair_demand",
    "hc_groups", "hc_layout", "hot_destinations_demand", "random_routing",
]


@dataclasses.dataclass(frozen=True)
class Topology:
    """PCIe cluster parameters (rank = ((node*S + socket)*W + switch)*g + local)."""
    n_nodes: int
    sockets_per_node: int = 2
    switches_per_socket: int = 2
    gpus_per_switch: int = 2
    nics_per_switch: int = 1
    pcie_bytes_per_ns: int = 32
    nic_bytes_per_ns: int = 25
    flags: int = 0           # bit 0: peer-to-peer between sockets of a node (SYS paths)

    @property
    def n_ranks(self) -> int:
        return (self.n_nodes * self.sockets_per_node * self.switches_per_socket
                * self.gpus_per_switch)

    def as_tuple(self):
        return (self.n_nodes, self.sockets_per_node, self.switches_per_socket,
                self.gpus_per_switch, self.nics_per_switch,
                self.pcie_bytes_per_ns, self.nic_bytes_per_ns, self.flags)


@dataclasses.dataclass(frozen=True)
class Workload:
    cid: int                 # 1..5
    name: str
    topo: Topology
    mode: str                # "moe" or "heads"
    tokens: int              # tokens per rank
    hidden: int              # MoE hidden size (bf16 elements)
    experts: int = 0
    top_k: int = 0
    law: str = "uniform"     # uniform | zipf | hot
    zipf_s: float = 0.0
    perm_per_matrix: bool = False
    hot_frac: float = 0.0
    hot_mass: float = 0.0
    heads: int = 0
    head_dim: int = 0
    n_matrices: int = 1

    @property
    def n_ranks(self) -> int:
        return self.topo.n_ranks

    @property
    def row_bytes(self) -> int:
        """Pack granule in bytes: one bf16 token row (MoE) or one head (Ulysses)."""
        if self.mode == "moe":
            return self.hidden * 2
        return self.head_dim * 2

    @property
    def token_stride(self) -> int:
        if self.mode == "moe":
            return self.hidden * 2
        return self.heads * self.head_dim * 2


CONFIGS = {
    1: Workload(1, "tiny-8gpu-moe", Topology(1), "moe", tokens=2048, hidden=2048,
                experts=32, top_k=2, law="uniform"),
    2: Workload(2, "qwen3-30b-a3b-like-16", Topology(2), "moe", tokens=8192, hidden=2048,
                experts=128, top_k=8, law="zipf", zipf_s=1.2),
    3: Workload(3, "dynamic-zipf-64", Topology(8), "moe", tokens=16384, hidden=4096,
                experts=256, top_k=8, law="zipf", zipf_s=1.0, perm_per_matrix=True,
                n_matrices=100),
    4: Workload(4, "ulysses-wan21-like-16", Topology(2), "heads", tokens=2048, hidden=0,
                heads=40, head_dim=128),
    5: Workload(5, "deepseek-v3-like-256", Topology(32), "moe", tokens=4096, hidden=7168,
                experts=256, top_k=8, law="hot", hot_frac=0.1, hot_mass=0.5,
                perm_per_matrix=True, n_matrices=1000),
}


def config(cid: int) -> Workload:
    return CONFIGS[cid]


def tiny_topology() -> Topology:
    """One node, one socket, two switches of two GPUs, one NIC per switch."""
    return Topology(1, sockets_per_node=1, switches_per_socket=2, gpus_per_switch=2)


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def expert_weights(w: Workload, matrix: int = 0) -> np.ndarray:
    """Per-draw expert popularity p(e) (sums to 1) for one demand matrix."""
    E = w.experts
    if w.law == "uniform":
        return np.full(E, 1.0 / E)
    m = matrix if w.perm_per_matrix else 0
    r = _rng(0, w.cid, m)
    if w.law == "zipf":
        perm = r.permutation(E)            # expert perm[i] has popularity rank i+1
        p = np.empty(E)
        p[perm] = (np.arange(1, E + 1, dtype=np.float64)) ** (-w.zipf_s)
        return p / p.sum()
    if w.law == "hot":
        n_hot = int(round(w.hot_frac * E))
        hot = r.permutation(E)[:n_hot]
        p = np.full(E, (1.0 - w.hot_mass) / (E - n_hot))
        p[hot] = w.hot_mass / n_hot
        return p
    raise ValueError(w.law)


def _topk_without_replacement(r: np.random.Generator, p: np.ndarray, T: int, k: int) -> np.ndarray:
    """Successive weighted draws without replacement, by rejection of repeats.

    Rejecting an already-drawn expert and redrawing from p is exactly a draw
    from p renormalised over the experts not yet drawn, so each row is a
    sequential sample without replacement (same law as Gumbel-top-k).
    """
    E = p.shape[0]
    cdf = np.cumsum(p)
    cdf /= cdf[-1]
    out = np.empty((T, k), dtype=np.int32)
    for d in range(k):
        need = np.arange(T)
        while need.size:
            c = np.searchsorted(cdf, r.random(need.size), side="right")
            c = np.minimum(c, E - 1).astype(np.int32)
            if d:
                dup = (out[need, :d] == c[:, None]).any(axis=1)
            else:
                dup = np.zeros(need.size, dtype=bool)
            out[need[~dup], d] = c[~dup]
            need = need[dup]
    return out


def routing(w: Workload, rank: int, matrix: int = 0, tokens: Optional[int] = None) -> np.ndarray:
    """int32 [T, k] expert ids of one source rank's tokens for one matrix."""
    if w.mode != "moe":
        raise ValueError("routing is defined for MoE workloads only")
    T = w.tokens if tokens is None else tokens
    r = _rng(0, w.cid, matrix, rank)
    p = expert_weights(w, matrix)
    return _topk_without_replacement(r, p, T, w.top_k)


def routing_all(w: Workload, matrix: int = 0, tokens: Optional[int] = None) -> np.ndarray:
    """int32 [N, T, k]: every rank's routing for one matrix."""
    return np.stack([routing(w, rk, matrix, tokens) for rk in range(w.n_ranks)])


def random_routing(seed: int, n_ranks: int, tokens: int, experts: int, top_k: int,
                   zipf_s: float) -> np.ndarray:
    """int32 [N, T, k]: every rank's top-k distinct experts per token, each
    draw weighted by popularity rank^-zipf_s over one random permutation of
    the experts shared by all ranks (zipf_s = 0 is uniform); for randomized
    shapes outside the named workloads."""
    r = _rng(7, seed)
    perm = r.permutation(experts)
    p = np.empty(experts)
    p[perm] = (np.arange(1, experts + 1, dtype=np.float64)) ** (-zipf_s)
    p /= p.sum()
    return np.stack([_topk_without_replacement(_rng(7, seed, rk), p, tokens, top_k) for rk in range(n_ranks)])


def bf16_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round to nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def tokens_bf16(w: Workload, rank: int = 0, tokens: Optional[int] = None) -> np.ndarray:
    """uint16 bf16 bits of one rank's activations.

    MoE: [T, hidden].  Ulysses: [T, heads, head_dim].  Values are N(0, 1).
    """
    T = w.tokens if tokens is None else tokens
    r = _rng(0, w.cid, 0, 1_000_000 + rank)
    if w.mode == "moe":
        shape = (T, w.hidden)
    else:
        shape = (T, w.heads, w.head_dim)
    return bf16_from_f32(r.standard_normal(shape, dtype=np.float32))


def head_split(heads: int, n_ranks: int) -> np.ndarray:
    """int64 [N+1] first head owned by each rank (contiguous ranges).

    The heads are spread as evenly as possible with the larger shares on the
    last ranks: 40 heads on 16 ranks gives 2 heads to ranks 0-7 and 3 to
    ranks 8-15.
    """
    base, extra = divmod(heads, n_ranks)
    counts = np.full(n_ranks, base, dtype=np.int64)
    if extra:
        counts[n_ranks - extra:] += 1
    return np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)


# ---------------------------------------------------------------------------
# Demand matrices given directly (AlltoAll / AlltoAllv microbenchmarks) and
# the Wan2.1 head/context layouts (Sec. 6 "Workloads", skew AlltoAllv,
# Sec. 6.2 Wan2.1, Sec. 6.3 ablation).  Only inputs: byte volumes drawn or
# laid out here are what a caller asks the scheduler to move.
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class DemandCase:
    name: str
    topo: Topology
    unit: int               # pack granule; every entry is a multiple of it
    kind: str               # "uniform" | "zipf_pairs" | "ulysses_hc"
    per_pair: int = 0       # uniform: bytes per ordered pair
    per_rank: int = 0       # zipf_pairs: bytes each source sends in total (before rounding)
    zipf_s: float = 0.0
    seq: int = 0            # ulysses_hc: global sequence length
    heads: int = 0
    head_dim: int = 0
    H: int = 0              # head-parallel degree (ranks of one all-to-all group)
    C: int = 0              # context-parallel degree (number of groups)


EXTRA = {
    "uniform-16": DemandCase("uniform-16", Topology(2), 4096, "uniform", per_pair=64 << 20),
    "zipf-pairs-16-s0.4": DemandCase("zipf-pairs-16-s0.4", Topology(2), 4096, "zipf_pairs", per_rank=1 << 30,
                                     zipf_s=0.4),
    "zipf-pairs-16-s0.6": DemandCase("zipf-pairs-16-s0.6", Topology(2), 4096, "zipf_pairs", per_rank=1 << 30,
                                     zipf_s=0.6),
    "zipf-pairs-16-s0.8": DemandCase("zipf-pairs-16-s0.8", Topology(2), 4096, "zipf_pairs", per_rank=1 << 30,
                                     zipf_s=0.8),
    # the same skew and layout on nodes whose sockets reach each other peer to
    # peer (SYS paths), where a path choice exists for every intra-node pair
    "zipf-pairs-16-s0.6-sys": DemandCase("zipf-pairs-16-s0.6-sys", Topology(2, flags=1), 4096, "zipf_pairs",
                                         per_rank=1 << 30, zipf_s=0.6),
    "wan21-H8C1-sys": DemandCase("wan21-H8C1-sys", Topology(1, flags=1), 256, "ulysses_hc", seq=75600, heads=40,
                                 head_dim=128, H=8, C=1),
    "wan21-H8C1": DemandCase("wan21-H8C1", Topology(1), 256, "ulysses_hc", seq=75600, heads=40, head_dim=128,
                             H=8, C=1),
    "wan21-H4C2": DemandCase("wan21-H4C2", Topology(1), 256, "ulysses_hc", seq=75600, heads=40, head_dim=128,
                             H=4, C=2),
    "wan21-H8C2": DemandCase("wan21-H8C2", Topology(2), 256, "ulysses_hc", seq=75600, heads=40, head_dim=128,
                             H=8, C=2),
    "wan21-H4C4": DemandCase("wan21-H4C4", Topology(2), 256, "ulysses_hc", seq=75600, heads=40, head_dim=128,
                             H=4, C=4),
}


def extra(name: str) -> DemandCase:
    return EXTRA[name]


def uniform_demand(case: DemandCase) -> np.ndarray:
    """int64 [N, N]: every rank sends case.per_pair bytes to every other rank."""
    N = case.topo.n_ranks
    D = np.full((N, N), case.per_pair, dtype=np.int64)
    np.fill_diagonal(D, 0)
    return D


def hot_destinations_demand(n_ranks: int = 1024, unit: int = 4096, seed: int = 1024) -> np.ndarray:
    """int64 [N, N] MoE-like skew at the planner's largest shape: 0-7 units
    between every pair plus 20-59 more toward a global hot tenth of the
    destinations, times 32 units (tens of units per quantum at K_target = 2N).
    numpy PCG64 seeded by `seed`."""
    rng = np.random.default_rng(seed)
    N = n_ranks
    D = rng.integers(0, 8, (N, N)).astype(np.int64)
    hot = rng.choice(N, N // 10, replace=False)
    D[:, hot] += rng.integers(20, 60, (N, hot.size))
    np.fill_diagonal(D, 0)
    return D * (32 * unit)


def zipf_pair_demand(case: DemandCase, matrix: int = 0) -> np.ndarray:
    """int64 [N, N] skew AlltoAllv demand: each source splits about
    case.per_rank bytes over its N - 1 destinations with Zipf(s) weights
    (1/rank^s) over a per-source random order of the destinations, each
    volume rounded down to the unit.  Seeded by (1, s in thousandths,
    matrix, source)."""
    N, u = case.topo.n_ranks, case.unit
    w = np.arange(1, N, dtype=np.float64) ** (-case.zipf_s)
    w /= w.sum()
    D = np.zeros((N, N), dtype=np.int64)
    for i in range(N):
        r = _rng(1, int(round(case.zipf_s * 1000)), matrix, i)
        dst = np.array([j for j in range(N) if j != i])
        order = r.permutation(N - 1)
        units = np.floor(w * (case.per_rank // u)).astype(np.int64)
        D[i, dst[order]] = units * u
    return D


def hc_groups(case: DemandCase) -> np.ndarray:
    """int64 [C, H]: the ranks of each head-parallel all-to-all group
    (contiguous blocks of H ranks)."""
    N = case.topo.n_ranks
    if case.H * case.C != N:
        raise ValueError("H * C must equal the rank count")
    return np.arange(N, dtype=np.int64).reshape(case.C, case.H)


def hc_layout(case: DemandCase):
    """(tokens per rank, head split of one group): each rank holds
    seq / (H*C) tokens of all heads; inside its group the heads are split
    evenly over the H ranks."""
    if case.seq % (case.H * case.C) or case.heads % case.H:
        raise ValueError("sequence and heads must divide evenly")
    return case.seq // (case.H * case.C), head_split(case.heads, case.H)
