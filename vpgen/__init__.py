"""Seeded synthetic inputs for the demand -> plan -> pack path.

This module is shared by the oracle side and the HIP side as a source of
*inputs only*.  It contains no arithmetic of the scheduling method: no demand
counting, no catalog, no planning, no packing.  It produces

* topology parameters (node / socket / switch / GPU counts and link rates),
* token -> expert routing tables (top-k without replacement under a stated
  expert-popularity law),
* bf16 token rows and Ulysses-style head splits,

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
    "expert_weights",
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

    @property
    def n_ranks(self) -> int:
        return (self.n_nodes * self.sockets_per_node * self.switches_per_socket
                * self.gpus_per_switch)

    def as_tuple(self):
        return (self.n_nodes, self.sockets_per_node, self.switches_per_socket,
                self.gpus_per_switch, self.nics_per_switch,
                self.pcie_bytes_per_ns, self.nic_bytes_per_ns)


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
