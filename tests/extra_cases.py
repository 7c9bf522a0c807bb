"""Demand of the extra cases (uniform AlltoAll, skew AlltoAllv, Wan2.1-like
head/context layouts) on each side: given matrices come from the seeded
generators; the head/context layouts are built per all-to-all group with the
oracle's or the library's head demand and placed on the block diagonal."""
import numpy as np

import vpgen

NAMES = list(vpgen.EXTRA)
ZIPF_MATRICES = 5   # the ablation replays five skew matrices


def oracle_demand(case, matrix=0):
    import oracle
    if case.kind == "uniform":
        return vpgen.uniform_demand(case)
    if case.kind == "zipf_pairs":
        return vpgen.zipf_pair_demand(case, matrix)
    N = case.topo.n_ranks
    T, hl = vpgen.hc_layout(case)
    D = np.zeros((N, N), np.int64)
    for grp in vpgen.hc_groups(case):
        for h, r in enumerate(grp):
            D[r, grp] = oracle.demand_heads(T, hl, case.unit, h)
    return D


def gpu_demand(vp, case, matrix=0):
    """int64 [N, N] on the GPU; head/context demand from vp_demand_heads."""
    import torch
    if case.kind != "ulysses_hc":
        D = vpgen.uniform_demand(case) if case.kind == "uniform" else vpgen.zipf_pair_demand(case, matrix)
        return torch.from_numpy(D).cuda()
    N = case.topo.n_ranks
    T, hl = vpgen.hc_layout(case)
    hl_d = torch.from_numpy(hl).cuda()
    D = torch.zeros((N, N), dtype=torch.int64, device="cuda")
    for grp in vpgen.hc_groups(case):
        lo, hi = int(grp[0]), int(grp[-1]) + 1
        blk = vp.demand_heads(T, hl_d, case.unit, first_rank=0, R=case.H)
        D[lo:hi, lo:hi] = blk
    return D
