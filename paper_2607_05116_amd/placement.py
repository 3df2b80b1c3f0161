"""Co-activation driven expert placement on the host (Sec. IV-B, Algorithm 1
and the node stage), plus the placement metrics of Eq. 2-4.

Input: the co-activation counts that cap_coactivation produces on a pruned
routing trace (Sec. VII: place on pruned traces).  Output: expert_rank and
expert_local arrays for cap_topology.

Readings of points the paper leaves open (one line each):
  p_ij        Jaccard ratio C_ij / (N_i + N_j - C_ij), 0 when never selected.
  seeds       the k largest weighted degrees; ties -> lower id.
  argmax      ties -> lower id.
  zero score  the first still-unassigned element of a caller-supplied uniform
              random permutation (the random draw is an input).
  node stage  group strength S_ab = sum_{i in a, j in b} p_ij, then Algorithm 1
              over groups with k = number of nodes.
  rank ids    node-major, groups in the order they join their node; local
              slots follow ascending expert id.
Sums run sequentially in a fixed order (insertion order for scores), so the
result is reproducible.
"""
from __future__ import annotations

import numpy as np


def coactivation_probability(C: np.ndarray) -> np.ndarray:
    C = np.asarray(C, dtype=np.float64)
    N = np.diag(C).copy()
    denom = (N[:, None] + N[None, :]) - C
    P = np.divide(C, denom, out=np.zeros_like(C), where=denom > 0)
    np.fill_diagonal(P, 0.0)
    return P


def greedy_groups(P: np.ndarray, k: int, rand_order) -> list[list[int]]:
    """Algorithm 1 on an n x n affinity matrix with zero diagonal."""
    P = np.asarray(P, dtype=np.float64)
    n = P.shape[0]
    deg = np.zeros(n)
    for j in range(n):                      # sequential accumulation over j
        deg = deg + P[:, j]
    order = sorted(range(n), key=lambda i: (-deg[i], i))
    groups = [[order[g]] for g in range(k)]
    unassigned = np.ones(n, dtype=bool)
    unassigned[order[:k]] = False
    score = np.zeros((k, n))
    for g in range(k):
        score[g] = score[g] + P[:, order[g]]
    rand_order = [int(e) for e in rand_order]
    g = 0
    for _ in range(n - k):
        cand = np.where(unassigned, score[g], -np.inf)
        best = int(np.argmax(cand))          # first maximum = lowest id
        if cand[best] == 0.0:
            best = next(e for e in rand_order if unassigned[e])
        groups[g].append(best)
        unassigned[best] = False
        score[g] = score[g] + P[:, best]
        g = (g + 1) % k
    return groups


def group_affinity(P: np.ndarray, groups: list[list[int]]) -> np.ndarray:
    m = len(groups)
    S = np.zeros((m, m))
    for a in range(m):
        for b in range(m):
            if a != b:
                block = P[np.ix_(groups[a], groups[b])].ravel()
                S[a, b] = np.cumsum(block)[-1] if block.size else 0.0
    return S


def coactivation_placement(C, R: int, ranks_per_node: int, rand_order_gpu, rand_order_node):
    """Two-stage placement -> (expert_rank, expert_local) int32 arrays.
    rand_order_gpu permutes range(E); rand_order_node permutes range(R)."""
    P = coactivation_probability(C)
    n = P.shape[0]
    groups = greedy_groups(P, R, rand_order_gpu)
    nodes = R // ranks_per_node
    node_groups = greedy_groups(group_affinity(P, groups), nodes, rand_order_node) if nodes > 1 \
        else [list(range(R))]
    expert_rank = np.zeros(n, np.int32)
    expert_local = np.zeros(n, np.int32)
    rank = 0
    for ng in node_groups:
        for g in ng:
            members = sorted(groups[g])
            expert_rank[members] = rank
            expert_local[members] = np.arange(len(members), dtype=np.int32)
            rank += 1
    return expert_rank, expert_local


def comm_objective(P: np.ndarray, expert_rank, ranks_per_node: int, c: float) -> float:
    """Eq. 2-3: sum_{i<j} p_ij d(pi(i), pi(j)) with d = 0 / 1 / c."""
    er = np.asarray(expert_rank)
    node = er // ranks_per_node
    dist = np.where(er[:, None] == er[None, :], 0.0, np.where(node[:, None] == node[None, :], 1.0, float(c)))
    return float(np.triu(np.asarray(P) * dist, 1).sum())


def load_imbalance(loads) -> float:
    """Eq. 4: max_g L_g / mean_g L_g."""
    loads = np.asarray(loads, dtype=np.float64)
    m = loads.mean()
    return float(loads.max() / m) if m > 0 else 0.0
