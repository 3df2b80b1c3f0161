"""Oracle co-activation placement (Sec. IV-B, Algorithm 1 and the node stage).

TEST INFRASTRUCTURE ONLY (see the package docstring).  Plain Python loops
written to be read against the paper; the product placement is separate code.

Readings of points the paper leaves open:
* p_ij is the Jaccard ratio C_ij / (N_i + N_j - C_ij): "times selected
  together" over "times either is selected" (Sec. IV-B); 0 if never selected.
* argmax ties pick the lower id; the weighted-degree order is descending degree
  then ascending id.
* The zero-score "uniformly at random" pick takes the first unassigned element
  of a uniform random permutation that the caller passes in.
* Node stage: the strength between GPU groups a and b is the sum of p_ij over
  i in a, j in b; Algorithm 1 then groups the GPU groups into nodes.  Ranks are
  numbered node-major in the order groups join a node; within a rank the local
  slot follows ascending expert id.
"""
from __future__ import annotations


def coactivation_probability(C):
    """p_ij from co-activation counts C (C[i][i] = N_i).  Diagonal is 0."""
    n = len(C)
    P = [[0.0] * n for _ in range(n)]
    for i in range(n):
        for j in range(n):
            if i == j:
                continue
            denom = float(C[i][i]) + float(C[j][j]) - float(C[i][j])
            P[i][j] = float(C[i][j]) / denom if denom > 0 else 0.0
    return P


def algorithm1(P, k, rand_order):
    """Algorithm 1: seeds = the k experts of largest weighted degree, then
    round-robin greedy growth by score(e, G[g]) = sum_{v in G[g]} p_ev."""
    n = len(P)
    deg = []
    for i in range(n):
        s = 0.0
        for j in range(n):
            if j != i:
                s += P[i][j]
        deg.append(s)
    by_degree = sorted(range(n), key=lambda i: (-deg[i], i))
    G = [[by_degree[g]] for g in range(k)]
    U = [e for e in range(n) if e not in by_degree[:k]]
    g = 0
    while U:
        best, best_score = None, None
        for e in U:                       # U is kept in ascending id order
            score = 0.0
            for v in G[g]:
                score += P[e][v]
            if best is None or score > best_score:
                best, best_score = e, score
        if best_score == 0.0:
            best = next(e for e in rand_order if e in U)
        G[g].append(best)
        U.remove(best)
        g = (g + 1) % k
    return G


def group_strength(P, groups):
    m = len(groups)
    S = [[0.0] * m for _ in range(m)]
    for a in range(m):
        for b in range(m):
            if a == b:
                continue
            s = 0.0
            for i in groups[a]:
                for j in groups[b]:
                    s += P[i][j]
            S[a][b] = s
    return S


def coactivation_placement(C, R, ranks_per_node, rand_order_gpu, rand_order_node):
    """Two-stage placement -> (expert_rank, expert_local) lists.
    rand_order_gpu permutes range(n experts); rand_order_node permutes range(R groups)."""
    n = len(C)
    P = coactivation_probability(C)
    groups = algorithm1(P, R, rand_order_gpu)
    nodes = R // ranks_per_node
    if nodes > 1:
        node_groups = algorithm1(group_strength(P, groups), nodes, rand_order_node)
    else:
        node_groups = [list(range(R))]
    expert_rank = [0] * n
    expert_local = [0] * n
    rank = 0
    for ng in node_groups:
        for g in ng:
            for l, e in enumerate(sorted(groups[g])):
                expert_rank[e] = rank
                expert_local[e] = l
            rank += 1
    return expert_rank, expert_local


def comm_objective(P, expert_rank, ranks_per_node, c):
    """Eq. 2-3: sum_{i<j} p_ij d(pi(i), pi(j))."""
    n = len(P)
    total = 0.0
    for i in range(n):
        for j in range(i + 1, n):
            a, b = expert_rank[i], expert_rank[j]
            if a == b:
                dist = 0.0
            elif a // ranks_per_node == b // ranks_per_node:
                dist = 1.0
            else:
                dist = float(c)
            total += P[i][j] * dist
    return total


def load_imbalance(loads):
    """Eq. 4: max_g L_g / mean_g L_g."""
    mean = sum(loads) / len(loads)
    return max(loads) / mean if mean > 0 else 0.0
