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


# ---------------------------------------------------------------- Adjustment Approach
# Comm.-comp. trade-off adjustment (Sec. V): starting from the communication-
# oriented placement, repeatedly swap a pair of experts between a high-load and
# a low-load device, reducing load imbalance while losing as little
# co-activation locality as possible; the successive placements form the
# placement spectrum.  The paper leaves the pair choice open; the reading here:
# * loads: L_g = sum of N_e over the experts on g, N_e = C[e][e] (kept
#   (token, expert) pairs, the rows device g computes);
# * each step swaps between the most loaded device (ties: lower id) and the
#   least loaded one (ties: lower id);
# * candidates: e on the most loaded device, f on the least loaded one, whose
#   swap lowers the larger of the two loads (N_e > N_f and
#   L_lo + N_e - N_f < L_hi);
# * the chosen pair has the smallest increase of the communication objective
#   (Eq. 2-3; ties: lower e, then lower f); e and f exchange devices and
#   local slots.  The increase is summed over the pairs whose distance the
#   swap changes -- (e, j) and (f, j) for every other expert j, in ascending
#   j, the e term before the f term -- which equals the difference of the two
#   objectives without the cancellation of subtracting two full sums (the
#   pair (e, f) keeps its distance);
# * the spectrum ends when no candidate remains (or after max_swaps).

def expert_loads(C):
    return [int(C[e][e]) for e in range(len(C))]


def device_loads(N, expert_rank, R):
    L = [0] * R
    for e, g in enumerate(expert_rank):
        L[g] += N[e]
    return L


def distance(a, b, ranks_per_node, c):
    """Eq. 3: d = 0 on one device, 1 within a node, c across nodes."""
    if a == b:
        return 0.0
    if a // ranks_per_node == b // ranks_per_node:
        return 1.0
    return float(c)


def swap_delta(P, expert_rank, e, f, ranks_per_node, c):
    """Increase of the Eq. 2-3 objective when e (on device hi) and f (on lo)
    exchange devices: sum over every other expert j, ascending, of
    p_ej (d(lo, pi_j) - d(hi, pi_j)) and then p_fj (d(hi, pi_j) - d(lo, pi_j))."""
    hi, lo = expert_rank[e], expert_rank[f]
    delta = 0.0
    for j in range(len(P)):
        if j == e or j == f:
            continue
        g = expert_rank[j]
        a = distance(lo, g, ranks_per_node, c) - distance(hi, g, ranks_per_node, c)
        delta += P[e][j] * a
        delta += P[f][j] * -a
    return delta


def adjust_step(P, N, expert_rank, expert_local, R, ranks_per_node, c):
    """One swap -> (expert_rank, expert_local, (e, f), delta_C), or None."""
    L = device_loads(N, expert_rank, R)
    hi = max(range(R), key=lambda g: (L[g], -g))
    lo = min(range(R), key=lambda g: (L[g], g))
    if L[hi] == L[lo]:
        return None
    best = None
    for e in range(len(N)):
        if expert_rank[e] != hi:
            continue
        for f in range(len(N)):
            if expert_rank[f] != lo:
                continue
            if not (N[e] > N[f] and L[lo] + N[e] - N[f] < L[hi]):
                continue
            delta = swap_delta(P, expert_rank, e, f, ranks_per_node, c)
            if best is None or delta < best[2]:
                best = (e, f, delta)
    if best is None:
        return None
    e, f, delta = best
    er = list(expert_rank)
    el = list(expert_local)
    er[e], er[f] = lo, hi
    el[e], el[f] = expert_local[f], expert_local[e]
    return er, el, (e, f), delta


def adjustment_spectrum(C, expert_rank, expert_local, R, ranks_per_node, c, max_swaps=1 << 30):
    """[(expert_rank, expert_local, swapped pair or None)] from the starting
    placement through every swap until none applies."""
    P = coactivation_probability(C)
    N = expert_loads(C)
    out = [(list(expert_rank), list(expert_local), None)]
    er, el = list(expert_rank), list(expert_local)
    for _ in range(max_swaps):
        step = adjust_step(P, N, er, el, R, ranks_per_node, c)
        if step is None:
            break
        er, el, pair, _ = step
        out.append((er, el, pair))
    return out
