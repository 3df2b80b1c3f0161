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


# ---------------------------------------------------------------- Adjustment Approach (Sec. V)
# Placement spectrum by load-balancing swaps, starting from the communication-
# oriented placement.  Readings of what the paper leaves open (one line each):
#   loads      L_g = sum of N_e over g's experts, N_e = C[e][e] (kept rows);
#   devices    each step swaps between the most loaded device and the least
#              loaded one (ties: lower id);
#   candidates e on the former, f on the latter, whose swap lowers the larger
#              of the two loads (N_e > N_f, L_lo + N_e - N_f < L_hi);
#   choice     smallest increase of the Eq. 2-3 objective (ties: lower e,
#              then lower f); e and f exchange local slots.  The increase is
#              summed over the pairs whose distance changes: for every other
#              expert j, ascending, p_ej (d(lo, pi_j) - d(hi, pi_j)) and then
#              p_fj (d(hi, pi_j) - d(lo, pi_j)), sequentially in fp64;
#   end        no candidate remains (or max_swaps).
# cap_adjustment_spectrum runs the same swaps on the GPU.

def _distance_matrix(R: int, ranks_per_node: int, c: float) -> np.ndarray:
    g = np.arange(R)
    same_node = (g[:, None] // ranks_per_node) == (g[None, :] // ranks_per_node)
    D = np.where(same_node, 1.0, float(c))
    np.fill_diagonal(D, 0.0)
    return D


def swap_deltas(P: np.ndarray, er: np.ndarray, E2: np.ndarray, F2: np.ndarray, hi: int, lo: int,
                ranks_per_node: int, c: float, R: int) -> np.ndarray:
    """Objective increase of each candidate swap (E2[k] on hi <-> F2[k] on lo),
    the terms of every other expert j in ascending j, e term then f term,
    summed sequentially (one running sum per candidate)."""
    D = _distance_matrix(R, ranks_per_node, c)
    a = D[lo, er] - D[hi, er]                                # per expert j
    n = P.shape[0]
    terms = np.empty((len(E2), 2 * n))
    terms[:, 0::2] = P[E2] * a[None, :]
    terms[:, 1::2] = P[F2] * -a[None, :]
    j = np.arange(n)
    skip = (j[None, :] == E2[:, None]) | (j[None, :] == F2[:, None])
    terms[:, 0::2][skip] = 0.0
    terms[:, 1::2][skip] = 0.0
    # a skipped term adds +0.0: the running sum is unchanged by it (x + 0.0 == x)
    return np.cumsum(terms, axis=1)[:, -1]


def adjustment_spectrum(C, expert_rank, expert_local, R: int, ranks_per_node: int, c: float,
                        max_swaps: int = 1 << 30):
    """[(expert_rank, expert_local, swapped pair or None)], the starting
    placement first, then one entry per swap."""
    P = coactivation_probability(C)
    N = np.diag(np.asarray(C, dtype=np.int64)).copy()
    er = np.asarray(expert_rank, dtype=np.int32).copy()
    el = np.asarray(expert_local, dtype=np.int32).copy()
    out = [(er.copy(), el.copy(), None)]
    for _ in range(max_swaps):
        L = np.bincount(er, weights=N, minlength=R).astype(np.int64)
        hi = int(np.flatnonzero(L == L.max())[0])
        lo = int(np.flatnonzero(L == L.min())[0])
        if L[hi] == L[lo]:
            break
        es, fs = np.flatnonzero(er == hi), np.flatnonzero(er == lo)
        E2, F2 = np.meshgrid(es, fs, indexing="ij")
        E2, F2 = E2.ravel(), F2.ravel()                     # (e asc, f asc) order
        ok = (N[E2] > N[F2]) & (L[lo] + N[E2] - N[F2] < L[hi])
        if not ok.any():
            break
        E2, F2 = E2[ok], F2[ok]
        delta = swap_deltas(P, er, E2, F2, hi, lo, ranks_per_node, c, R)
        k = int(np.argmin(delta))                           # first minimum: lower e, then f
        e, f = int(E2[k]), int(F2[k])
        er[e], er[f] = lo, hi
        el[e], el[f] = el[f], el[e]
        out.append((er.copy(), el.copy(), (e, f)))
    return out


def adjustment_spectrum_gpu(coact, expert_rank, expert_local, R: int, ranks_per_node: int, c: float,
                            max_swaps: int = 4096, stream=None):
    """The Adjustment Approach on the GPU (cap_adjustment_spectrum): coact is
    the int32/uint32 [E][E] co-activation counts on the device.  Returns the
    same list as adjustment_spectrum (the placements are rebuilt on the host
    from the swap sequence the kernel chose) and the per-swap increases."""
    import torch
    from . import capi
    E = int(coact.shape[0])
    dev = coact.device
    er_d = torch.as_tensor(np.asarray(expert_rank, np.int32)).to(dev)
    el_d = torch.as_tensor(np.asarray(expert_local, np.int32)).to(dev)
    swaps = torch.empty((max(max_swaps, 1), 2), dtype=torch.int32, device=dev)
    deltas = torch.empty(max(max_swaps, 1), dtype=torch.float64, device=dev)
    n_swaps = torch.zeros(1, dtype=torch.int32, device=dev)
    topo = capi.Topology(E=E, R=R, ranks_per_node=ranks_per_node, T=R, tokens_per_rank=1, k=1)
    ws = torch.empty(capi.cap_workspace_size(capi.CAP_OP_ADJUSTMENT, topo), dtype=torch.uint8, device=dev)
    capi.cap_adjustment_spectrum(coact, E, R, ranks_per_node, c, er_d, el_d, max_swaps, swaps, deltas, n_swaps,
                                 ws, stream=stream)
    n = int(n_swaps.item())
    pairs = swaps[:n].cpu().numpy()
    er = np.asarray(expert_rank, np.int32).copy()
    el = np.asarray(expert_local, np.int32).copy()
    out = [(er.copy(), el.copy(), None)]
    for e, f in pairs:
        e, f = int(e), int(f)
        er[e], er[f] = er[f], er[e]
        el[e], el[f] = el[f], el[e]
        out.append((er.copy(), el.copy(), (e, f)))
    assert np.array_equal(er, er_d.cpu().numpy()) and np.array_equal(el, el_d.cpu().numpy())
    return out, deltas[:n].cpu().numpy()


def spectrum_points(n_placements: int, points: int = 7) -> list[int]:
    """Indices of `points` placements evenly spread over a spectrum of
    n_placements (first and last included)."""
    if n_placements <= points:
        return list(range(n_placements))
    return sorted({round(i * (n_placements - 1) / (points - 1)) for i in range(points)})
