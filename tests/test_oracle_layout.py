"""Pins of the oracle's layout, volume and co-activation steps.

Checked against: the paper's Device-per-Token Default column and its closed
form (uniform routing), the toy example of Sec. II-C, the inter-node cost
direction of Sec. VIII-E, and independent library derivations (numpy sorts,
one-hot matrix products) on small inputs.
"""
import json
import math
import os

import numpy as np
import pytest

from workloads import generator as gen

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _layout(orc, r, er, el, R, rpn, tpr, E):
    return orc.dispatch_layout(r["idx"], r["keep"], r["mask"], er, el, R, rpn, tpr, E)


def test_device_per_token_closed_form_matches_paper(orc):
    """Uniform routing, sequential placement, no pruning: mean distinct devices
    per token = R(1 - C(E-E/R,k)/C(E,k)) = 5.3394, and the paper's Default
    column (tab:cross-domain-dpt) sits at 5.33-5.35, so its Device per Token
    counts the token's own device."""
    g = json.load(open(os.path.join(GOLDEN, "device_per_token_default.json")))
    E, R, k = g["E"], g["R"], g["k"]
    closed = R * (1 - math.comb(E - E // R, k) / math.comb(E, k))
    assert abs(closed - 5.3394) < 1e-4
    for v in g["default_device_per_token"].values():
        assert abs(v - closed) < 0.015
    T = 32768
    L = gen.iid_logits(T, E, seed=11)
    er = (np.arange(E) // (E // R)).astype(np.int32)
    el = (np.arange(E) % (E // R)).astype(np.int32)
    r = orc.route_prune(L, k, er, R, T // R, 5.0, 0.0)
    lay = _layout(orc, r, er, el, R, R, T // R, E)
    n_dev = lay["vol"][:, 0].astype(np.float64)
    assert abs(n_dev.mean() - closed) < 0.02          # ~4.5 standard errors
    assert lay["totals"][0] == n_dev.sum()


def test_toy_example_one_copy_per_device(orc):
    """Sec. II-C: a token routed to experts 0 and 2, both on device 0, is sent
    to device 0 once, and both experts use that copy."""
    E, R = 4, 2
    er = np.array([0, 1, 0, 1], np.int32)            # experts 0 and 2 on device 0
    el = np.array([0, 0, 1, 1], np.int32)
    idx = np.array([[0, 2]], np.int32)
    keep = np.ones((1, 2), np.uint8)
    mask = np.array([1], np.uint64)
    lay = orc.dispatch_layout(idx, keep, mask, er, el, R, R, 1, E)
    assert lay["vol"][0].tolist() == [1, 0, 0, 1]
    assert lay["send_counts"].tolist() == [[1, 0], [0, 0]]
    assert lay["recv_offsets"].tolist() == [0, 1, 1]
    assert lay["copy_row"].tolist() == [[0, 0]]      # both experts share row 0
    assert lay["slot_pos"].tolist() == [[0, 1]]      # two expert rows
    assert lay["expert_counts"].tolist() == [1, 1, 0, 0]


def _independent_layout(r, er, el, R, rpn, tpr, E):
    """Library derivation: stable sorts and set arithmetic."""
    idx, keep, mask = r["idx"], r["keep"], r["mask"]
    T, k = idx.shape
    E_loc = E // R
    pos = er * E_loc + el
    t_of = np.repeat(np.arange(T), k)
    q_of = np.arange(T * k)
    kept = keep.ravel() == 1
    P = pos[idx.ravel()]
    order = np.lexsort((t_of[kept], P[kept]))     # by slot position, then token
    slot_pos = np.full(T * k, -1, np.int64)
    slot_pos[q_of[kept][order]] = np.arange(kept.sum())
    counts = np.bincount(P[kept], minlength=E)
    bits = ((mask[:, None] >> np.arange(R, dtype=np.uint64)) & np.uint64(1)).astype(bool)  # [T][R]
    src = np.arange(T) // tpr
    send_counts = np.zeros((R, R), np.int64)
    for s in range(R):
        send_counts[s] = bits[src == s].sum(0)
    copy = np.cumsum(bits, 0) - bits                # rank of t among tokens sent to d
    dev = er[idx]
    copy_row = np.where(keep == 1, np.take_along_axis(copy, dev, 1), -1)
    node = np.arange(R) // rpn
    n_dev = bits.sum(1)
    same_node = node[None, :] == node[src][:, None]
    n_intra = (bits & same_node & (np.arange(R)[None, :] != src[:, None])).sum(1)
    n_inter = (bits & ~same_node).sum(1)
    n_nodes = np.array([len(set(node[b])) for b in bits])
    return dict(slot_pos=slot_pos.reshape(T, k), expert_counts=counts, send_counts=send_counts,
                copy_row=copy_row, vol=np.stack([n_dev, n_intra, n_inter, n_nodes], 1))


@pytest.mark.parametrize("cfgname,p,c", [("c1", 0.3, 5.0), ("c3", 0.1, 5.0), ("c3", 0.2, 1.0), ("c4", 0.1, 5.0)])
def test_layout_matches_independent_derivation(orc, cfgname, p, c):
    cfg = gen.CONFIGS[cfgname]
    T = min(cfg.T, 4096)
    tpr = T // cfg.R
    L = gen.logits(cfg)[:T]
    rng = np.random.default_rng(5)
    perm = rng.permutation(cfg.E)                    # a scrambled placement
    er = (perm // cfg.E_loc).astype(np.int32)
    el = (perm % cfg.E_loc).astype(np.int32)
    r = orc.route_prune(L, cfg.k, er, cfg.ranks_per_node, tpr, c, p)
    lay = _layout(orc, r, er, el, cfg.R, cfg.ranks_per_node, tpr, cfg.E)
    ind = _independent_layout(r, er, el, cfg.R, cfg.ranks_per_node, tpr, cfg.E)
    assert np.array_equal(lay["slot_pos"], ind["slot_pos"])
    assert np.array_equal(lay["expert_counts"], ind["expert_counts"])
    assert np.array_equal(lay["send_counts"], ind["send_counts"])
    assert np.array_equal(lay["copy_row"], ind["copy_row"])
    assert np.array_equal(lay["vol"], ind["vol"])
    # invariants
    n_pruned = int((r["keep"] == 0).sum())
    assert lay["expert_offsets"][-1] == T * cfg.k - n_pruned
    assert np.array_equal(np.diff(lay["expert_offsets"]), lay["expert_counts"])
    assert lay["expert_offsets"][0] == 0
    for s in range(cfg.R):
        assert lay["send_counts"][s].sum() == lay["vol"][s * tpr:(s + 1) * tpr, 0].astype(int).sum()
        assert np.array_equal(lay["send_offsets"][s], np.cumsum(lay["send_counts"][s]) - lay["send_counts"][s])
    U = lay["send_counts"].sum(0)
    assert np.array_equal(lay["recv_offsets"], np.concatenate([[0], np.cumsum(U)]))
    kept = r["keep"] == 1
    sp = lay["slot_pos"][kept]
    assert np.array_equal(np.sort(sp), np.arange(kept.sum()))      # bijection
    assert np.all(lay["slot_pos"][~kept] == -1) and np.all(lay["copy_row"][~kept] == -1)
    # recv_token inverts copy_row
    dev = er[r["idx"]]
    t_idx = np.broadcast_to(np.arange(T)[:, None], r["idx"].shape)
    rows = lay["recv_offsets"][dev[kept]] + lay["copy_row"][kept]
    assert np.array_equal(lay["recv_token"][rows], t_idx[kept])
    assert lay["totals"].tolist() == lay["vol"].astype(np.int64).sum(0).tolist()


def test_inter_node_cost_direction(orc):
    """tab:inter-node-cost: with c=5 tokens visit fewer nodes than with c=1."""
    g = json.load(open(os.path.join(GOLDEN, "inter_node_cost.json")))
    assert g["node_per_token"]["c=5"] < g["node_per_token"]["c=1"]
    cfg = gen.CONFIGS["c3"]
    L = gen.logits(cfg)
    er, el = gen.sequential_placement(cfg)
    res = {}
    for c in (1.0, 5.0):
        r = orc.route_prune(L, cfg.k, er, cfg.ranks_per_node, cfg.tokens_per_rank, c, 0.2)
        lay = _layout(orc, r, er, el, cfg.R, cfg.ranks_per_node, cfg.tokens_per_rank, cfg.E)
        res[c] = lay["vol"].astype(np.float64).mean(0)
    assert res[5.0][3] < res[1.0][3]        # nodes per token
    assert res[5.0][2] < res[1.0][2]        # inter-node copies per token


# ---------------------------------------------------------------- co-activation
def test_coactivation_pins(orc):
    cfg = gen.CONFIGS["c2"]
    L = gen.logits(cfg)[:4096]
    er, _ = gen.sequential_placement(cfg)
    r = orc.route_prune(L, cfg.k, er, 8, 512, 5.0, 0.3)
    C = orc.coactivation(r["idx"], r["keep"], cfg.E).astype(np.int64)
    # one-hot matrix product B^T B (library matmul) on the kept routing
    B = np.zeros((L.shape[0], cfg.E), np.int64)
    for s in range(cfg.k):
        np.add.at(B, (np.arange(L.shape[0]), r["idx"][:, s]), r["keep"][:, s].astype(np.int64))
    assert B.max() <= 1
    assert np.array_equal(C, B.T @ B)
    assert np.array_equal(C, C.T)
    N = np.diag(C)
    assert N.sum() == int(r["keep"].sum())
    m = r["keep"].sum(1).astype(np.int64)
    assert np.array_equal(C.sum(1) - N, B.T @ (m - 1))
    # accumulate mode adds
    C2 = orc.coactivation(r["idx"], r["keep"], cfg.E, C.astype(np.uint32).copy())
    assert np.array_equal(C2.astype(np.int64), 2 * C)


def test_coactivation_tiny_brute_force(orc):
    idx = np.array([[0, 2, 1], [2, 0, 3], [3, 1, 0]], np.int32)
    keep = np.array([[1, 1, 0], [1, 1, 1], [0, 0, 1]], np.uint8)
    C = orc.coactivation(idx, keep, 4)
    want = np.zeros((4, 4), np.int64)
    # token 0 keeps {0,2}; token 1 keeps {2,0,3}; token 2 keeps {0}
    for kept in ({0, 2}, {0, 2, 3}, {0}):
        for i in kept:
            for j in kept:
                want[i, j] += 1
    assert np.array_equal(C, want)
