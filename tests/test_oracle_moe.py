"""Pins of the oracle's permutation, expert FFN and combine, and of the oracle
placement (Algorithm 1 + node stage).

Checked against: hand-worked SwiGLU values, a closed form (identity weights),
the independent dense path of Eq. 1 (no permutation at all), a constant-row
case where the renormalised weights must return the row unchanged, and block
structured co-activation that Algorithm 1 must recover.
"""
import math

import numpy as np
import pytest

from oracle import placement as oplace
from workloads import generator as gen


# ---------------------------------------------------------------- SwiGLU
def test_swiglu_hand_worked(orc):
    # g = W1 x = 1, u = W3 x = 3, h = silu(1) * 3 = 3 / (1 + e^-1), y = W2 h = (h, 2h)
    x = np.array([[1.0, 3.0]], np.float32)
    W1 = np.array([[1.0, 0.0]], np.float32)
    W3 = np.array([[0.0, 1.0]], np.float32)
    W2 = np.array([[1.0], [2.0]], np.float32)
    h = 3.0 / (1.0 + math.exp(-1.0))
    y = orc.swiglu_rows(x, W1, W3, W2)
    assert np.allclose(y, [[h, 2 * h]], rtol=1e-15, atol=0)


def test_swiglu_identity_weights_closed_form(orc):
    d = 64
    x = np.random.default_rng(0).standard_normal((5, d)).astype(np.float32)
    I = np.eye(d, dtype=np.float32)
    y = orc.swiglu_rows(x, I, I, I)
    xd = x.astype(np.float64)
    assert np.allclose(y, xd * xd / (1 + np.exp(-xd)), rtol=1e-14, atol=1e-300)


def test_swiglu_rank_one_non_square(orc):
    # W1 = a b^T, W3 = c b^T, W2 = e f^T with d != inter: closed form
    rng = np.random.default_rng(1)
    d, inter = 12, 5
    # small integers keep every outer product exact in fp32
    a, c, f = (rng.integers(-4, 5, inter).astype(np.float64) for _ in range(3))
    b, e = rng.integers(-4, 5, d).astype(np.float64), rng.integers(-4, 5, d).astype(np.float64)
    x = (rng.standard_normal((3, d)) * 0.1).astype(np.float32).astype(np.float64)
    W1, W3, W2 = np.outer(a, b), np.outer(c, b), np.outer(e, f)
    y = orc.swiglu_rows(x.astype(np.float32), W1.astype(np.float32), W3.astype(np.float32), W2.astype(np.float32))
    s = x @ b                                            # b.x per row
    g, u = s[:, None] * a[None, :], s[:, None] * c[None, :]
    h = g / (1 + np.exp(-g)) * u
    want = (h @ f)[:, None] * e[None, :]
    assert np.allclose(y, want, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- whole layer on the tiny config
def _tiny(orc, cfgname, p, placement="seq"):
    cfg = gen.CONFIGS[cfgname]
    L = gen.logits(cfg)
    if placement == "seq":
        er, el = gen.sequential_placement(cfg)
    else:
        perm = np.random.default_rng(7).permutation(cfg.E)
        er, el = (perm // cfg.E_loc).astype(np.int32), (perm % cfg.E_loc).astype(np.int32)
    r = orc.route_prune(L, cfg.k, er, cfg.ranks_per_node, cfg.tokens_per_rank, 5.0, p)
    lay = orc.dispatch_layout(r["idx"], r["keep"], r["mask"], er, el, cfg.R, cfg.ranks_per_node,
                              cfg.tokens_per_rank, cfg.E)
    x = gen.activations_f32(cfg)
    wts = {e: gen.expert_weights_f32(cfg, e) for e in range(cfg.E)}
    return cfg, er, el, r, lay, x, wts


def _permuted_path(orc, cfg, er, el, r, lay, x, wts, shared=None):
    """gather -> per-rank expert FFN -> destination reduce -> source reduce."""
    parts = np.zeros((int(lay["recv_offsets"][-1]), cfg.d), np.float32)
    for rank in range(cfg.R):
        xs = orc.expert_gather(x, r["idx"], r["keep"], lay["slot_pos"], lay["expert_offsets"], er, cfg.R, rank)
        local = [int(np.where((er == rank) & (el == l))[0][0]) for l in range(cfg.E_loc)]
        offs = lay["expert_offsets"][rank * cfg.E_loc:(rank + 1) * cfg.E_loc + 1]
        Y = orc.expert_ffn(xs, offs, [wts[e] for e in local])
        part = orc.dest_reduce(Y, r, lay, er, cfg.R, rank, cfg.d)
        a, b = lay["recv_offsets"][rank], lay["recv_offsets"][rank + 1]
        parts[a:b] = part
    ys = []
    for s in range(cfg.R):
        sh = None if shared is None else shared[s * cfg.tokens_per_rank:(s + 1) * cfg.tokens_per_rank]
        ys.append(orc.src_reduce(parts, r, lay, er, cfg.R, cfg.tokens_per_rank, s, cfg.d, sh))
    return np.concatenate(ys)


@pytest.mark.parametrize("cfgname,p,placement", [("c1", 0.3, "seq"), ("c1", 0.0, "seq"),
                                                 ("c1u", 0.3, "scrambled"), ("c1u", 0.0, "seq")])
def test_permuted_path_equals_dense_eq1(orc, cfgname, p, placement):
    cfg, er, el, r, lay, x, wts = _tiny(orc, cfgname, p, placement)
    y = _permuted_path(orc, cfg, er, el, r, lay, x, wts)
    dense = orc.dense_moe_rows(np.arange(cfg.T), x, r, lambda e: wts[e])
    ref = np.abs(dense).max()
    assert np.abs(y - dense).max() <= 1e-6 * ref


def test_no_pruning_single_rank_is_dense_moe(orc):
    """p = 0 and a trivial placement (one rank holds every expert): the layer is
    the dense Eq. 1 MoE over the top-k gates, with no copy sent anywhere."""
    cfg0 = gen.CONFIGS["c1u"]
    L = gen.logits(cfg0)
    E = cfg0.E
    er = np.zeros(E, np.int32)
    el = np.arange(E, dtype=np.int32)
    r = orc.route_prune(L, cfg0.k, er, 1, cfg0.T, 5.0, 0.0)
    assert r["keep"].all() and np.allclose(r["wp"], r["w"], rtol=2.5e-7, atol=0)
    lay = orc.dispatch_layout(r["idx"], r["keep"], r["mask"], er, el, 1, 1, cfg0.T, E)
    assert lay["totals"].tolist() == [cfg0.T, 0, 0, cfg0.T]
    x = gen.activations_f32(cfg0)
    wts = {e: gen.expert_weights_f32(cfg0, e) for e in range(E)}
    xs = orc.expert_gather(x, r["idx"], r["keep"], lay["slot_pos"], lay["expert_offsets"], er, 1, 0)
    Y = orc.expert_ffn(xs, lay["expert_offsets"], [wts[e] for e in range(E)])
    part = orc.dest_reduce(Y, r, lay, er, 1, 0, cfg0.d)
    y = orc.src_reduce(part, r, lay, er, 1, cfg0.T, 0, cfg0.d)
    # dense MoE written with a library matmul over every expert, gates scattered
    G = np.zeros((cfg0.T, E))
    np.put_along_axis(G, r["idx"], r["w"].astype(np.float64), 1)
    xd = x.astype(np.float64)
    ref = np.zeros_like(xd)
    for e in range(E):
        W1, W3, W2 = (w.astype(np.float64) for w in wts[e])
        g, u = xd @ W1.T, xd @ W3.T
        ref += G[:, e:e + 1] * ((g / (1 + np.exp(-g)) * u) @ W2.T)
    assert np.abs(y - ref).max() <= 2e-6 * np.abs(ref).max()


def test_combine_constant_rows_renormalised(orc):
    """If every expert returns the same row v, renormalised weights (sum 1 over
    kept experts) make the layer return v for every token."""
    cfg, er, el, r, lay, x, wts = _tiny(orc, "c1u", 0.3, "scrambled")
    v = np.linspace(-1, 1, cfg.d).astype(np.float32)
    parts = np.zeros((int(lay["recv_offsets"][-1]), cfg.d), np.float32)
    for rank in range(cfg.R):
        rows = int(lay["expert_offsets"][(rank + 1) * cfg.E_loc] - lay["expert_offsets"][rank * cfg.E_loc])
        Y = np.tile(v, (rows, 1))
        a, b = lay["recv_offsets"][rank], lay["recv_offsets"][rank + 1]
        parts[a:b] = orc.dest_reduce(Y, r, lay, er, cfg.R, rank, cfg.d)
    for s in range(cfg.R):
        y = orc.src_reduce(parts, r, lay, er, cfg.R, cfg.tokens_per_rank, s, cfg.d)
        assert np.abs(y - v[None, :]).max() <= 1e-6
        sh = np.ones((cfg.tokens_per_rank, cfg.d), np.float32)
        y2 = orc.src_reduce(parts, r, lay, er, cfg.R, cfg.tokens_per_rank, s, cfg.d, sh)
        assert np.abs(y2 - (v[None, :] + 1)).max() <= 1e-6


def test_send_pack_rows(orc):
    cfg, er, el, r, lay, x, wts = _tiny(orc, "c1", 0.3, "scrambled")
    for s in range(cfg.R):
        out = orc.send_pack(x, r["mask"], lay["send_offsets"], lay["send_counts"], cfg.R, cfg.tokens_per_rank, s)
        row = 0
        for dd in range(cfg.R):
            for t in range(s * cfg.tokens_per_rank, (s + 1) * cfg.tokens_per_rank):
                if (int(r["mask"][t]) >> dd) & 1:
                    assert np.array_equal(out[row], x[t])
                    row += 1
        assert row == out.shape[0]


def test_send_pack_matches_receive_buffers(orc):
    """Independent of the send-pack enumeration: the rows source s sends to
    device d are the rows of d's receive buffer that come from s, in the
    buffer's order (recv_token of the layout, Sec. II-C one copy per device)."""
    for cfgname, p, placement in [("c1", 0.3, "scrambled"), ("c1u", 0.0, "seq")]:
        cfg, er, el, r, lay, x, wts = _tiny(orc, cfgname, p, placement)
        T_loc = cfg.tokens_per_rank
        for s in range(cfg.R):
            out = orc.send_pack(x, r["mask"], lay["send_offsets"], lay["send_counts"], cfg.R, T_loc, s)
            for dd in range(cfg.R):
                a, b = lay["recv_offsets"][dd], lay["recv_offsets"][dd + 1]
                toks = lay["recv_token"][a:b]
                mine = toks[(toks >= s * T_loc) & (toks < (s + 1) * T_loc)]
                o = int(np.asarray(lay["send_offsets"]).reshape(cfg.R, cfg.R)[s, dd])
                assert len(mine) == int(np.asarray(lay["send_counts"]).reshape(cfg.R, cfg.R)[s, dd])
                assert np.array_equal(out[o:o + len(mine)], x[mine])


# ---------------------------------------------------------------- placement (Algorithm 1 + node stage)
def _hub_block_counts(n, groups):
    """Co-activation counts with one hub per group: the hub co-activates more
    with its group than any other expert, so the n/len(groups) largest weighted
    degrees are the hubs, one per group, and Algorithm 1 seeds one per group."""
    C = np.zeros((n, n), np.int64)
    for g in groups:
        hub = g[0]
        for i in g:
            for j in g:
                C[i, j] = 80 if hub in (i, j) else 50
    C[np.diag_indices(n)] = 100
    return C


def test_algorithm1_recovers_blocks(orc):
    rng = np.random.default_rng(4)
    n, R = 32, 4
    perm = rng.permutation(n)
    groups = [perm[i * 8:(i + 1) * 8].tolist() for i in range(R)]
    C = _hub_block_counts(n, groups)
    er, el = oplace.coactivation_placement(C, R, R, list(range(n)), list(range(R)))
    got = sorted(sorted(e for e in range(n) if er[e] == r) for r in range(R))
    assert got == sorted(sorted(g) for g in groups)
    for r in range(R):       # local slots follow ascending expert id within a rank
        mine = sorted(e for e in range(n) if er[e] == r)
        assert [el[e] for e in mine] == list(range(8))
    P = oplace.coactivation_probability(C)
    assert oplace.comm_objective(P, er, R, 5.0) == 0.0


def test_algorithm1_node_stage_pairs_groups():
    """Node stage = Algorithm 1 over group strengths: groups 2g and 2g+1 are
    strongly linked; even groups carry a weak extra link to each other, so the
    seeds are the even groups and each pulls in its partner."""
    m = 8
    S = [[0.0] * m for _ in range(m)]
    for g in range(0, m, 2):
        S[g][g + 1] = S[g + 1][g] = 1.0
        for h in range(0, m, 2):
            if h != g:
                S[g][h] = 0.01
    G = oplace.algorithm1(S, 4, list(range(m)))
    assert G == [[0, 1], [2, 3], [4, 5], [6, 7]]


def test_placement_ranks_are_node_major():
    """Two nodes x 2 ranks: ranks 0,1 form node 0, ranks 2,3 node 1, and the
    GPU groups that co-activate across groups share a node.  A weak 0-2 link
    makes groups {0,1} and {2,3} the two node-stage seeds."""
    n, R, rpn = 8, 4, 2
    groups = [[0, 1], [2, 3], [4, 5], [6, 7]]
    C = _hub_block_counts(n, groups)
    C[0, 4] = C[4, 0] = 40              # groups {0,1} and {4,5} co-activate
    C[2, 6] = C[6, 2] = 40              # groups {2,3} and {6,7} co-activate
    C[0, 2] = C[2, 0] = 10
    er, el = oplace.coactivation_placement(C, R, rpn, list(range(n)), list(range(R)))
    rank_groups = {r: sorted(e for e in range(n) if er[e] == r) for r in range(R)}
    assert sorted(rank_groups.values()) == groups
    node_of = {tuple(v): r // rpn for r, v in rank_groups.items()}
    assert node_of[(0, 1)] == node_of[(4, 5)]
    assert node_of[(2, 3)] == node_of[(6, 7)]


def test_algorithm1_zero_score_uses_given_random_order():
    n, R = 8, 2
    P = [[0.0] * n for _ in range(n)]
    order = [5, 3, 7, 1, 0, 2, 4, 6]
    G = oplace.algorithm1(P, R, order)
    # all degrees 0 -> seeds 0 and 1 (lower ids); then every score is 0 and the
    # groups take turns drawing the next unassigned expert of `order`:
    # 5, 3, 7, (1, 0 taken) 2, 4, 6
    assert G == [[0, 5, 7, 4], [1, 3, 2, 6]]


def _placement_from_trace(orc, cfg, p=0.0):
    er0, _ = gen.sequential_placement(cfg)
    tr = orc.route_prune(gen.trace_logits(cfg), cfg.k, er0, cfg.ranks_per_node,
                         cfg.trace_tokens // cfg.R, 5.0, p)
    C = orc.coactivation(tr["idx"], tr["keep"], cfg.E)
    er, el = oplace.coactivation_placement(C, cfg.R, cfg.ranks_per_node,
                                           gen.random_order(cfg.E, 0, 0).tolist(),
                                           gen.random_order(cfg.R, 0, 1).tolist())
    return np.array(er, np.int32), np.array(el, np.int32)


def _device_per_token(orc, cfg, L, er, el):
    tpr = L.shape[0] // cfg.R
    r = orc.route_prune(L, cfg.k, er, cfg.ranks_per_node, tpr, 5.0, 0.0)
    lay = orc.dispatch_layout(r["idx"], r["keep"], r["mask"], er, el, cfg.R, cfg.ranks_per_node, tpr, cfg.E)
    return lay["vol"][:, 0].mean()


def test_coactivation_placement_lowers_device_per_token(orc):
    """tab:cross-domain-dpt direction: grouping co-activated experts lowers
    Device per Token below sequential placement (5.3 -> 4.1-4.5 in the paper).
    Checked on the Qwen3-shaped latent-topic workload with flatter popularity
    (Zipf 0.3), where co-activation structure rather than a few hot experts
    drives routing -- the premise of Sec. IV-A."""
    import dataclasses
    cfg = dataclasses.replace(gen.CONFIGS["c2"], zipf_s=0.3)
    er, el = _placement_from_trace(orc, cfg)
    assert sorted(np.bincount(er).tolist()) == [cfg.E_loc] * cfg.R
    L = gen.logits(cfg)[:8192]
    seq = _device_per_token(orc, cfg, L, *gen.sequential_placement(cfg))
    coact = _device_per_token(orc, cfg, L, er, el)
    assert coact < seq - 1.0, (coact, seq)


def test_coactivation_placement_is_balanced_on_stated_workloads(orc):
    for name in ("c2", "c3", "c5"):
        cfg = gen.CONFIGS[name]
        er, el = _placement_from_trace(orc, cfg, 0.1)
        assert sorted(np.bincount(er, minlength=cfg.R).tolist()) == [cfg.E_loc] * cfg.R
        for r in range(cfg.R):
            assert sorted(el[er == r].tolist()) == list(range(cfg.E_loc))
