"""The product placement (host code of the package) equals the oracle
placement on the same co-activation counts and random orders."""
import numpy as np
import pytest

import oracle
from oracle import placement as oplace
from paper_2607_05116_amd import placement as pplace
from workloads import generator as gen


@pytest.mark.parametrize("name,p", [("c2", 0.3), ("c3", 0.1), ("c4", 0.1), ("c5", 0.1), ("c1", 0.3)])
def test_product_placement_matches_oracle(name, p):
    cfg = gen.CONFIGS[name]
    er0, _ = gen.sequential_placement(cfg)
    tr = oracle.route_prune(gen.trace_logits(cfg), cfg.k, er0, cfg.ranks_per_node,
                            cfg.trace_tokens // cfg.R, 5.0, p)
    C = oracle.coactivation(tr["idx"], tr["keep"], cfg.E)
    ro_g, ro_n = gen.random_order(cfg.E, 0, 0), gen.random_order(cfg.R, 0, 1)
    er_o, el_o = oplace.coactivation_placement(C, cfg.R, cfg.ranks_per_node, ro_g.tolist(), ro_n.tolist())
    er_p, el_p = pplace.coactivation_placement(C, cfg.R, cfg.ranks_per_node, ro_g, ro_n)
    assert er_p.tolist() == er_o and el_p.tolist() == el_o
    P = oplace.coactivation_probability(C)
    assert np.allclose(pplace.comm_objective(np.array(P), er_p, cfg.ranks_per_node, 5.0),
                       oplace.comm_objective(P, er_o, cfg.ranks_per_node, 5.0), rtol=1e-12)


def test_product_placement_zero_scores_follow_random_order():
    P = np.zeros((8, 8))
    G = pplace.greedy_groups(P, 2, [5, 3, 7, 1, 0, 2, 4, 6])
    assert G == oplace.algorithm1(P.tolist(), 2, [5, 3, 7, 1, 0, 2, 4, 6])


@pytest.mark.parametrize("name,p,swaps", [("c1", 0.3, 64), ("c2", 0.3, 8), ("c3", 0.1, 6), ("c4", 0.1, 8)])
def test_product_adjustment_matches_oracle(name, p, swaps):
    """The product Adjustment Approach takes the same swaps as the oracle,
    starting from the co-activation placement of a pruned trace."""
    cfg = gen.CONFIGS[name]
    er0, _ = gen.sequential_placement(cfg)
    tr = oracle.route_prune(gen.trace_logits(cfg), cfg.k, er0, cfg.ranks_per_node,
                            cfg.trace_tokens // cfg.R, 5.0, p)
    C = oracle.coactivation(tr["idx"], tr["keep"], cfg.E)
    ro_g, ro_n = gen.random_order(cfg.E, 0, 0), gen.random_order(cfg.R, 0, 1)
    er, el = pplace.coactivation_placement(C, cfg.R, cfg.ranks_per_node, ro_g, ro_n)
    spec_p = pplace.adjustment_spectrum(C, er, el, cfg.R, cfg.ranks_per_node, 5.0, max_swaps=swaps)
    spec_o = oplace.adjustment_spectrum(C.tolist(), er.tolist(), el.tolist(), cfg.R, cfg.ranks_per_node, 5.0,
                                        max_swaps=swaps)
    assert len(spec_p) == len(spec_o)
    for (rp, lp, pair_p), (ro, lo, pair_o) in zip(spec_p, spec_o):
        assert pair_p == pair_o
        assert rp.tolist() == ro and lp.tolist() == lo


def test_spectrum_points_spread():
    assert pplace.spectrum_points(3) == [0, 1, 2]
    assert pplace.spectrum_points(63) == [0, 10, 21, 31, 41, 52, 62]
    pts = pplace.spectrum_points(8)
    assert pts[0] == 0 and pts[-1] == 7 and len(pts) == 7
