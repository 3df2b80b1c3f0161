"""GPU Adjustment Approach (cap_adjustment_spectrum, Sec. V) against the
oracle: the same swap sequence, the same increases of the Eq. 2-3 objective
bit for bit, and the same final placement, from the co-activation placement of
each workload's pruned routing trace (Algorithm 1 + node stage on the oracle's
co-activation counts), and on random counts with exact ties."""
import numpy as np
import pytest

from oracle import placement as oplace
from tests import cases as C
from workloads import generator as gen

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle  # noqa: E402
from paper_2607_05116_amd import placement as pplace  # noqa: E402


def _oracle_spectrum(counts, er, el, R, rpn, c, max_swaps):
    P = oplace.coactivation_probability(counts.tolist())
    N = oplace.expert_loads(counts.tolist())
    er, el = list(map(int, er)), list(map(int, el))
    pairs, deltas = [], []
    for _ in range(max_swaps):
        step = oplace.adjust_step(P, N, er, el, R, rpn, c)
        if step is None:
            break
        er, el, pair, d = step
        pairs.append(pair)
        deltas.append(d)
    return pairs, np.array(deltas, np.float64), er, el


def _check(counts, er, el, R, rpn, c, max_swaps):
    dev = torch.from_numpy(counts.astype(np.uint32).view(np.int32)).cuda()
    spec, deltas = pplace.adjustment_spectrum_gpu(dev, er, el, R, rpn, c, max_swaps=max_swaps)
    pairs, want_d, er_o, el_o = _oracle_spectrum(counts, er, el, R, rpn, c, max_swaps)
    got_pairs = [s[2] for s in spec[1:]]
    assert got_pairs == pairs
    assert np.array_equal(deltas.view(np.uint64), want_d.view(np.uint64))
    assert spec[-1][0].tolist() == er_o and spec[-1][1].tolist() == el_o
    return len(pairs)


@pytest.mark.parametrize("name,p,c", [("c1", 0.3, 5.0), ("c2", 0.3, 5.0), ("c3", 0.1, 5.0), ("c3", 0.1, 1.0),
                                      ("c4", 0.1, 5.0), ("c5", 0.1, 5.0)])
def test_adjustment_spectrum_matches_oracle(name, p, c):
    cfg = gen.CONFIGS[name]
    er0, _ = gen.sequential_placement(cfg)
    tr = oracle.route_prune(gen.trace_logits(cfg), cfg.k, er0, cfg.ranks_per_node, cfg.trace_tokens // cfg.R,
                            c, p)
    counts = oracle.coactivation(tr["idx"], tr["keep"], cfg.E)
    er, el = oplace.coactivation_placement(counts.tolist(), cfg.R, cfg.ranks_per_node,
                                           gen.random_order(cfg.E, 0, 0).tolist(),
                                           gen.random_order(cfg.R, 0, 1).tolist())
    n = _check(counts, er, el, cfg.R, cfg.ranks_per_node, c, max_swaps=400)
    print(f"[{name} p={p} c={c}] {n} swaps", flush=True)
    assert n > 0


@pytest.mark.parametrize("seed,E,R,rpn,c", [(0, 16, 4, 2, 5.0), (1, 32, 8, 4, 3.0), (2, 24, 2, 1, 5.0),
                                            (3, 64, 4, 4, 1.0)])
def test_adjustment_ties_and_idle_experts(seed, E, R, rpn, c):
    """Random counts where a third of the experts never co-activate (their
    rows of p are 0, so many candidates tie exactly): the tie rule (lower e,
    then lower f) picks the same swap on both sides; also max_swaps = 0 and a
    cap of 3 swaps."""
    rng = np.random.default_rng(seed)
    counts = np.zeros((E, E), np.int64)
    active = rng.permutation(E)[: 2 * E // 3]
    for _ in range(40 * E):
        sel = rng.choice(active, size=3, replace=False)
        for a in sel:
            for b in sel:
                counts[a, b] += 1
    idle = np.setdiff1d(np.arange(E), active)
    counts[idle, idle] = rng.integers(1, 5, size=len(idle))       # selected alone now and then
    perm = rng.permutation(E)
    er, el = (perm // (E // R)).astype(np.int32), (perm % (E // R)).astype(np.int32)
    _check(counts, er, el, R, rpn, c, max_swaps=1000)
    assert _check(counts, er, el, R, rpn, c, max_swaps=0) == 0
    assert _check(counts, er, el, R, rpn, c, max_swaps=3) <= 3
