"""Pins of the oracle's Adjustment Approach (Sec. V: load-balancing swaps that
keep as much co-activation locality as possible, producing the placement
spectrum).  The oracle recomputes the Eq. 2-3 objective in floating point; the
pins check its choices against exact rational arithmetic, invariants of the
spectrum, and a hand-worked case."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import placement as op


def _random_counts(rng, n, tokens=40, k=3):
    C = np.zeros((n, n), np.int64)
    for _ in range(tokens):
        w = rng.random(n) ** 3
        sel = rng.choice(n, size=k, replace=False, p=w / w.sum())
        for a in sel:
            for b in sel:
                C[a, b] += 1
    return C


def _exact_objective(C, ranks, rpn, c):
    n = len(C)
    tot = Fraction(0)
    for i in range(n):
        for j in range(i + 1, n):
            den = C[i][i] + C[j][j] - C[i][j]
            p = Fraction(int(C[i][j]), int(den)) if den > 0 else Fraction(0)
            a, b = ranks[i], ranks[j]
            d = 0 if a == b else (1 if a // rpn == b // rpn else Fraction(c).limit_denominator(1000))
            tot += p * d
    return tot


@pytest.mark.parametrize("seed,R,rpn,c", [(0, 4, 4, 5.0), (1, 4, 2, 5.0), (2, 4, 2, 3.0), (3, 2, 1, 5.0),
                                          (4, 4, 2, 1.0), (5, 4, 4, 1.0)])
def test_each_swap_is_an_exact_minimum(seed, R, rpn, c):
    rng = np.random.default_rng(seed)
    n = 8
    C = _random_counts(rng, n)
    er = [e // (n // R) for e in range(n)]
    el = [e % (n // R) for e in range(n)]
    P = op.coactivation_probability(C.tolist())
    N = op.expert_loads(C.tolist())
    steps = 0
    while True:
        step = op.adjust_step(P, N, er, el, R, rpn, c)
        L = op.device_loads(N, er, R)
        hi = max(range(R), key=lambda g: (L[g], -g))
        lo = min(range(R), key=lambda g: (L[g], g))
        cands = [(e, f) for e in range(n) for f in range(n)
                 if er[e] == hi and er[f] == lo and N[e] > N[f] and L[lo] + N[e] - N[f] < L[hi]]
        if step is None:
            assert not cands or L[hi] == L[lo]
            break
        e, f = step[2]
        assert (e, f) in cands
        base = _exact_objective(C, er, rpn, c)
        def delta(pair):
            t = list(er)
            t[pair[0]], t[pair[1]] = lo, hi
            return _exact_objective(C, t, rpn, c) - base
        best = min(delta(p) for p in cands)
        # the choice is an exact minimum (floating point may only split exact ties)
        assert delta((e, f)) == best
        # and the reported increase is the exact objective difference, rounded
        assert abs(float(delta((e, f))) - step[3]) <= 1e-12
        er, el = step[0], step[1]
        steps += 1
        assert steps < 100


def test_spectrum_invariants():
    rng = np.random.default_rng(7)
    n, R, rpn = 16, 4, 2
    C = _random_counts(rng, n, tokens=300, k=4)
    er = [e // (n // R) for e in range(n)]
    el = [e % (n // R) for e in range(n)]
    spec = op.adjustment_spectrum(C.tolist(), er, el, R, rpn, 5.0)
    N = op.expert_loads(C.tolist())
    prev_max = prev_sq = None
    for ranks, local, _ in spec:
        for g in range(R):
            members = [e for e in range(n) if ranks[e] == g]
            assert len(members) == n // R                                   # equal expert counts
            assert sorted(local[e] for e in members) == list(range(n // R))  # slots a permutation
        mx = max(op.device_loads(N, ranks, R))
        assert prev_max is None or mx <= prev_max                           # max load never grows
        sq = sum(v * v for v in op.device_loads(N, ranks, R))
        assert prev_sq is None or sq < prev_sq                              # spread falls strictly
        prev_max, prev_sq = mx, sq
    # the spectrum ends where no swap applies
    P = op.coactivation_probability(C.tolist())
    assert op.adjust_step(P, N, spec[-1][0], spec[-1][1], R, rpn, 5.0) is None


def test_hand_worked_swap():
    """Two devices of four experts.  Device 0 holds the hot experts 0 and 1
    (N = 50) with partners 2 and 3; device 1 holds 4..7 (N = 10).  Only a hot
    expert can move (N_e > N_f), and 0 and 1 cost the same unless co-activated:
    expert 1 is tied to 3 (p = 0.5) and expert 0 to nothing, so expert 0 moves;
    among the four f (all N = 10), expert 4 is tied to 5 and the rest to nothing,
    so the lowest-cost f is the first of 6 and 7: 6."""
    n = 8
    C = np.zeros((n, n), np.int64)
    N = [50, 50, 10, 10, 10, 10, 10, 10]
    for e in range(n):
        C[e, e] = N[e]
    C[1, 3] = C[3, 1] = 20          # p_13 = 20 / (50 + 10 - 20) = 0.5
    C[4, 5] = C[5, 4] = 5           # p_45 = 5 / 15
    er = [0, 0, 0, 0, 1, 1, 1, 1]
    el = [0, 1, 2, 3, 0, 1, 2, 3]
    P = op.coactivation_probability(C.tolist())
    step = op.adjust_step(P, N, er, el, 2, 2, 5.0)
    assert step[2] == (0, 6)
    assert step[0][0] == 1 and step[0][6] == 0
    assert step[1][0] == 2 and step[1][6] == 0          # slots exchanged
    assert step[3] == 0.0                               # neither endpoint had a partner
