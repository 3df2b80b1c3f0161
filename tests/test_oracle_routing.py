"""Pins of the oracle's routing steps: gate exponential, top-k, gates, pruning.

Each check is tied to something other than the oracle itself: fp64 library
exp, a library sort, closed forms, brute force over Eq. 6 on tiny inputs, and
hand-worked cases of the greedy rule of Sec. VI.
"""
import itertools
import math

import numpy as np
import pytest

from workloads import generator as gen


def _ulp_f32(x: np.ndarray) -> np.ndarray:
    x = np.abs(x.astype(np.float32))
    return np.spacing(x).astype(np.float64)


# ---------------------------------------------------------------- exp
def test_exp_within_2ulp_of_fp64(orc):
    z = np.concatenate([
        np.linspace(-87.33, 0.0, 200001, dtype=np.float64).astype(np.float32),
        -np.abs(np.random.default_rng(1).standard_normal(100000).astype(np.float32)) * 10,
        np.array([0.0, -0.0, -1e-30, -1e-7, -0.34657359, -0.34657360, -0.6931472, -87.3], np.float32),
    ])
    got = orc.exp_f32(z).astype(np.float64)
    ref = np.exp(z.astype(np.float64))
    err = np.abs(got - ref) / _ulp_f32(ref.astype(np.float32))
    assert err.max() <= 2.0, (err.max(), z[np.argmax(err)])


def test_exp_special_values(orc):
    assert orc.exp_f32(0.0)[0] == 1.0
    assert orc.exp_f32(-0.0)[0] == 1.0
    assert orc.exp_f32(-87.34)[0] == 0.0
    assert orc.exp_f32(-1000.0)[0] == 0.0
    v = orc.exp_f32(np.float32(-87.33))[0]
    assert v >= np.finfo(np.float32).tiny           # never subnormal
    # near -n ln2 the result is 2^-n up to the rounding of the fp32 argument
    for n in range(0, 126, 5):
        z = np.float32(-n * math.log(2))
        assert abs(orc.exp_f32(z)[0] / math.exp(float(z)) - 1) < 2.5e-7
        assert abs(math.exp(float(z)) / 2.0 ** -n - 1) < n * 2.0 ** -24 + 1e-12


def test_exp_monotone(orc):
    z = np.sort(-np.abs(np.random.default_rng(2).standard_normal(200000).astype(np.float32)) * 20)
    v = orc.exp_f32(z)
    assert np.all(np.diff(v) >= 0)


# ---------------------------------------------------------------- top-k
def _lib_topk(L, k):
    # library stable sort by (value desc, index asc); -0.0 and +0.0 compare equal
    return np.stack([np.lexsort((np.arange(L.shape[1]), -row))[:k] for row in L]).astype(np.int32)


@pytest.mark.parametrize("E,k", [(16, 2), (64, 6), (128, 8), (256, 8), (7, 7), (5, 1)])
def test_topk_matches_library_sort(orc, E, k):
    L = gen.iid_logits(300, E, seed=E + k)
    assert np.array_equal(orc.topk(L, k), _lib_topk(L, k))


def test_topk_ties_and_signed_zero(orc):
    rng = np.random.default_rng(3)
    # bf16-quantised logits: many exact ties
    L = gen.bf16_bits_to_f32(gen.f32_to_bf16_bits(rng.standard_normal((500, 64)).astype(np.float32) * 0.05))
    assert np.array_equal(orc.topk(L, 8), _lib_topk(L, 8))
    # all-equal rows pick 0..k-1
    assert np.array_equal(orc.topk(np.zeros((3, 16), np.float32), 4), np.tile(np.arange(4, dtype=np.int32), (3, 1)))
    # -0.0 and +0.0 are equal: lower index first
    row = np.full((1, 8), -1.0, np.float32)
    row[0, 5] = 0.0
    row[0, 2] = -0.0
    assert orc.topk(row, 2).tolist() == [[2, 5]]


# ---------------------------------------------------------------- gates
def test_gates_sum_to_one_and_match_full_softmax(orc):
    for E, k in [(16, 2), (128, 8), (256, 8), (64, 6)]:
        L = gen.iid_logits(2000, E, seed=E) * np.float32(3.0)
        idx = orc.topk(L, k)
        w = orc.gates(L, idx)
        s = w.astype(np.float64).sum(1)
        assert np.abs(s - 1).max() <= k * 2 ** -23
        # fp64: softmax over all experts, then top-k, then renormalise
        Ld = L.astype(np.float64)
        full = np.exp(Ld - Ld.max(1, keepdims=True))
        full /= full.sum(1, keepdims=True)
        sel = np.take_along_axis(full, idx, 1)
        ref = sel / sel.sum(1, keepdims=True)
        assert np.abs(w - ref).max() <= 4e-7
        assert np.all(np.diff(w, axis=1) <= 0)        # slot order = descending gate


def test_gates_closed_forms(orc):
    L = np.array([[math.log(3.0), 0.0, -5.0, -6.0]], np.float32)
    w = orc.gates(L, orc.topk(L, 2))
    assert abs(w[0, 0] - 0.75) < 1e-7 and abs(w[0, 1] - 0.25) < 1e-7
    L = np.array([[1.5, 1.5, 0.0]], np.float32)
    assert orc.gates(L, orc.topk(L, 2)).tolist() == [[0.5, 0.5]]
    L = np.array([[0.3, 2.0, 1.0]], np.float32)
    assert orc.gates(L, orc.topk(L, 1)).tolist() == [[1.0]]


def test_gates_large_logit_gaps(orc):
    """Gaps to the top logit far beyond the fp32 range of exp: the gates stay
    finite.  A slot whose gap is at or above -87.33 gets exp(gap) / S (fp64
    reference, S within one ulp of 1 here), one below the cutoff gets exactly 0
    (the specified exponential never returns a subnormal), and the top slot
    takes the rest."""
    gaps = [0.0, -20.0, -80.0, -86.0, -87.33, -87.34, -88.0, -90.0, -150.0, -1e4]
    base = np.float32(3.5)
    L = (base + np.array([gaps], np.float32)).astype(np.float32)
    real_gaps = (L[0].astype(np.float64) - float(L[0, 0]))
    k = len(gaps)
    w = orc.gates(L, orc.topk(L, k))[0]
    assert np.all(np.isfinite(w))
    assert w[0] == 1.0
    for s in range(1, k):
        g = np.float32(L[0, s] - L[0, 0])
        if g >= np.float32(-87.33):
            ref = math.exp(float(real_gaps[s]))
            assert abs(float(w[s]) - ref) <= 2 * ref * 2.0 ** -23, (s, w[s], ref)
            assert w[s] >= np.finfo(np.float32).tiny
        else:
            assert w[s] == 0.0, (s, w[s])
    # the same gaps from the bottom of the fp32 range and from a large positive
    # top logit (the shift is by the top logit, so nothing overflows)
    for top in (np.float32(-3e4), np.float32(3e4)):
        L2 = (top + np.array([[0.0, -10.0, -1e4]], np.float32)).astype(np.float32)
        w2 = orc.gates(L2, orc.topk(L2, 3))[0]
        assert np.all(np.isfinite(w2)) and w2[2] == 0.0
        assert abs(float(w2.sum()) - 1.0) <= 3 * 2.0 ** -23


# ---------------------------------------------------------------- pruning: hand-worked cases
def _prune1(orc, experts, w, expert_rank, rpn, tpr, c, p, t=0):
    """Prune a single token t whose slots are `experts` with gates `w`."""
    T = t + 1
    idx = np.zeros((T, len(experts)), np.int32)
    ww = np.zeros((T, len(experts)), np.float32)
    idx[t] = experts
    ww[t] = w
    ww[:t] = np.float32(1.0 / len(experts))
    keep, wp, mask = orc.prune(idx, ww, np.asarray(expert_rank, np.int32), rpn, tpr, c, p)
    return keep[t], wp[t], int(mask[t])


def test_prune_worked_examples(orc):
    # Sec. VI greedy: keep devices in descending a_d/c_d until the kept sum >= 1-p.
    # 16 ranks, 8 per node, one expert per rank; the token lives on rank 0.
    er = list(range(16))
    # a = (0.3 own, 0.3 same-node rank 1, 0.4 other-node rank 8); p = 0.4 -> target 0.6
    # c=5: ratios inf, 0.3, 0.08 -> keep 0 (0.3), 1 (0.6 >= 0.6) -> drop rank 8
    keep, wp, mask = _prune1(orc, [8, 0, 1], [0.4, 0.3, 0.3], er, 8, 1, 5.0, 0.4)
    assert keep.tolist() == [0, 1, 1] and mask == 0b11
    assert wp.tolist() == [0.0, 0.5, 0.5]
    # c=1: ratios inf, 0.3, 0.4 -> keep 0 (0.3), 8 (0.7 >= 0.6) -> drop rank 1
    keep, wp, mask = _prune1(orc, [8, 0, 1], [0.4, 0.3, 0.3], er, 8, 1, 1.0, 0.4)
    assert keep.tolist() == [1, 1, 0] and mask == (1 | 1 << 8)
    # sum exactly at the target: a = 0.5, 0.25, 0.25 on remote ranks 1,2,3; p = 0.25
    # -> 0.5, then 0.75 >= 0.75 stops: ranks 1 and 2 kept (tie 2 vs 3 -> lower id)
    keep, wp, mask = _prune1(orc, [1, 2, 3], [0.5, 0.25, 0.25], er, 8, 1, 5.0, 0.25)
    assert keep.tolist() == [1, 1, 0] and mask == 0b110
    assert abs(wp[0] - 2 / 3) < 1e-7 and abs(wp[1] - 1 / 3) < 1e-7
    # own device always kept even with the smallest score
    keep, wp, mask = _prune1(orc, [1, 2, 0], [0.6, 0.3, 0.1], er, 8, 1, 5.0, 0.5)
    assert keep.tolist() == [1, 0, 1] and mask == 0b11
    # p = 0 keeps everything, even a negligible device
    keep, wp, mask = _prune1(orc, [1, 2, 9], [0.98, 0.01, 0.01], er, 8, 1, 5.0, 0.0)
    assert keep.tolist() == [1, 1, 1]
    # two experts on one device are kept or dropped together (device-level pruning)
    er2 = [0, 1, 1, 2]                 # experts 1 and 2 live on rank 1
    keep, wp, mask = _prune1(orc, [3, 1, 2], [0.5, 0.3, 0.2], er2, 8, 1, 1.0, 0.5)
    # a_1 = 0.5 (0.3+0.2), a_2 = 0.5: tie -> rank 1 first -> 0.5 >= 0.5 stop
    assert keep.tolist() == [0, 1, 1] and mask == 0b10


def _ilp_min_remote(a_local, a_remote, cost, target):
    """Brute force of Eq. 6 over all subsets of remote devices (own device free)."""
    best = None
    n = len(a_remote)
    for bits in itertools.product([0, 1], repeat=n):
        s = a_local + sum(a for a, b in zip(a_remote, bits) if b)
        if s >= target - 1e-12:
            c = sum(cc for cc, b in zip(cost, bits) if b)
            best = c if best is None else min(best, c)
    return best


def _token_devices(expert_rank, idx_row, w_row):
    a = {}
    for e, ww in zip(idx_row, w_row):
        d = int(expert_rank[e])
        a[d] = a.get(d, 0.0) + float(ww)
    return a


@pytest.mark.parametrize("p", [0.05, 0.1, 0.2, 0.3, 0.5])
def test_prune_single_node_is_ilp_optimal(orc, p):
    """Single node: costs are 0/1, so Eq. 6 minimises the number of remote
    devices and the greedy (largest a_d first) is optimal; brute force agrees."""
    cfg = gen.CONFIGS["c2"]
    L = gen.logits(cfg)[:3000]
    er, _ = gen.sequential_placement(cfg)
    r = orc.route_prune(L, cfg.k, er, 8, 375, 5.0, p)
    ambiguous = 0
    for t in range(L.shape[0]):
        src = t // 375
        a = _token_devices(er, r["idx"][t], r["w"][t])
        a_local = a.pop(src, 0.0)
        devs = sorted(a)
        kept_remote = sum(1 for d in devs if (int(r["mask"][t]) >> d) & 1)
        # skip tokens whose greedy sum lands within float noise of the target
        prefix = np.cumsum([a_local] + sorted(a.values(), reverse=True))
        if np.min(np.abs(prefix - (1 - p))) < 1e-5:
            ambiguous += 1
            continue
        opt = _ilp_min_remote(a_local, [a[d] for d in devs], [1.0] * len(devs), 1 - p)
        assert kept_remote == opt, (t, a_local, a, r["mask"][t])
    assert ambiguous < 30


def test_prune_multi_node_feasible_and_gap_reported(orc):
    """Multi-node (costs 1 and c): greedy by ratio is a heuristic; every kept
    set is feasible and never cheaper than the ILP optimum."""
    cfg = gen.CONFIGS["c3"]
    L = gen.logits(cfg)[:2000]
    er, _ = gen.sequential_placement(cfg)
    p, c = 0.2, 5.0
    r = orc.route_prune(L, cfg.k, er, 8, 1024, c, p)
    gaps = []
    for t in range(L.shape[0]):
        src = t // 1024
        a = _token_devices(er, r["idx"][t], r["w"][t])
        a_local = a.pop(src, 0.0)
        devs = sorted(a)
        cost = [1.0 if d // 8 == src // 8 else c for d in devs]
        kept = [(int(r["mask"][t]) >> d) & 1 for d in devs]
        assert a_local + sum(a[d] for d, k_ in zip(devs, kept) if k_) >= (1 - p) - 1e-6
        greedy_cost = sum(cc for cc, k_ in zip(cost, kept) if k_)
        opt = _ilp_min_remote(a_local, [a[d] for d in devs], cost, 1 - p)
        assert greedy_cost >= opt - 1e-9
        gaps.append(greedy_cost - opt)
    assert np.mean(gaps) < 1.0     # reported gap: heuristic close to optimum on average


def test_prune_properties(orc):
    cfg = gen.CONFIGS["c3"]
    L = gen.logits(cfg)[:4096]
    er, _ = gen.sequential_placement(cfg)
    masks = {}
    for p in [0.0, 0.05, 0.1, 0.2, 0.4]:
        r = orc.route_prune(L, cfg.k, er, 8, 1024, 5.0, p)
        masks[p] = r["mask"]
        srcs = np.arange(L.shape[0]) // 1024
        cand = np.zeros(L.shape[0], np.uint64)
        for s in range(cfg.k):
            cand |= np.left_shift(np.uint64(1), er[r["idx"][:, s]].astype(np.uint64))
        own = np.left_shift(np.uint64(1), srcs.astype(np.uint64))
        # the own device is never dropped when it is a candidate
        assert np.all(((cand & own) == 0) | ((r["mask"] & own) != 0))
        # kept weights renormalise to 1; pruned slots have w' = 0
        s = r["wp"].astype(np.float64).sum(1)
        assert np.abs(s - 1).max() <= cfg.k * 2 ** -23
        assert np.all((r["wp"] == 0) == (r["keep"] == 0))
        # a slot is kept iff its device is kept
        dev = er[r["idx"]]
        assert np.array_equal(r["keep"] == 1, ((r["mask"][:, None] >> dev.astype(np.uint64)) & np.uint64(1)) == 1)
        if p == 0.0:
            assert np.array_equal(r["mask"], cand)
    # monotone in p: kept(p2) is a subset of kept(p1) for p2 > p1
    ps = sorted(masks)
    for p1, p2 in zip(ps, ps[1:]):
        assert np.all((masks[p2] & ~masks[p1]) == 0)


def test_naive_pruning_keeps_prefix(orc):
    L = gen.iid_logits(500, 64, seed=9) * np.float32(2)
    idx = orc.topk(L, 6)
    w = orc.gates(L, idx)
    er = (np.arange(64) // 8).astype(np.int32)
    keep, wp, mask = orc.prune_naive(idx, w, er, 0.3)
    for t in range(500):
        n = int(keep[t].sum())
        assert keep[t, :n].all() and not keep[t, n:].any()
        assert w[t, :n].astype(np.float64).sum() >= 0.7 - 1e-6
        if n > 1:
            cum = np.float32(0)
            for v in w[t, :n - 1]:
                cum = np.float32(cum + v)
            assert cum < np.float32(0.7)


def test_naive_pruning_mask_and_renormalised_gates(orc):
    """Naive expert-level pruning (Sec. II-D; the baseline of Sec. VIII-D) on
    random tokens: the device mask is the OR of the devices of the kept slots
    only; kept gates are w / (sum of kept w) (fp64 reference, within the
    rounding of an fp32 slot-order sum and one division), pruned slots are 0,
    and the kept gates sum to 1."""
    rng = np.random.default_rng(31)
    L = gen.iid_logits(3000, 64, seed=13) * np.float32(2.5)
    er = (rng.permutation(64) % 8).astype(np.int32)          # 8 experts per device, scrambled
    for k, p in [(6, 0.3), (8, 0.1), (4, 0.5), (8, 0.45)]:
        idx = orc.topk(L, k)
        w = orc.gates(L, idx)
        keep, wp, mask = orc.prune_naive(idx, w, er, p)
        kept = keep == 1
        assert kept[:, 0].all()
        bits = np.where(kept, np.left_shift(np.uint64(1), er[idx].astype(np.uint64)), np.uint64(0))
        assert np.array_equal(mask, np.bitwise_or.reduce(bits, axis=1))
        assert np.all(wp[~kept] == 0)
        S = np.where(kept, w.astype(np.float64), 0.0).sum(1)
        ref = w.astype(np.float64) / S[:, None]
        rel = np.abs(wp.astype(np.float64) - ref)[kept] / ref[kept]
        assert rel.max() <= (k + 1) * 2.0 ** -24
        assert np.abs(wp.astype(np.float64).sum(1) - 1).max() <= k * 2.0 ** -23
        # some slot is pruned while its device stays kept (another kept slot
        # shares it): the expert-level rule prunes slots, not devices
        dev_kept = ((mask[:, None] >> er[idx].astype(np.uint64)) & np.uint64(1)) == 1
        if p >= 0.3:
            assert np.any(dev_kept & ~kept)


def test_naive_pruning_hand_worked(orc):
    """Hand-worked tokens of the expert-level rule.
    Token 0: gates 0.5 / 0.3 / 0.2 on devices 0 / 1 / 2, p = 0.3: the running
    sum 0.5 < 0.7, then 0.8 >= 0.7, so two slots stay, w' = 0.625 / 0.375 / 0
    and the mask is {0, 1}.
    Token 1: gates 0.5 / 0.25 / 0.25 on devices 1 / 0 / 1, p = 0.25: the sum
    reaches 0.75 exactly at the second slot (exact in fp32), so the third slot
    is pruned although its device 1 stays in the mask; w' = 2/3, 1/3, 0."""
    er = np.array([0, 1, 2, 1, 3, 1], np.int32)
    idx = np.array([[0, 1, 2]], np.int32)
    w = np.array([[0.5, 0.3, 0.2]], np.float32)
    keep, wp, mask = orc.prune_naive(idx, w, er, 0.3)
    assert keep.tolist() == [[1, 1, 0]]
    assert np.allclose(wp, [[0.625, 0.375, 0.0]], rtol=2 ** -23, atol=0)
    assert int(mask[0]) == 0b011
    idx = np.array([[3, 0, 5]], np.int32)
    w = np.array([[0.5, 0.25, 0.25]], np.float32)
    keep, wp, mask = orc.prune_naive(idx, w, er, 0.25)
    assert keep.tolist() == [[1, 1, 0]]
    assert np.allclose(wp, [[2 / 3, 1 / 3, 0.0]], rtol=2 ** -23, atol=0)
    assert int(mask[0]) == 0b011
    # p = 0 keeps every slot whatever the sum
    keep, wp, mask = orc.prune_naive(idx, w, er, 0.0)
    assert keep.tolist() == [[1, 1, 1]] and int(mask[0]) == 0b011


def test_router_logits_definition(orc):
    """x W_g^T: explicit dot products (exact sums), and identity rows pick columns."""
    import fractions
    rng = np.random.default_rng(5)
    x = rng.standard_normal((5, 7)).astype(np.float32)
    wg = rng.standard_normal((3, 7)).astype(np.float32)
    got = orc.router_logits(x, wg)
    assert got.shape == (5, 3)
    for t in range(5):
        for e in range(3):
            exact = sum(fractions.Fraction(float(x[t, q])) * fractions.Fraction(float(wg[e, q])) for q in range(7))
            assert abs(got[t, e] - float(exact)) <= 1e-12
    eye = np.eye(7, dtype=np.float32)[[4, 0, 6]]
    assert np.array_equal(orc.router_logits(x, eye), x[:, [4, 0, 6]].astype(np.float64))
