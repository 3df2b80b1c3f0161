"""GPU parity: every C-ABI call against the CPU oracle on the same seeded inputs.

Bit-exact: routing indices, gates, keep masks, device masks, every layout
array, volumes, co-activation counts, permuted rows.  FFN and combine:
|gpu - ref| <= 1e-3 + 2e-2 |ref| element-wise against the fp64 oracle, plus a
normalised Frobenius error gate (1e-2 bf16, 1e-5 fp32).
"""
import dataclasses
import os

import numpy as np
import pytest

from tests import cases as C
from workloads import generator as gen

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2607_05116_amd import capi  # noqa: E402
from paper_2607_05116_amd.layer import DeviceLayer  # noqa: E402

import oracle  # noqa: E402


def _layer(case: C.Case, x=None, **kw) -> DeviceLayer:
    """Device layer of a case; without x, a narrow dummy activation (routing-only tests)."""
    cfg = case.cfg
    er, el = C.placement(case.name, case.placement, case.p, case.c)
    if x is None:
        dd = 8 if cfg.dtype == "bf16" else 4
        x = np.zeros((cfg.T, dd), np.uint16 if cfg.dtype == "bf16" else np.float32)
        cfg = dataclasses.replace(cfg, d=dd)
    return DeviceLayer(cfg, C.logits(case.name), x, er, el, case.p, case.c, **kw)


@pytest.mark.parametrize("case", C.ROUTE_CASES, ids=lambda c: c.id)
def test_route_layout_coact_bit_exact(case):
    L = _layer(case, row_cap=8, recv_cap=8)
    L.front()
    torch.cuda.synchronize()
    r, lay = C.oracle_routing(case.name, case.placement, case.p, case.c)
    assert np.array_equal(L.host("idx"), r["idx"])
    assert np.array_equal(L.host("w").view(np.uint32), r["wp"].view(np.uint32))
    assert np.array_equal(L.host("keep"), r["keep"])
    assert np.array_equal(L.host("mask").view(np.uint64), r["mask"])
    for name in ("send_counts", "send_offsets", "recv_offsets", "expert_counts", "expert_offsets",
                 "slot_pos", "copy_row", "vol", "totals"):
        assert np.array_equal(L.host(name), lay[name]), name
    n_recv = int(lay["recv_offsets"][-1])
    assert np.array_equal(L.host("recv_token")[:n_recv], lay["recv_token"])
    coact = oracle.coactivation(r["idx"], r["keep"], case.cfg.E)
    assert np.array_equal(L.host("coact").view(np.uint32), coact)


@pytest.mark.parametrize("case", C.ROUTE_CASES, ids=lambda c: c.id)
def test_route_layout_fused_bit_exact(case):
    """cap_route_layout (routing, layout and co-activation in three launches)
    gives the oracle's routing, layout, volumes and co-activation bit for bit,
    and the separate calls' bits; without a co-activation output it leaves
    the counts alone."""
    L = _layer(case, row_cap=8, recv_cap=8)
    L.coact.fill_(-1)
    L.route_layout(True)
    torch.cuda.synchronize()
    r, lay = C.oracle_routing(case.name, case.placement, case.p, case.c)
    assert np.array_equal(L.host("idx"), r["idx"])
    assert np.array_equal(L.host("w").view(np.uint32), r["wp"].view(np.uint32))
    assert np.array_equal(L.host("keep"), r["keep"])
    assert np.array_equal(L.host("mask").view(np.uint64), r["mask"])
    for name in ("send_counts", "send_offsets", "recv_offsets", "expert_counts", "expert_offsets",
                 "slot_pos", "copy_row", "vol", "totals"):
        assert np.array_equal(L.host(name), lay[name]), name
    n_recv = int(lay["recv_offsets"][-1])
    assert np.array_equal(L.host("recv_token")[:n_recv], lay["recv_token"])
    coact = oracle.coactivation(r["idx"], r["keep"], case.cfg.E)
    assert np.array_equal(L.host("coact").view(np.uint32), coact)
    L.coact.fill_(7)
    L.route_layout(False)
    torch.cuda.synchronize()
    assert int((L.coact != 7).sum()) == 0
    assert np.array_equal(L.host("slot_pos"), lay["slot_pos"])


@pytest.mark.parametrize("E,k,R,rpn,p,c,T_loc", [
    (16, 2, 4, 4, 0.3, 5.0, 160), (64, 6, 8, 4, 0.25, 5.0, 300), (128, 8, 16, 8, 0.1, 5.0, 129),
    (256, 8, 32, 8, 0.2, 3.0, 97), (7, 3, 1, 1, 0.4, 5.0, 1000), (24, 5, 6, 2, 0.5, 2.0, 256),
    (128, 8, 64, 8, 0.3, 5.0, 64), (96, 1, 8, 8, 0.0, 5.0, 385), (40, 8, 4, 2, 0.05, 5.0, 1)])
def test_route_layout_fused_odd_shapes(E, k, R, rpn, p, c, T_loc):
    """The fused front end on adversarial logits (ties, +-0) and ragged token
    counts per rank (empty and partial 32-token parts), against the oracle."""
    T = R * T_loc
    L0 = _adversarial_logits(T, E, E + k + T_loc)
    perm = np.random.default_rng(R + T_loc).permutation(E)
    er, el = (perm // (E // R)).astype(np.int32), (perm % (E // R)).astype(np.int32)
    cfg = gen.Config("adv", T=T, d=8, E=E, k=k, inter=128, R=R, ranks_per_node=rpn, n_clusters=1,
                     zipf_s=0.0, dtype="bf16")
    Ld = DeviceLayer(cfg, L0, np.zeros((T, 8), np.uint16), er, el, p, c, row_cap=8, recv_cap=8)
    Ld.route_layout(True)
    torch.cuda.synchronize()
    r = oracle.route_prune(L0, k, er, rpn, T // R, c, p)
    lay = oracle.dispatch_layout(r["idx"], r["keep"], r["mask"], er, el, R, rpn, T // R, E)
    assert np.array_equal(Ld.host("idx"), r["idx"])
    assert np.array_equal(Ld.host("w").view(np.uint32), r["wp"].view(np.uint32))
    assert np.array_equal(Ld.host("mask").view(np.uint64), r["mask"])
    for name in ("slot_pos", "copy_row", "vol", "expert_offsets", "expert_counts", "send_counts",
                 "send_offsets", "recv_offsets", "totals"):
        assert np.array_equal(Ld.host(name), lay[name]), name
    n_recv = int(lay["recv_offsets"][-1])
    assert np.array_equal(Ld.host("recv_token")[:n_recv], lay["recv_token"])
    assert np.array_equal(Ld.host("coact").view(np.uint32), oracle.coactivation(r["idx"], r["keep"], E))


@pytest.mark.parametrize("case", C.ROUTE_CASES, ids=lambda c: c.id)
def test_naive_pruning_bit_exact(case):
    """Expert-level threshold pruning (the comparison baseline) against the
    oracle: routing outputs and the layout built from them."""
    L = _layer(case, row_cap=8, recv_cap=8)
    L.naive = True
    L.route()
    L.layout()
    torch.cuda.synchronize()
    cfg = case.cfg
    er, el = C.placement(case.name, case.placement, case.p, case.c)
    logits = C.logits(case.name)
    idx = oracle.topk(logits, cfg.k)
    w = oracle.gates(logits, idx)
    keep, wp, mask = oracle.prune_naive(idx, w, er, case.p)
    assert np.array_equal(L.host("idx"), idx)
    assert np.array_equal(L.host("w").view(np.uint32), wp.view(np.uint32))
    assert np.array_equal(L.host("keep"), keep)
    assert np.array_equal(L.host("mask").view(np.uint64), mask)
    lay = oracle.dispatch_layout(idx, keep, mask, er, el, cfg.R, cfg.ranks_per_node, cfg.tokens_per_rank, cfg.E)
    for name in ("send_counts", "expert_offsets", "slot_pos", "copy_row", "vol", "totals"):
        assert np.array_equal(L.host(name), lay[name]), name


def test_coactivation_accumulate():
    case = C.ROUTE_CASES[3]
    L = _layer(case, row_cap=8, recv_cap=8)
    L.route()
    L.coactivation(False)
    L.coactivation(True)
    torch.cuda.synchronize()
    r, _ = C.oracle_routing(case.name, case.placement, case.p, case.c)
    coact = oracle.coactivation(r["idx"], r["keep"], case.cfg.E)
    assert np.array_equal(L.host("coact").view(np.uint32), 2 * coact)


@pytest.mark.parametrize("case", C.ROUTE_CASES[:3], ids=lambda c: c.id)
def test_front_with_side_stream_matches_serial(case):
    """Co-activation on a side stream (beside the layout) gives the same bits."""
    L = _layer(case)
    L.front()
    torch.cuda.synchronize()
    want = {n: L.host(n).copy() for n in ("coact", "slot_pos", "expert_offsets", "totals", "copy_row")}
    L.coact.zero_()
    L.lay_t["slot_pos"].fill_(-7)
    side = torch.cuda.Stream()
    for _ in range(2):
        L.front(side=side)
    torch.cuda.synchronize()
    for n, v in want.items():
        assert np.array_equal(L.host(n), v), n


@pytest.mark.parametrize("name", ["c4", "c2"])
def test_step_with_side_stream_matches_serial(name):
    """The step with the shared experts and the co-activation counts on a side
    stream (joined before the source reduce) gives the serial step's bits."""
    case = C.Case(name, gen.CONFIGS[name], "coact", 0.1)
    cfg = case.cfg
    er, el = C.placement(name, "coact", 0.1, 5.0)
    L = _layer(case, x=gen.activations(cfg))
    L.set_rank_weights(0, *C.rank_weights(cfg, er, el, 0))
    if cfg.n_shared:
        L.set_shared_weights(*gen.shared_weights(cfg))
    g0 = torch.Generator(device="cuda").manual_seed(3)
    L.parts.copy_((torch.randn(L.parts.shape, generator=g0, device="cuda") * 0.05).to(L.tdt))
    # Y holds only the rows the FFN does not combine into parts itself: start
    # every run from the same contents
    L.Y.zero_()
    L.step(0)
    torch.cuda.synchronize()
    rows = L.rank_rows(0)
    names = ("y", "Y", "parts", "coact") + (("shared_out",) if cfg.n_shared else ())

    def snap(n):
        v = L.host(n)
        return v[:rows].copy() if n == "Y" else v.copy()

    want = {n: snap(n) for n in names}
    side = torch.cuda.Stream()
    for rep in range(2):
        L.y.zero_()
        L.Y.zero_()
        L.coact.zero_()
        if cfg.n_shared:
            L.shared_out.zero_()
        L.step(0, side=side)
        torch.cuda.synchronize()
        for n in names:
            assert np.array_equal(snap(n).view(np.uint8), want[n].view(np.uint8)), (rep, n)


def _check_router_route(L, cfg, x_bits, wg_bits, er, rows=None):
    """Fused router + routing: the decisions equal the logits-in kernel's (and
    the oracle's) on the logits the fused kernel used, and those logits equal
    x W_g^T within the fp32 accumulation bound d * 2^-24 * sum |x_k w_k|."""
    from paper_2607_05116_amd.layer import to_device_rows
    wg = to_device_rows(wg_bits, "bf16", "cuda")
    lg = torch.empty((cfg.T, cfg.E), dtype=torch.float32, device="cuda")
    L.router_route(wg, lg)
    torch.cuda.synchronize()
    fused = {n: L.host(n).copy() for n in ("idx", "w", "keep", "mask")}
    L.logits.copy_(lg)
    L.route()
    torch.cuda.synchronize()
    for n, v in fused.items():
        assert np.array_equal(L.host(n).view(np.uint8), v.view(np.uint8)), n
    lg_h = lg.cpu().numpy()
    r = oracle.route_prune(lg_h, cfg.k, er, cfg.ranks_per_node, cfg.tokens_per_rank, L.topo.inter_node_cost,
                           L.p)
    assert np.array_equal(fused["idx"], r["idx"])
    assert np.array_equal(fused["w"].view(np.uint32), r["wp"].view(np.uint32))
    assert np.array_equal(fused["mask"].view(np.uint64), r["mask"])
    rows = np.arange(cfg.T) if rows is None else rows
    xf = gen.bf16_bits_to_f32(x_bits[rows]).astype(np.float64)
    wf = gen.bf16_bits_to_f32(wg_bits).astype(np.float64)
    ref = oracle.router_logits(xf, wf)
    bound = cfg.d * 2.0 ** -24 * (np.abs(xf) @ np.abs(wf).T)
    err = np.abs(lg_h[rows].astype(np.float64) - ref)
    assert np.all(err <= bound), float((err / np.maximum(bound, 1e-300)).max())


@pytest.mark.parametrize("name,kind,p", [("c2", "coact", 0.3), ("c3", "seq", 0.1), ("c4", "coact", 0.1),
                                         ("c5", "coact", 0.1)])
def test_router_route_fused(name, kind, p):
    cfg = gen.CONFIGS[name]
    er, el = C.placement(name, kind, p, 5.0)
    x = gen.activations(cfg)
    L = DeviceLayer(cfg, np.zeros((cfg.T, cfg.E), np.float32), x, er, el, p, 5.0, row_cap=8, recv_cap=8)
    rows = np.random.default_rng(3).choice(cfg.T, size=4096, replace=False) if cfg.d * cfg.E > 2 ** 20 else None
    _check_router_route(L, cfg, x, gen.router_weights(cfg), er, rows)


@pytest.mark.parametrize("T,E,k,R,rpn,d,p", [(1000, 40, 3, 8, 4, 192, 0.2), (264, 256, 8, 8, 8, 128, 0.3),
                                             (130, 24, 2, 2, 2, 64, 0.0), (4096, 64, 6, 8, 8, 2048, 0.1)])
def test_router_route_odd_shapes(T, E, k, R, rpn, d, p):
    """Ragged token tails, E not a power of two times 8, k = 2..8."""
    cfg = gen.Config("rt", T=T, d=d, E=E, k=k, inter=128, R=R, ranks_per_node=rpn, n_clusters=1,
                     zipf_s=0.0, dtype="bf16")
    rng = np.random.default_rng(T + E)
    x = gen.f32_to_bf16_bits(rng.standard_normal((T, d)).astype(np.float32))
    wg = gen.f32_to_bf16_bits((rng.standard_normal((E, d)) / np.sqrt(d)).astype(np.float32))
    perm = rng.permutation(E)
    er, el = (perm // (E // R)).astype(np.int32), (perm % (E // R)).astype(np.int32)
    L = DeviceLayer(cfg, np.zeros((T, E), np.float32), x, er, el, p, 5.0, row_cap=8, recv_cap=8)
    _check_router_route(L, cfg, x, wg, er)


def test_graph_replay_matches_eager():
    """The captured step, replayed three times with eager work and host syncs
    in between, reproduces the eager step's outputs bit for bit each time."""
    name, kind, p = "c4", "coact", 0.1
    case = C.Case(name, gen.CONFIGS[name], kind, p)
    cfg = case.cfg
    er, el = C.placement(name, kind, p, 5.0)
    L = _layer(case, x=gen.activations(cfg))
    L.set_rank_weights(0, *C.rank_weights(cfg, er, el, 0))
    L.set_shared_weights(*gen.shared_weights(cfg))
    g0 = torch.Generator(device="cuda").manual_seed(11)
    L.parts.copy_((torch.randn(L.parts.shape, generator=g0, device="cuda") * 0.05).to(L.tdt))
    side = torch.cuda.Stream()
    L.Y.zero_()                                    # rows combined into parts by the FFN stay as they are
    L.front(side=side)
    L.rank_path(0)
    torch.cuda.synchronize()
    names = ("y", "Y", "parts", "coact", "idx", "w", "mask", "row_src", "row_dst", "row_w")
    rows = L.rank_rows(0)                          # Y and the row plan past this are capacity, never written

    def snap(n):
        v = L.host(n)
        return v[:rows].copy() if n in ("Y", "row_src", "row_dst", "row_w") else v.copy()

    want = {n: snap(n) for n in names}
    graph = L.capture_step(0, side=side)
    for rep in range(3):
        L.y.zero_()
        L.Y.zero_()
        L.coact.zero_()
        L.idx.fill_(-1)
        L.route()                                   # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for n in names:
            assert np.array_equal(snap(n).view(np.uint8), want[n].view(np.uint8)), (rep, n)


def _adversarial_logits(T, E, seed):
    rng = np.random.default_rng(seed)
    L = rng.standard_normal((T, E)).astype(np.float32)
    L[: T // 4] = gen.bf16_bits_to_f32(gen.f32_to_bf16_bits(L[: T // 4] * 0.02))  # heavy ties
    L[T // 4: T // 4 + 8] = 0.0                                                    # all equal
    L[T // 4 + 8: T // 4 + 16] = -0.0
    L[T // 4 + 16: T // 4 + 24, ::2] = -0.0                                        # +-0 mix
    tiny = np.array([1e-45, 1e-40, 1e-38, 0.0, -0.0, -1e-45, -1e-40, -1e-38], np.float32)
    huge = np.array([8.5e37, 3e36, 1e30, -1e30, -3e36, -8.5e37], np.float32)
    blk = L[T // 4 + 24: T // 4 + 32]
    blk[:] = rng.choice(tiny, size=blk.shape)                                      # subnormal ties
    blk = L[T // 4 + 32: T // 4 + 40]
    blk[:] = rng.choice(huge, size=blk.shape)                                      # extreme exponents
    return L


ADV_SHAPES = [
    (16, 2, 4, 4, 0.3, 5.0), (64, 6, 8, 4, 0.25, 5.0), (128, 8, 16, 8, 0.1, 5.0),
    (256, 8, 32, 8, 0.2, 3.0), (7, 3, 1, 1, 0.4, 5.0), (24, 5, 6, 2, 0.5, 2.0),
    (128, 8, 64, 8, 0.3, 5.0), (96, 1, 8, 8, 0.0, 5.0), (40, 8, 4, 2, 0.05, 5.0),
    # the four-lane kernel with one slot per lane (k <= 4) and a partly filled second slot
    (64, 4, 8, 4, 0.2, 5.0), (256, 3, 16, 8, 0.3, 3.0), (128, 1, 8, 8, 0.1, 5.0), (128, 5, 16, 4, 0.25, 5.0)]


@pytest.mark.parametrize("E,k,R,rpn,p,c", ADV_SHAPES)
def test_route_adversarial_and_odd_shapes(E, k, R, rpn, p, c):
    T = R * 160
    L = _adversarial_logits(T, E, E + k)
    perm = np.random.default_rng(R).permutation(E)
    er, el = (perm // (E // R)).astype(np.int32), (perm % (E // R)).astype(np.int32)
    cfg = gen.Config("adv", T=T, d=8, E=E, k=k, inter=128, R=R, ranks_per_node=rpn, n_clusters=1,
                     zipf_s=0.0, dtype="bf16")
    Ld = DeviceLayer(cfg, L, np.zeros((T, 8), np.uint16), er, el, p, c, row_cap=8, recv_cap=8)
    Ld.front()
    torch.cuda.synchronize()
    r = oracle.route_prune(L, k, er, rpn, T // R, c, p)
    lay = oracle.dispatch_layout(r["idx"], r["keep"], r["mask"], er, el, R, rpn, T // R, E)
    assert np.array_equal(Ld.host("idx"), r["idx"])
    assert np.array_equal(Ld.host("w").view(np.uint32), r["wp"].view(np.uint32))
    assert np.array_equal(Ld.host("mask").view(np.uint64), r["mask"])
    for name in ("slot_pos", "copy_row", "vol", "expert_offsets", "send_counts", "totals"):
        assert np.array_equal(Ld.host(name), lay[name]), name
    assert np.array_equal(Ld.host("coact").view(np.uint32), oracle.coactivation(r["idx"], r["keep"], E))


@pytest.mark.parametrize("E,k,R,rpn,p,c", ADV_SHAPES)
def test_route_naive_adversarial_and_odd_shapes(E, k, R, rpn, p, c):
    """Expert-level pruning (cap_route_prune_naive) on the adversarial logits
    and shapes, against the oracle's top-k, gates and naive pruning."""
    T = R * 160
    L = _adversarial_logits(T, E, E + k + 1)
    perm = np.random.default_rng(R + 1).permutation(E)
    er, el = (perm // (E // R)).astype(np.int32), (perm % (E // R)).astype(np.int32)
    cfg = gen.Config("adv", T=T, d=8, E=E, k=k, inter=128, R=R, ranks_per_node=rpn, n_clusters=1,
                     zipf_s=0.0, dtype="bf16")
    Ld = DeviceLayer(cfg, L, np.zeros((T, 8), np.uint16), er, el, p, c, row_cap=8, recv_cap=8)
    Ld.naive = True
    Ld.route()
    torch.cuda.synchronize()
    idx = oracle.topk(L, k)
    w = oracle.gates(L, idx)
    keep, wp, mask = oracle.prune_naive(idx, w, er, p)
    assert np.array_equal(Ld.host("idx"), idx)
    assert np.array_equal(Ld.host("w").view(np.uint32), wp.view(np.uint32))
    assert np.array_equal(Ld.host("keep"), keep)
    assert np.array_equal(Ld.host("mask").view(np.uint64), mask)


def _edge_logits(T, E, k, seed):
    """Rows whose gaps to the top logit span [-90, -80] (including exactly
    -87.33 in fp32, the exponential's cutoff, and gaps whose 2^n scaling is
    near the bottom of the normal range), with top logits 0 (so the gap is the
    logit itself, exactly) or large."""
    rng = np.random.default_rng(seed)
    L = np.full((T, E), -1e4, np.float32)
    edge = np.array([-80.0, -84.5, -86.0, -87.0, -87.33, -87.34, -88.0, -89.5, -90.0], np.float32)
    for t in range(T):
        top = np.float32(0.0) if t % 3 else np.float32(rng.uniform(-40, 40))
        g = np.concatenate([[np.float32(0.0)], rng.permutation(edge)[:k - 1]]).astype(np.float32)
        if t % 2:
            g[1:] = g[1:] + rng.uniform(-0.5, 0.5, size=k - 1).astype(np.float32)
        cols = rng.permutation(E)[:k]
        L[t, cols] = (top + g).astype(np.float32) if top != 0 else g
    return L


def _exact_sum_logits(T, E, k, er, tokens_per_rank, rpn, seed):
    """Tokens whose k selected logits are equal (gates exactly 1/k) and whose
    experts sit two on one remote device and one on each of k - 2 other
    remote devices of the same node: device scores 2/k, 1/k, ..., so the
    greedy's fp32 running sum lands exactly on 1 - p for p = 1 - m/k."""
    rng = np.random.default_rng(seed)
    L = np.full((T, E), -5.0, np.float32)
    R = int(er.max()) + 1
    for t in range(T):
        src = t // tokens_per_rank
        node = src // rpn
        others = [d for d in range(node * rpn, (node + 1) * rpn) if d != src]
        devs = rng.permutation(others)[:k - 1]
        chosen = []
        for j, d in enumerate(devs):
            pool = [e for e in np.flatnonzero(er == d) if e not in chosen]
            take = 2 if j == 0 else 1
            chosen += list(rng.choice(pool, size=take, replace=False))
        L[t, chosen] = 5.0
    return L


@pytest.mark.parametrize("kind,p", [("cutoff", 0.3), ("cutoff", 0.0), ("exact", 0.25), ("exact", 0.5),
                                    ("exact", 0.75)])
def test_route_gate_cutoff_and_exact_greedy_sum(kind, p):
    """Bit-exact routing where the arithmetic is at its edges: gate
    exponentials around the -87.33 cutoff (returned as 0 below it, scaled by
    2^n with n near -126 above it), and pruning whose fp32 running sum reaches
    1 - p exactly (Eq. 6 keeps the device that makes it reach the target and
    no more)."""
    E, R, rpn = 64, 8, 8
    k = 8 if kind == "cutoff" else 4
    T = R * 96
    perm = np.random.default_rng(5).permutation(E)
    er, el = (perm // (E // R)).astype(np.int32), (perm % (E // R)).astype(np.int32)
    if kind == "cutoff":
        L = _edge_logits(T, E, k, 11)
    else:
        L = _exact_sum_logits(T, E, k, er, T // R, rpn, 12)
    cfg = gen.Config("edge", T=T, d=8, E=E, k=k, inter=128, R=R, ranks_per_node=rpn, n_clusters=1,
                     zipf_s=0.0, dtype="bf16")
    Ld = DeviceLayer(cfg, L, np.zeros((T, 8), np.uint16), er, el, p, 5.0, row_cap=8, recv_cap=8)
    Ld.front()
    torch.cuda.synchronize()
    r = oracle.route_prune(L, k, er, rpn, T // R, 5.0, p)
    assert np.array_equal(Ld.host("idx"), r["idx"])
    assert np.array_equal(Ld.host("w").view(np.uint32), r["wp"].view(np.uint32))
    assert np.array_equal(Ld.host("keep"), r["keep"])
    assert np.array_equal(Ld.host("mask").view(np.uint64), r["mask"])
    if kind == "cutoff":
        w = oracle.gates(L, r["idx"])
        assert np.any(w == 0.0) and np.any((w > 0) & (w < 1e-35))      # both sides of the cutoff reached
    else:
        # the target is reached exactly: kept devices = the fewest whose score reaches 1 - p
        n_dev = np.array([bin(int(m)).count("1") for m in r["mask"]])
        want = {0.25: 2, 0.5: 1, 0.75: 1}[p]
        assert np.all(n_dev == want), np.unique(n_dev)


@pytest.mark.parametrize("T,k,E", [(600_000, 8, 256), (200_000, 8, 128), (1000, 3, 7), (1, 1, 1)])
def test_coactivation_duplicates_and_many_splits(T, k, E):
    """Random expert ids (duplicates within a token included) and random keep
    flags, up to 600k tokens (the largest split size), straight through the
    C-ABI, accumulating onto a nonzero start."""
    rng = np.random.default_rng(T + E)
    idx = rng.integers(0, E, (T, k), dtype=np.int32)
    keep = (rng.random((T, k)) < 0.7).astype(np.uint8)
    start = rng.integers(0, 1000, (E, E)).astype(np.uint32)
    dev = torch.device("cuda:0")
    idx_d = torch.from_numpy(idx).to(dev)
    keep_d = torch.from_numpy(keep).to(dev)
    coact_d = torch.from_numpy(start.view(np.int32)).to(dev)
    ws_bytes = capi.cap_workspace_size(capi.CAP_OP_COACTIVATION, _coact_topo(T, E))
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=dev)
    capi.cap_coactivation(T, k, E, idx_d, keep_d, coact_d, True, ws, ws_bytes)
    torch.cuda.synchronize()
    want = start + oracle.coactivation(idx, keep, E)
    assert np.array_equal(coact_d.cpu().numpy().view(np.uint32), want)


def _coact_topo(T, E):
    return capi.Topology(E=E, R=1, ranks_per_node=1, T=T, tokens_per_rank=T, k=1)


def test_determinism_front_end():
    case = C.ROUTE_CASES[5]
    L = _layer(case, row_cap=8, recv_cap=8)
    outs = []
    for _ in range(3):
        L.front()
        torch.cuda.synchronize()
        outs.append([L.host(n).copy() for n in ("idx", "w", "keep", "mask", "slot_pos", "copy_row", "coact")])
    for a, b in zip(outs[0], outs[1]):
        assert np.array_equal(a, b)
    for a, b in zip(outs[0], outs[2]):
        assert np.array_equal(a, b)


# ---------------------------------------------------------------- permutation
@pytest.mark.parametrize("name,kind,p", [("c1", "seq", 0.3), ("c2", "coact", 0.3), ("c3", "coact", 0.1),
                                         ("c4", "coact", 0.1), ("c5", "coact", 0.1)])
def test_permute_exact(name, kind, p):
    case = C.Case(name, gen.CONFIGS[name], kind, p)
    cfg = case.cfg
    x = gen.activations(cfg)
    L = _layer(case, x=x)
    L.front()
    r, lay = C.oracle_routing(name, kind, p, 5.0)
    er, _ = C.placement(name, kind, p, 5.0)
    ranks = range(cfg.R) if cfg.R <= 4 else [0, cfg.R - 1]
    for rank in ranks:
        L.gather(rank)
        torch.cuda.synchronize()
        want = oracle.expert_gather(x, r["idx"], r["keep"], lay["slot_pos"], lay["expert_offsets"], er, cfg.R, rank)
        got = L.host("xs")[: want.shape[0]]
        assert np.array_equal(got.view(np.uint8), want.view(np.uint8)), rank
        out = torch.empty((int(lay["send_counts"][rank].sum()), cfg.d), dtype=L.tdt, device="cuda")
        L.send_pack(rank, out)
        torch.cuda.synchronize()
        want = oracle.send_pack(x, r["mask"], lay["send_offsets"], lay["send_counts"], cfg.R,
                                cfg.tokens_per_rank, rank)
        got = out.view(torch.int16).cpu().numpy() if cfg.dtype == "bf16" else out.cpu().numpy()
        assert np.array_equal(got.view(np.uint8), want.view(np.uint8)), rank


@pytest.mark.parametrize("case", C.ROUTE_CASES, ids=lambda c: c.id)
def test_row_source_bit_exact(case):
    """CAP_PERMUTE_ROW_SOURCE is the expert gather of the token index."""
    cfg = case.cfg
    L = _layer(case)
    L.front()
    r, lay = C.oracle_routing(case.name, case.placement, case.p, case.c)
    er, _ = C.placement(case.name, case.placement, case.p, case.c)
    tok = np.arange(cfg.T, dtype=np.int32)[:, None]
    for rank in sorted({0, cfg.R - 1}):
        L.row_source(rank)
        torch.cuda.synchronize()
        want = oracle.expert_gather(tok, r["idx"], r["keep"], lay["slot_pos"], lay["expert_offsets"], er, cfg.R,
                                    rank)[:, 0]
        got = L.row_src[: len(want)].cpu().numpy()
        assert np.array_equal(got, want), rank


@pytest.mark.parametrize("name,kind,p", [("c1", "seq", 0.3), ("c2", "coact", 0.3), ("c4", "coact", 0.1),
                                         ("c5", "coact", 0.1)])
def test_ffn_gather_equals_ffn_on_gathered_rows(name, kind, p):
    """Reading x through row_src gives the same bits as the FFN on the gathered copy."""
    case = C.Case(name, gen.CONFIGS[name], kind, p)
    cfg = case.cfg
    er, el = C.placement(name, kind, p, 5.0)
    L = _layer(case, x=gen.activations(cfg))
    for rank in sorted({0, cfg.R - 1}):
        L.set_rank_weights(rank, *C.rank_weights(cfg, er, el, rank))
        L.front()
        L.gather(rank)
        L.ffn(rank)
        torch.cuda.synchronize()
        rows = L.rank_rows(rank)
        want = L.Y[:rows].clone()
        L.Y.zero_()
        L.row_source(rank)
        L.ffn_gather(rank)
        torch.cuda.synchronize()
        assert torch.equal(L.Y[:rows].view(torch.uint8), want.view(torch.uint8)), rank
        del L.weights[rank]


@pytest.mark.parametrize("dtype,d,inter,counts", [("bf16", 512, 384, [300, 1, 0, 513]),
                                                  ("bf16", 256, 128, [0, 700, 40]),
                                                  ("bf16", 256, 128, [3000, 1, 0, 5200]),  # fused kernel
                                                  ("f32", 128, 256, [70, 0, 131])])
def test_ffn_gather_ragged_with_repeats_and_clamping(dtype, d, inter, counts):
    """Ragged experts, repeated source rows and out-of-range indices (clamped
    into [0, x_rows)) against cap_expert_ffn on the explicitly gathered rows."""
    rng = np.random.default_rng(len(counts) + d)
    E_loc, rows = len(counts), int(sum(counts))
    offs = torch.from_numpy(np.concatenate([[0], np.cumsum(counts)]).astype(np.int32) + 9).cuda()
    x_rows = 97
    max_rows = rows + 3
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    cdt = capi.CAP_DTYPE_BF16 if dtype == "bf16" else capi.CAP_DTYPE_F32
    x = torch.from_numpy(rng.standard_normal((x_rows, d)).astype(np.float32)).to(tdt).cuda()
    src = rng.integers(-3, x_rows + 3, size=max_rows).astype(np.int32)
    row_src = torch.from_numpy(src).cuda()
    xs = x[torch.from_numpy(np.clip(src, 0, x_rows - 1).astype(np.int64)).cuda()].contiguous()
    w1 = (torch.randn(E_loc, inter, d, device="cuda") / d ** 0.5).to(tdt)
    w3 = (torch.randn(E_loc, inter, d, device="cuda") / d ** 0.5).to(tdt)
    w2 = (torch.randn(E_loc, d, inter, device="cuda") / (12 * inter ** 0.5)).to(tdt)
    ws = torch.empty(capi.cap_workspace_size(capi.CAP_OP_EXPERT_FFN, None, d, inter, max_rows, cdt),
                     dtype=torch.uint8, device="cuda")
    y_ref = torch.zeros((max_rows, d), dtype=tdt, device="cuda")
    y = torch.zeros((max_rows, d), dtype=tdt, device="cuda")
    capi.cap_expert_ffn(cdt, E_loc, d, inter, max_rows, xs, offs, w1, w3, w2, y_ref, ws)
    capi.cap_expert_ffn_gather(cdt, E_loc, d, inter, max_rows, x, x_rows, row_src, offs, w1, w3, w2, y, ws)
    torch.cuda.synchronize()
    assert torch.equal(y[:rows].view(torch.uint8), y_ref[:rows].view(torch.uint8))


# Row capacity from which a bf16 call runs the fused kernel (both GEMMs in one
# launch, a tile queue per XCD); below it the two-kernel path runs.
FUSED_MIN_ROWS = 8192


def test_ffn_gather_offsets_near_4gib():
    """Gathered rows at the far end of an x of just under 4 GiB (the limit the
    C ABI states: x_rows * d * 2 < 2^32): the 32-bit byte offsets of the
    gathered loads reach the last rows exactly; the result equals the FFN on
    the explicitly gathered rows, on the fused kernel's path (row capacity
    >= 8192) and on the two-kernel path."""
    d, inter = 2048, 256
    x_rows = (1 << 32) // (d * 2) - 1                       # 1,048,575 rows, 4 GiB - 4 KiB
    counts = [3000, 0, 2000, 3100]                           # 8100 rows: < 8192 for the two-kernel path
    E_loc, rows = len(counts), sum(counts)
    g = torch.Generator(device="cuda").manual_seed(17)
    x = torch.randn((x_rows, d), generator=g, device="cuda").to(torch.bfloat16)
    src = torch.randint(x_rows - 20000, x_rows, (rows,), generator=g, device="cuda", dtype=torch.int32)
    src[:8] = x_rows - 1                                     # the very last row
    offs = torch.tensor(np.concatenate([[0], np.cumsum(counts)]).astype(np.int32), device="cuda")
    w1 = (torch.randn((E_loc, inter, d), generator=g, device="cuda") / d ** 0.5).to(torch.bfloat16)
    w3 = (torch.randn((E_loc, inter, d), generator=g, device="cuda") / d ** 0.5).to(torch.bfloat16)
    w2 = (torch.randn((E_loc, d, inter), generator=g, device="cuda") / (12 * inter ** 0.5)).to(torch.bfloat16)
    cdt = capi.CAP_DTYPE_BF16
    for max_rows in (FUSED_MIN_ROWS + 64, rows):
        row_src = torch.zeros(max_rows, dtype=torch.int32, device="cuda")
        row_src[:rows] = src
        xs = torch.zeros((max_rows, d), dtype=torch.bfloat16, device="cuda")
        xs[:rows] = x[src.long()]
        ws = torch.empty(capi.cap_workspace_size(capi.CAP_OP_EXPERT_FFN, None, d, inter, max_rows, cdt),
                         dtype=torch.uint8, device="cuda")
        y_ref = torch.zeros((max_rows, d), dtype=torch.bfloat16, device="cuda")
        y = torch.zeros((max_rows, d), dtype=torch.bfloat16, device="cuda")
        capi.cap_expert_ffn(cdt, E_loc, d, inter, max_rows, xs, offs, w1, w3, w2, y_ref, ws)
        capi.cap_expert_ffn_gather(cdt, E_loc, d, inter, max_rows, x, x_rows, row_src, offs, w1, w3, w2, y, ws)
        torch.cuda.synchronize()
        assert torch.equal(y[:rows].view(torch.int16), y_ref[:rows].view(torch.int16)), max_rows
    del x


# ---------------------------------------------------------------- expert FFN
def _ffn_direct(dtype, E_loc, d, inter, counts, seed=0, max_rows=None):
    """cap_expert_ffn on synthetic ragged experts; returns (gpu Y, oracle Y)."""
    rng = np.random.default_rng(seed)
    rows = int(sum(counts))
    offs = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32) + 17    # non-zero base
    x32 = rng.standard_normal((rows, d)).astype(np.float32)
    w1 = (rng.standard_normal((E_loc, inter, d)) / np.sqrt(d)).astype(np.float32)
    w3 = (rng.standard_normal((E_loc, inter, d)) / np.sqrt(d)).astype(np.float32)
    w2 = (rng.standard_normal((E_loc, d, inter)) / (12 * np.sqrt(inter))).astype(np.float32)
    if dtype == "bf16":
        q = lambda a: gen.f32_to_bf16_bits(a)
        x32, w1, w3, w2 = (gen.bf16_bits_to_f32(q(a)) for a in (x32, w1, w3, w2))
        tdt, cdt = torch.bfloat16, capi.CAP_DTYPE_BF16
        dev = lambda a: torch.from_numpy(q(a).view(np.int16)).view(torch.bfloat16).cuda()
    else:
        tdt, cdt = torch.float32, capi.CAP_DTYPE_F32
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    max_rows = rows + 5 if max_rows is None else max_rows
    xs = torch.zeros((max_rows, d), dtype=tdt, device="cuda")
    xs[:rows] = dev(x32)
    y = torch.zeros((max_rows, d), dtype=tdt, device="cuda")
    ws = torch.empty(capi.cap_workspace_size(capi.CAP_OP_EXPERT_FFN, None, d, inter, max_rows, cdt),
                     dtype=torch.uint8, device="cuda")
    capi.cap_expert_ffn(cdt, E_loc, d, inter, max_rows, xs, torch.from_numpy(offs).cuda(), dev(w1), dev(w3),
                        dev(w2), y, ws)
    torch.cuda.synchronize()
    got = y[:rows].float().cpu().numpy()
    ref = oracle.expert_ffn(x32, offs, [(w1[l], w3[l], w2[l]) for l in range(E_loc)])
    return got, ref


@pytest.mark.parametrize("counts", [[300, 1, 0, 513], [256, 256], [1], [0, 0, 700, 40, 1000, 3]])
def test_ffn_bf16_ragged_experts(counts):
    got, ref = _ffn_direct("bf16", len(counts), 512, 384, counts, seed=len(counts))
    ok, worst = C.within_tol(got, ref)
    assert ok, worst
    assert C.rel_fro(got, ref) <= 1e-2


@pytest.mark.parametrize("d,inter,counts", [
    (256, 128, [3000, 0, 1, 257, 4100, 0, 900, 2000]),   # down GEMM of two K stages
    (512, 256, [9000]),                                   # every m-tile on one expert
    (256, 384, [40] * 200 + [0] * 56),                    # 256 experts, one partial m-tile each
    (256, 128, [100, 0, 200]),                            # two m-tiles: most XCD queues empty
    (512, 384, []),                                       # no rows at all
])
def test_ffn_fused_ragged_experts(d, inter, counts):
    counts = counts or [0, 0, 0]
    rows = int(sum(counts))
    got, ref = _ffn_direct("bf16", len(counts), d, inter, counts, seed=len(counts) + d,
                           max_rows=max(FUSED_MIN_ROWS, rows + 5))
    if rows == 0:
        return
    ok, worst = C.within_tol(got, ref)
    assert ok, worst
    assert C.rel_fro(got, ref) <= 1e-2


def test_ffn_fused_equals_two_kernel_path():
    """The same rows with row capacities on either side of the fused kernel's
    threshold give identical bits, and repeated fused calls (its counters are
    cleared by every call) give the same bits again."""
    rng = np.random.default_rng(5)
    d, inter, counts = 512, 256, [700, 0, 1500, 3, 2000, 257]
    E_loc, rows = len(counts), sum(counts)
    offs = torch.from_numpy(np.concatenate([[0], np.cumsum(counts)]).astype(np.int32) + 4).cuda()
    cdt = capi.CAP_DTYPE_BF16
    bf = lambda a: torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16).cuda()
    w1 = bf(rng.standard_normal((E_loc, inter, d)) / np.sqrt(d))
    w3 = bf(rng.standard_normal((E_loc, inter, d)) / np.sqrt(d))
    w2 = bf(rng.standard_normal((E_loc, d, inter)) / (12 * np.sqrt(inter)))
    x = bf(rng.standard_normal((FUSED_MIN_ROWS, d)))
    outs = []
    for max_rows in (FUSED_MIN_ROWS - 1, FUSED_MIN_ROWS, FUSED_MIN_ROWS):
        ws = torch.full((capi.cap_workspace_size(capi.CAP_OP_EXPERT_FFN, None, d, inter, max_rows, cdt),), 0xA5,
                        dtype=torch.uint8, device="cuda")          # non-zero: the call clears its counters
        y = torch.zeros((max_rows, d), dtype=torch.bfloat16, device="cuda")
        for _ in range(2):
            capi.cap_expert_ffn(cdt, E_loc, d, inter, max_rows, x[:max_rows], offs, w1, w3, w2, y, ws)
        torch.cuda.synchronize()
        outs.append(y[:rows].view(torch.int16).cpu().numpy())
    assert np.array_equal(outs[0], outs[1])
    assert np.array_equal(outs[1], outs[2])


def test_ffn_fused_repeated_calls_identical():
    """Forty fused-kernel calls give the same bits each time, half of them
    while a large elementwise kernel on another stream holds compute units
    (workgroups then start late and unevenly, so the per-XCD queues and the
    waits for an m-tile's H rows run in other orders)."""
    rng = np.random.default_rng(9)
    d, inter = 512, 256
    counts = list(rng.integers(0, 2500, size=16))
    E_loc, rows = len(counts), int(sum(counts))
    max_rows = max(FUSED_MIN_ROWS, rows)
    offs = torch.tensor(np.concatenate([[0], np.cumsum(counts)]).astype(np.int32), device="cuda")
    g = torch.Generator(device="cuda").manual_seed(9)
    x = torch.randn((max_rows, d), generator=g, device="cuda").to(torch.bfloat16)
    w1 = (torch.randn((E_loc, inter, d), generator=g, device="cuda") / d ** 0.5).to(torch.bfloat16)
    w3 = (torch.randn((E_loc, inter, d), generator=g, device="cuda") / d ** 0.5).to(torch.bfloat16)
    w2 = (torch.randn((E_loc, d, inter), generator=g, device="cuda") / (12 * inter ** 0.5)).to(torch.bfloat16)
    cdt = capi.CAP_DTYPE_BF16
    ws = torch.empty(capi.cap_workspace_size(capi.CAP_OP_EXPERT_FFN, None, d, inter, max_rows, cdt),
                     dtype=torch.uint8, device="cuda")
    y = torch.zeros((max_rows, d), dtype=torch.bfloat16, device="cuda")
    capi.cap_expert_ffn(cdt, E_loc, d, inter, max_rows, x, offs, w1, w3, w2, y, ws)
    torch.cuda.synchronize()
    want = y[:rows].clone()
    want_sum = want.view(torch.int16).to(torch.int64).sum()
    other = torch.cuda.Stream()
    big = torch.zeros(1 << 28, dtype=torch.float32, device="cuda")
    sums = []
    for it in range(40):
        y.zero_()
        if it % 2:
            with torch.cuda.stream(other):
                big.add_(1.0)
        capi.cap_expert_ffn(cdt, E_loc, d, inter, max_rows, x, offs, w1, w3, w2, y, ws)
        sums.append(y[:rows].view(torch.int16).to(torch.int64).sum())
    torch.cuda.synchronize()
    assert all(int(v) == int(want_sum) for v in sums), [int(v) for v in sums]
    assert torch.equal(y[:rows].view(torch.int16), want.view(torch.int16))
    del big


@pytest.mark.parametrize("grid", [1, 3])
def test_ffn_fused_with_fewer_workgroups_than_xcds(grid):
    """With the fused kernel's grid capped below the XCD count, the queues of
    XCDs that ran no workgroup are run by the last workgroup to finish: the
    result is still complete and identical to the full grid's, and no wait
    gives up."""
    rng = np.random.default_rng(grid)
    d, inter, counts = 256, 128, [2000, 0, 3000, 1, 4000]
    E_loc, rows = len(counts), sum(counts)
    max_rows = FUSED_MIN_ROWS + 100
    offs = torch.from_numpy(np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)).cuda()
    bf = lambda a: torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16).cuda()
    w1 = bf(rng.standard_normal((E_loc, inter, d)) / np.sqrt(d))
    w3 = bf(rng.standard_normal((E_loc, inter, d)) / np.sqrt(d))
    w2 = bf(rng.standard_normal((E_loc, d, inter)) / (12 * np.sqrt(inter)))
    x = bf(rng.standard_normal((max_rows, d)))
    cdt = capi.CAP_DTYPE_BF16
    ws = torch.empty(capi.cap_workspace_size(capi.CAP_OP_EXPERT_FFN, None, d, inter, max_rows, cdt),
                     dtype=torch.uint8, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    outs = []
    for cap in (0, grid):
        y = torch.zeros((max_rows, d), dtype=torch.bfloat16, device="cuda")
        opts = capi.make_ffn_options(err, max_workgroups=cap)
        capi.cap_expert_ffn_ex(cdt, E_loc, d, inter, max_rows, x, 0, None, offs, w1, w3, w2, y, ws, options=opts)
        torch.cuda.synchronize()
        outs.append(y[:rows].view(torch.int16).cpu().numpy())
    assert int(err.item()) == 0
    assert np.array_equal(outs[0], outs[1])


@pytest.mark.parametrize("gathered", [False, True])
def test_ffn_fused_wait_give_up_is_counted(gathered):
    """The fused kernel's bounded waits report giving up.  The host makes every
    wait's target unreachable with a spin limit of 1 poll: each of the
    m-tiles x (d / 256) down tiles waits once and gives up, every kernel
    finishes, and the caller's counter holds exactly that many.  A normal call
    afterwards on the same workspace adds nothing and matches the two-kernel
    path's bits."""
    rng = np.random.default_rng(7)
    d, inter, counts = 512, 256, [3000, 4000, 700]
    E_loc, rows = len(counts), sum(counts)
    max_rows = FUSED_MIN_ROWS + 108
    assert rows < FUSED_MIN_ROWS <= max_rows
    m_tiles = sum((c + 255) // 256 for c in counts)
    offs = torch.from_numpy(np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)).cuda()
    bf = lambda a: torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16).cuda()
    w1 = bf(rng.standard_normal((E_loc, inter, d)) / np.sqrt(d))
    w3 = bf(rng.standard_normal((E_loc, inter, d)) / np.sqrt(d))
    w2 = bf(rng.standard_normal((E_loc, d, inter)) / (12 * np.sqrt(inter)))
    x = bf(rng.standard_normal((max_rows + 50, d)))
    src = torch.from_numpy(rng.permutation(max_rows + 50)[:max_rows].astype(np.int32)).cuda()
    cdt = capi.CAP_DTYPE_BF16
    ws = torch.empty(capi.cap_workspace_size(capi.CAP_OP_EXPERT_FFN, None, d, inter, max_rows, cdt),
                     dtype=torch.uint8, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    y = torch.zeros((max_rows, d), dtype=torch.bfloat16, device="cuda")

    def call(opts, cap_rows=max_rows, out=y):
        if gathered:
            capi.cap_expert_ffn_ex(cdt, E_loc, d, inter, cap_rows, x, x.shape[0], src, offs, w1, w3, w2, out, ws,
                                   options=opts)
        else:
            capi.cap_expert_ffn_ex(cdt, E_loc, d, inter, cap_rows, x, 0, None, offs, w1, w3, w2, out, ws,
                                   options=opts)
        torch.cuda.synchronize()

    call(capi.make_ffn_options(err, spin_limit=1, force_wait_timeout=True))
    assert int(err.item()) == m_tiles * (d // 256)
    err.zero_()
    call(capi.make_ffn_options(err))
    assert int(err.item()) == 0
    # the two-kernel path (capacity below the fused threshold) on the same rows
    y2 = torch.zeros((max_rows, d), dtype=torch.bfloat16, device="cuda")
    call(None, cap_rows=rows, out=y2)
    assert torch.equal(y[:rows].view(torch.int16), y2[:rows].view(torch.int16))


def test_ffn_f32_ragged_experts():
    got, ref = _ffn_direct("f32", 3, 128, 256, [70, 0, 131], seed=3)
    ok, worst = C.within_tol(got, ref, atol=1e-5, rtol=1e-4)
    assert ok, worst
    assert C.rel_fro(got, ref) <= 1e-5


ORACLE_THREADS = max(1, min(16, os.cpu_count() or 1))


def _m_tile_sample(eo, E_loc, rng, per_tile=2):
    """Rows of a rank's expert-sorted buffer: per_tile random rows of every
    256-row m-tile of every expert, plus each expert's first and last row."""
    rows = []
    base = int(eo[0])
    for l in range(E_loc):
        a, b = int(eo[l]) - base, int(eo[l + 1]) - base
        if b <= a:
            continue
        rows += [a, b - 1]
        for m0 in range(a, b, 256):
            m1 = min(b, m0 + 256)
            rows += list(rng.integers(m0, m1, size=per_tile))
    return np.unique(np.asarray(rows, np.int64))


def _oracle_ffn_rows(cfg, er, el, r, lay, x, rank, rows):
    """fp64 oracle SwiGLU of the given rows of a rank's expert-sorted buffer."""
    eo = lay["expert_offsets"][rank * cfg.E_loc:(rank + 1) * cfg.E_loc + 1].astype(np.int64)
    xs = oracle.expert_gather(x, r["idx"], r["keep"], lay["slot_pos"], lay["expert_offsets"], er, cfg.R, rank)
    xs32 = gen.bf16_bits_to_f32(xs) if cfg.dtype == "bf16" else xs
    ids = C.local_experts(er, el, rank, cfg.E_loc)
    ref = np.zeros((len(rows), cfg.d), np.float64)
    for l in range(cfg.E_loc):
        a, b = eo[l] - eo[0], eo[l + 1] - eo[0]
        sel = np.flatnonzero((rows >= a) & (rows < b))
        if len(sel):
            W1, W3, W2 = (gen.expert_weights_f32(cfg, ids[l]))
            ref[sel] = oracle.swiglu_rows(xs32[rows[sel]], W1, W3, W2, nthreads=ORACLE_THREADS)
    return ref


@pytest.mark.parametrize("name,kind,p,all_rows", [("c2", "coact", 0.3, True), ("c2", "seq", 0.0, True),
                                                  ("c4", "coact", 0.1, True), ("c3", "coact", 0.1, True),
                                                  ("c5", "coact", 0.1, False)])
def test_ffn_full_size_benched_path(name, kind, p, all_rows):
    """Rank 0's expert FFN at the workload's real shape through the benched
    path (row source + the gathered FFN, which reads x in place), against the
    fp64 oracle (Eq. 1 Expert_i): every row of the rank, or for the
    DeepSeek-V3-shaped layer two rows of every 256-row m-tile plus each
    expert's first and last row.  No wait of the fused kernel gave up."""
    case = C.Case(name, gen.CONFIGS[name], kind, p)
    cfg = case.cfg
    er, el = C.placement(name, kind, p, 5.0)
    r, lay = C.oracle_routing(name, kind, p, 5.0)
    x = gen.activations(cfg)
    L = _layer(case, x=x)
    L.set_rank_weights(0, *C.rank_weights(cfg, er, el, 0))
    L.front()
    L.row_source(0)
    L.ffn_gather(0)
    torch.cuda.synchronize()
    assert L.ffn_wait_errors() == 0
    n = L.rank_rows(0)
    eo = lay["expert_offsets"][:cfg.E_loc + 1]
    rows = np.arange(n) if all_rows else _m_tile_sample(eo, cfg.E_loc, np.random.default_rng(1))
    print(f"[{name} {kind} p={p}] rank-0 rows {n}, compared {len(rows)}", flush=True)
    got = L.Y[:n].float().cpu().numpy()[rows]
    ref = _oracle_ffn_rows(cfg, er, el, r, lay, x, 0, rows)
    ok, worst = C.within_tol(got, ref)
    assert ok, worst
    assert C.rel_fro(got, ref) <= 1e-2


def test_step_bf16_end_to_end_all_received_rows():
    """The whole benched step (DeviceLayer.step: routing, layout, co-activation,
    row source, gathered FFN, destination reduce, source reduce) on the
    Qwen3-shaped layer (coact, p = 0.3), bf16: every row rank 0 returns
    (all of its received tokens) against the oracle's destination reduce of
    the oracle FFN (Eq. 1 over the kept experts on rank 0; Sec. II-C local
    aggregation), and rank 0's source-reduced output against the oracle's
    source reduce of those rows (other ranks' returned rows zero here)."""
    name, kind, p = "c2", "coact", 0.3
    cfg = gen.CONFIGS[name]
    case = C.Case(name, cfg, kind, p)
    er, el = C.placement(name, kind, p, 5.0)
    r, lay = C.oracle_routing(name, kind, p, 5.0)
    x = gen.activations(cfg)
    L = _layer(case, x=x)
    L.set_rank_weights(0, *C.rank_weights(cfg, er, el, 0))
    L.parts.zero_()
    L.step(0)
    torch.cuda.synchronize()
    assert L.ffn_wait_errors() == 0
    n = L.rank_rows(0)
    U0 = int(lay["recv_offsets"][1])
    print(f"[c2 step] rank-0 rows {n}, received tokens {U0}", flush=True)
    Y = _oracle_ffn_rows(cfg, er, el, r, lay, x, 0, np.arange(n)).astype(np.float32)
    ref = oracle.dest_reduce(Y, r, lay, er, cfg.R, 0, cfg.d)
    got = L.parts[:U0].float().cpu().numpy()
    ok, worst = C.within_tol(got, ref)
    assert ok, worst
    assert C.rel_fro(got, ref) <= 1e-2
    parts = np.zeros((int(lay["recv_offsets"][-1]), cfg.d), np.float32)
    parts[:U0] = got
    ref_y = oracle.src_reduce(parts, r, lay, er, cfg.R, cfg.tokens_per_rank, 0, cfg.d)
    got_y = L.y.float().cpu().numpy()
    ok, worst = C.within_tol(got_y, ref_y)
    assert ok, worst
    assert C.rel_fro(got_y, ref_y) <= 1e-2


@pytest.mark.parametrize("name", ["c4", "c5"])
def test_shared_experts_and_src_reduce(name):
    """Shared experts at the workload's real shape: the shared SwiGLU (one FFN
    over the concatenated intermediate size) on sampled rank-0 tokens against
    the oracle, then the source reduce with the shared output added."""
    cfg = gen.CONFIGS[name]
    kind, p = "coact", 0.1
    case = C.Case(name, cfg, kind, p)
    er, el = C.placement(name, kind, p, 5.0)
    r, lay = C.oracle_routing(name, kind, p, 5.0)
    x = gen.activations(cfg)
    L = _layer(case, x=x)
    L.set_shared_weights(*gen.shared_weights(cfg))
    L.front()
    L.shared_ffn(0)
    torch.cuda.synchronize()
    T_loc = cfg.tokens_per_rank
    rng = np.random.default_rng(4)
    sample = np.sort(rng.choice(T_loc, size=48, replace=False))
    got = L.shared_out[torch.from_numpy(sample).cuda()].float().cpu().numpy()
    W1, W3, W2 = gen.shared_weights_f32(cfg)
    ref = oracle.swiglu_rows(gen.bf16_bits_to_f32(x[sample]), W1, W3, W2)
    ok, worst = C.within_tol(got, ref)
    assert ok, worst
    assert C.rel_fro(got, ref) <= 1e-2
    n_recv = int(lay["recv_offsets"][-1])
    parts = gen.random_rows(n_recv, cfg.d, "bf16", salt=5)
    L.parts[:n_recv] = torch.from_numpy(parts.view(np.int16)).view(torch.bfloat16).cuda()
    L.src_reduce(0)
    torch.cuda.synchronize()
    shared = L.shared_out.float().cpu().numpy()
    ref = oracle.src_reduce(gen.bf16_bits_to_f32(parts), r, lay, er, cfg.R, T_loc, 0, cfg.d, shared=shared)
    got = L.y.float().cpu().numpy()
    ok, worst = C.within_tol(got, ref)
    assert ok, worst
    assert C.rel_fro(got, ref) <= 1e-2


# ---------------------------------------------------------------- combine / whole layer
@pytest.mark.parametrize("cfgname,kind,p", [("c1", "seq", 0.3), ("c1u", "seq", 0.3), ("c1u", "coact", 0.0)])
def test_layer_tiny_fp32_end_to_end(cfgname, kind, p):
    """All 4 ranks on the GPU: gather -> FFN -> dest reduce; then every source
    rank's src reduce, against the oracle's independent dense Eq. 1 path."""
    cfg = gen.CONFIGS[cfgname]
    case = C.Case(cfgname, cfg, kind, p)
    er, el = C.placement(cfgname, kind, p, 5.0)
    x = gen.activations(cfg)
    L = DeviceLayer(cfg, gen.logits(cfg), x, er, el, p, 5.0)
    for rank in range(cfg.R):
        L.set_rank_weights(rank, *C.rank_weights(cfg, er, el, rank))
    L.front()
    for rank in range(cfg.R):
        L.gather(rank)
        L.ffn(rank)
        L.dest_reduce(rank)
    r = oracle.route_prune(gen.logits(cfg), cfg.k, er, cfg.ranks_per_node, cfg.tokens_per_rank, 5.0, p)
    wts = {e: gen.expert_weights_f32(cfg, e) for e in range(cfg.E)}
    for s in range(cfg.R):
        L.src_reduce(s)
        torch.cuda.synchronize()
        toks = np.arange(s * cfg.tokens_per_rank, (s + 1) * cfg.tokens_per_rank)
        ref = oracle.dense_moe_rows(toks, x[toks], r, lambda e: wts[e])
        got = L.host("y")
        ok, worst = C.within_tol(got, ref, atol=1e-6 if cfgname == "c1" else 1e-5, rtol=1e-4)
        assert ok, (s, worst)
        assert C.rel_fro(got, ref) <= 1e-5


@pytest.mark.parametrize("fused", [False, True])
def test_rank_with_no_rows(fused):
    """A degenerate placement: one rank's experts are never selected, so it
    computes no expert rows and receives no tokens.  Its permutation, FFN and
    destination reduce are empty calls; every source rank's result still
    equals the dense Eq. 1 path (c1u shape, fp32)."""
    cfg = gen.CONFIGS["c1u"]
    p = 0.3
    er, el = gen.sequential_placement(cfg)
    logits = gen.logits(cfg).copy()
    idle = cfg.R - 1
    logits[:, er == idle] -= 60.0                     # never in any token's top k
    x = gen.activations(cfg)
    L = DeviceLayer(cfg, logits, x, er, el, p, 5.0)
    L.fused_gather = fused
    for rank in range(cfg.R):
        L.set_rank_weights(rank, *C.rank_weights(cfg, er, el, rank))
    L.front()
    torch.cuda.synchronize()
    assert L.rank_rows(idle) == 0
    rec = L.host("recv_offsets")
    assert rec[idle + 1] == rec[idle]
    for rank in range(cfg.R):
        if fused:
            L.row_source(rank)
            L.ffn_gather(rank)
        else:
            L.gather(rank)
            L.ffn(rank)
        L.dest_reduce(rank)
    r = oracle.route_prune(logits, cfg.k, er, cfg.ranks_per_node, cfg.tokens_per_rank, 5.0, p)
    assert not np.isin(r["idx"], np.flatnonzero(er == idle)).any()
    wts = {e: gen.expert_weights_f32(cfg, e) for e in range(cfg.E)}
    for s in range(cfg.R):
        L.src_reduce(s)
        torch.cuda.synchronize()
        toks = np.arange(s * cfg.tokens_per_rank, (s + 1) * cfg.tokens_per_rank)
        ref = oracle.dense_moe_rows(toks, x[toks], r, lambda e: wts[e])
        got = L.host("y")
        ok, worst = C.within_tol(got, ref, atol=1e-5, rtol=1e-4)
        assert ok, (s, worst)
        assert C.rel_fro(got, ref) <= 1e-5


def test_combine_bf16_full_size_sampled():
    """C2 coact p=0.3, rank 0: destination reduce of the real FFN output on
    sampled received tokens, and source reduce of seeded returned rows."""
    name, kind, p = "c2", "coact", 0.3
    cfg = gen.CONFIGS[name]
    case = C.Case(name, cfg, kind, p)
    er, el = C.placement(name, kind, p, 5.0)
    r, lay = C.oracle_routing(name, kind, p, 5.0)
    x = gen.activations(cfg)
    L = _layer(case, x=x)
    L.set_rank_weights(0, *C.rank_weights(cfg, er, el, 0))
    L.front()
    L.gather(0)
    L.ffn(0)
    L.dest_reduce(0)
    torch.cuda.synchronize()
    U0 = int(lay["recv_offsets"][1])
    rng = np.random.default_rng(2)
    sample = np.sort(rng.choice(U0, size=32, replace=False))
    got = L.parts[torch.from_numpy(sample).cuda()].float().cpu().numpy()
    ref = np.zeros(got.shape, np.float64)
    for i, u in enumerate(sample):
        t = int(lay["recv_token"][u])
        for s in range(cfg.k):
            if r["keep"][t, s] and er[r["idx"][t, s]] == 0:
                W1, W3, W2 = gen.expert_weights_f32(cfg, int(r["idx"][t, s]))
                xt = gen.bf16_bits_to_f32(x[t:t + 1])
                ref[i] += float(r["wp"][t, s]) * oracle.swiglu_rows(xt, W1, W3, W2)[0]
    ok, worst = C.within_tol(got, ref)
    assert ok, worst
    assert C.rel_fro(got, ref) <= 1e-2
    # source reduce over seeded returned rows for every device
    n_recv = int(lay["recv_offsets"][-1])
    parts = gen.random_rows(n_recv, cfg.d, "bf16", salt=3)
    L.parts[:n_recv] = torch.from_numpy(parts.view(np.int16)).view(torch.bfloat16).cuda()
    L.src_reduce(0)
    torch.cuda.synchronize()
    ref = oracle.src_reduce(gen.bf16_bits_to_f32(parts), r, lay, er, cfg.R, cfg.tokens_per_rank, 0, cfg.d)
    got = L.y.float().cpu().numpy()
    ok, worst = C.within_tol(got, ref)
    assert ok, worst
    assert C.rel_fro(got, ref) <= 1e-2
