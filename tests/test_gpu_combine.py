"""The destination combine folded into the FFN (cap_row_plan,
cap_expert_ffn_combine, CAP_COMBINE_DEST_REDUCE_MULTI), through the C ABI.

A received token whose kept experts on the rank reduce to one row has a
one-term local aggregation (Sec. II-C; Eq. 1): the FFN's down GEMM writes
w' * y for it straight into the receive-side buffer, and the destination
reduce then handles only the tokens with two or more rows.  Checked against:
the plan's definition computed in numpy from the oracle's layout (bit-exact),
and the separate path (row source, gathered FFN, destination reduce) on the
same inputs: the receive-side rows are identical bit for bit, because the
epilogue does the single-term reduce's arithmetic.  The separate path itself
is checked against the fp64 oracle elsewhere; so is the step, which now takes
this path.
"""
import dataclasses

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


def _plan_ref(cfg, r, lay, rank, rows_cap, parts_rows):
    """(row_src, row_dst, row_w) of the plan's definition, for rows [0, rows used)."""
    E_loc, k = cfg.E_loc, cfg.k
    eo, ro = lay["expert_offsets"], lay["recv_offsets"]
    base = int(eo[rank * E_loc])
    rows_r = min(int(eo[(rank + 1) * E_loc]) - base, rows_cap)
    r0, U = int(ro[rank]), int(ro[rank + 1] - ro[rank])
    src = np.full(rows_r, -7, np.int32)
    dst = np.full(rows_r, -7, np.int32)
    wgt = np.full(rows_r, np.nan, np.float32)
    rt = lay["recv_token"]
    sp = lay["slot_pos"].astype(np.int64) - base
    for u in range(U):
        t = int(rt[r0 + u])
        mine = [s for s in range(k) if 0 <= sp[t, s] < rows_r]
        single = len(mine) == 1 and r0 + u < parts_rows
        for s in mine:
            i = int(sp[t, s])
            src[i] = t
            dst[i] = r0 + u if single else -1
            wgt[i] = r["wp"][t, s] if single else 0.0
    return src, dst, wgt


def _layer(name, kind, p, x=None, **kw):
    cfg = gen.CONFIGS[name]
    er, el = C.placement(name, kind, p, 5.0)
    if x is None:
        x = np.zeros((cfg.T, 8), np.uint16)
        cfg = dataclasses.replace(cfg, d=8)
    return DeviceLayer(cfg, C.logits(name), x, er, el, p, 5.0, **kw)


@pytest.mark.parametrize("name,kind,p", [("c2", "coact", 0.3), ("c2", "seq", 0.0), ("c3", "coact", 0.1),
                                         ("c4", "coact", 0.1), ("c5", "coact", 0.1), ("c5", "seq", 0.1)])
def test_row_plan_matches_definition(name, kind, p):
    cfg = gen.CONFIGS[name]
    r, lay = C.oracle_routing(name, kind, p, 5.0)
    L = _layer(name, kind, p)
    L.front()
    for rank in sorted({0, cfg.R - 1}):
        r0, U = int(lay["recv_offsets"][rank]), int(lay["recv_offsets"][rank + 1] - lay["recv_offsets"][rank])
        for parts_rows in (L.recv_cap, r0 + U // 2):
            L.row_src.fill_(-7)
            L.row_dst.fill_(-7)
            L.row_w.fill_(float("nan"))
            capi.cap_row_plan(L.topo, rank, L.w, L.lay, L.row_src, L.row_dst, L.row_w, L.row_cap, parts_rows)
            torch.cuda.synchronize()
            src, dst, wgt = _plan_ref(cfg, r, lay, rank, L.row_cap, parts_rows)
            n = len(src)
            assert np.array_equal(L.row_src[:n].cpu().numpy(), src), (rank, parts_rows)
            assert np.array_equal(L.row_dst[:n].cpu().numpy(), dst), (rank, parts_rows)
            assert np.array_equal(L.row_w[:n].cpu().numpy().view(np.uint32), wgt.view(np.uint32)), (rank, parts_rows)
            single = int((dst >= 0).sum())
            print(f"[{name} {kind} p={p} rank {rank} parts_rows {parts_rows}] rows {n}, single-expert {single}",
                  flush=True)


def _separate_and_fused(L, rank, parts_rows):
    """parts rows [0, parts_rows) and Y of the separate path, then of the fused one."""
    sentinel = torch.full_like(L.parts, 0)
    sentinel.view(torch.int16).fill_(0x7F7F)
    L.parts.copy_(sentinel)
    L.Y.view(torch.int16).fill_(0x7F7F)
    L.row_source(rank)
    L.ffn_gather(rank)
    capi.cap_combine(L.topo, capi.CAP_COMBINE_DEST_REDUCE, rank, L.dt, L.d, L.Y, L.row_cap, L.idx, L.w, L.keep,
                     L.mask, L.lay, None, L.parts, parts_rows)
    torch.cuda.synchronize()
    parts_a, y_a = L.parts[:parts_rows].clone(), L.Y.clone()
    L.parts.copy_(sentinel)
    L.Y.view(torch.int16).fill_(0x7F7F)
    capi.cap_row_plan(L.topo, rank, L.w, L.lay, L.row_src, L.row_dst, L.row_w, L.row_cap, parts_rows)
    w1, w3, w2 = L.weights[rank]
    E_loc = L.cfg.E_loc
    offs = L.lay_t["expert_offsets"][rank * E_loc:(rank + 1) * E_loc + 1]
    capi.cap_expert_ffn_combine(L.dt, E_loc, L.d, L.cfg.inter, L.row_cap, L.x, L.x.shape[0], L.row_src, offs,
                                w1, w3, w2, L.Y, L.row_dst, L.row_w, L.parts, parts_rows, L.ws_ffn,
                                options=L.ffn_opts)
    capi.cap_combine(L.topo, capi.CAP_COMBINE_DEST_REDUCE_MULTI, rank, L.dt, L.d, L.Y, L.row_cap, L.idx, L.w,
                     L.keep, L.mask, L.lay, None, L.parts, parts_rows)
    torch.cuda.synchronize()
    return parts_a, y_a, L.parts[:parts_rows].clone(), L.Y.clone()


# (workload, placement, p, ranks, row capacity): the last case's capacity is
# the rank's own row count, below the fused kernel's 8192, so the two-kernel
# path runs the plan.
@pytest.mark.parametrize("name,kind,p,ranks,own_cap", [("c2", "coact", 0.3, (0, 7), False),
                                                       ("c4", "coact", 0.1, (0, 7), False),
                                                       ("c5", "coact", 0.1, (0,), False),
                                                       ("c3", "coact", 0.1, (0,), True)])
def test_ffn_combine_equals_separate_path(name, kind, p, ranks, own_cap):
    cfg = gen.CONFIGS[name]
    er, el = C.placement(name, kind, p, 5.0)
    _, lay = C.oracle_routing(name, kind, p, 5.0)
    kw = {}
    if own_cap:
        eo = lay["expert_offsets"]
        kw["row_cap"] = int(eo[cfg.E_loc] - eo[0])
        assert kw["row_cap"] < 8192
    L = _layer(name, kind, p, x=gen.activations(cfg), **kw)
    L.front()
    for rank in ranks:
        L.set_rank_weights(rank, *C.rank_weights(cfg, er, el, rank))
        r0 = int(lay["recv_offsets"][rank])
        U = int(lay["recv_offsets"][rank + 1]) - r0
        for parts_rows in (L.recv_cap, r0 + U // 2):
            pa, ya, pb, yb = _separate_and_fused(L, rank, parts_rows)
            assert torch.equal(pa.view(torch.int16), pb.view(torch.int16)), (rank, parts_rows)
            dst = L.row_dst.cpu().numpy()
            n = min(L.rank_rows(rank), L.row_cap)
            multi = np.nonzero(dst[:n] < 0)[0]
            idx = torch.from_numpy(multi).to(L.Y.device)
            assert torch.equal(ya[idx].view(torch.int16), yb[idx].view(torch.int16)), (rank, parts_rows)
            print(f"[{name} rank {rank} parts_rows {parts_rows}] rows {n}, rows through Y {len(multi)}", flush=True)
        assert L.ffn_wait_errors() == 0
        del L.weights[rank]


def test_idle_rank_combine_calls_are_empty():
    """A rank whose experts are never selected: its row plan, combining FFN
    and multi-term destination reduce write nothing."""
    name, p = "c2", 0.3
    cfg = gen.CONFIGS[name]
    er, el = gen.sequential_placement(cfg)
    logits = C.logits(name).copy()
    idle = cfg.R - 1
    logits[:, er == idle] -= 60.0                     # never in any token's top k
    L = DeviceLayer(cfg, logits, gen.activations(cfg), er, el, p, 5.0)
    L.set_rank_weights(idle, *C.rank_weights(cfg, er, el, idle))
    L.front()
    torch.cuda.synchronize()
    assert L.rank_rows(idle) == 0
    L.parts.view(torch.int16).fill_(0x1234)
    L.Y.view(torch.int16).fill_(0x1234)
    L.row_dst.fill_(-5)
    L.row_plan(idle)
    L.ffn_combine(idle)
    L.dest_reduce_multi(idle)
    torch.cuda.synchronize()
    assert bool((L.parts.view(torch.int16) == 0x1234).all())
    assert bool((L.Y.view(torch.int16) == 0x1234).all())
    assert bool((L.row_dst == -5).all())
    assert L.ffn_wait_errors() == 0


def test_c5_step_receive_rows_against_oracle():
    """The DeepSeek-V3-shaped step (folded combine) against the fp64 oracle on
    sampled received tokens of rank 0: 200 whose only kept expert on the rank
    makes the FFN's epilogue write their row, and 200 with several, which the
    multi-term reduce sums (Eq. 1 over the kept experts on the rank, Sec. II-C)."""
    name, kind, p = "c5", "coact", 0.1
    cfg = gen.CONFIGS[name]
    er, el = C.placement(name, kind, p, 5.0)
    r, lay = C.oracle_routing(name, kind, p, 5.0)
    x = gen.activations(cfg)
    L = _layer(name, kind, p, x=x)
    L.set_rank_weights(0, *C.rank_weights(cfg, er, el, 0))
    L.set_shared_weights(*gen.shared_weights(cfg))
    L.parts.zero_()
    L.step(0)
    torch.cuda.synchronize()
    assert L.ffn_wait_errors() == 0
    eo = lay["expert_offsets"].astype(np.int64)
    base, rows_r = int(eo[0]), int(eo[cfg.E_loc] - eo[0])
    U0 = int(lay["recv_offsets"][1])
    sp = lay["slot_pos"].astype(np.int64) - base
    toks = lay["recv_token"][:U0].astype(np.int64)
    mine = (sp[toks] >= 0) & (sp[toks] < rows_r)              # [U0][k]
    n = mine.sum(axis=1)
    rng = np.random.default_rng(5)
    single = rng.choice(np.flatnonzero(n == 1), 200, replace=False)
    multi = rng.choice(np.flatnonzero(n >= 2), 200, replace=False)
    us = np.concatenate([single, multi])
    row_tok = {}
    for u in us:
        for s in range(cfg.k):
            if mine[u, s]:
                row_tok[int(sp[toks[u], s])] = int(toks[u])
    rows = np.array(sorted(row_tok), np.int64)
    Y = dict(zip(rows.tolist(), _oracle_rows(cfg, er, el, lay, x, rows, [row_tok[i] for i in rows.tolist()])))
    ref = np.zeros((len(us), cfg.d), np.float64)
    for i, u in enumerate(us):
        t = toks[u]
        for s in range(cfg.k):
            if mine[u, s]:
                ref[i] += float(r["wp"][t, s]) * Y[int(sp[t, s])]
    got = L.parts[torch.from_numpy(us).to(L.parts.device)].float().cpu().numpy()
    print(f"[c5 step] received {U0}, sampled {len(us)} tokens over {len(rows)} expert rows", flush=True)
    ok, worst = C.within_tol(got, ref)
    assert ok, worst
    assert C.rel_fro(got, ref) <= 1e-2


def _oracle_rows(cfg, er, el, lay, x, rows, tokens):
    """fp64 oracle SwiGLU of the given rows of rank 0's expert-sorted buffer
    (row i holds x of token tokens[i], the expert gather's definition)."""
    import oracle
    eo = lay["expert_offsets"][: cfg.E_loc + 1].astype(np.int64)
    xs32 = gen.bf16_bits_to_f32(x[np.asarray(tokens, np.int64)])
    ids = C.local_experts(er, el, 0, cfg.E_loc)
    out = np.zeros((len(rows), cfg.d), np.float64)
    for l in range(cfg.E_loc):
        a, b = eo[l] - eo[0], eo[l + 1] - eo[0]
        sel = np.flatnonzero((rows >= a) & (rows < b))
        if len(sel):
            W1, W3, W2 = gen.expert_weights_f32(cfg, ids[l])
            out[sel] = oracle.swiglu_rows(xs32[sel], W1, W3, W2)
    return out
