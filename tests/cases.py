"""Parity cases: a workload config, a placement, p and c, with the oracle's
results.  Every oracle input comes from the seeded generator or from the
oracle itself (the co-activation placement is built by the oracle pipeline:
pruned trace under sequential placement -> co-activation counts -> Algorithm 1
+ node stage)."""
from __future__ import annotations

import dataclasses
import functools

import numpy as np

import oracle
from oracle import placement as oplace
from workloads import generator as gen


@dataclasses.dataclass
class Case:
    name: str
    cfg: gen.Config
    placement: str   # "seq" or "coact"
    p: float
    c: float = 5.0

    @property
    def id(self) -> str:
        return f"{self.name}-{self.placement}-p{self.p}-c{self.c:g}"


# Routing / layout / co-activation cases over the five workloads (sizes as stated).
ROUTE_CASES = [
    Case("c1", gen.CONFIGS["c1"], "seq", 0.3), Case("c1", gen.CONFIGS["c1"], "seq", 0.0),
    Case("c2", gen.CONFIGS["c2"], "seq", 0.0), Case("c2", gen.CONFIGS["c2"], "seq", 0.3),
    Case("c2", gen.CONFIGS["c2"], "coact", 0.0), Case("c2", gen.CONFIGS["c2"], "coact", 0.3),
    Case("c3", gen.CONFIGS["c3"], "seq", 0.0), Case("c3", gen.CONFIGS["c3"], "seq", 0.05),
    Case("c3", gen.CONFIGS["c3"], "seq", 0.1), Case("c3", gen.CONFIGS["c3"], "seq", 0.2),
    Case("c3", gen.CONFIGS["c3"], "seq", 0.2, 1.0), Case("c3", gen.CONFIGS["c3"], "coact", 0.1),
    Case("c4", gen.CONFIGS["c4"], "seq", 0.0), Case("c4", gen.CONFIGS["c4"], "seq", 0.1),
    Case("c4", gen.CONFIGS["c4"], "coact", 0.1),
    Case("c5", gen.CONFIGS["c5"], "coact", 0.1), Case("c5", gen.CONFIGS["c5"], "seq", 0.1),
]


@functools.lru_cache(maxsize=None)
def logits(name: str) -> np.ndarray:
    return gen.logits(gen.CONFIGS[name])


@functools.lru_cache(maxsize=None)
def placement(name: str, kind: str, p: float, c: float):
    cfg = gen.CONFIGS[name]
    er0, el0 = gen.sequential_placement(cfg)
    if kind == "seq":
        return er0, el0
    tr = oracle.route_prune(gen.trace_logits(cfg), cfg.k, er0, cfg.ranks_per_node,
                            cfg.trace_tokens // cfg.R, c, p)
    C = oracle.coactivation(tr["idx"], tr["keep"], cfg.E)
    er, el = oplace.coactivation_placement(C, cfg.R, cfg.ranks_per_node,
                                           gen.random_order(cfg.E, 0, 0).tolist(),
                                           gen.random_order(cfg.R, 0, 1).tolist())
    return np.array(er, np.int32), np.array(el, np.int32)


@functools.lru_cache(maxsize=None)
def oracle_routing(name: str, kind: str, p: float, c: float):
    cfg = gen.CONFIGS[name]
    er, el = placement(name, kind, p, c)
    r = oracle.route_prune(logits(name), cfg.k, er, cfg.ranks_per_node, cfg.tokens_per_rank, c, p)
    lay = oracle.dispatch_layout(r["idx"], r["keep"], r["mask"], er, el, cfg.R, cfg.ranks_per_node,
                                 cfg.tokens_per_rank, cfg.E)
    return r, lay


def local_experts(er, el, rank, E_loc):
    """Expert ids of `rank` in local-slot order."""
    out = [-1] * E_loc
    for e in range(len(er)):
        if er[e] == rank:
            out[el[e]] = e
    return out


def rank_weights(cfg, er, el, rank):
    """(W1, W3, W2) stacked in local-slot order, storage type."""
    ids = local_experts(er, el, rank, cfg.E_loc)
    ws = [gen.expert_weights(cfg, e) for e in ids]
    return tuple(np.stack([w[i] for w in ws]) for i in range(3))


def within_tol(got, ref, atol=1e-3, rtol=2e-2):
    """Element-wise |got - ref| <= atol + rtol*|ref|; returns (ok, worst ratio)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    bound = atol + rtol * np.abs(ref)
    ratio = np.abs(got - ref) / bound
    return bool(np.all(ratio <= 1.0)), float(ratio.max() if ratio.size else 0.0)


def rel_fro(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    n = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / n) if n > 0 else float(np.linalg.norm(got))
