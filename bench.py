#!/usr/bin/env python3
"""Benchmark of the CAP expert-parallel MoE layer hot path on one MI355X.

One step = the whole hot path over one batch of synthetic input, inputs
resident in HBM (DeviceLayer.step):
  route + prune (all T tokens of all virtual ranks), dispatch layout,
  co-activation counts, rank 0's row source (the expert gather as indices),
  rank 0's grouped SwiGLU FFN reading x rows in place, destination reduce for
  rank 0, [shared experts, on a side stream], source reduce for rank 0.
The step is captured once as a HIP graph and replayed; --warmup untimed steps
(eager and replayed) let the GPU clock settle before --steps timed ones.
`value` = rank 0's tokens carried through the layer per second
(tokens_per_rank / step time; the step also routes every other virtual rank's
tokens, which a real rank would not do).

The rows every other rank returns to rank 0 are stand-in values in HBM (on a
real system they arrive by all-to-all); rank 0's own rows are recomputed every
step.  The dominant kernel is the grouped FFN (one fused launch for both GEMMs
on the bench workloads), timed live with HIP events on the stream it runs on.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "routed tokens/s per MoE layer (1 GPU) + %HBM/%MFMA peak; send bytes/token"
PEAK_BF16_TFLOPS = 2500.0          # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0              # MI355X HBM3E
PROFILES = os.path.join(ROOT, "profiles")
FFN_SOURCE = os.path.join(ROOT, "paper_2607_05116_amd", "csrc", "expert_ffn.hip")


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100,
                    help="untimed steps before each timed loop (eager and graph): the GPU clock "
                         "rises over the first ~20 ms of sustained work")
    ap.add_argument("--config", default="c5",
                    help="workload: c1..c5 (default c5, the DeepSeek-V3-shaped layer, the largest)")
    ap.add_argument("--placement", default="coact", choices=["coact", "seq"])
    ap.add_argument("--p", type=float, default=None,
                    help="pruning threshold (default: the workload's; the paper uses 0.3 for Qwen3 "
                         "and 0.1 for DeepSeek-V2-Lite)")
    ap.add_argument("--c", type=float, default=5.0, help="inter-node cost")
    ap.add_argument("--rank", type=int, default=0)
    ap.add_argument("--eager", action="store_true",
                    help="time eager launches (default: the step captured once as a HIP graph, replayed)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--cpu-stride", type=int, default=4, help="oracle FFN runs every n-th rank-0 row")
    ap.add_argument("--separate-combine", action="store_true",
                    help="run the destination combine as its own kernel after the FFN (for comparison; default: "
                         "single-expert tokens combined in the FFN's epilogue)")
    ap.add_argument("--quick", action="store_true",
                    help="only the timed step and its FFN timing (no stage times, cold-cache replays, "
                         "sweeps, spectrum, second workload): for profiler runs")
    ap.add_argument("--aux-config", default="c2",
                    help="second workload measured briefly into aux (graph-replayed step and FFN); "
                         "'none' to skip")
    ap.add_argument("--vendor", action="store_true",
                    help="also time the vendor library (torch.matmul, hipBLASLt) on the same rank's grouped "
                         "SwiGLU FFN, one GEMM pair per expert, into aux.vendor_grouped_ffn (for comparison)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run 3 device-to-device copies of MIB MiB (HBM counter calibration) and exit")
    return ap.parse_args()


def calibrate_copy(mib: int):
    """A plain copy of known size: reads and writes mib MiB per launch, so HBM
    byte counters of other kernels can be scaled against it."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes": n * 4, "launches": 3}), flush=True)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def rank_weights(gen, cfg, er, el, rank):
    import numpy as np
    ids = [-1] * cfg.E_loc
    for e in range(cfg.E):
        if er[e] == rank:
            ids[el[e]] = e
    ws = [gen.expert_weights(cfg, e) for e in ids]
    return tuple(np.stack([w[i] for w in ws]) for i in range(3))


def product_placement(cfg, p, c):
    """CAP offline steps 1-2 on the GPU path: pruned routing trace under
    sequential placement -> co-activation counts -> Algorithm 1 + node stage."""
    import dataclasses
    import numpy as np
    from paper_2607_05116_amd import placement
    from paper_2607_05116_amd.layer import DeviceLayer
    from workloads import generator as gen
    er0, el0 = gen.sequential_placement(cfg)
    tcfg = dataclasses.replace(cfg, T=cfg.trace_tokens, d=8)
    trace = gen.trace_logits(cfg)
    Lt = DeviceLayer(tcfg, trace, np.zeros((tcfg.T, 8), np.uint16), er0, el0, p, c, row_cap=8, recv_cap=8)
    Lt.route()
    Lt.coactivation()
    C = Lt.host("coact").view(np.uint32)
    er, el = placement.coactivation_placement(C, cfg.R, cfg.ranks_per_node, gen.random_order(cfg.E, 0, 0),
                                              gen.random_order(cfg.R, 0, 1))
    return er, el, C


def placement_spectrum(cfg, p, c):
    """CAP offline step 3 (Sec. V) on this workload: the Adjustment Approach's
    swap sequence computed on the GPU (cap_adjustment_spectrum) from the
    co-activation placement of the pruned trace, timed; then 7 points of the
    spectrum and the sequential placement, each re-routed and re-laid-out on
    the GPU over the evaluated batch (devices per token, load imbalance of kept
    rows, send volume) with C(pi) on the trace's p_ij.  Untimed otherwise."""
    import dataclasses
    import numpy as np
    import torch
    from paper_2607_05116_amd import placement
    from paper_2607_05116_amd.layer import DeviceLayer
    from workloads import generator as gen
    er0, el0 = gen.sequential_placement(cfg)
    tcfg = dataclasses.replace(cfg, T=cfg.trace_tokens, d=8)
    Lt = DeviceLayer(tcfg, gen.trace_logits(cfg), np.zeros((tcfg.T, 8), np.uint16), er0, el0, p, c,
                     row_cap=8, recv_cap=8)
    Lt.route()
    Lt.coactivation()
    torch.cuda.synchronize()
    C = Lt.host("coact").view(np.uint32)
    er, el = placement.coactivation_placement(C, cfg.R, cfg.ranks_per_node, gen.random_order(cfg.E, 0, 0),
                                              gen.random_order(cfg.R, 0, 1))
    placement.adjustment_spectrum_gpu(Lt.coact, er, el, cfg.R, cfg.ranks_per_node, c)      # warm
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    spec, deltas = placement.adjustment_spectrum_gpu(Lt.coact, er, el, cfg.R, cfg.ranks_per_node, c)
    build_s = time.perf_counter() - t0
    P = placement.coactivation_probability(C)
    ecfg = dataclasses.replace(cfg, d=8)
    Le = DeviceLayer(ecfg, gen.logits(cfg), np.zeros((cfg.T, 8), np.uint16), er, el, p, c, row_cap=8, recv_cap=8)

    def evaluate(ranks, local):
        Le.set_placement(ranks, local)
        Le.route()
        Le.layout()
        torch.cuda.synchronize()
        tot = Le.host("totals").astype(np.int64)
        rows = np.diff(Le.host("expert_offsets")[:: cfg.E_loc]).astype(np.float64)
        return {"comm_objective": float(placement.comm_objective(P, np.asarray(ranks), cfg.ranks_per_node, c)),
                "device_per_token": int(tot[0]) / cfg.T,
                "load_imbalance": float(rows.max() / rows.mean()),
                "send_bytes_per_token": int(tot[1] + tot[2]) * cfg.d * cfg.elem_bytes / cfg.T}
    points = []
    for i in placement.spectrum_points(len(spec)):
        pt = evaluate(spec[i][0], spec[i][1])
        pt["swaps"] = i
        points.append(pt)
    seq = evaluate(er0, el0)
    return {"zipf_s": cfg.zipf_s, "total_swaps": len(spec) - 1, "gpu_build_s": build_s,
            "objective_increase_total": float(np.sum(deltas)), "points": points, "sequential": seq}


def fused_front_end(L, cfg, stream, reps=20):
    """The router GEMM x W_g^T fused with routing and pruning
    (cap_router_route_prune), timed against the logits-in route kernel
    (untimed by the step; seeded router weights, so its routing differs from
    the step's).  Leaves the layer's routing state as the step left it."""
    import torch
    from paper_2607_05116_amd.layer import to_device_rows
    from workloads import generator as gen
    if cfg.dtype != "bf16":
        return None
    wg = to_device_rows(gen.router_weights(cfg), "bf16", L.dev)

    def timed(fn):
        for _ in range(3):
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    fused_ms = timed(lambda: L.router_route(wg))
    route_ms = timed(L.route)
    L.layout()
    torch.cuda.synchronize()
    x_bytes = cfg.T * cfg.d * 2 + cfg.E * cfg.d * 2 + cfg.T * cfg.k * 9 + cfg.T * 8
    return {"router_route_ms": fused_ms, "route_from_logits_ms": route_ms,
            "router_flops": 2.0 * cfg.T * cfg.d * cfg.E,
            "router_route_hbm_GBs": x_bytes / (fused_ms * 1e-3) / 1e9,
            "logits_bytes_not_written": cfg.T * cfg.E * 4}


def file_hash(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def traffic_from_profile(workload_key: str):
    """HBM bytes per FFN call from a committed rocprofv3 counter summary, if it
    was taken on the current FFN source (else None)."""
    path = os.path.join(PROFILES, f"expert_ffn_{workload_key}_hbm_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256_16") != file_hash(FFN_SOURCE):
        return None
    return rec.get("bytes_per_call")


def cpu_baseline(cfg, p, c, logits, x, stride):
    """The oracle as it stands, timed on this host on a bounded sample."""
    import numpy as np
    import oracle
    from oracle import placement as oplace
    from workloads import generator as gen
    # the FFN's OpenMP threads: the host's CPUs, capped at the 16 a GPU job
    # gets on the box (cores = the threads it actually used)
    threads = min(16, os.cpu_count() or 1)
    er0, _ = gen.sequential_placement(cfg)
    tr = oracle.route_prune(gen.trace_logits(cfg), cfg.k, er0, cfg.ranks_per_node,
                            cfg.trace_tokens // cfg.R, c, p)
    C = oracle.coactivation(tr["idx"], tr["keep"], cfg.E)
    er, el = oplace.coactivation_placement(C, cfg.R, cfg.ranks_per_node, gen.random_order(cfg.E, 0, 0).tolist(),
                                           gen.random_order(cfg.R, 0, 1).tolist())
    er, el = np.array(er, np.int32), np.array(el, np.int32)
    t0 = time.perf_counter()
    r = oracle.route_prune(logits, cfg.k, er, cfg.ranks_per_node, cfg.tokens_per_rank, c, p)
    lay = oracle.dispatch_layout(r["idx"], r["keep"], r["mask"], er, el, cfg.R, cfg.ranks_per_node,
                                 cfg.tokens_per_rank, cfg.E)
    oracle.coactivation(r["idx"], r["keep"], cfg.E)
    t_front = time.perf_counter() - t0
    t0 = time.perf_counter()
    xs = oracle.expert_gather(x, r["idx"], r["keep"], lay["slot_pos"], lay["expert_offsets"], er, cfg.R, 0)
    t_gather = time.perf_counter() - t0
    xs32 = gen.bf16_bits_to_f32(xs) if cfg.dtype == "bf16" else xs
    eo = lay["expert_offsets"]
    rows0 = int(eo[cfg.E_loc] - eo[0])
    ids = [-1] * cfg.E_loc
    for e in range(cfg.E):
        if er[e] == 0:
            ids[el[e]] = e
    t_ffn, n_sample = 0.0, 0
    for l in range(cfg.E_loc):
        a, b = int(eo[l] - eo[0]), int(eo[l + 1] - eo[0])
        rows = np.arange(a, b)[::stride]
        if len(rows) == 0:
            continue
        W = gen.expert_weights_f32(cfg, ids[l])
        t0 = time.perf_counter()
        oracle.swiglu_rows(xs32[rows], *W, nthreads=threads)
        t_ffn += time.perf_counter() - t0
        n_sample += len(rows)
    t_ffn_full = t_ffn * rows0 / max(1, n_sample)
    Y = np.zeros((rows0, cfg.d), np.float32)
    t0 = time.perf_counter()
    oracle.dest_reduce(Y, r, lay, er, cfg.R, 0, cfg.d)
    t_dest = time.perf_counter() - t0
    parts = np.zeros((int(lay["recv_offsets"][-1]), cfg.d), np.float32)
    t0 = time.perf_counter()
    oracle.src_reduce(parts, r, lay, er, cfg.R, cfg.tokens_per_rank, 0, cfg.d)
    t_src = time.perf_counter() - t0
    total = t_front + t_gather + t_ffn_full + t_dest + t_src
    return {
        "value": cfg.tokens_per_rank / total,
        "unit": "tokens/s",
        "cores": threads,
        "threads_by_stage": {"routing_layout_coactivation": 1, "gather": 1, "ffn": threads, "combine": 1},
        "host_logical_cpus": os.cpu_count(),
        "kind": "oracle",
        "sample": (f"full routing/layout/co-activation of all {cfg.T} tokens ({t_front:.2f} s, 1 thread), "
                   f"rank-0 gather ({t_gather:.2f} s), fp64 SwiGLU on every {stride}th of {rows0} rank-0 rows "
                   f"({n_sample} rows, {t_ffn:.2f} s on {threads} threads, scaled x{rows0 / max(1, n_sample):.2f}), "
                   f"destination + source reduce of rank 0 ({t_dest + t_src:.2f} s, 1 thread); "
                   f"host: {cpu_model()}"),
    }


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# Pruning threshold of each workload when --p is not given: the paper's 0.3
# for the Qwen3-shaped layers and 0.1 for the DeepSeek-shaped ones
# (Sec. VIII-A); the 16-rank layer is swept, 0.1 is its middle point.
DEFAULT_P = {"c1": 0.3, "c1u": 0.3, "c2": 0.3, "c3": 0.1, "c4": 0.1, "c5": 0.1}


def build_layer(cfg, placement_kind, p, c, rank):
    """Inputs, placement, weights and buffers of one workload, resident in HBM;
    the front end has run once and the rows other ranks return are seeded
    stand-in values."""
    import numpy as np
    import torch
    from paper_2607_05116_amd.layer import DeviceLayer
    from workloads import generator as gen
    t_setup = time.perf_counter()
    logits = gen.logits(cfg)
    x = gen.activations(cfg)
    coact_counts = None
    if placement_kind == "coact":
        er, el, coact_counts = product_placement(cfg, p, c)
    else:
        er, el = gen.sequential_placement(cfg)
    L = DeviceLayer(cfg, logits, x, er, el, p, c)
    L.set_rank_weights(rank, *rank_weights(gen, cfg, er, el, rank))
    if cfg.n_shared:
        L.set_shared_weights(*gen.shared_weights(cfg))
    L.front()
    torch.cuda.synchronize()
    n_recv = int(L.host("recv_offsets")[-1])
    g = torch.Generator(device="cuda").manual_seed(1234)
    L.parts[:n_recv] = (torch.randn((n_recv, cfg.d), generator=g, device="cuda") * 0.05).to(L.tdt)
    log(f"{cfg.name}: setup {time.perf_counter() - t_setup:.1f} s; rank-{rank} rows {L.rank_rows(rank)}, "
        f"received rows {n_recv}")
    return L, logits, x, er, el, coact_counts


def check_ffn_waits(L):
    """The fused FFN's bounded cross-workgroup waits never gave up (the
    counter the layer passes to every FFN call)."""
    n = L.ffn_wait_errors()
    if n:
        raise RuntimeError(f"fused FFN: {n} cross-workgroup waits gave up (results of those calls are invalid)")
    return n


def time_graph(graph, stream, steps, warmup):
    import torch
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    g0.record(stream)
    for _ in range(steps):
        graph.replay()
    g1.record(stream)
    torch.cuda.synchronize()
    return g0.elapsed_time(g1) / steps, time.perf_counter() - wall0


def aux_workload(name, rank, steps, warmup, c):
    """A second workload measured briefly: its graph-replayed step and the
    FFN call inside it (HIP events on the FFN's stream)."""
    import torch
    from workloads import generator as gen
    cfg = gen.CONFIGS[name]
    p = DEFAULT_P[name]
    L, *_ = build_layer(cfg, "coact", p, c, rank)
    stream = torch.cuda.current_stream()
    side = torch.cuda.Stream() if cfg.n_shared else None
    graph = L.capture_step(rank, side=side)
    for _ in range(warmup):
        L.step(rank, side=side)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for i in range(steps):
        L.step(rank, side=side, ffn_events=ev[i])
    torch.cuda.synchronize()
    ffn_ms = sum(a.elapsed_time(b) for a, b in ev) / steps
    ms, _ = time_graph(graph, stream, steps, warmup)
    check_ffn_waits(L)
    rows = L.rank_rows(rank)
    flops = 6.0 * cfg.d * cfg.inter * rows
    out = {"workload": f"{name}: T={cfg.T}, d={cfg.d}, E={cfg.E} top-{cfg.k}, inter={cfg.inter}, R={cfg.R}, "
                       f"coact placement, p={p:g}, rank {rank}",
           "ms_per_step": ms, "tokens_per_s": cfg.tokens_per_rank / (ms * 1e-3),
           "ffn_ms": ffn_ms, "ffn_rows": rows, "ffn_tflops": flops / (ffn_ms * 1e-3) / 1e12,
           "ffn_frac_bf16_peak": flops / (ffn_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}
    del graph, L
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures the hot path on one GPU (virtual expert-parallel ranks); "
              f"--gpus {args.gpus} / WORLD_SIZE={world} is not supported", file=sys.stderr)
        sys.exit(2)

    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return

    import numpy as np
    import torch

    from workloads import generator as gen

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    cfg = gen.CONFIGS[args.config]
    if args.p is None:
        args.p = DEFAULT_P[args.config]
    rank = args.rank
    L, logits, x, er, el, coact_counts = build_layer(cfg, args.placement, args.p, args.c, rank)
    if args.separate_combine:
        L.fused_combine = False

    stream = torch.cuda.current_stream()
    # a side stream for the shared experts and the co-activation counts when
    # there are shared experts; without them the co-activation counts run in
    # line (in a replayed graph each dependency between streams costs ~10 us)
    side = torch.cuda.Stream() if cfg.n_shared else None

    def one_step(ev=None):
        """The whole hot path once: front end over all tokens, then rank r's
        row plan, gathered FFN (which writes single-expert tokens' weighted
        rows into the receive buffer), destination reduce of the other tokens
        and source reduce, with the shared experts on the side stream."""
        L.step(rank, side=side, ffn_events=ev)

    # the graph is captured first, so that the eager loop, the graph warmup
    # and the timed replays follow each other without an idle gap
    graph = None if args.eager else L.capture_step(rank, side=side)
    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()

    K = args.steps
    ffn_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for i in range(K):
        one_step(ffn_ev[i])
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_per_step = t_start.elapsed_time(t_end) / K
    ffn_ms = sum(a.elapsed_time(b) for a, b in ffn_ev) / K
    log(f"timed {K} steps: {ms_per_step:.4f} ms/step (host wall {1e3 * wall / K:.4f} ms/step), FFN {ffn_ms:.4f} ms")
    eager_ms_per_step = ms_per_step
    graph_ms_per_step = cold_ms_per_step = cold_dirty_ms_per_step = composite = None
    if graph is not None:
        # the same step captured once as a HIP graph and replayed K times
        graph_ms_per_step, wall = time_graph(graph, stream, K, args.warmup)
        ms_per_step = graph_ms_per_step
        log(f"graph replays: {graph_ms_per_step:.4f} ms/step (host wall {1e3 * wall / K:.4f} ms/step)")
    check_ffn_waits(L)
    if graph is not None and not args.quick:
        # the same replays with the caches cold: 512 MB (twice the 256 MB
        # Infinity Cache) read before each, outside its timed window, which
        # leaves the caches full of clean lines of other data; and the same
        # after 512 MB are rewritten, whose dirty lines the step also writes back
        flush = torch.zeros(512 << 20, dtype=torch.uint8, device="cuda")

        def cold_replays(evict):
            times = []
            for _ in range(min(K, 10)):
                evict()
                c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                c0.record(stream)
                graph.replay()
                c1.record(stream)
                torch.cuda.synchronize()
                times.append(c0.elapsed_time(c1))
            return float(np.median(times))

        cold_ms_per_step = cold_replays(lambda: flush.sum(dtype=torch.int64))
        cold_dirty_ms_per_step = cold_replays(lambda: flush.add_(1))
        del flush
        log(f"cold-cache replays: {cold_ms_per_step:.4f} ms/step after a 512 MB read, "
            f"{cold_dirty_ms_per_step:.4f} after a 512 MB rewrite (medians of {min(K, 10)})")
        # the front end alone (route, layout, co-activation of all T tokens),
        # for the composite rank-0 rate that charges rank 0 its 1/R share of it
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        with torch.cuda.stream(cap):
            L.front(side=side)
        stream.wait_stream(cap)
        fg = torch.cuda.CUDAGraph()
        with torch.cuda.graph(fg):
            L.front(side=side)
        front_ms, _ = time_graph(fg, stream, K, args.warmup)
        composite = {
            "front_graph_ms": front_ms,
            "rank0_step_ms": graph_ms_per_step - front_ms * (1.0 - 1.0 / cfg.R),
            "tokens_per_s": cfg.tokens_per_rank / ((graph_ms_per_step - front_ms * (1.0 - 1.0 / cfg.R)) * 1e-3),
            "definition": "tokens_per_rank / (step - (1 - 1/R) * front end): rank 0's own share of routing, "
                          "layout and co-activation plus its whole rank path",
        }
        log(f"front end alone: {front_ms:.4f} ms; composite rank-0 rate {composite['tokens_per_s'] / 1e6:.2f} M tokens/s")

    rows = L.rank_rows(rank)
    flops = 6.0 * cfg.d * cfg.inter * rows
    achieved = flops / (ffn_ms * 1e-3) / 1e12
    workload_key = f"{cfg.name}_{args.placement}_p{args.p:g}"
    traffic = traffic_from_profile(workload_key)
    totals = L.host("totals").astype(np.int64)
    eb = cfg.elem_bytes
    send_copies = int(totals[1] + totals[2])
    loads = np.diff(L.host("expert_offsets")[:: cfg.E_loc]).astype(np.float64)
    result = {
        "metric": METRIC,
        "value": cfg.tokens_per_rank / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded latent-topic router logits, N(0,1) activations, scaled random-init weights)",
        "config": {
            "workload": (f"{cfg.name}: MoE layer T={cfg.T} tokens ({cfg.R} virtual ranks x {cfg.tokens_per_rank}), "
                         f"d={cfg.d}, E={cfg.E} top-{cfg.k}, SwiGLU inter={cfg.inter}"
                         + (f" + {cfg.n_shared} shared x {cfg.shared_inter}" if cfg.n_shared else "")
                         + f", {args.placement} placement, p={args.p:g}, c={args.c:g}, FFN/combine on rank {rank}"),
            "name": cfg.name,
            "T": cfg.T, "tokens_per_rank": cfg.tokens_per_rank, "d": cfg.d, "E": cfg.E, "k": cfg.k,
            "inter": cfg.inter, "R": cfg.R, "ranks_per_node": cfg.ranks_per_node,
            "n_shared": cfg.n_shared, "shared_inter": cfg.shared_inter,
            "placement": args.placement, "p": args.p, "c": args.c, "rank": rank,
            "parallelism": "1 GPU, virtual EP ranks",
        },
        "roofline": {
            "kernel": (("cap_expert_ffn_combine" if L.fused_combine else "cap_expert_ffn_gather")
                       + ", rank 0: one fused gate/up + down launch reading x rows in place"
                       + (" and writing single-expert tokens' weighted rows into the receive buffer"
                          if L.fused_combine else "")
                       + " (the call's events also hold its one-block counter clear, a few us)"),
            "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic,
            "flops_per_call": flops, "rows": rows, "avg_call_ms": ffn_ms,
        },
        "aux": {
            "send_bytes_per_token": send_copies * cfg.d * eb / cfg.T,
            "send_bytes_per_token_intra": int(totals[1]) * cfg.d * eb / cfg.T,
            "send_bytes_per_token_inter": int(totals[2]) * cfg.d * eb / cfg.T,
            "device_per_token": int(totals[0]) / cfg.T,
            "node_per_token": int(totals[3]) / cfg.T,
            "load_imbalance_max_over_mean": float(loads.max() / loads.mean()),
            "rank_rows": rows,
            "host_wall_ms_per_step": 1e3 * wall / K,
            "eager_ms_per_step": eager_ms_per_step, "graph_ms_per_step": graph_ms_per_step,
            "cold_cache_ms_per_step": cold_ms_per_step,
            "cold_cache_dirty_ms_per_step": cold_dirty_ms_per_step,
            "composite_rank0": composite,
            "ffn_wait_errors": 0,
        },
    }
    if not args.quick:
        result["aux"].update(detail_measurements(args, L, cfg, rank, stream, totals))
    if args.vendor:
        log("vendor library on the same grouped FFN ...")
        result["aux"]["vendor_grouped_ffn"] = vendor_grouped_ffn(L, cfg, rank, flops)
    if not args.no_cpu:
        log("timing the CPU oracle on a bounded sample ...")
        result["cpu_baseline"] = cpu_baseline(cfg, args.p, args.c, logits, x, args.cpu_stride)
    if not args.quick and args.aux_config not in ("none", "", args.config):
        del graph, L
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        log(f"second workload {args.aux_config} ...")
        result["aux"]["second_workload"] = aux_workload(args.aux_config, rank, K, args.warmup, args.c)
    print(json.dumps(result), flush=True)


def vendor_grouped_ffn(L, cfg, rank, flops, reps=20, warmup=30):
    """The vendor library on the rank's FFN: for each local expert, torch.matmul
    (hipBLASLt) of its gathered rows with [W1; W3] (one GEMM), SiLU(gate) * up,
    and the down GEMM with W2, on the same rows and weights as the fused call;
    timed with HIP events after a warmup long enough for the clock to settle.
    For comparison only: the product path never calls it."""
    import torch
    E_loc = cfg.E_loc
    eo = L.host("expert_offsets")[rank * E_loc:(rank + 1) * E_loc + 1].astype("int64")
    rows = int(eo[-1] - eo[0])
    L.row_source(rank)
    xs = L.x.index_select(0, L.row_src[:rows].long())
    w1, w3, w2 = L.weights[rank]
    w13 = [torch.cat([w1[l], w3[l]], 0).contiguous() for l in range(E_loc)]
    w2c = [w2[l].contiguous() for l in range(E_loc)]
    inter = cfg.inter
    spans = [(int(eo[l] - eo[0]), int(eo[l + 1] - eo[0])) for l in range(E_loc)]

    def ffn():
        for l, (a, b) in enumerate(spans):
            if b > a:
                h = torch.matmul(xs[a:b], w13[l].t())
                torch.matmul(torch.nn.functional.silu(h[:, :inter]) * h[:, inter:], w2c[l].t())

    def gemms_only():
        for l, (a, b) in enumerate(spans):
            if b > a:
                h = torch.matmul(xs[a:b], w13[l].t())
                torch.matmul(h[:, :inter], w2c[l].t())

    out = {"library": "torch.matmul (hipBLASLt), one [W1; W3] GEMM and one W2 GEMM per expert",
           "experts": E_loc, "rows": rows}
    for fn, key in ((ffn, "swiglu"), (gemms_only, "gemms_only")):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        out[f"{key}_ms"] = ms
        out[f"{key}_tflops"] = flops / (ms * 1e-3) / 1e12
        out[f"{key}_frac_bf16_peak"] = flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS
    del xs, w13, w2c
    torch.cuda.empty_cache()
    return out


def detail_measurements(args, L, cfg, rank, stream, totals):
    """Untimed detail of the headline workload: per-stage device times and
    HBM rates, CAP against expert-level pruning, the pruning sweep, the
    placement spectrum and the fused router front end."""
    import numpy as np
    import torch
    # per-stage device times (separate, untimed): each stage captured as a graph
    # of 20 back-to-back calls (every stage rewrites the same buffers from
    # unchanged inputs) and replayed, so launch gaps do not enter the times
    stages = ["front_fused", "route", "layout", "coact", "row_source", "ffn", "dest", "shared", "src", "gather",
              "ffn_rows", "row_plan", "ffn_combine", "dest_multi"]
    fns = [L.route_layout, L.route, L.layout, L.coactivation, lambda: L.row_source(rank), lambda: L.ffn_gather(rank),
           lambda: L.dest_reduce(rank), lambda: L.shared_ffn(rank), lambda: L.src_reduce(rank),
           lambda: L.gather(rank), lambda: L.ffn(rank), lambda: L.row_plan(rank), lambda: L.ffn_combine(rank),
           lambda: L.dest_reduce_multi(rank)]

    def stage_time(fn, n=20, reps=5):
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        with torch.cuda.stream(cap):
            fn()
        stream.wait_stream(cap)
        sg = torch.cuda.CUDAGraph()
        with torch.cuda.graph(sg):
            for _ in range(n):
                fn()
        sg.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            sg.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / (n * reps)

    stage_ms = {}
    for s_name, fn in zip(stages, fns):
        if (s_name == "shared" and not cfg.n_shared) or (s_name in ("row_plan", "ffn_combine", "dest_multi")
                                                         and not L.fused_combine):
            stage_ms[s_name] = 0.0
            continue
        stage_ms[s_name] = round(stage_time(fn), 5)
    check_ffn_waits(L)

    rows = L.rank_rows(rank)
    eb = cfg.elem_bytes
    # HBM roofline context for the row movers (algorithmic bytes / measured time)
    U = int(L.host("recv_offsets")[rank + 1] - L.host("recv_offsets")[rank])
    mask = L.host("mask").view(np.uint64)[rank * cfg.tokens_per_rank:(rank + 1) * cfg.tokens_per_rank]
    n_dev_src = int(sum(bin(int(m)).count("1") for m in mask))
    kbytes = {
        "route": cfg.T * cfg.E * 4 + cfg.T * cfg.k * 9 + cfg.T * 8,
        "gather": (U + rows) * cfg.d * eb + rows * 4,
        "dest": rows * (cfg.d * eb + 8) + U * cfg.d * eb,
        "src": (n_dev_src + cfg.tokens_per_rank * (2 if cfg.n_shared else 1)) * cfg.d * eb,
    }
    hbm = {s: round(kbytes[s] / (stage_ms[s] * 1e-3) / 1e9, 1) for s in kbytes if stage_ms[s] > 0}

    # CAP's device-level pruning against expert-level threshold pruning at the
    # same p (untimed): kept slots, destinations and send volume per token
    def volume(tot, kept):
        return {"kept_slot_frac": kept / (cfg.T * cfg.k), "device_per_token": int(tot[0]) / cfg.T,
                "node_per_token": int(tot[3]) / cfg.T,
                "send_bytes_per_token": int(tot[1] + tot[2]) * cfg.d * eb / cfg.T,
                "send_bytes_per_token_inter": int(tot[2]) * cfg.d * eb / cfg.T}
    pruning = {"p": args.p, "cap": volume(totals, int(L.host("keep").sum()))}
    L.naive = True
    L.route()
    L.layout()
    torch.cuda.synchronize()
    pruning["naive"] = volume(L.host("totals").astype(np.int64), int(L.host("keep").sum()))
    L.naive = False
    # CAP's volumes over the pruning threshold (untimed), and on multi-node
    # layers the same with c = 1 (the inter-node cost orders remote devices)
    sweep = []
    c_values = [args.c] + ([1.0] if cfg.R > cfg.ranks_per_node and args.c != 1.0 else [])
    for cc in c_values:
        L.topo.inter_node_cost = cc
        for pp in (0.0, 0.05, 0.1, 0.2, 0.3):
            L.p = pp
            L.route()
            L.layout()
            torch.cuda.synchronize()
            tot = L.host("totals").astype(np.int64)
            v = volume(tot, int(L.host("keep").sum()))
            v.update({"p": pp, "c": cc, "intra_copies_per_token": int(tot[1]) / cfg.T,
                      "inter_copies_per_token": int(tot[2]) / cfg.T})
            sweep.append(v)
    L.topo.inter_node_cost = args.c
    L.p = args.p
    L.route()
    L.layout()
    torch.cuda.synchronize()
    # the Adjustment Approach's spectrum on the stated workload and on the same
    # layer with flatter expert popularity (Zipf 0.3)
    import dataclasses
    spectrum = {}
    for label, scfg in (("stated", cfg), ("zipf_0.3", dataclasses.replace(cfg, zipf_s=0.3))):
        t_spec = time.perf_counter()
        spectrum[label] = placement_spectrum(scfg, args.p, args.c)
        log(f"placement spectrum ({label}): {spectrum[label]['total_swaps']} swaps in "
            f"{spectrum[label]['gpu_build_s'] * 1e3:.2f} ms on the GPU; evaluated in {time.perf_counter() - t_spec:.1f} s")

    front_end = fused_front_end(L, cfg, stream)
    return {"stage_ms": stage_ms, "stage_hbm_GBs": hbm, "pruning_cap_vs_naive": pruning,
            "pruning_sweep": sweep, "placement_spectrum": spectrum, "fused_router_front_end": front_end,
            "rank_received_tokens": U}


if __name__ == "__main__":
    main()
