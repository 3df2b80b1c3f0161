"""One expert-parallel MoE layer step on one GPU with virtual ranks.

Owns the device buffers (torch) and chains the C-ABI calls in the order of the
layer (Sec. II-B/II-C; Sec. VI):

  route_prune (all T tokens)  -> dispatch_layout -> coactivation
  expert_gather(rank) -> expert_ffn(rank) -> dest_reduce(rank)
  [shared experts on the source rank's tokens] -> src_reduce(rank)

Every step runs in libcap.so's HIP kernels; this module only allocates and
passes pointers.  All calls are asynchronous on the current stream.
"""
from __future__ import annotations

import numpy as np
import torch

from . import capi

_BF16 = torch.bfloat16


def to_device_rows(a: np.ndarray, dtype: str, device) -> torch.Tensor:
    """numpy rows (uint16 bf16 bits or float32) -> device tensor of that storage type."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(_BF16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


class DeviceLayer:
    """Buffers and calls for one layer configuration.

    cfg: workloads.generator.Config (shapes only).  logits / x are numpy arrays
    (x as uint16 bf16 bits for bf16 configs).  expert_rank / expert_local: int32
    numpy [E].  row_cap: rows allocated per rank for expert rows (None = the
    T*min(k, E_loc) bound).
    """

    def __init__(self, cfg, logits: np.ndarray, x: np.ndarray, expert_rank, expert_local, p: float,
                 c: float = 5.0, device: str = "cuda", row_cap: int | None = None,
                 recv_cap: int | None = None):
        self.cfg = cfg
        self.dev = torch.device(device)
        self.p = float(p)
        self.dt = capi.CAP_DTYPE_BF16 if cfg.dtype == "bf16" else capi.CAP_DTYPE_F32
        self.tdt = _BF16 if cfg.dtype == "bf16" else torch.float32
        T, E, k, R = cfg.T, cfg.E, cfg.k, cfg.R
        d = self.d = cfg.d
        i32 = dict(dtype=torch.int32, device=self.dev)
        self.expert_rank = torch.as_tensor(np.asarray(expert_rank, np.int32)).to(self.dev)
        self.expert_local = torch.as_tensor(np.asarray(expert_local, np.int32)).to(self.dev)
        self.topo = capi.make_topology(E, R, cfg.ranks_per_node, T, k, self.expert_rank,
                                       self.expert_local, c)
        self.logits = torch.from_numpy(np.ascontiguousarray(logits, np.float32)).to(self.dev)
        self.x = to_device_rows(x, cfg.dtype, self.dev)
        # routing
        self.idx = torch.empty((T, k), **i32)
        self.w = torch.empty((T, k), dtype=torch.float32, device=self.dev)
        self.keep = torch.empty((T, k), dtype=torch.uint8, device=self.dev)
        self.mask = torch.empty(T, dtype=torch.int64, device=self.dev)
        # layout
        self.lay_t = dict(
            send_counts=torch.empty((R, R), **i32), send_offsets=torch.empty((R, R), **i32),
            recv_offsets=torch.empty(R + 1, **i32), recv_token=torch.empty(T * k, **i32),
            expert_counts=torch.empty(E, **i32), expert_offsets=torch.empty(E + 1, **i32),
            slot_pos=torch.empty((T, k), **i32), copy_row=torch.empty((T, k), **i32),
            vol=torch.empty((T, 4), dtype=torch.uint8, device=self.dev),
            totals=torch.empty(4, dtype=torch.int64, device=self.dev))
        self.lay = capi.make_layout(self.lay_t)
        self.ws_layout = self._ws(capi.cap_workspace_size(capi.CAP_OP_DISPATCH_LAYOUT, self.topo))
        self.coact = torch.zeros((E, E), dtype=torch.int32, device=self.dev)
        self.ws_coact = self._ws(capi.cap_workspace_size(capi.CAP_OP_COACTIVATION, self.topo))
        self.ws_front = self._ws(capi.cap_workspace_size(capi.CAP_OP_ROUTE_LAYOUT, self.topo))
        self.fused_front = True         # routing, layout and co-activation in three launches (CAP pruning)
        # rank-side buffers
        self.row_cap = row_cap if row_cap is not None else T * min(k, cfg.E_loc)
        self.recv_cap = recv_cap if recv_cap is not None else T * min(k, R)
        self.xs = torch.empty((self.row_cap, d), dtype=self.tdt, device=self.dev)
        self.row_src = torch.empty(self.row_cap, **i32)
        self.row_dst = torch.empty(self.row_cap, **i32)
        self.row_w = torch.empty(self.row_cap, dtype=torch.float32, device=self.dev)
        self.Y = torch.empty((self.row_cap, d), dtype=self.tdt, device=self.dev)
        self.parts = torch.zeros((self.recv_cap, d), dtype=self.tdt, device=self.dev)
        self.y = torch.empty((cfg.tokens_per_rank, d), dtype=self.tdt, device=self.dev)
        self.ws_ffn = self._ws(capi.cap_workspace_size(capi.CAP_OP_EXPERT_FFN, None, d, cfg.inter,
                                                       self.row_cap, self.dt))
        # waits of the fused FFN kernel that gave up (every FFN call adds to it)
        self.ffn_err = torch.zeros(1, **i32)
        self.ffn_opts = capi.make_ffn_options(self.ffn_err)
        self.weights: dict[int, tuple] = {}
        self.naive = False              # expert-level threshold pruning instead of CAP's
        self.fused_gather = True        # FFN reads x through row_src instead of a gathered copy
        # bf16: single-expert tokens' destination combine in the FFN's epilogue
        self.fused_combine = cfg.dtype == "bf16"
        # with a side stream: start the shared experts after the routing front
        # end (True) or with it (False)
        self.shared_after_front = False
        self.shared = None
        self.shared_out = None
        self.ws_shared = None

    def _ws(self, nbytes: int) -> torch.Tensor:
        # 256-byte aligned by the caching allocator
        return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=self.dev)

    # ------------------------------------------------------------ weights
    def set_rank_weights(self, rank: int, w1: np.ndarray, w3: np.ndarray, w2: np.ndarray):
        """w1, w3 [E_loc][inter][d], w2 [E_loc][d][inter] in local-slot order (storage type)."""
        self.weights[rank] = tuple(to_device_rows(w, self.cfg.dtype, self.dev) for w in (w1, w3, w2))

    def set_placement(self, expert_rank, expert_local):
        """Replace the placement in place (the topology keeps pointing at the
        same device arrays)."""
        self.expert_rank.copy_(torch.as_tensor(np.asarray(expert_rank, np.int32)))
        self.expert_local.copy_(torch.as_tensor(np.asarray(expert_local, np.int32)))

    def set_shared_weights(self, w1, w3, w2):
        self.shared = tuple(to_device_rows(w, self.cfg.dtype, self.dev) for w in (w1, w3, w2))
        inter = self.shared[0].shape[0]
        T_loc = self.cfg.tokens_per_rank
        self.shared_out = torch.empty((T_loc, self.d), dtype=self.tdt, device=self.dev)
        self.ws_shared = self._ws(capi.cap_workspace_size(capi.CAP_OP_EXPERT_FFN, None, self.d, inter,
                                                          T_loc, self.dt))
        self.shared_offsets = torch.tensor([0, T_loc], dtype=torch.int32, device=self.dev)

    # ------------------------------------------------------------ steps
    def route(self, stream=None):
        fn = capi.cap_route_prune_naive if self.naive else capi.cap_route_prune
        fn(self.topo, self.logits, self.p, self.idx, self.w, self.keep, self.mask, stream)

    def router_route(self, w_gate: torch.Tensor, logits_out: torch.Tensor | None = None, stream=None):
        """Router GEMM x W_g^T fused with top-k routing and pruning (bf16 x)."""
        capi.cap_router_route_prune(self.topo, self.dt, self.d, self.x, w_gate, self.p, self.idx, self.w,
                                    self.keep, self.mask, logits_out, stream)

    def route_layout(self, coactivation=True, stream=None):
        """Routing, pruning, layout and (optionally) co-activation counts in
        the fused three-launch front end."""
        capi.cap_route_layout(self.topo, self.logits, self.p, self.idx, self.w, self.keep, self.mask, self.lay,
                              self.coact if coactivation else None, self.ws_front, stream=stream)

    def layout(self, stream=None):
        capi.cap_dispatch_layout(self.topo, self.idx, self.keep, self.mask, self.lay, self.ws_layout,
                                 stream=stream)

    def coactivation(self, accumulate=False, stream=None):
        capi.cap_coactivation(self.cfg.T, self.cfg.k, self.cfg.E, self.idx, self.keep, self.coact,
                              accumulate, self.ws_coact, stream=stream)

    def gather(self, rank: int, stream=None):
        capi.cap_permute(self.topo, capi.CAP_PERMUTE_EXPERT_GATHER, rank, self.dt, self.d, self.x,
                         self.idx, self.keep, self.mask, self.lay, self.xs, self.row_cap, stream)

    def row_source(self, rank: int, stream=None):
        capi.cap_permute(self.topo, capi.CAP_PERMUTE_ROW_SOURCE, rank, self.dt, self.d, None,
                         self.idx, self.keep, self.mask, self.lay, self.row_src, self.row_cap, stream)

    def row_plan(self, rank: int, stream=None):
        """Row source plus the receive row and gate weight of each row whose
        token has no other kept expert on the rank."""
        capi.cap_row_plan(self.topo, rank, self.w, self.lay, self.row_src, self.row_dst, self.row_w,
                          self.row_cap, self.recv_cap, stream)

    def send_pack(self, rank: int, out: torch.Tensor, stream=None):
        capi.cap_permute(self.topo, capi.CAP_PERMUTE_SEND_PACK, rank, self.dt, self.d, self.x,
                         self.idx, self.keep, self.mask, self.lay, out, out.shape[0], stream)

    def ffn(self, rank: int, stream=None):
        w1, w3, w2 = self.weights[rank]
        E_loc = self.cfg.E_loc
        offs = self.lay_t["expert_offsets"][rank * E_loc:(rank + 1) * E_loc + 1]
        capi.cap_expert_ffn_ex(self.dt, E_loc, self.d, self.cfg.inter, self.row_cap, self.xs, 0, None, offs,
                               w1, w3, w2, self.Y, self.ws_ffn, options=self.ffn_opts, stream=stream)

    def ffn_gather(self, rank: int, stream=None):
        """The rank's expert FFN reading its rows from x through row_src."""
        w1, w3, w2 = self.weights[rank]
        E_loc = self.cfg.E_loc
        offs = self.lay_t["expert_offsets"][rank * E_loc:(rank + 1) * E_loc + 1]
        capi.cap_expert_ffn_ex(self.dt, E_loc, self.d, self.cfg.inter, self.row_cap, self.x,
                               self.x.shape[0], self.row_src, offs, w1, w3, w2, self.Y, self.ws_ffn,
                               options=self.ffn_opts, stream=stream)

    def ffn_combine(self, rank: int, stream=None):
        """ffn_gather with the single-expert tokens' destination combine in the
        down GEMM's epilogue (their rows go to parts, scaled; the rest to Y)."""
        w1, w3, w2 = self.weights[rank]
        E_loc = self.cfg.E_loc
        offs = self.lay_t["expert_offsets"][rank * E_loc:(rank + 1) * E_loc + 1]
        capi.cap_expert_ffn_combine(self.dt, E_loc, self.d, self.cfg.inter, self.row_cap, self.x,
                                    self.x.shape[0], self.row_src, offs, w1, w3, w2, self.Y, self.row_dst,
                                    self.row_w, self.parts, self.recv_cap, self.ws_ffn, options=self.ffn_opts,
                                    stream=stream)

    def shared_ffn(self, rank: int, stream=None):
        if self.shared is None:
            return
        w1, w3, w2 = self.shared
        T_loc = self.cfg.tokens_per_rank
        xs = self.x[rank * T_loc:(rank + 1) * T_loc]
        capi.cap_expert_ffn_ex(self.dt, 1, self.d, w1.shape[0], T_loc, xs, 0, None, self.shared_offsets,
                               w1, w3, w2, self.shared_out, self.ws_shared, options=self.ffn_opts, stream=stream)

    def dest_reduce(self, rank: int, stream=None):
        capi.cap_combine(self.topo, capi.CAP_COMBINE_DEST_REDUCE, rank, self.dt, self.d, self.Y,
                         self.row_cap, self.idx, self.w, self.keep, self.mask, self.lay, None,
                         self.parts, self.recv_cap, stream)

    def dest_reduce_multi(self, rank: int, stream=None):
        """The destination reduce of the tokens with two or more kept experts
        on the rank (after ffn_combine)."""
        capi.cap_combine(self.topo, capi.CAP_COMBINE_DEST_REDUCE_MULTI, rank, self.dt, self.d, self.Y,
                         self.row_cap, self.idx, self.w, self.keep, self.mask, self.lay, None,
                         self.parts, self.recv_cap, stream)

    def src_reduce(self, rank: int, stream=None):
        capi.cap_combine(self.topo, capi.CAP_COMBINE_SRC_REDUCE, rank, self.dt, self.d, self.parts,
                         self.recv_cap, self.idx, self.w, self.keep, self.mask, self.lay,
                         self.shared_out if self.shared is not None else None, self.y,
                         self.y.shape[0], stream)

    def front(self, stream=None, side=None):
        """Routing front end over all virtual ranks' tokens: the fused
        three-launch front end (CAP pruning), or route, layout and
        co-activation as separate calls (naive pruning, or fused_front off).
        In the separate form, with a side stream the co-activation counts
        (which only feed placement) run there beside the layout; the main
        stream waits for them before returning control to later work."""
        if self.fused_front and not self.naive:
            self.route_layout(True, stream)
            return
        if side is None:
            self.route(stream)
            self.layout(stream)
            self.coactivation(False, stream)
            return
        self.route(stream)
        main = stream if stream is not None else torch.cuda.current_stream()
        if not hasattr(self, "_fork"):
            self._fork, self._join = torch.cuda.Event(), torch.cuda.Event()
        self._fork.record(main)
        side.wait_event(self._fork)
        self.coactivation(False, side)
        self._join.record(side)
        self.layout(main)
        main.wait_event(self._join)

    def rank_path(self, rank: int, stream=None, ffn_events=None, join=None):
        """The destination and source work of one rank.  ffn_events: an
        optional pair of events recorded around the routed FFN.  join: an event
        the source reduce waits for, when the shared experts ran on another
        stream; without it they run here, before the source reduce."""
        main = stream if stream is not None else torch.cuda.current_stream()
        combine = self.fused_gather and self.fused_combine
        if combine:
            self.row_plan(rank, main)
        elif self.fused_gather:
            self.row_source(rank, main)
        else:
            self.gather(rank, main)
        if ffn_events is not None:
            ffn_events[0].record(main)
        if combine:
            self.ffn_combine(rank, main)
        elif self.fused_gather:
            self.ffn_gather(rank, main)
        else:
            self.ffn(rank, main)
        if ffn_events is not None:
            ffn_events[1].record(main)
        if combine:
            self.dest_reduce_multi(rank, main)
        else:
            self.dest_reduce(rank, main)
        if join is None:
            self.shared_ffn(rank, main)
        else:
            main.wait_event(join)
        self.src_reduce(rank, main)

    def capture_step(self, rank: int = 0, side=None, warmup: int = 2) -> torch.cuda.CUDAGraph:
        """The whole step (step(rank, side=side)) as one HIP graph.
        Every call writes fixed buffers and allocates nothing, so replays redo
        exactly the eager work."""
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap):
            for _ in range(warmup):
                self.step(rank, side=side)
        torch.cuda.current_stream().wait_stream(cap)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.step(rank, side=side)
        return g

    def step(self, rank: int = 0, stream=None, side=None, ffn_events=None):
        """One layer step: the front end over all virtual ranks' tokens, then
        rank `rank`'s path.  With a side stream, the work that no later
        main-stream kernel reads runs there: the shared experts (they read only
        x) from the start of the step, the co-activation counts once routing
        is done; the main stream joins it before the source reduce, which adds
        the shared output.  ffn_events: as in rank_path."""
        main = stream if stream is not None else torch.cuda.current_stream()
        if side is None or (self.fused_front and not self.naive):
            # the fused front end, then (beside it on the side stream, when
            # there is one) the shared experts, which read only x
            if side is not None:
                if not hasattr(self, "_step_ev"):
                    self._step_ev = [torch.cuda.Event() for _ in range(3)]
                start, _, side_done = self._step_ev
                if self.shared_after_front:
                    self.front(main)
                start.record(main)
                side.wait_event(start)
                self.shared_ffn(rank, side)
                side_done.record(side)
                if not self.shared_after_front:
                    self.front(main)
                self.rank_path(rank, main, ffn_events, join=side_done)
                return
            self.front(main)
            self.rank_path(rank, main, ffn_events)
            return
        if not hasattr(self, "_step_ev"):
            self._step_ev = [torch.cuda.Event() for _ in range(3)]
        start, routed, side_done = self._step_ev
        start.record(main)
        side.wait_event(start)
        self.shared_ffn(rank, side)
        self.route(main)
        routed.record(main)
        side.wait_event(routed)
        self.coactivation(False, side)
        side_done.record(side)
        self.layout(main)
        self.rank_path(rank, main, ffn_events, join=side_done)

    def ffn_wait_errors(self) -> int:
        """Waits of the fused FFN kernel that gave up since the layer was made
        (0 unless an FFN output is invalid).  Synchronises."""
        torch.cuda.synchronize()
        return int(self.ffn_err.item())

    # ------------------------------------------------------------ host views
    def host(self, name: str) -> np.ndarray:
        if name in self.lay_t:
            return self.lay_t[name].cpu().numpy()
        t = getattr(self, name)
        if t.dtype == _BF16:
            return t.view(torch.int16).cpu().numpy().view(np.uint16)
        return t.cpu().numpy()

    def rank_rows(self, rank: int) -> int:
        eo = self.lay_t["expert_offsets"].cpu().numpy()
        E_loc = self.cfg.E_loc
        return int(eo[(rank + 1) * E_loc] - eo[rank * E_loc])
