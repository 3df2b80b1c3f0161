"""Thin ctypes binding of libcap.so (include/cap.h).

Argument marshalling only: torch tensors in, device pointers and sizes out;
every computation runs in the HIP kernels of libcap.so.  There is no CPU
fallback: importing this module raises if the library is missing, and every
call raises CapError on a non-zero status.

Function names follow the C ABI: cap_route_prune, cap_route_prune_naive, cap_router_route_prune,
cap_dispatch_layout,
cap_permute, cap_row_plan, cap_expert_ffn, cap_expert_ffn_gather, cap_expert_ffn_ex, cap_expert_ffn_combine,
cap_combine, cap_coactivation, cap_workspace_size, cap_status_string, cap_version.
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (loads the HIP runtime that libcap.so binds to)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcap.so")

CAP_OK, CAP_ERR_INVALID_ARG, CAP_ERR_UNSUPPORTED, CAP_ERR_WORKSPACE, CAP_ERR_HIP = 0, -1, -2, -3, -4
CAP_DTYPE_F32, CAP_DTYPE_BF16 = 0, 1
CAP_PERMUTE_EXPERT_GATHER, CAP_PERMUTE_SEND_PACK, CAP_PERMUTE_ROW_SOURCE = 0, 1, 2
CAP_COMBINE_DEST_REDUCE, CAP_COMBINE_SRC_REDUCE, CAP_COMBINE_DEST_REDUCE_MULTI = 0, 1, 2
(CAP_OP_ROUTE_PRUNE, CAP_OP_DISPATCH_LAYOUT, CAP_OP_PERMUTE, CAP_OP_EXPERT_FFN,
 CAP_OP_COMBINE, CAP_OP_COACTIVATION, CAP_OP_ADJUSTMENT, CAP_OP_ROUTE_LAYOUT) = range(8)

EXPORTS = ["cap_status_string", "cap_version", "cap_workspace_size", "cap_route_prune", "cap_route_prune_naive",
           "cap_router_route_prune",
           "cap_dispatch_layout", "cap_permute", "cap_expert_ffn", "cap_expert_ffn_gather", "cap_expert_ffn_ex",
           "cap_combine", "cap_coactivation", "cap_dispatch_layout_static",
           "cap_dispatch_layout_static_max_bytes", "cap_adjustment_spectrum", "cap_route_layout",
           "cap_row_plan", "cap_expert_ffn_combine"]


class CapError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {status_string(status)} ({status})")
        self.status = status


class Topology(ctypes.Structure):
    _fields_ = [("E", ctypes.c_int32), ("R", ctypes.c_int32), ("ranks_per_node", ctypes.c_int32),
                ("T", ctypes.c_int32), ("tokens_per_rank", ctypes.c_int32), ("k", ctypes.c_int32),
                ("expert_rank", ctypes.c_void_p), ("expert_local", ctypes.c_void_p),
                ("inter_node_cost", ctypes.c_float)]


class FfnOptions(ctypes.Structure):
    _fields_ = [("wait_errors", ctypes.c_void_p), ("max_workgroups", ctypes.c_int32),
                ("spin_limit", ctypes.c_int32), ("force_wait_timeout", ctypes.c_int32)]


class Layout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "send_counts", "send_offsets", "recv_offsets", "recv_token", "expert_counts",
        "expert_offsets", "slot_pos", "copy_row", "vol", "totals")]


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2607_05116_amd.build` "
                          "(or __graft_entry__.build()); there is no CPU fallback")
    L = ctypes.CDLL(path)
    vp, i32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    P = ctypes.POINTER
    sig = {
        "cap_status_string": ([ctypes.c_int], ctypes.c_char_p),
        "cap_version": ([], i32),
        "cap_workspace_size": ([ctypes.c_int, P(Topology), i32, i32, i32, ctypes.c_int], sz),
        "cap_route_prune": ([P(Topology), vp, f32, vp, vp, vp, vp, vp], ctypes.c_int),
        "cap_route_prune_naive": ([P(Topology), vp, f32, vp, vp, vp, vp, vp], ctypes.c_int),
        "cap_router_route_prune": ([P(Topology), ctypes.c_int, i32, vp, vp, f32, vp, vp, vp, vp, vp, vp],
                                   ctypes.c_int),
        "cap_dispatch_layout": ([P(Topology), vp, vp, vp, P(Layout), vp, sz, vp], ctypes.c_int),
        "cap_dispatch_layout_static": ([P(Topology), vp, vp, vp, P(Layout), vp], ctypes.c_int),
        "cap_dispatch_layout_static_max_bytes": ([], sz),
        "cap_permute": ([P(Topology), ctypes.c_int, i32, ctypes.c_int, i32, vp, vp, vp, vp, P(Layout),
                         vp, i32, vp], ctypes.c_int),
        "cap_expert_ffn": ([ctypes.c_int, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp],
                           ctypes.c_int),
        "cap_expert_ffn_gather": ([ctypes.c_int, i32, i32, i32, i32, vp, i32, vp, vp, vp, vp, vp, vp, vp, sz,
                                   vp], ctypes.c_int),
        "cap_expert_ffn_ex": ([ctypes.c_int, i32, i32, i32, i32, vp, i32, vp, vp, vp, vp, vp, vp, vp, sz,
                               P(FfnOptions), vp], ctypes.c_int),
        "cap_expert_ffn_combine": ([ctypes.c_int, i32, i32, i32, i32, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp,
                                    vp, i32, vp, sz, P(FfnOptions), vp], ctypes.c_int),
        "cap_row_plan": ([P(Topology), i32, vp, P(Layout), vp, vp, vp, i32, i32, vp], ctypes.c_int),
        "cap_combine": ([P(Topology), ctypes.c_int, i32, ctypes.c_int, i32, vp, i32, vp, vp, vp, vp,
                         P(Layout), vp, vp, i32, vp], ctypes.c_int),
        "cap_coactivation": ([i32, i32, i32, vp, vp, vp, i32, vp, sz, vp], ctypes.c_int),
        "cap_route_layout": ([P(Topology), vp, f32, vp, vp, vp, vp, P(Layout), vp, vp, sz, vp], ctypes.c_int),
        "cap_adjustment_spectrum": ([vp, i32, i32, i32, f32, vp, vp, i32, vp, vp, vp, vp, sz, vp], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    return L


_lib = load_library()


def status_string(s: int) -> str:
    return _lib.cap_status_string(int(s)).decode()


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _check(fn: str, st: int):
    if st != CAP_OK:
        raise CapError(fn, st)


def make_topology(E, R, ranks_per_node, T, k, expert_rank, expert_local, inter_node_cost=5.0) -> Topology:
    """expert_rank / expert_local: int32 device tensors [E] (kept alive by the caller)."""
    return Topology(E, R, ranks_per_node, T, T // R, k, _ptr(expert_rank), _ptr(expert_local),
                    float(inter_node_cost))


def make_layout(t: dict) -> Layout:
    return Layout(*[_ptr(t[n]) for n, _ in Layout._fields_])


def cap_version() -> int:
    return _lib.cap_version()


def cap_workspace_size(op: int, topo: Topology | None, d: int = 0, inter: int = 0, max_rows: int = 0,
                       dtype: int = CAP_DTYPE_BF16) -> int:
    return _lib.cap_workspace_size(op, ctypes.byref(topo) if topo is not None else None,
                                   d, inter, max_rows, dtype)


def cap_route_prune_naive(topo, logits, p, idx, w, keep, dst_mask, stream=None):
    _check("cap_route_prune_naive", _lib.cap_route_prune_naive(
        ctypes.byref(topo), _ptr(logits), float(p), _ptr(idx), _ptr(w), _ptr(keep), _ptr(dst_mask),
        _stream(stream)))


def cap_route_prune(topo, logits, p, idx, w, keep, dst_mask, stream=None):
    _check("cap_route_prune", _lib.cap_route_prune(
        ctypes.byref(topo), _ptr(logits), float(p), _ptr(idx), _ptr(w), _ptr(keep), _ptr(dst_mask),
        _stream(stream)))


def cap_router_route_prune(topo, dtype, d, x, w_gate, p, idx, w, keep, dst_mask, logits=None, stream=None):
    _check("cap_router_route_prune", _lib.cap_router_route_prune(
        ctypes.byref(topo), dtype, int(d), _ptr(x), _ptr(w_gate), float(p), _ptr(idx), _ptr(w), _ptr(keep),
        _ptr(dst_mask), _ptr(logits), _stream(stream)))


def cap_dispatch_layout(topo, idx, keep, dst_mask, layout: Layout, ws, ws_bytes=None, stream=None):
    nbytes = ws_bytes if ws_bytes is not None else ws.numel() * ws.element_size()
    _check("cap_dispatch_layout", _lib.cap_dispatch_layout(
        ctypes.byref(topo), _ptr(idx), _ptr(keep), _ptr(dst_mask), ctypes.byref(layout), _ptr(ws), nbytes,
        _stream(stream)))


def cap_route_layout(topo, logits, p, idx, w, keep, dst_mask, layout: Layout, coact, ws, ws_bytes=None,
                     stream=None):
    nbytes = ws_bytes if ws_bytes is not None else ws.numel() * ws.element_size()
    _check("cap_route_layout", _lib.cap_route_layout(
        ctypes.byref(topo), _ptr(logits), float(p), _ptr(idx), _ptr(w), _ptr(keep), _ptr(dst_mask),
        ctypes.byref(layout), _ptr(coact), _ptr(ws), nbytes, _stream(stream)))


def cap_dispatch_layout_static(topo, idx, keep, dst_mask, layout: Layout, stream=None):
    _check("cap_dispatch_layout_static", _lib.cap_dispatch_layout_static(
        ctypes.byref(topo), _ptr(idx), _ptr(keep), _ptr(dst_mask), ctypes.byref(layout), _stream(stream)))


def cap_dispatch_layout_static_max_bytes() -> int:
    return int(_lib.cap_dispatch_layout_static_max_bytes())


def cap_permute(topo, mode, rank, dtype, d, x, idx, keep, dst_mask, layout: Layout, out, out_rows,
                stream=None):
    _check("cap_permute", _lib.cap_permute(
        ctypes.byref(topo), mode, rank, dtype, d, _ptr(x), _ptr(idx), _ptr(keep), _ptr(dst_mask),
        ctypes.byref(layout), _ptr(out), int(out_rows), _stream(stream)))


def cap_expert_ffn(dtype, E_loc, d, inter, max_rows, xs, row_offsets, w1, w3, w2, y, ws, ws_bytes=None,
                   stream=None):
    nbytes = ws_bytes if ws_bytes is not None else ws.numel() * ws.element_size()
    _check("cap_expert_ffn", _lib.cap_expert_ffn(
        dtype, E_loc, d, inter, max_rows, _ptr(xs), _ptr(row_offsets), _ptr(w1), _ptr(w3), _ptr(w2),
        _ptr(y), _ptr(ws), nbytes, _stream(stream)))


def cap_expert_ffn_gather(dtype, E_loc, d, inter, max_rows, x, x_rows, row_src, row_offsets, w1, w3, w2, y, ws,
                          ws_bytes=None, stream=None):
    nbytes = ws_bytes if ws_bytes is not None else ws.numel() * ws.element_size()
    _check("cap_expert_ffn_gather", _lib.cap_expert_ffn_gather(
        dtype, E_loc, d, inter, max_rows, _ptr(x), int(x_rows), _ptr(row_src), _ptr(row_offsets), _ptr(w1),
        _ptr(w3), _ptr(w2), _ptr(y), _ptr(ws), nbytes, _stream(stream)))


def make_ffn_options(wait_errors=None, max_workgroups=0, spin_limit=0, force_wait_timeout=False) -> FfnOptions:
    """wait_errors: an int32 device tensor the fused kernel adds its given-up waits to."""
    return FfnOptions(_ptr(wait_errors), int(max_workgroups), int(spin_limit), int(bool(force_wait_timeout)))


def cap_expert_ffn_ex(dtype, E_loc, d, inter, max_rows, x, x_rows, row_src, row_offsets, w1, w3, w2, y, ws,
                      ws_bytes=None, options: FfnOptions | None = None, stream=None):
    nbytes = ws_bytes if ws_bytes is not None else ws.numel() * ws.element_size()
    _check("cap_expert_ffn_ex", _lib.cap_expert_ffn_ex(
        dtype, E_loc, d, inter, max_rows, _ptr(x), int(x_rows), _ptr(row_src), _ptr(row_offsets), _ptr(w1),
        _ptr(w3), _ptr(w2), _ptr(y), _ptr(ws), nbytes, ctypes.byref(options) if options is not None else None,
        _stream(stream)))


def cap_expert_ffn_combine(dtype, E_loc, d, inter, max_rows, x, x_rows, row_src, row_offsets, w1, w3, w2, y,
                           row_dst, row_w, parts, parts_rows, ws, ws_bytes=None, options: FfnOptions | None = None,
                           stream=None):
    nbytes = ws_bytes if ws_bytes is not None else ws.numel() * ws.element_size()
    _check("cap_expert_ffn_combine", _lib.cap_expert_ffn_combine(
        dtype, E_loc, d, inter, max_rows, _ptr(x), int(x_rows), _ptr(row_src), _ptr(row_offsets), _ptr(w1),
        _ptr(w3), _ptr(w2), _ptr(y), _ptr(row_dst), _ptr(row_w), _ptr(parts), int(parts_rows), _ptr(ws), nbytes,
        ctypes.byref(options) if options is not None else None, _stream(stream)))


def cap_row_plan(topo, rank, w, layout: Layout, row_src, row_dst, row_w, rows_cap, parts_rows, stream=None):
    _check("cap_row_plan", _lib.cap_row_plan(
        ctypes.byref(topo), int(rank), _ptr(w), ctypes.byref(layout), _ptr(row_src), _ptr(row_dst), _ptr(row_w),
        int(rows_cap), int(parts_rows), _stream(stream)))


def cap_combine(topo, mode, rank, dtype, d, inp, in_rows, idx, w, keep, dst_mask, layout: Layout,
                shared_out, out, out_rows, stream=None):
    _check("cap_combine", _lib.cap_combine(
        ctypes.byref(topo), mode, rank, dtype, d, _ptr(inp), int(in_rows), _ptr(idx), _ptr(w), _ptr(keep),
        _ptr(dst_mask), ctypes.byref(layout), _ptr(shared_out), _ptr(out), int(out_rows), _stream(stream)))


def cap_coactivation(T, k, E, idx, keep, coact, accumulate, ws, ws_bytes=None, stream=None):
    nbytes = ws_bytes if ws_bytes is not None else ws.numel() * ws.element_size()
    _check("cap_coactivation", _lib.cap_coactivation(
        T, k, E, _ptr(idx), _ptr(keep), _ptr(coact), int(accumulate), _ptr(ws), nbytes, _stream(stream)))


def cap_adjustment_spectrum(coact, E, R, ranks_per_node, inter_node_cost, expert_rank, expert_local, max_swaps,
                            swaps, deltas, n_swaps, ws, ws_bytes=None, stream=None):
    nbytes = ws_bytes if ws_bytes is not None else ws.numel() * ws.element_size()
    _check("cap_adjustment_spectrum", _lib.cap_adjustment_spectrum(
        _ptr(coact), int(E), int(R), int(ranks_per_node), float(inter_node_cost), _ptr(expert_rank),
        _ptr(expert_local), int(max_swaps), _ptr(swaps), _ptr(deltas), _ptr(n_swaps), _ptr(ws), nbytes,
        _stream(stream)))
