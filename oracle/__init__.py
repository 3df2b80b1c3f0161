"""CPU oracle of the CAP MoE layer hot path (numpy + a plain C library).

TEST INFRASTRUCTURE ONLY: only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the GPU product path and never serves as its fallback.

Each function wraps one step of ``cap_oracle.c`` (which cites the paper) or
composes them in the paper's order.  Inputs are numpy arrays; bf16 data enters
as exact fp32 values (bf16 bits widened by the caller).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

_lib = None

_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_u8p = np.ctypeslib.ndpointer(dtype=np.uint8, flags="C_CONTIGUOUS")
_u32p = np.ctypeslib.ndpointer(dtype=np.uint32, flags="C_CONTIGUOUS")
_u64p = np.ctypeslib.ndpointer(dtype=np.uint64, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")
_vp = ctypes.c_void_p
_i = ctypes.c_int
_f = ctypes.c_float
_sz = ctypes.c_size_t


def lib():
    global _lib
    if _lib is None:
        L = ctypes.CDLL(_build.ensure_built())
        sig = {
            "orc_exp": ([_f], _f),
            "orc_exp_array": ([ctypes.c_int64, _f32p, _f32p], None),
            "orc_topk": ([_i, _i, _i, _f32p, _i32p], None),
            "orc_gates": ([_i, _i, _i, _f32p, _i32p, _f32p], None),
            "orc_prune": ([_i, _i, _i, _i, _f, _f, _i32p, _i32p, _f32p, _u8p, _f32p, _u64p], None),
            "orc_prune_naive": ([_i, _i, _i32p, _f, _i32p, _f32p, _u8p, _f32p, _u64p], None),
            "orc_dispatch_layout": ([_i, _i, _i, _i, _i, _i, _i32p, _i32p, _i32p, _u8p, _u64p,
                                     _i32p, _i32p, _i32p, _i32p, _i32p, _i32p, _i32p, _i32p,
                                     _u8p, _i64p], None),
            "orc_expert_gather": ([_i, _i, _i, _i, _i, _sz, _i32p, _i32p, _u8p, _i32p, _i32p,
                                   _vp, _vp], None),
            "orc_send_pack": ([_i, _i, _i, _sz, _u64p, _i32p, _vp, _vp], None),
            "orc_swiglu_rows": ([_i, _i, _i, _f32p, _f32p, _f32p, _f32p, _f64p, _i], None),
            "orc_dest_reduce": ([_i, _i, _i, _i, _i, _i32p, _i32p, _f32p, _u8p, _i32p, _i32p,
                                 _i32p, _i32p, _f32p, _f32p], None),
            "orc_src_reduce": ([_i, _i, _i, _i, _i, _i32p, _i32p, _u8p, _u64p, _i32p, _i32p,
                                _f32p, _vp, _f32p], None),
            "orc_coactivation": ([_i, _i, _i, _i32p, _u8p, _u32p, _i], None),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ------------------------------------------------------------------ routing
def exp_f32(z) -> np.ndarray:
    z = _c(np.atleast_1d(z), np.float32)
    out = np.empty_like(z)
    lib().orc_exp_array(z.size, z.ravel(), out.ravel())
    return out


def topk(logits: np.ndarray, k: int) -> np.ndarray:
    L = _c(logits, np.float32)
    T, E = L.shape
    idx = np.empty((T, k), np.int32)
    lib().orc_topk(T, E, k, L, idx)
    return idx


def gates(logits: np.ndarray, idx: np.ndarray) -> np.ndarray:
    L = _c(logits, np.float32)
    idx = _c(idx, np.int32)
    T, E = L.shape
    k = idx.shape[1]
    w = np.empty((T, k), np.float32)
    lib().orc_gates(T, E, k, L, idx, w)
    return w


def prune(idx, w, expert_rank, ranks_per_node, tokens_per_rank, c, p):
    idx = _c(idx, np.int32)
    w = _c(w, np.float32)
    T, k = idx.shape
    keep = np.empty((T, k), np.uint8)
    wp = np.empty((T, k), np.float32)
    mask = np.empty(T, np.uint64)
    lib().orc_prune(T, k, ranks_per_node, tokens_per_rank, float(c), float(p),
                    _c(expert_rank, np.int32), idx, w, keep, wp, mask)
    return keep, wp, mask


def prune_naive(idx, w, expert_rank, p):
    idx = _c(idx, np.int32)
    w = _c(w, np.float32)
    T, k = idx.shape
    keep = np.empty((T, k), np.uint8)
    wp = np.empty((T, k), np.float32)
    mask = np.empty(T, np.uint64)
    lib().orc_prune_naive(T, k, _c(expert_rank, np.int32), float(p), idx, w, keep, wp, mask)
    return keep, wp, mask


def router_logits(x, w_gate) -> np.ndarray:
    """Router logits of Eq. 1, x W_g^T, in fp64 (x [T][d], w_gate [E][d])."""
    return np.asarray(x, np.float64) @ np.asarray(w_gate, np.float64).T


def route_prune(logits, k, expert_rank, ranks_per_node, tokens_per_rank, c, p):
    """Top-k, gates, then communication-aware pruning (the paper's order)."""
    idx = topk(logits, k)
    w = gates(logits, idx)
    keep, wp, mask = prune(idx, w, expert_rank, ranks_per_node, tokens_per_rank, c, p)
    return dict(idx=idx, w=w, keep=keep, wp=wp, mask=mask)


# ------------------------------------------------------------------ layout
def dispatch_layout(idx, keep, mask, expert_rank, expert_local, R, ranks_per_node, tokens_per_rank, E):
    idx = _c(idx, np.int32)
    keep = _c(keep, np.uint8)
    mask = _c(mask, np.uint64)
    T, k = idx.shape
    out = dict(
        send_counts=np.empty((R, R), np.int32),
        send_offsets=np.empty((R, R), np.int32),
        recv_offsets=np.empty(R + 1, np.int32),
        recv_token=np.full(T * k, -1, np.int32),
        expert_counts=np.empty(E, np.int32),
        expert_offsets=np.empty(E + 1, np.int32),
        slot_pos=np.empty((T, k), np.int32),
        copy_row=np.empty((T, k), np.int32),
        vol=np.empty((T, 4), np.uint8),
        totals=np.empty(4, np.int64),
    )
    lib().orc_dispatch_layout(T, E, k, R, ranks_per_node, tokens_per_rank,
                              _c(expert_rank, np.int32), _c(expert_local, np.int32),
                              idx, keep, mask,
                              out["send_counts"], out["send_offsets"], out["recv_offsets"],
                              out["recv_token"], out["expert_counts"], out["expert_offsets"],
                              out["slot_pos"], out["copy_row"], out["vol"], out["totals"])
    out["recv_token"] = out["recv_token"][: int(out["recv_offsets"][R])]
    return out


# ------------------------------------------------------------------ permutation
def expert_gather(x, idx, keep, slot_pos, expert_offsets, expert_rank, R, rank):
    x = np.ascontiguousarray(x)
    idx = _c(idx, np.int32)
    T, k = idx.shape
    E = len(expert_rank)
    E_loc = E // R
    rows = int(expert_offsets[(rank + 1) * E_loc] - expert_offsets[rank * E_loc])
    out = np.zeros((rows,) + x.shape[1:], x.dtype)
    row_bytes = x[0].nbytes
    lib().orc_expert_gather(T, k, E, R, rank, row_bytes, _c(expert_rank, np.int32), idx,
                            _c(keep, np.uint8), _c(slot_pos, np.int32),
                            _c(expert_offsets, np.int32), x.ctypes.data, out.ctypes.data)
    return out


def send_pack(x, mask, send_offsets, send_counts, R, tokens_per_rank, src):
    x = np.ascontiguousarray(x)
    rows = int(np.asarray(send_counts)[src].sum())
    out = np.zeros((rows,) + x.shape[1:], x.dtype)
    lib().orc_send_pack(R, tokens_per_rank, src, x[0].nbytes, _c(mask, np.uint64),
                        _c(send_offsets, np.int32), x.ctypes.data, out.ctypes.data)
    return out


# ------------------------------------------------------------------ expert FFN
def swiglu_rows(X, W1, W3, W2, nthreads: int | None = None) -> np.ndarray:
    """fp64 SwiGLU of each row of X (exact fp32 inputs); returns float64 [n][d]."""
    X = _c(X, np.float32)
    n, d = X.shape
    inter = W1.shape[0]
    Y = np.empty((n, d), np.float64)
    if n:
        lib().orc_swiglu_rows(n, d, inter, X, _c(W1, np.float32), _c(W3, np.float32),
                              _c(W2, np.float32), Y, nthreads or (os.cpu_count() or 1))
    return Y


def expert_ffn(xs, row_offsets, weights, nthreads: int | None = None) -> np.ndarray:
    """SwiGLU over a rank's expert-sorted rows: expert l owns rows
    [row_offsets[l]-row_offsets[0], row_offsets[l+1]-row_offsets[0]).
    weights[l] = (W1, W3, W2) as fp32.  Returns fp32 [rows][d]."""
    xs = _c(xs, np.float32)
    base = int(row_offsets[0])
    Y = np.zeros(xs.shape, np.float32)
    for l, (W1, W3, W2) in enumerate(weights):
        a, b = int(row_offsets[l]) - base, int(row_offsets[l + 1]) - base
        if b > a:
            Y[a:b] = swiglu_rows(xs[a:b], W1, W3, W2, nthreads).astype(np.float32)
    return Y


# ------------------------------------------------------------------ combine
def dest_reduce(Y, route, layout, expert_rank, R, rank, d):
    U = int(layout["recv_offsets"][rank + 1] - layout["recv_offsets"][rank])
    part = np.zeros((U, d), np.float32)
    T, k = route["idx"].shape
    lib().orc_dest_reduce(k, len(expert_rank), R, rank, d, _c(expert_rank, np.int32),
                          _c(route["idx"], np.int32), _c(route["wp"], np.float32),
                          _c(route["keep"], np.uint8), _c(layout["slot_pos"], np.int32),
                          _c(layout["expert_offsets"], np.int32),
                          _c(layout["recv_offsets"], np.int32),
                          _c(layout["recv_token"], np.int32), _c(Y, np.float32), part)
    return part


def src_reduce(parts, route, layout, expert_rank, R, tokens_per_rank, src, d, shared=None):
    T, k = route["idx"].shape
    y = np.zeros((tokens_per_rank, d), np.float32)
    sh = None if shared is None else _c(shared, np.float32)
    lib().orc_src_reduce(k, R, tokens_per_rank, src, d, _c(expert_rank, np.int32),
                         _c(route["idx"], np.int32), _c(route["keep"], np.uint8),
                         _c(route["mask"], np.uint64), _c(layout["copy_row"], np.int32),
                         _c(layout["recv_offsets"], np.int32), _c(parts, np.float32),
                         None if sh is None else sh.ctypes.data, y)
    return y


def dense_moe_rows(tokens, x_rows, route, expert_weights_f32, shared_f32=None, nthreads=None):
    """Independent dense path of Eq. 1 for the given tokens, with no permutation:
    y[t] = sum over kept slots of w'_s * SwiGLU_{idx_s}(x_t) + shared(x_t).
    ``expert_weights_f32(e)`` returns (W1, W3, W2) fp32.  fp64 result."""
    x_rows = _c(x_rows, np.float64)
    out = np.zeros(x_rows.shape, np.float64)
    by_expert: dict[int, list[tuple[int, float]]] = {}
    for i, t in enumerate(tokens):
        for s in range(route["idx"].shape[1]):
            if route["keep"][t, s]:
                by_expert.setdefault(int(route["idx"][t, s]), []).append((i, float(route["wp"][t, s])))
    for e, uses in sorted(by_expert.items()):
        W1, W3, W2 = expert_weights_f32(e)
        rows = [i for i, _ in uses]
        Y = swiglu_rows(x_rows[rows].astype(np.float32), W1, W3, W2, nthreads)
        for j, (i, wgt) in enumerate(uses):
            out[i] += wgt * Y[j]
    if shared_f32 is not None:
        out += swiglu_rows(x_rows.astype(np.float32), *shared_f32, nthreads)
    return out


# ------------------------------------------------------------------ co-activation
def coactivation(idx, keep, E, C=None):
    idx = _c(idx, np.int32)
    T, k = idx.shape
    acc = C is not None
    if C is None:
        C = np.zeros((E, E), np.uint32)
    lib().orc_coactivation(T, k, E, idx, _c(keep, np.uint8), C, int(acc))
    return C
