"""Host-side checks that need no GPU: the C ABI library loads and exports
every symbol include/cap.h declares, argument validation rejects bad calls
before launching anything, and bench.py refuses more than one GPU."""
import ctypes
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cap.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(cap_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def capi():
    from paper_2607_05116_amd import capi as c
    return c


def test_library_exports_every_declared_symbol(capi):
    names = _declared()
    assert "cap_route_prune" in names and len(names) >= 9
    lib = ctypes.CDLL(capi.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(capi.EXPORTS) == names


def test_status_strings_and_version(capi):
    assert capi.status_string(0) == "CAP_OK"
    assert "workspace" in capi.status_string(-3)
    assert capi.cap_version() >= 100


def _topo(capi, **over):
    kw = dict(E=16, R=4, ranks_per_node=4, T=256, k=2)
    kw.update(over)
    t = capi.make_topology(kw["E"], kw["R"], kw["ranks_per_node"], kw["T"], kw["k"], 0x1000, 0x2000, 5.0)
    return t


ROUTE_FNS = ["cap_route_prune", "cap_route_prune_naive"]


@pytest.mark.parametrize("fn", ROUTE_FNS)
@pytest.mark.parametrize("over", [dict(k=0), dict(k=9), dict(E=300), dict(E=18), dict(R=65, E=130, T=260),
                                  dict(T=255), dict(ranks_per_node=3)])
def test_route_prune_rejects_bad_topology(capi, fn, over):
    t = _topo(capi, **over)
    st = getattr(capi._lib, fn)(ctypes.byref(t), 0x3000, 0.3, 0x4000, 0x5000, 0x6000, 0x7000, None)
    assert st == capi.CAP_ERR_INVALID_ARG


@pytest.mark.parametrize("fn", ROUTE_FNS)
@pytest.mark.parametrize("p", [-0.1, 1.0, 1.5, float("nan")])
def test_route_prune_rejects_bad_threshold(capi, fn, p):
    t = _topo(capi)
    st = getattr(capi._lib, fn)(ctypes.byref(t), 0x3000, p, 0x4000, 0x5000, 0x6000, 0x7000, None)
    assert st == capi.CAP_ERR_INVALID_ARG


@pytest.mark.parametrize("fn", ROUTE_FNS)
def test_route_prune_rejects_null_and_bad_cost(capi, fn):
    t = _topo(capi)
    f = getattr(capi._lib, fn)
    assert f(ctypes.byref(t), None, 0.3, 0x4000, 0x5000, 0x6000, 0x7000, None) == -1
    t.inter_node_cost = 0.5
    assert f(ctypes.byref(t), 0x3000, 0.3, 0x4000, 0x5000, 0x6000, 0x7000, None) == -1


def test_router_route_validation(capi):
    f = capi._lib.cap_router_route_prune
    B, F = capi.CAP_DTYPE_BF16, capi.CAP_DTYPE_F32
    out = (0x4000, 0x5000, 0x6000, 0x7000, None, None)
    t = _topo(capi, E=32, R=4)
    assert f(ctypes.byref(t), F, 128, 0x1000, 0x2000, 0.3, *out) == capi.CAP_ERR_UNSUPPORTED     # dtype
    assert f(ctypes.byref(t), B, 96, 0x1000, 0x2000, 0.3, *out) == capi.CAP_ERR_UNSUPPORTED      # d % 64
    assert f(ctypes.byref(t), B, 128, None, 0x2000, 0.3, *out) == capi.CAP_ERR_INVALID_ARG       # x
    assert f(ctypes.byref(t), B, 128, 0x1008, 0x2000, 0.3, *out) == capi.CAP_ERR_INVALID_ARG     # alignment
    assert f(ctypes.byref(t), B, 128, 0x1000, 0x2000, 1.0, *out) == capi.CAP_ERR_INVALID_ARG     # p
    small = _topo(capi, E=16, R=4)
    assert f(ctypes.byref(small), B, 128, 0x1000, 0x2000, 0.3, *out) == capi.CAP_ERR_UNSUPPORTED  # E <= 16


def test_workspace_checks(capi):
    t = _topo(capi)
    need = capi.cap_workspace_size(capi.CAP_OP_DISPATCH_LAYOUT, t)
    assert need > 0
    lay = capi.Layout(*([0x10000] * 10))
    st = capi._lib.cap_dispatch_layout(ctypes.byref(t), 0x3000, 0x4000, 0x5000, ctypes.byref(lay), 0x8000,
                                       need - 1, None)
    assert st == capi.CAP_ERR_WORKSPACE
    n = capi.cap_workspace_size(capi.CAP_OP_EXPERT_FFN, None, 2048, 768, 1000, capi.CAP_DTYPE_BF16)
    # H [max_rows][inter] bf16, then the fused kernel's counters (a few KiB)
    assert 1000 * 768 * 2 < n < 1000 * 768 * 2 + 8192
    assert capi.cap_workspace_size(capi.CAP_OP_EXPERT_FFN, None, 128, 256, 1000, capi.CAP_DTYPE_F32) == 1000 * 256 * 4
    st = capi._lib.cap_expert_ffn(capi.CAP_DTYPE_BF16, 4, 2048, 768, 1000, 0x1000, 0x2000, 0x3000, 0x4000,
                                  0x5000, 0x6000, 0x7000, n - 1, None)
    assert st == capi.CAP_ERR_WORKSPACE


def test_ffn_rejects_unsupported_shapes(capi):
    args = (0x1000, 0x2000, 0x3000, 0x4000, 0x5000, 0x6000, 0x7000, 1 << 30, None)
    assert capi._lib.cap_expert_ffn(capi.CAP_DTYPE_BF16, 4, 2000, 768, 100, *args) == capi.CAP_ERR_UNSUPPORTED
    # K beyond the 24-bit block offsets of the direct loads
    assert capi._lib.cap_expert_ffn(capi.CAP_DTYPE_BF16, 4, 1 << 20, 768, 100, *args) == capi.CAP_ERR_UNSUPPORTED
    assert capi._lib.cap_expert_ffn(capi.CAP_DTYPE_BF16, 4, 2048, 1 << 20, 100, *args) == capi.CAP_ERR_UNSUPPORTED
    assert capi._lib.cap_expert_ffn(capi.CAP_DTYPE_BF16, 4, 2048, 700, 100, *args) == capi.CAP_ERR_UNSUPPORTED
    assert capi._lib.cap_expert_ffn(7, 4, 2048, 768, 100, *args) == capi.CAP_ERR_UNSUPPORTED
    assert capi._lib.cap_expert_ffn(capi.CAP_DTYPE_BF16, 0, 2048, 768, 100, *args) == capi.CAP_ERR_INVALID_ARG


def test_ffn_gather_validation(capi):
    f = capi._lib.cap_expert_ffn_gather
    B = capi.CAP_DTYPE_BF16
    ws = 1 << 30
    ok = (0x1000, 512, 0x2000, 0x3000, 0x4000, 0x5000, 0x6000, 0x7000, 0x8000, ws, None)
    assert f(B, 4, 2048, 768, 100, None, *ok[1:]) == capi.CAP_ERR_INVALID_ARG             # x
    assert f(B, 4, 2048, 768, 100, 0x1000, 512, None, *ok[3:]) == capi.CAP_ERR_INVALID_ARG  # row_src
    assert f(B, 4, 2048, 768, 100, 0x1000, 0, *ok[2:]) == capi.CAP_ERR_INVALID_ARG         # x_rows
    assert f(B, 4, 2000, 768, 100, *ok) == capi.CAP_ERR_UNSUPPORTED                         # d
    big = (0x1000, (1 << 32) // 4096) + ok[2:]
    assert f(B, 4, 2048, 768, 100, *big) == capi.CAP_ERR_UNSUPPORTED                        # 32-bit offsets
    small_ws = ok[:-2] + (100 * 768 * 2 - 1, None)
    assert f(B, 4, 2048, 768, 100, *small_ws) == capi.CAP_ERR_WORKSPACE


def test_permute_and_combine_validation(capi):
    t = _topo(capi)
    lay = capi.Layout(*([0x10000] * 10))
    bad_rank = capi._lib.cap_permute(ctypes.byref(t), 0, 4, 1, 128, 0x1000, 0x2000, 0x3000, 0x4000,
                                     ctypes.byref(lay), 0x5000, 10, None)
    assert bad_rank == capi.CAP_ERR_INVALID_ARG
    bad_mode = capi._lib.cap_permute(ctypes.byref(t), 5, 0, 1, 128, 0x1000, 0x2000, 0x3000, 0x4000,
                                     ctypes.byref(lay), 0x5000, 10, None)
    assert bad_mode == capi.CAP_ERR_UNSUPPORTED
    bad_d = capi._lib.cap_permute(ctypes.byref(t), 0, 0, 1, 12, 0x1000, 0x2000, 0x3000, 0x4000,
                                  ctypes.byref(lay), 0x5000, 10, None)
    assert bad_d == capi.CAP_ERR_INVALID_ARG
    no_x = capi._lib.cap_permute(ctypes.byref(t), 0, 0, 1, 128, None, 0x2000, 0x3000, 0x4000,
                                 ctypes.byref(lay), 0x5000, 10, None)
    assert no_x == capi.CAP_ERR_INVALID_ARG
    rs_bad_rank = capi._lib.cap_permute(ctypes.byref(t), capi.CAP_PERMUTE_ROW_SOURCE, 4, 1, 0, None, 0x2000,
                                        0x3000, 0x4000, ctypes.byref(lay), 0x5000, 10, None)
    assert rs_bad_rank == capi.CAP_ERR_INVALID_ARG
    rs_misaligned = capi._lib.cap_permute(ctypes.byref(t), capi.CAP_PERMUTE_ROW_SOURCE, 0, 1, 0, None, 0x2000,
                                          0x3000, 0x4000, ctypes.byref(lay), 0x5002, 10, None)
    assert rs_misaligned == capi.CAP_ERR_INVALID_ARG
    small_out = capi._lib.cap_combine(ctypes.byref(t), 1, 0, 1, 128, 0x1000, 10, 0x2000, 0x3000, 0x4000,
                                      0x5000, ctypes.byref(lay), None, 0x6000, 63, None)
    assert small_out == capi.CAP_ERR_INVALID_ARG


def test_row_plan_and_ffn_combine_validation(capi):
    """The folded destination combine's calls reject bad arguments before
    launching anything."""
    t = _topo(capi)
    lay = capi.Layout(*([0x10000] * 10))
    plan = capi._lib.cap_row_plan
    by = ctypes.byref
    assert plan(by(t), 0, None, by(lay), 0x2000, 0x3000, 0x4000, 100, 100, None) == capi.CAP_ERR_INVALID_ARG
    assert plan(by(t), 4, 0x1000, by(lay), 0x2000, 0x3000, 0x4000, 100, 100, None) == capi.CAP_ERR_INVALID_ARG
    assert plan(by(t), 0, 0x1000, by(lay), 0x2000, 0x3001, 0x4000, 100, 100, None) == capi.CAP_ERR_INVALID_ARG
    assert plan(by(t), 0, 0x1000, by(lay), 0x2000, 0x3000, 0x4000, -1, 100, None) == capi.CAP_ERR_INVALID_ARG
    assert plan(by(t), 0, 0x1000, by(lay), 0x2000, 0x3000, None, 100, 100, None) == capi.CAP_ERR_INVALID_ARG
    f = capi._lib.cap_expert_ffn_combine
    B, F = capi.CAP_DTYPE_BF16, capi.CAP_DTYPE_F32
    head = (0x10000, 512, 0x20000, 0x30000, 0x40000, 0x50000, 0x60000, 0x70000)
    ws = (0x80000, 1 << 30, None, None)
    assert f(F, 4, 128, 256, 100, *head, 0x90000, 0xA0000, 0xB0000, 100, *ws) == capi.CAP_ERR_UNSUPPORTED
    assert f(B, 4, 2048, 768, 100, *head, None, 0xA0000, 0xB0000, 100, *ws) == capi.CAP_ERR_INVALID_ARG
    assert f(B, 4, 2048, 768, 100, *head, 0x90000, 0xA0000, 0xB0008, 100, *ws) == capi.CAP_ERR_INVALID_ARG
    assert f(B, 4, 2048, 768, 100, *head, 0x90000, 0xA0000, 0xB0000, -1, *ws) == capi.CAP_ERR_INVALID_ARG
    assert f(B, 4, 2000, 768, 100, *head, 0x90000, 0xA0000, 0xB0000, 100, *ws) == capi.CAP_ERR_UNSUPPORTED
    multi_no_w = capi._lib.cap_combine(by(t), capi.CAP_COMBINE_DEST_REDUCE_MULTI, 0, 1, 128, 0x1000, 10, 0x2000,
                                       None, 0x4000, 0x5000, by(lay), None, 0x6000, 63, None)
    assert multi_no_w == capi.CAP_ERR_INVALID_ARG


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_dispatch_layout_static_rejects_topologies_past_its_array(capi):
    """The allocation-free layout refuses, before touching the device, a
    topology whose workspace would not fit its fixed per-GPU array."""
    cap = capi.cap_dispatch_layout_static_max_bytes()
    assert cap == 4 << 20
    small = _topo(capi, E=128, R=8, ranks_per_node=8, T=32768, k=8)
    assert 0 < capi.cap_workspace_size(capi.CAP_OP_DISPATCH_LAYOUT, small) <= cap
    big = _topo(capi, E=256, R=64, ranks_per_node=8, T=64 * 16384, k=8)
    assert capi.cap_workspace_size(capi.CAP_OP_DISPATCH_LAYOUT, big) > cap
    lay = capi.Layout(*([0x9000] * 10))
    st = capi._lib.cap_dispatch_layout_static(ctypes.byref(big), 0x3000, 0x4000, 0x5000, ctypes.byref(lay), None)
    assert st == capi.CAP_ERR_WORKSPACE
    bad = _topo(capi, k=0)
    st = capi._lib.cap_dispatch_layout_static(ctypes.byref(bad), 0x3000, 0x4000, 0x5000, ctypes.byref(lay), None)
    assert st == capi.CAP_ERR_INVALID_ARG


@pytest.mark.parametrize("over", [dict(E=0), dict(E=300), dict(R=3), dict(R=65, E=130), dict(rpn=3),
                                  dict(c=0.5), dict(max_swaps=-1)])
def test_adjustment_rejects_bad_arguments(capi, over):
    kw = dict(E=16, R=4, rpn=2, c=5.0, max_swaps=4)
    kw.update(over)
    st = capi._lib.cap_adjustment_spectrum(0x1000, kw["E"], kw["R"], kw["rpn"], kw["c"], 0x2000, 0x3000,
                                           kw["max_swaps"], 0x4000, None, 0x5000, 0x6000, 1 << 20, None)
    assert st == capi.CAP_ERR_INVALID_ARG
    st = capi._lib.cap_adjustment_spectrum(0x1000, 16, 4, 2, 5.0, 0x2000, 0x3000, 4, 0x4000, None, 0x5000,
                                           0x6000, 16 * 16 * 8 - 1, None)
    assert st == capi.CAP_ERR_WORKSPACE


def test_route_layout_validation(capi):
    """The fused front end validates like the separate calls, and sizes its
    workspace for eight count rows per 256-token chunk plus co-activation."""
    t = _topo(capi, E=128, R=8, ranks_per_node=8, T=32768, k=8)
    need = capi.cap_workspace_size(capi.CAP_OP_ROUTE_LAYOUT, t)
    assert need > capi.cap_workspace_size(capi.CAP_OP_DISPATCH_LAYOUT, t)
    lay = capi.Layout(*([0x9000] * 10))
    f = capi._lib.cap_route_layout
    assert f(ctypes.byref(t), 0x3000, 0.3, 0x4000, 0x5000, 0x6000, 0x7000, ctypes.byref(lay), None, 0x10000,
             need - 1, None) == capi.CAP_ERR_WORKSPACE
    assert f(ctypes.byref(t), 0x3000, 1.0, 0x4000, 0x5000, 0x6000, 0x7000, ctypes.byref(lay), None, 0x10000,
             need, None) == capi.CAP_ERR_INVALID_ARG
    bad = _topo(capi, k=0)
    assert f(ctypes.byref(bad), 0x3000, 0.3, 0x4000, 0x5000, 0x6000, 0x7000, ctypes.byref(lay), None, 0x10000,
             need, None) == capi.CAP_ERR_INVALID_ARG
