"""cap_dispatch_layout_static (the allocation-free layout) against
cap_dispatch_layout on the same routing, through the C ABI: bit-identical
outputs on two calls in a row, the second with a smaller input, so the fixed
per-GPU array's leftovers from the first call must not leak into the second."""
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

NAMES = ("send_counts", "send_offsets", "recv_offsets", "recv_token", "expert_counts", "expert_offsets",
         "slot_pos", "copy_row", "vol", "totals")


def _routed(name, kind, p):
    cfg = dataclasses.replace(gen.CONFIGS[name], d=8)
    er, el = C.placement(name, kind, p, 5.0)
    L = DeviceLayer(cfg, C.logits(name), np.zeros((cfg.T, 8), np.uint16), er, el, p, 5.0, row_cap=8, recv_cap=8)
    L.route()
    return L


def _static_layout(L):
    """A second set of layout buffers filled by the allocation-free call."""
    out = {n: torch.full_like(t, -7) for n, t in L.lay_t.items()}
    lay = capi.make_layout(out)
    capi.cap_dispatch_layout_static(L.topo, L.idx, L.keep, L.mask, lay)
    return out


@pytest.mark.parametrize("first,second", [(("c5", "coact", 0.1), ("c2", "coact", 0.3)),
                                          (("c2", "seq", 0.0), ("c1", "seq", 0.3))])
def test_static_layout_matches_workspace_layout(first, second):
    for name, kind, p in (first, second):
        L = _routed(name, kind, p)
        got = _static_layout(L)
        L.layout()                                   # the existing entry point, own workspace
        torch.cuda.synchronize()
        n_recv = int(L.lay_t["recv_offsets"][-1].item())
        for n in NAMES:
            a, b = got[n].cpu().numpy(), L.lay_t[n].cpu().numpy()
            if n == "recv_token":
                a, b = a[:n_recv], b[:n_recv]
            assert np.array_equal(a, b), (name, n)
        # and against the oracle
        r, lay = C.oracle_routing(name, kind, p, 5.0)
        assert np.array_equal(got["slot_pos"].cpu().numpy(), lay["slot_pos"]), name
        assert np.array_equal(got["totals"].cpu().numpy(), lay["totals"]), name
