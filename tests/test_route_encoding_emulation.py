"""CPU emulation of two pieces of integer/float arithmetic the routing kernels
rely on, checked against their plain definitions on the host.

* The selection key (route_device.hpp, pack_key): a (logit x, expert e) pair
  becomes the fp64 whose high word holds the bits of x + 0.0f and whose low
  word holds 255 - e, all 32 bits complemented when x is negative.  The
  kernels select and order the top k by fp64 max / min on these keys, so fp64
  order on the keys must be the selection order of the definition (Eq. 1's top
  k): logit descending, -0.0 equal to +0.0, ties to the lower expert id.  The
  expert and the logit must come back out of a key unchanged.
* The small quotient (cap_device.hpp, small_quotient): floor(n / d) from the
  fp32 estimate n * rcp(d), truncated, then one correction step each way.  The
  hardware reciprocal is within one ulp of 1/d, so the emulation tries the
  correctly rounded reciprocal and its two neighbours.

Both are emulated in numpy with the kernels' operations, none of the
kernels' code.
"""
from __future__ import annotations

import numpy as np


def pack_keys(x: np.ndarray, e: np.ndarray) -> np.ndarray:
    hi = (x.astype(np.float32) + np.float32(0.0)).view(np.uint32).astype(np.uint64)
    sm = ((hi >> np.uint64(31)) * np.uint64(0xFFFFFFFF)).astype(np.uint64)      # 0 or all ones
    lo = sm ^ (np.uint64(255) - e.astype(np.uint64))
    return ((hi << np.uint64(32)) | lo).view(np.float64)


def key_expert(k: np.ndarray) -> np.ndarray:
    b = k.view(np.uint64)
    sm = ((b >> np.uint64(63)) * np.uint64(0xFFFFFFFF)).astype(np.uint64)
    lo = (b & np.uint64(0xFFFFFFFF)) ^ sm
    return (255 - (lo & np.uint64(255))).astype(np.int64)


def key_logit(k: np.ndarray) -> np.ndarray:
    return (k.view(np.uint64) >> np.uint64(32)).astype(np.uint32).view(np.float32)


def _value_pool(rng):
    tiny = np.array([1e-45, 3e-45, 1e-40, 1e-38, 1.1754944e-38], np.float32)
    huge = np.array([3.4028235e38, 1e38, 8.5e37, 1e30], np.float32)
    return np.concatenate([tiny, -tiny, huge, -huge, np.float32([0.0, -0.0, 1.0, -1.0, 0.5, -0.5]),
                           rng.standard_normal(16).astype(np.float32),
                           (rng.standard_normal(8) * 1e-3).astype(np.float32)])


def test_selection_key_order_is_the_selection_order():
    rng = np.random.default_rng(7)
    pool = _value_pool(rng)
    for trial in range(200):
        E = int(rng.integers(1, 257))
        x = rng.choice(pool, size=E)                 # heavy ties, +-0, subnormals, extremes
        e = np.arange(E)
        keys = pack_keys(x, e)
        assert np.all(np.isfinite(keys)), trial
        # definition: logit descending (-0 == +0), then expert ascending
        xf = x + np.float32(0.0)
        want = np.lexsort((e, -xf.astype(np.float64)))
        got = np.argsort(-keys, kind="stable")
        assert np.array_equal(got, want), trial
        assert np.unique(keys).size == E              # no two pairs share a key
        assert np.array_equal(key_expert(keys), e)
        assert np.array_equal(key_logit(keys).view(np.uint32), xf.view(np.uint32))
        assert np.all(keys > -np.inf)                 # the empty key sorts below every key


def test_selection_key_ties_across_zero_and_sign():
    # equal logits on both sides of zero, and the two zeros
    e = np.arange(6)
    for v in (np.float32(2.5), np.float32(-2.5), np.float32(1e-45), np.float32(-1e-45)):
        keys = pack_keys(np.full(6, v, np.float32), e)
        assert np.array_equal(np.argsort(-keys, kind="stable"), e)   # lower expert first
    x = np.float32([-0.0, 0.0, -0.0, 0.0])
    keys = pack_keys(x, np.arange(4))
    assert np.array_equal(np.argsort(-keys, kind="stable"), np.arange(4))
    x = np.float32([-1e-45, 0.0, 1e-45, -0.0])
    keys = pack_keys(x, np.arange(4))
    assert np.array_equal(np.argsort(-keys, kind="stable"), [2, 1, 3, 0])


def small_quotient(n: np.ndarray, d: np.ndarray, rcp: np.ndarray) -> np.ndarray:
    q = (n.astype(np.float32) * rcp).astype(np.float64)
    q = np.trunc(q).astype(np.int64)
    r = n.astype(np.int64) - q * d.astype(np.int64)
    return q + (r >= d) - (r < 0)


def _rcp_variants(d):
    r = (np.float32(1.0) / d.astype(np.float32)).astype(np.float32)
    return [r, np.nextafter(r, np.float32(0)), np.nextafter(r, np.float32(np.inf))]


def test_small_quotient_is_floor_division():
    # device and node indices: n < 4096, d <= 64
    n = np.arange(4096, dtype=np.int64)
    for d0 in range(1, 65):
        d = np.full_like(n, d0)
        for rcp in _rcp_variants(d):
            assert np.array_equal(small_quotient(n, d, rcp), n // d), d0
    # token -> source rank: n < 2^31, quotient below 2^16
    rng = np.random.default_rng(3)
    d = rng.integers(1, 1 << 31, size=200_000, dtype=np.int64)
    qmax = np.minimum((1 << 16) - 1, ((1 << 31) - 1) // d)
    q = (rng.random(d.size) * (qmax + 1)).astype(np.int64)
    n = np.minimum(q * d + rng.integers(0, 1 << 31, size=d.size) % d, (1 << 31) - 1)
    edge = np.minimum(q * d, (1 << 31) - 1)                 # exact multiples and their neighbours
    for nn in (n, edge, np.maximum(edge - 1, 0)):
        for rcp in _rcp_variants(d):
            assert np.array_equal(small_quotient(nn, d, rcp), nn // d)
