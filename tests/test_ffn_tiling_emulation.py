"""CPU emulation of the bf16 expert FFN kernels' tile schedule and addresses.

The direct-to-LDS loads of the GEMM kernels form their global offsets in
inline assembly (32-bit per-lane offsets added to a scalar base), where an
index slip faults the GPU instead of failing a comparison.  This test replays,
in numpy, every index computation of the kernels for real call shapes and
checks it on the host:

* the tile schedule over ragged experts (row bounds clamped to the capacity,
  m-tiles per expert, the expert of an m-tile);
* the fused kernel's queues: the split of m-tiles over XCD queues and the
  grouped entry order (entry -> m-tile, n-tile) are bijections onto the tiles
  of each GEMM, and every ready counter index lies in the counter array;
* the two-kernel path's block -> worker map is a permutation;
* for every tile of both GEMMs, the first and last K stage of every direct load
  of every loader wave and lane: the global byte offset stays inside its
  operand (x or the expert-sorted rows, W1 / W3 / W2, H), fits in 32 bits, the
  24-bit multiplies stay below 2^24, and the LDS destination stays inside the
  two stage buffers;
* the epilogue's output rows and 8-column chunks stay inside H / Y.

Shapes: rank 0 and the last rank of the Qwen3-, DeepSeek-V2-Lite- and
DeepSeek-V3-shaped workloads (their routing from the oracle), the shared
experts, ragged synthetic experts (empty experts, one-row experts, capacity
cuts) and gathered rows at the 4 GiB limit of x.
"""
from __future__ import annotations

import numpy as np
import pytest

from tests import cases as C
from workloads import generator as gen

# kernel constants (expert_ffn.hip)
BM = BN = 256
STAGE_K = 64
ROW_B = STAGE_K * 2
ROWS_PER_LOAD = 1024 // ROW_B
NW, NL = 8, 4
ALD = BM // ROWS_PER_LOAD // NL
BLD = BN // ROWS_PER_LOAD // NL
BRUN = BLD // 2
STAGE_BYTES = (BM + BN) * ROW_B
STAGES = 2
WAVES_N = 2
WM, WN = 64, 128
MI, NJ = WM // 16, WN // 16          # 16 x 16 MFMA blocks per wave
GROUP_M = 4
N_XCC = 8
SYNC_READY = 8 * 32 + 32
MAX_E = 256

LANE = np.arange(64)
LD_ROW = LANE >> 3
_PC = LANE & 7


def _swz(r):
    return (r & 7) ^ ((r >> 3) & 1)


FR_ROW, FR_KC = LANE & 15, ((LANE >> 3) & 2) | (LANE >> 5)   # fragment reads: row, 16-byte K chunk
EP_C = 2 * ((LANE >> 4) & 1) + (LANE >> 5)          # epilogue: a lane's chunk within a pair's four


COL_B = np.stack([(_PC ^ _swz(LD_ROW)) * 16, (_PC ^ _swz(ROWS_PER_LOAD + LD_ROW)) * 16]).astype(np.int64)


def schedule(row_offsets, max_rows):
    ro = np.asarray(row_offsets, np.int64)
    base = ro[0]
    b = np.clip(ro[:-1] - base, 0, max_rows)
    e = np.maximum(b, np.clip(ro[1:] - base, 0, max_rows))
    mt = (e - b + BM - 1) // BM
    pref = np.concatenate([[0], np.cumsum(mt)])
    return b, e, pref


def tiles_of(pref, b, e, m):
    """expert, first row and valid rows of m-tiles m (find_expert + row bounds)."""
    E_loc = len(b)
    lo = np.zeros_like(m)
    hi = np.full_like(m, E_loc - 1)
    while np.any(lo < hi):                   # the kernel's binary search
        mid = (lo + hi + 1) >> 1
        go = pref[mid] <= m
        lo = np.where((lo < hi) & go, mid, lo)
        hi = np.where((lo < hi) & ~go, mid - 1, hi)
    l = lo
    row0 = b[l] + (m - pref[l]) * BM
    rows = np.minimum(BM, e[l] - row0)
    return l, row0, rows


def fused_queue_tiles(MT, n_gu, n_dn):
    """(gemm, m, nt) of every queue entry of every XCD queue, in queue order."""
    out = []
    for xs in range(N_XCC):
        mb = xs * MT // N_XCC
        MX = (xs + 1) * MT // N_XCC - mb
        for gu, nn in ((1, n_gu), (0, n_dn)):
            for u in range(MX * nn):
                g = u // (GROUP_M * nn)
                v = u - g * GROUP_M * nn
                gm = min(GROUP_M, MX - g * GROUP_M)
                out.append((gu, mb + g * GROUP_M + v % gm, v // gm))
    return out


def check_loads(gu, l, row0, rows, nt, K, N_rows_b, a_rows_cap, gathered, row_src, x_rows, inter, d):
    """Every direct load of the tiles (vectors over tiles) at stages 0 and KT-1."""
    pitch = K * 2
    blk = ROWS_PER_LOAD * pitch
    assert blk < (1 << 24) and pitch < (1 << 24)
    KT = K // STAGE_K
    for kt in (0, KT - 1):
        kb = kt * STAGE_K * 2
        for lw in range(NL):
            a_first = lw * ALD * ROWS_PER_LOAD
            for i in range(ALD):
                cb = COL_B[(lw * ALD + i) & 1]
                if gathered:
                    r = np.minimum(a_first + i * ROWS_PER_LOAD + LD_ROW[None, :], rows[:, None] - 1)
                    tok = np.clip(row_src[row0[:, None] + r], 0, x_rows - 1)
                    off = tok * pitch + cb[None, :] + kb
                    assert off.max() < (1 << 32)
                    assert off.min() >= 0 and off.max() + 16 <= x_rows * pitch
                else:
                    full = (a_first + ALD * ROWS_PER_LOAD) <= rows
                    r_full = a_first + i * ROWS_PER_LOAD + LD_ROW[None, :]
                    r_clamp = np.minimum(r_full, rows[:, None] - 1)
                    r = np.where(full[:, None], r_full, r_clamp)
                    assert np.all(r <= rows[:, None] - 1)
                    off = (row0[:, None] + r) * pitch + cb[None, :] + kb
                    assert off.min() >= 0 and off.max() + 16 <= a_rows_cap * pitch
                    # the 32-bit voffset inside the statement (relative to the tile's first row)
                    assert (i * blk + LD_ROW.max() * pitch + cb.max()) < (1 << 32)
                lds = (kt % STAGES) * STAGE_BYTES + lw * ALD * 1024 + i * 1024
                assert 0 <= lds and lds + 1024 <= STAGES * STAGE_BYTES
            for i in range(BLD):
                cb = COL_B[(lw * BLD + i) & 1]
                if gu:
                    first = l * inter + nt * (BN // 2) + lw * 32          # W1 and W3 runs
                    brow = first[:, None] + (i % BRUN) * ROWS_PER_LOAD + LD_ROW[None, :]
                else:
                    first = l * d + nt * BN + lw * BLD * ROWS_PER_LOAD + (i // BRUN) * 32
                    brow = first[:, None] + (i % BRUN) * ROWS_PER_LOAD + LD_ROW[None, :]
                off = brow * pitch + cb[None, :] + kb
                assert brow.min() >= 0 and brow.max() < N_rows_b
                assert off.max() + 16 <= N_rows_b * pitch
                lds = (kt % STAGES) * STAGE_BYTES + BM * ROW_B + lw * BLD * 1024 + i * 1024
                assert lds + 1024 <= STAGES * STAGE_BYTES


def check_stores(gu, row0, rows, nt, N_out, out_rows_cap):
    OUT_C = WN // 2 if gu else WN
    NP = OUT_C // 32
    for w in range(NW):
        wm, wn = w // WAVES_N, w % WAVES_N
        c0 = (nt * (BN // 2) if gu else nt * BN) + wn * OUT_C
        for i in range(MI):
            r = wm * WM + i * 16 + (LANE & 15)
            ok = r[None, :] < rows[:, None]
            grow = np.where(ok, row0[:, None] + r[None, :], 0)
            assert grow.max() < out_rows_cap
            for pr in range(NP):
                c = 4 * pr + EP_C
                col = c0[:, None] + 8 * c[None, :]
                assert col.min() >= 0 and col.max() + 8 <= N_out


def emulate_call(row_offsets, max_rows, d, inter, gathered=False, row_src=None, x_rows=0):
    E_loc = len(row_offsets) - 1
    b, e, pref = schedule(row_offsets, max_rows)
    MT = int(pref[-1])
    n_gu, n_dn = inter // (BN // 2), d // BN
    assert MT <= (max_rows + BM - 1) // BM + MAX_E      # ready counters fit the workspace
    if MT == 0:
        return 0
    # fused queues: bijection onto the tiles of each GEMM
    q = fused_queue_tiles(MT, n_gu, n_dn)
    for gu, nn in ((1, n_gu), (0, n_dn)):
        got = sorted((m, nt) for g, m, nt in q if g == gu)
        assert got == [(m, nt) for m in range(MT) for nt in range(nn)]
    assert max(m for _, m, _ in q) + SYNC_READY < SYNC_READY + (max_rows + BM - 1) // BM + MAX_E + 1
    # two-kernel path: block -> worker is a permutation for every grid size
    for G in (1, 3, 8, 200, 256):
        wid = [((bb % 8) * (G // 8) + bb // 8) if G % 8 == 0 else bb for bb in range(G)]
        assert sorted(wid) == list(range(G))
    if gathered:
        assert x_rows * d * 2 < (1 << 32)
        row_src = np.asarray(row_src, np.int64)
        assert len(row_src) >= max_rows
    for gu, nn, K, N_out, nb_rows in ((1, n_gu, d, inter, E_loc * inter), (0, n_dn, inter, d, E_loc * d)):
        m = np.repeat(np.arange(MT), nn)
        nt = np.tile(np.arange(nn), MT)
        l, row0, rows = tiles_of(pref, b, e, m)
        assert np.all(rows >= 1) and np.all(row0 + rows <= max_rows)
        check_loads(gu, l, row0, rows, nt, K, nb_rows, max_rows, gathered and gu == 1, row_src, x_rows, inter, d)
        check_stores(gu, row0, rows, nt, N_out, max_rows)
    return MT


def _rank_call(name, kind, p, rank):
    cfg = gen.CONFIGS[name]
    r, lay = C.oracle_routing(name, kind, p, 5.0)
    eo = lay["expert_offsets"].astype(np.int64)
    offs = eo[rank * cfg.E_loc:(rank + 1) * cfg.E_loc + 1]
    base = int(offs[0])
    n = int(offs[-1] - base)
    # row source of the rank (token of each expert-sorted row)
    sp = lay["slot_pos"].astype(np.int64)
    er, _ = C.placement(name, kind, p, 5.0)
    on = (r["keep"] == 1) & (er[r["idx"]] == rank)
    src = np.zeros(max(n, 1), np.int64)
    tt = np.repeat(np.arange(cfg.T), cfg.k).reshape(cfg.T, cfg.k)
    src[sp[on] - base] = tt[on]
    return cfg, offs, n, src


@pytest.mark.parametrize("name,kind,p", [("c2", "coact", 0.3), ("c2", "seq", 0.0), ("c3", "coact", 0.1),
                                         ("c4", "coact", 0.1), ("c5", "coact", 0.1), ("c5", "seq", 0.1)])
def test_workload_calls_in_bounds(name, kind, p):
    cfg0 = gen.CONFIGS[name]
    for rank in (0, cfg0.R - 1):
        cfg, offs, n, src = _rank_call(name, kind, p, rank)
        cap = cfg.T * min(cfg.k, cfg.E_loc)                  # the layer's row capacity
        src_cap = np.zeros(cap, np.int64)
        src_cap[:len(src)] = src
        for max_rows in (cap, max(n, 1)):
            emulate_call(offs, max_rows, cfg.d, cfg.inter)
            emulate_call(offs, max_rows, cfg.d, cfg.inter, gathered=True, row_src=src_cap, x_rows=cfg.T)
        if cfg.n_shared:
            T_loc = cfg.tokens_per_rank
            emulate_call([0, T_loc], T_loc, cfg.d, cfg.n_shared * cfg.shared_inter)


@pytest.mark.parametrize("counts,max_rows,d,inter", [
    ([300, 1, 0, 513], 814, 512, 384),
    ([0, 0, 700, 40, 1000, 3], 1743, 256, 128),
    ([2000, 0, 3000, 1, 4000], 8292, 256, 128),          # capacity cuts the last expert
    ([1] * 256, 8300, 256, 128),                          # 256 experts of one row
    ([9000], 8192, 256, 256),                             # one expert past the capacity
    ([3000, 4000, 700], 8300, 512, 256),
    ([0, 0, 0], 9000, 256, 128),                          # no rows
])
def test_ragged_calls_in_bounds(counts, max_rows, d, inter):
    offs = np.concatenate([[0], np.cumsum(counts)])
    rng = np.random.default_rng(len(counts))
    x_rows = max_rows + 37
    src = rng.integers(-5, x_rows + 5, size=max_rows)       # out-of-range sources are clamped
    emulate_call(offs, max_rows, d, inter)
    emulate_call(offs, max_rows, d, inter, gathered=True, row_src=src, x_rows=x_rows)
    # a non-zero first offset (a rank's slice of the global offsets)
    emulate_call(offs + 12345, max_rows, d, inter)


def test_gathered_rows_at_the_4gib_limit():
    """x of 2^20 - 1 rows of d = 2048 bf16 (4 GiB - 4 KiB, the largest the C
    ABI accepts): byte offsets of rows near the end exceed 2^31 and stay below
    2^32."""
    d, inter = 2048, 768
    x_rows = (1 << 20) - 1
    counts = [5000, 4000, 3000]
    max_rows = sum(counts)
    rng = np.random.default_rng(3)
    src = x_rows - 1 - rng.integers(0, 20000, size=max_rows)
    src[-1] = x_rows - 1
    emulate_call(np.concatenate([[0], np.cumsum(counts)]), max_rows, d, inter, gathered=True,
                 row_src=src, x_rows=x_rows)
    assert (x_rows - 1) * d * 2 > (1 << 31)


def test_queue_order_groups_m_tiles():
    """The grouped order: the first CUs-per-XCD entries of a queue cover
    GROUP_M m-tiles x (32 / GROUP_M) n-tiles when there are enough of both."""
    q = fused_queue_tiles(8 * 16, 16, 28)
    first = q[:32]
    assert len({m for _, m, _ in first}) == GROUP_M
    assert len({nt for _, _, nt in first}) == 32 // GROUP_M


def test_combine_plan_indices_in_bounds():
    """The combine plan's indices (cap_expert_ffn_combine): every storer lane's
    LDS table slot, every epilogue read of the table (own rows and staged
    rows) lies in [0, BM); a receive row is used only when it lies in
    [0, parts_rows) (the kernel's unsigned compare), and then every 16-byte
    store of the row lies inside parts; other rows go to Y as before."""
    lane = np.arange(64)
    # table writes: storer waves NL..NW-1, one row per lane
    q = np.concatenate([(w - NL) * 64 + lane for w in range(NL, NW)])
    assert q.min() == 0 and q.max() == BM - 1 and len(set(q.tolist())) == BM
    # own-row reads (storer waves) and staged-row reads (storer w reads loader w - NL's rows)
    for w in range(NW):
        wm = w // WAVES_N
        r = np.arange(MI)[:, None] * 16 + (lane & 15)[None, :]
        assert (wm * WM + r).min() >= 0 and (wm * WM + r).max() < BM
    for gu, out_rb in ((0, (WN) * 2),):
        rows_per_read = 1024 // out_rb
        for w in range(NL, NW):
            lw = w - NL
            lwm = lw // WAVES_N
            r = np.arange(0, WM, rows_per_read)[:, None] + (lane // (out_rb // 16))[None, :]
            assert (lwm * WM + r).max() < BM
    # receive rows: the unsigned compare keeps [0, parts_rows); stores stay in parts
    d = 7168
    for parts_rows in (0, 1, 1000):
        dst = np.array([-1, 0, parts_rows - 1, parts_rows, 2 ** 31 - 1], np.int64)
        used = (dst.astype(np.uint32) < np.uint32(parts_rows)) if parts_rows > 0 else np.zeros(len(dst), bool)
        for nt in range(d // BN):
            for wn in range(WAVES_N):
                c0 = nt * BN + wn * WN
                chunks = c0 + 8 * np.arange(WN // 8)
                for v in dst[used]:
                    assert 0 <= v < parts_rows
                    assert v * d + chunks.max() + 8 <= parts_rows * d


def test_fragment_reads_inside_the_stage():
    """k_step's LDS fragment reads (K steps 0 and 1 of either stage buffer):
    every A read lies in the stage's A rows, every B read in its B rows, at a
    16-byte chunk of the 128-byte row; each lane group's 8 K values are one
    chunk and the four groups cover the step's four chunks.  Banks (64 banks
    of 4 bytes, a 256-byte window, two 128-byte rows): the 16 lanes of one
    group, and lanes 8k .. 8k + 7 together with 8k + 32 .. 8k + 39 (the pairs
    one pass of a 16-byte read serves), hit 16 distinct 16-byte bank slots."""
    for st in range(STAGES):
        for ks in range(2):
            pc = ((4 * ks + FR_KC) ^ _swz(FR_ROW)) * 16
            logical = (pc // 16) ^ _swz(FR_ROW)
            for g in range(4):
                assert len(set(logical[16 * g:16 * g + 16].tolist())) == 1
            assert sorted(set(logical.tolist())) == list(range(4 * ks, 4 * ks + 4))
            assert pc.min() >= 0 and pc.max() + 16 <= ROW_B
            for w in range(NW):
                wm, wn = w // WAVES_N, w % WAVES_N
                for i in range(MI):
                    off = st * STAGE_BYTES + (wm * WM + i * 16 + FR_ROW) * ROW_B + pc
                    assert off.min() >= st * STAGE_BYTES and off.max() + 16 <= st * STAGE_BYTES + BM * ROW_B
                for j in range(NJ):
                    off = st * STAGE_BYTES + (BM + wn * WN + j * 16 + FR_ROW) * ROW_B + pc
                    assert off.min() >= st * STAGE_BYTES + BM * ROW_B
                    assert off.max() + 16 <= (st + 1) * STAGE_BYTES
            slot = (FR_ROW & 1) * 8 + pc // 16            # 16-byte slot in the 256-byte window
            for g in range(4):
                assert len(set(slot[16 * g:16 * g + 16].tolist())) == 16
            for k in range(4):
                lanes = np.r_[8 * k:8 * k + 8, 8 * k + 32:8 * k + 40]
                assert len(set(slot[lanes].tolist())) == 16


def _permlane16_swap(x, y):
    """v_permlane16_swap on 64-lane values: rows of 16 lanes; odd rows of the
    first operand trade places with even rows of the second."""
    x, y = x.copy(), y.copy()
    for lo in (0, 32):
        a, b = slice(lo + 16, lo + 32), slice(lo, lo + 16)
        x[a], y[b] = y[b].copy(), x[a].copy()
    return x, y


@pytest.mark.parametrize("gu", [True, False])
def test_epilogue_lane_layout_writes_each_output_once(gu):
    """The epilogue's register-to-column map (store_tile): with the 16 x 16
    MFMA output layout (lane (r, q) holds columns 4 q + 0..3 of row r of each
    block, the weight fragment being the first operand), the permlane16_swap of
    a block pair and the chunk index 4 pr + EP_C put every output column of
    every row of the wave tile in exactly one 16-byte piece, at its own column;
    for gate/up, each H column takes the gate from W1 block 4 pr + {0, 1} and
    the up value from W3 block 4 pr + {2, 3} of the same B rows (the B tile
    interleaves 32-row blocks of W1 and W3)."""
    OUT_C = WN // 2 if gu else WN
    NP = OUT_C // 32
    r16, q = LANE & 15, LANE >> 4
    # B-tile rows (wave-relative) that are W1 (gate) or W3 (up), and their H column
    b_rows = np.arange(WN)
    is_w3 = (b_rows // 32) % 2 == 1
    h_col = (b_rows // 64) * 32 + b_rows % 32
    seen = np.zeros((MI * 16, OUT_C), np.int64)
    for i in range(MI):
        for pr in range(NP):
            pieces = []
            for half in (0, 1):                     # packed pairs (e = 0, 1) and (e = 2, 3)
                blocks = [4 * pr + 0, 4 * pr + 1] if gu else [2 * pr + 0, 2 * pr + 1]
                # each packed value is tagged with the B row of its first element
                x = 16 * blocks[0] + 4 * q + 2 * half
                y = 16 * blocks[1] + 4 * q + 2 * half
                pieces.append(_permlane16_swap(x, y))
            (ra0, ra1), (rb0, rb1) = pieces
            o = np.stack([ra0, rb0, ra1, rb1], 1)   # four packed pairs = 8 columns
            c = 4 * pr + EP_C
            for lane in range(64):
                row = i * 16 + r16[lane]
                for t in range(4):
                    src = o[lane, t]
                    for k in range(2):
                        b = src + k
                        col = 8 * c[lane] + 2 * t + k
                        if gu:
                            assert not is_w3[b] and h_col[b] == col
                            assert is_w3[b + 32] and h_col[b + 32] == col    # its up partner block
                        else:
                            assert b == col
                        seen[row, col] += 1
    assert np.all(seen == 1)
