// Kernels of the device-centric all-to-all layout, shared by the layout call
// and the fused front end (see dispatch_layout.hip for the method).
#pragma once

#include "cap_device.hpp"

namespace cap {
namespace {


constexpr int kChunk = 256;        // tokens per chunk = threads per block
constexpr int kWavesPerChunk = kChunk / kWave;
constexpr int kMaxW = kMaxE + kMaxR;

// C chunks of up to kChunk tokens within one source rank (cpr per rank); the
// per-chunk counts may come in `sub` partial rows per chunk (Cs = C * sub rows
// of the workspace), each counting a consecutive part of the chunk.
struct Geom {
    int T, E, k, R, rpn, tpr, E_loc, cpr, C, W, sub, Cs;
};

struct Workspace {
    int32_t* part;     // [Cs][W]
    int32_t* coltot;   // [W]
    int64_t* volpart;  // [Cs][4]
};

inline size_t align256(size_t b) { return (b + 255) & ~static_cast<size_t>(255); }

__device__ __forceinline__ void chunk_range(const Geom& g, int c, int& t0, int& t1, int& src) {
    src = c / g.cpr;
    t0 = src * g.tpr + (c % g.cpr) * kChunk;
    t1 = min(t0 + kChunk, (src + 1) * g.tpr);
}

// Slot position r * E_loc + l of an expert on rank r at local index l, or -1
// when the placement entry is out of range.
__device__ __forceinline__ int slot_position_of(int r, int l, const Geom& g) {
    const bool ok = (static_cast<unsigned>(r) < static_cast<unsigned>(g.R)) &
                    (static_cast<unsigned>(l) < static_cast<unsigned>(g.E_loc));
    return ok ? r * g.E_loc + l : -1;
}
// Both table entries are read before either is tested, so the two loads are
// in flight together.
__device__ __forceinline__ int slot_position(const int32_t* er, const int32_t* el, int e, const Geom& g) {
    if (static_cast<unsigned>(e) >= static_cast<unsigned>(g.E)) return -1;
    return slot_position_of(er[e], el[e], g);
}

__device__ __forceinline__ uint64_t device_bits(uint64_t m, int R) {
    return R >= 64 ? m : (m & ((1ull << R) - 1));
}

// Slot positions (-1 when pruned or invalid) and device mask of token t.
__device__ __forceinline__ void load_token(const Geom& g, int t, const int32_t* __restrict__ idx,
                                           const uint8_t* __restrict__ keep, const uint64_t* __restrict__ mask,
                                           const int* pos_lds, int (&P)[kMaxK], uint64_t& m) {
    int e[kMaxK];
    uint8_t kp[kMaxK];
    // every slot loaded unconditionally (slots past k reload slot k - 1 and are
    // dropped below), so all the loads go out before the first wait
    const size_t q0 = static_cast<size_t>(t) * g.k;
#pragma unroll
    for (int s = 0; s < kMaxK; ++s) {
        const size_t q = q0 + min(s, g.k - 1);
        e[s] = idx[q];
        kp[s] = keep[q];
    }
    m = device_bits(mask[t], g.R);
#pragma unroll
    for (int s = 0; s < kMaxK; ++s)
        P[s] = (kp[s] && s < g.k && static_cast<unsigned>(e[s]) < static_cast<unsigned>(g.E)) ? pos_lds[e[s]] : -1;
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

// Exclusive scan over the 256 threads of a block; *total gets the sum.
template <int NW = kWavesPerChunk>
__device__ __forceinline__ int block_exclusive_scan(int v, int* wsum, int* total) {
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    int inc = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int n = __shfl_up(inc, off);
        if (lane >= off) inc += n;
    }
    if (lane == kWave - 1) wsum[wave] = inc;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        if (w < wave) before += wsum[w];
        all += wsum[w];
    }
    __syncthreads();
    *total = all;
    return before + inc - v;
}

// ---------------------------------------------------------------- 1. count
__global__ __launch_bounds__(kChunk) void layout_count_kernel(
    Geom g, const int32_t* __restrict__ idx, const uint8_t* __restrict__ keep,
    const uint64_t* __restrict__ mask, const int32_t* __restrict__ er, const int32_t* __restrict__ el,
    Workspace ws, uint8_t* __restrict__ vol) {
    // one partial row per chunk (sub == 1)
    __shared__ int cnt[kMaxW];
    __shared__ int pos_lds[kMaxE];
    __shared__ int vsum[kWavesPerChunk][4];
    for (int i = threadIdx.x; i < g.W; i += kChunk) cnt[i] = 0;
    for (int e = threadIdx.x; e < g.E; e += kChunk) pos_lds[e] = slot_position(er, el, e, g);
    __syncthreads();

    int t0, t1, src;
    chunk_range(g, blockIdx.x, t0, t1, src);
    const int t = t0 + threadIdx.x;
    int v[4] = {0, 0, 0, 0};       // n_dev, n_intra_remote, n_inter, n_nodes
    if (t < t1) {
        int P[kMaxK];
        uint64_t m;
        load_token(g, t, idx, keep, mask, pos_lds, P, m);
#pragma unroll
        for (int s = 0; s < kMaxK; ++s)
            if (P[s] >= 0) atomicAdd(&cnt[P[s]], 1);
        const int src_node = src / g.rpn;
        uint64_t nodes = 0;
        for (uint64_t b = m; b; b &= b - 1) {
            const int d = __ffsll(static_cast<unsigned long long>(b)) - 1;
            atomicAdd(&cnt[g.E + d], 1);
            ++v[0];
            const int nd = d / g.rpn;
            if (nd != src_node) ++v[2];
            else if (d != src) ++v[1];
            nodes |= 1ull << nd;
        }
        v[3] = __popcll(nodes);
        reinterpret_cast<uint32_t*>(vol)[t] = static_cast<uint32_t>(v[0]) | (static_cast<uint32_t>(v[1]) << 8) |
                                              (static_cast<uint32_t>(v[2]) << 16) | (static_cast<uint32_t>(v[3]) << 24);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int s = wave_sum(v[j]);
        if (lane_id() == 0) vsum[threadIdx.x / kWave][j] = s;
    }
    __syncthreads();
    int32_t* out = ws.part + static_cast<size_t>(blockIdx.x) * g.W;
    for (int i = threadIdx.x; i < g.W; i += kChunk) out[i] = cnt[i];
    if (threadIdx.x < 4) {
        int64_t s = 0;
#pragma unroll
        for (int w = 0; w < kWavesPerChunk; ++w) s += vsum[w][threadIdx.x];
        ws.volpart[blockIdx.x * 4 + threadIdx.x] = s;
    }
}

// ---------------------------------------------------------------- 2. colscan
constexpr int kScanBatch = 8;

// Column scan, block bid of g.W + 1: one block of NT threads per column scans
// it over the Cs partial rows (in place: counts -> exclusive bases) and writes
// its total; block g.W sums the volumes.  When a thread's rows fit one batch
// (Cs <= 8 NT) they are read once, clamped rather than tested, so the block
// waits for one round of loads.
template <int NT>
__device__ __forceinline__ void layout_colscan_block(const Geom& g, const Workspace& ws, int64_t* __restrict__ totals,
                                                     int bid) {
    constexpr int NW = NT / kWave;
    __shared__ int wsum[NW];
    if (bid == g.W) {
        // volume totals: wave j < 4 sums column j of volpart
        const int j = threadIdx.x / kWave;
        if (j >= 4) return;
        int64_t s = 0;
        for (int c = lane_id(); c < g.Cs; c += kWave) s += ws.volpart[c * 4 + j];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
        if (lane_id() == 0) totals[j] = s;
        return;
    }
    const int col = bid;
    const int per = (g.Cs + NT - 1) / NT;                 // partial rows per thread, consecutive
    const int c0 = min(g.Cs, static_cast<int>(threadIdx.x) * per);
    const int c1 = min(g.Cs, c0 + per);
    int total;
    if (per <= kScanBatch) {
        int x[kScanBatch];
#pragma unroll
        for (int i = 0; i < kScanBatch; ++i) {
            x[i] = ws.part[static_cast<size_t>(min(c0 + i, g.Cs - 1)) * g.W + col];
            if (c0 + i >= c1) x[i] = 0;
        }
        int mine = 0;
#pragma unroll
        for (int i = 0; i < kScanBatch; ++i) mine += x[i];
        int run = block_exclusive_scan<NW>(mine, wsum, &total);
#pragma unroll
        for (int i = 0; i < kScanBatch; ++i) {
            if (c0 + i < c1) ws.part[static_cast<size_t>(c0 + i) * g.W + col] = run;
            run += x[i];
        }
    } else {
        int mine = 0;
        for (int b = c0; b < c1; b += kScanBatch) {
            int x[kScanBatch];
#pragma unroll
            for (int i = 0; i < kScanBatch; ++i)
                x[i] = (b + i < c1) ? ws.part[static_cast<size_t>(b + i) * g.W + col] : 0;
#pragma unroll
            for (int i = 0; i < kScanBatch; ++i) mine += x[i];
        }
        int run = block_exclusive_scan<NW>(mine, wsum, &total);
        for (int b = c0; b < c1; b += kScanBatch) {
            int x[kScanBatch];
#pragma unroll
            for (int i = 0; i < kScanBatch; ++i)
                x[i] = (b + i < c1) ? ws.part[static_cast<size_t>(b + i) * g.W + col] : 0;
#pragma unroll
            for (int i = 0; i < kScanBatch; ++i) {
                if (b + i < c1) ws.part[static_cast<size_t>(b + i) * g.W + col] = run;
                run += x[i];
            }
        }
    }
    if (threadIdx.x == 0) ws.coltot[col] = total;
}

__global__ __launch_bounds__(kChunk) void layout_colscan_kernel(Geom g, Workspace ws, int64_t* __restrict__ totals) {
    layout_colscan_block<kChunk>(g, ws, totals, blockIdx.x);
}

// ---------------------------------------------------------------- 3. scatter
// Exclusive scans of two values over the 256 threads of a block in one pass;
// *total_a / *total_b get the sums.
__device__ __forceinline__ void block_exclusive_scan2(int a, int b, int (*wsum)[kWavesPerChunk], int& ea, int& eb,
                                                      int* total_a, int* total_b) {
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    int ia = a, ib = b;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int na = __shfl_up(ia, off), nb = __shfl_up(ib, off);
        if (lane >= off) {
            ia += na;
            ib += nb;
        }
    }
    if (lane == kWave - 1) {
        wsum[0][wave] = ia;
        wsum[1][wave] = ib;
    }
    __syncthreads();
    int before_a = 0, before_b = 0, all_a = 0, all_b = 0;
#pragma unroll
    for (int w = 0; w < kWavesPerChunk; ++w) {
        if (w < wave) {
            before_a += wsum[0][w];
            before_b += wsum[1][w];
        }
        all_a += wsum[0][w];
        all_b += wsum[1][w];
    }
    __syncthreads();
    *total_a = all_a;
    *total_b = all_b;
    ea = before_a + ia - a;
    eb = before_b + ib - b;
}

// Scatter of chunk bid (one block of kChunk threads per chunk).  Every global
// load that does not depend on another is issued first, so the block waits
// for one round of memory latency before its LDS work: the placement tables,
// the column totals, the chunk's column bases, the token's slots and mask, and
// in block 0 the rank-boundary bases that give send_counts (send_offsets then
// come from one block scan over the (s, d) pairs).
constexpr int kSendPerThread = kMaxR * kMaxR / kChunk;   // (s, d) pairs per thread in block 0
static_assert(kMaxR * kMaxR % kChunk == 0, "send-count pairs split evenly over the block");

__device__ __forceinline__ void layout_scatter_block(
    const Geom& g, const int32_t* __restrict__ idx, const uint8_t* __restrict__ keep,
    const uint64_t* __restrict__ mask, const int32_t* __restrict__ er, const int32_t* __restrict__ el,
    const Workspace& ws, int32_t* __restrict__ send_counts, int32_t* __restrict__ send_offsets,
    int32_t* __restrict__ recv_offsets, int32_t* __restrict__ expert_counts,
    int32_t* __restrict__ expert_offsets, int32_t* __restrict__ slot_pos,
    int32_t* __restrict__ copy_row, int32_t* __restrict__ recv_token, int bid) {
    __shared__ unsigned long long bits[kWavesPerChunk][kMaxW];
    __shared__ int32_t pre[kWavesPerChunk][kMaxW];
    __shared__ int pos_lds[kMaxE];
    __shared__ int32_t gbase[kMaxW];
    __shared__ int32_t roff[kMaxR + 1];
    __shared__ int wsum[2][kWavesPerChunk];
    __shared__ int32_t sc_lds[kMaxR * kMaxR];
    const int i = threadIdx.x;                  // E <= 256 = kChunk threads
    const int wave = i / kWave;

    // ---- one round of independent loads (indices clamped rather than tested,
    // so that no branch splits the loads and they all go out before the first
    // wait; what a clamped lane loaded is dropped after the wait)
    const int32_t* cb = ws.part + static_cast<size_t>(bid) * g.sub * g.W;     // the chunk's first partial row
    const int ie = min(i, g.E - 1), ir = min(i, g.R - 1);
    int er_i = er[ie], el_i = el[ie], tot_e = ws.coltot[ie], cb_e = cb[ie];
    int tot_d = ws.coltot[g.E + ir], cb_d = cb[g.E + ir];
    int t0, t1, src;
    chunk_range(g, bid, t0, t1, src);
    const int t = t0 + i;
    const bool live = t < t1;
    const int tc = min(t, t1 - 1);              // chunks are never empty
    int e_raw[kMaxK];
    uint8_t kp_raw[kMaxK];
    {
        const size_t q0 = static_cast<size_t>(tc) * g.k;
#pragma unroll
        for (int s = 0; s < kMaxK; ++s) {
            const size_t q = q0 + min(s, g.k - 1);
            e_raw[s] = idx[q];
            kp_raw[s] = keep[q];
        }
    }
    const uint64_t m_raw = mask[tc];
    // block 0: send_counts[s][d] = rows of column E + d from the chunks of rank
    // s = (base at rank s + 1's first chunk, or the total) - (base at rank s's)
    // (thread i takes the consecutive pairs q = i * kSendPerThread + j, those
    // past R * R clamped to the last one)
    int sc_hi[kSendPerThread], sc_lo[kSendPerThread];
    if (bid == 0) {
#pragma unroll
        for (int j = 0; j < kSendPerThread; ++j) {
            const int q = min(i * kSendPerThread + j, g.R * g.R - 1);
            const int s = small_quotient(q, g.R), d = q - s * g.R;
            const int32_t* lp = ws.part + static_cast<size_t>(s * g.cpr * g.sub) * g.W + g.E + d;
            const int32_t* hp = (s + 1 < g.R) ? lp + static_cast<size_t>(g.cpr * g.sub) * g.W : ws.coltot + g.E + d;
            sc_hi[j] = *hp;
            sc_lo[j] = *lp;
        }
    }

    // ---- LDS work
#pragma unroll
    for (int w = 0; w < kWavesPerChunk; ++w)
        for (int c = i; c < g.W; c += kChunk) bits[w][c] = 0ull;
    if (i >= g.E) tot_e = 0;
    if (i >= g.R) tot_d = 0;
#pragma unroll
    for (int s = 0; s < kMaxK; ++s)
        if (!live || s >= g.k) {
            e_raw[s] = -1;
            kp_raw[s] = 0;
        }
    const uint64_t m = live ? device_bits(m_raw, g.R) : 0ull;
    if (i < g.E) {
        const bool ok = (static_cast<unsigned>(er_i) < static_cast<unsigned>(g.R)) &
                        (static_cast<unsigned>(el_i) < static_cast<unsigned>(g.E_loc));
        pos_lds[i] = ok ? er_i * g.E_loc + el_i : -1;
    }
    // expert offsets (slot-position order) and receive offsets from the column totals
    int eoff, doff, rows_total, recv_total;
    block_exclusive_scan2(tot_e, tot_d, wsum, eoff, doff, &rows_total, &recv_total);
    if (i < g.E) gbase[i] = cb_e + eoff;
    if (i < g.R) {
        gbase[g.E + i] = cb_d;
        roff[i] = doff;
    }
    if (i == 0) roff[g.R] = recv_total;
    if (bid == 0) {
        if (i < g.E) {
            expert_counts[i] = tot_e;
            expert_offsets[i] = eoff;
        }
        if (i == 0) expert_offsets[g.E] = rows_total;
        if (i < g.R) recv_offsets[i] = doff;
        if (i == 0) recv_offsets[g.R] = recv_total;
        // send_offsets[s][d] = sum of send_counts[s][d'] over d' < d: the
        // exclusive scan over all pairs in row-major order, less its value at
        // the row's first pair
        const int nq = g.R * g.R;
        int sc[kSendPerThread];
#pragma unroll
        for (int j = 0; j < kSendPerThread; ++j) sc[j] = sc_hi[j] - sc_lo[j];
        int local[kSendPerThread];
        int mine = 0;
#pragma unroll
        for (int j = 0; j < kSendPerThread; ++j) {
            local[j] = mine;
            mine += (i * kSendPerThread + j < nq) ? sc[j] : 0;
        }
        int all;
        const int base = block_exclusive_scan(mine, wsum[0], &all);
#pragma unroll
        for (int j = 0; j < kSendPerThread; ++j) {
            const int q = i * kSendPerThread + j;
            if (q < nq) sc_lds[q] = base + local[j];
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kSendPerThread; ++j) {
            const int q = i * kSendPerThread + j;
            if (q < nq) {
                const int row0 = q - (q - small_quotient(q, g.R) * g.R);   // s * R
                send_counts[q] = sc[j];
                send_offsets[q] = base + local[j] - sc_lds[row0];
            }
        }
    }
    __syncthreads();

    const unsigned long long me = 1ull << lane_id();
    int P[kMaxK];
#pragma unroll
    for (int s = 0; s < kMaxK; ++s)
        P[s] = (kp_raw[s] && static_cast<unsigned>(e_raw[s]) < static_cast<unsigned>(g.E)) ? pos_lds[e_raw[s]] : -1;
    if (live) {
#pragma unroll
        for (int s = 0; s < kMaxK; ++s)
            if (P[s] >= 0) atomicOr(&bits[wave][P[s]], me);
        for (uint64_t b = m; b; b &= b - 1)
            atomicOr(&bits[wave][g.E + __ffsll(static_cast<unsigned long long>(b)) - 1], me);
    }
    __syncthreads();
    for (int col = threadIdx.x; col < g.W; col += kChunk) {
        int run = 0;
#pragma unroll
        for (int w = 0; w < kWavesPerChunk; ++w) {
            pre[w][col] = run;
            run += __popcll(bits[w][col]);
        }
    }
    __syncthreads();
    if (!live) return;
    const unsigned long long below = lanemask_lt();
#pragma unroll
    for (int s = 0; s < kMaxK; ++s) {
        if (s >= g.k) break;
        const size_t q = static_cast<size_t>(t) * g.k + s;
        int sp = -1, cr = -1;
        if (P[s] >= 0) {
            const int Pe = P[s];
            sp = gbase[Pe] + pre[wave][Pe] + __popcll(bits[wave][Pe] & below);
            const int d = small_quotient(Pe, g.E_loc);
            const int col = g.E + d;
            if ((m >> d) & 1ull) cr = gbase[col] + pre[wave][col] + __popcll(bits[wave][col] & below);
        }
        slot_pos[q] = sp;
        copy_row[q] = cr;
    }
    for (uint64_t b = m; b; b &= b - 1) {
        const int d = __ffsll(static_cast<unsigned long long>(b)) - 1;
        const int col = g.E + d;
        const int row = gbase[col] + pre[wave][col] + __popcll(bits[wave][col] & below);
        const long long at = static_cast<long long>(roff[d]) + row;
        if (at >= 0 && at < static_cast<long long>(g.T) * g.k) recv_token[at] = t;   // malformed masks stay in bounds
    }
}

__global__ __launch_bounds__(kChunk) void layout_scatter_kernel(
    Geom g, const int32_t* __restrict__ idx, const uint8_t* __restrict__ keep,
    const uint64_t* __restrict__ mask, const int32_t* __restrict__ er, const int32_t* __restrict__ el,
    Workspace ws, int32_t* __restrict__ send_counts, int32_t* __restrict__ send_offsets,
    int32_t* __restrict__ recv_offsets, int32_t* __restrict__ expert_counts,
    int32_t* __restrict__ expert_offsets, int32_t* __restrict__ slot_pos,
    int32_t* __restrict__ copy_row, int32_t* __restrict__ recv_token) {
    layout_scatter_block(g, idx, keep, mask, er, el, ws, send_counts, send_offsets, recv_offsets, expert_counts,
                         expert_offsets, slot_pos, copy_row, recv_token, blockIdx.x);
}

inline Geom make_geom(const cap_topology* tp, int sub) {
    Geom g;
    g.T = tp->T; g.E = tp->E; g.k = tp->k; g.R = tp->R; g.rpn = tp->ranks_per_node;
    g.tpr = tp->tokens_per_rank; g.E_loc = tp->E / tp->R;
    g.cpr = (tp->tokens_per_rank + kChunk - 1) / kChunk;
    g.C = g.R * g.cpr;
    g.W = g.E + g.R;
    g.sub = sub;
    g.Cs = g.C * sub;
    return g;
}

inline Workspace carve(const Geom& g, void* base, size_t* bytes) {
    char* p = static_cast<char*>(base);
    Workspace w;
    size_t off = 0;
    w.part = reinterpret_cast<int32_t*>(p + off);
    off += align256(static_cast<size_t>(g.Cs) * g.W * sizeof(int32_t));
    w.coltot = reinterpret_cast<int32_t*>(p + off);
    off += align256(static_cast<size_t>(g.W) * sizeof(int32_t));
    w.volpart = reinterpret_cast<int64_t*>(p + off);
    off += static_cast<size_t>(g.Cs) * 4 * sizeof(int64_t);
    if (bytes) *bytes = off;
    return w;
}

}  // namespace
}  // namespace cap
