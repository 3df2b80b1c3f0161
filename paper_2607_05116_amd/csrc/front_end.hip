// Fused front end: top-k routing, gates and communication-aware pruning
// (Eq. 1; Sec. VI, Eq. 6), the all-to-all and expert-sorted layout with the
// per-token send volume (Sec. II-C; Eq. 3), and the co-activation counts on
// the pruned routing (Sec. IV-B), in three launches instead of six.  The
// outputs are those of cap_route_prune, cap_dispatch_layout and
// cap_coactivation, bit for bit.
//
//   1. route + count   one workgroup of 256 threads per eighth of a chunk (32
//                      tokens of one source rank, 8 lanes per token): the
//                      routing of route_prune.hip, then, from the results
//                      each lane holds, the part's column counts (the
//                      kept slots' experts in slot-position order, the kept
//                      devices), the per-token volume and the volume sums.
//                      Each wave adds its tokens' counts into a histogram of
//                      its own with integer LDS adds (exact, so the counts do
//                      not depend on the order they land in), and the 4 wave
//                      histograms are summed in a fixed order; the volume
//                      sums go through wave shuffles; no global atomics.
//   2. tiles + scan    the co-activation tile blocks (one per split of
//                      tokens, dispatched first: the longer work), beside
//                      the column scans over the part rows (exclusive bases
//                      in place) and the volume totals.
//   3. scatter + sum   the stable scatter of each 256-token chunk (its base is
//                      the scanned row of its first part), beside the
//                      co-activation reduce blocks.
// Workspace: the layout's, with eight partial rows per chunk, then the
// co-activation partials.
#pragma clang fp contract(off)

#include <math.h>

#include "coact_device.hpp"
#include "layout_device.hpp"
#include "route_device.hpp"

namespace cap {
namespace {

constexpr int kPart = 32;                              // tokens per route + count workgroup
constexpr int kParts = kChunk / kPart;                 // partial count rows per chunk
constexpr int kRcThreads = kPart * kGroup;             // 256
constexpr int kRcWaves = kRcThreads / kWave;           // 4
static_assert(kChunk % kPart == 0 && kRcThreads == 256, "one 8-lane group per token of a part");
static_assert(kThreads == kChunk, "co-activation reduce and scatter blocks share one block size");

template <int V, int K, bool VEC>
__global__ __launch_bounds__(kRcThreads) void route_count_kernel(
    Geom g, const float* __restrict__ logits, float inter_node_cost, float p,
    const int32_t* __restrict__ expert_rank, const int32_t* __restrict__ expert_local,
    int32_t* __restrict__ out_idx, float* __restrict__ out_w, uint8_t* __restrict__ out_keep,
    uint64_t* __restrict__ out_mask, Workspace ws, uint8_t* __restrict__ vol) {
    __shared__ int er_lds[kMaxE];
    __shared__ int pos_lds[kMaxE];
    __shared__ int hist[kRcWaves][kMaxW];
    __shared__ uint64_t vsum[kRcWaves];
    // expert tables in LDS, one entry per thread; their loads are issued
    // together with the logit loads (no branch, so no early wait)
    static_assert(kMaxE <= kRcThreads, "one table entry per thread");
    const int e_me = min(static_cast<int>(threadIdx.x), g.E - 1);
    const int er_v = expert_rank[e_me], el_v = expert_local[e_me];
    const int wave = threadIdx.x / kWave;
#pragma unroll
    for (int w = 0; w < kRcWaves; ++w)
        for (int i = threadIdx.x; i < g.W; i += kRcThreads) hist[w][i] = 0;

    // part h of chunk c
    const int sc = blockIdx.x;
    int c0, c1, src;
    chunk_range(g, sc / kParts, c0, c1, src);
    const int t0 = c0 + (sc % kParts) * kPart;
    const int t1 = min(t0 + kPart, c1);
    const int grp = threadIdx.x >> 3;
    const int lg = threadIdx.x & (kGroup - 1);
    const int t = t0 + grp;
    const bool live = t < t1;
    const float* row = logits + static_cast<size_t>(live ? t : g.T - 1) * g.E;

    constexpr int CW = V < 4 ? V : 4;
    float vals[V];
    if constexpr (VEC) {
#pragma unroll
        for (int c = 0; c < V / CW; ++c) {
            const int e0 = c * (kGroup * CW) + lg * CW;
            if constexpr (CW == 4) {
                const float4 q = *reinterpret_cast<const float4*>(row + e0);
                vals[c * 4 + 0] = q.x; vals[c * 4 + 1] = q.y; vals[c * 4 + 2] = q.z; vals[c * 4 + 3] = q.w;
            } else if constexpr (CW == 2) {
                const float2 q = *reinterpret_cast<const float2*>(row + e0);
                vals[c * 2 + 0] = q.x; vals[c * 2 + 1] = q.y;
            } else {
                vals[c] = row[e0];
            }
        }
    } else {
#pragma unroll
        for (int c = 0; c < V / CW; ++c)
#pragma unroll
            for (int i = 0; i < CW; ++i) {
                const int e = c * (kGroup * CW) + lg * CW + i;
                vals[c * CW + i] = row[e < g.E ? e : g.E - 1];
            }
    }
    er_lds[threadIdx.x] = er_v & 63;               // entries past E are never read
    pos_lds[threadIdx.x] = slot_position_of(er_v, el_v, g);
    __syncthreads();                               // er_lds, pos_lds, zeroed histograms ready
    const RouteResult res = route_token<V, K, VEC, false>(vals, lg, t, live, g.E, g.R, g.rpn, g.tpr,
                                                            inter_node_cost, p, er_lds, out_idx, out_w, out_keep,
                                                            out_mask);

    // the counters this lane adds to: its slot's expert (if kept) and the
    // lg-th kept device of the token
    const uint64_t m = device_bits(res.mask, g.R);
    int col_e = -1, col_d = -1;
    if (live) {
        if (res.has_slot && res.keep && static_cast<unsigned>(res.e) < static_cast<unsigned>(g.E))
            col_e = pos_lds[res.e];
        uint64_t b = m;
        for (int i = 0; i < lg && b; ++i) b &= b - 1;
        if (b) col_d = g.E + __ffsll(static_cast<unsigned long long>(b)) - 1;
    }
    // into the wave's own histogram (integer LDS adds: the sums do not depend
    // on the order the hardware applies them in)
    if (col_e >= 0) atomicAdd(&hist[wave][col_e], 1);
    if (col_d >= 0) atomicAdd(&hist[wave][col_d], 1);
    // per-token volume (lane 0 of the token's group): n_dev, n_intra_remote,
    // n_inter, n_nodes, and their sums over the part (the four packed as
    // 16-bit fields: a part's sums stay below 32 * 64 = 2^11)
    int v[4] = {0, 0, 0, 0};
    uint64_t vp = 0;
    if (live && lg == 0) {
        // devices of one node: rpn consecutive bits; the source's node is `home`
        const uint64_t node_bits = (g.rpn >= 64) ? ~0ull : ((1ull << g.rpn) - 1);
        const uint64_t home = node_bits << ((src / g.rpn) * g.rpn);
        v[0] = __popcll(m);
        v[1] = __popcll(m & home & ~(1ull << src));
        v[2] = __popcll(m & ~home);
        for (uint64_t b = m; b; ++v[3]) {        // one step per node: drop all of its devices
            const int d = __ffsll(static_cast<unsigned long long>(b)) - 1;
            b &= ~(node_bits << (small_quotient(d, g.rpn) * g.rpn));
        }
        reinterpret_cast<uint32_t*>(vol)[t] = static_cast<uint32_t>(v[0]) | (static_cast<uint32_t>(v[1]) << 8) |
                                              (static_cast<uint32_t>(v[2]) << 16) | (static_cast<uint32_t>(v[3]) << 24);
        vp = static_cast<uint64_t>(v[0]) | (static_cast<uint64_t>(v[1]) << 16) |
             (static_cast<uint64_t>(v[2]) << 32) | (static_cast<uint64_t>(v[3]) << 48);
    }
    // the wave's 8 tokens (lanes 0, 8, ..., 56) summed by butterfly shuffles
#pragma unroll
    for (int off = kGroup; off < kWave; off <<= 1) {
        const uint32_t lo = __shfl_xor(static_cast<uint32_t>(vp), off);
        const uint32_t hi = __shfl_xor(static_cast<uint32_t>(vp >> 32), off);
        vp += static_cast<uint64_t>(lo) | (static_cast<uint64_t>(hi) << 32);
    }
    if (lane_id() == 0) vsum[wave] = vp;
    __syncthreads();
    if (threadIdx.x < 4) {
        uint64_t all = 0;
#pragma unroll
        for (int w = 0; w < kRcWaves; ++w) all += vsum[w];
        ws.volpart[sc * 4 + threadIdx.x] = static_cast<int64_t>((all >> (16 * threadIdx.x)) & 0xFFFFu);
    }
    // the part's row: the waves' histograms summed (W <= 2 * 256: two
    // columns per thread, the second clamped, all LDS reads issued together)
    static_assert(kMaxW <= 2 * kRcThreads, "two columns per thread");
    int32_t* out = ws.part + static_cast<size_t>(sc) * g.W;
    const int col0 = threadIdx.x, col1 = min(static_cast<int>(threadIdx.x) + kRcThreads, g.W - 1);
    int s0 = 0, s1 = 0;
#pragma unroll
    for (int w = 0; w < kRcWaves; ++w) {
        s0 += hist[w][col0];
        s1 += hist[w][col1];
    }
    if (col0 < g.W) out[col0] = s0;
    if (col0 + kRcThreads < g.W) out[col1] = s1;
}

// Launch 2 (blocks of kTileThreads): the first `splits` blocks count the
// co-activation tiles (the longer work, so it starts first), the remaining
// W + 1 scan the columns and sum the volumes.
__global__ __launch_bounds__(kTileThreads) void front_scan_tile_kernel(Geom g, Workspace ws, int64_t* __restrict__ totals,
                                                                 const int32_t* __restrict__ idx,
                                                                 const uint8_t* __restrict__ keep, int per,
                                                                 uint32_t* __restrict__ coact_part) {
    const int splits = static_cast<int>(gridDim.x) - (g.W + 1);
    const int b = static_cast<int>(blockIdx.x);
    if (b < splits) coact_tile_block(g.T, g.k, g.E, per, idx, keep, coact_part, b);
    else layout_colscan_block<kTileThreads>(g, ws, totals, b - splits);
}

// Launch 3: blocks [0, C) scatter the chunks; the rest reduce the
// co-activation partials.
__global__ __launch_bounds__(kChunk) void front_scatter_reduce_kernel(
    Geom g, const int32_t* __restrict__ idx, const uint8_t* __restrict__ keep, const uint64_t* __restrict__ mask,
    const int32_t* __restrict__ er, const int32_t* __restrict__ el, Workspace ws, int32_t* __restrict__ send_counts,
    int32_t* __restrict__ send_offsets, int32_t* __restrict__ recv_offsets, int32_t* __restrict__ expert_counts,
    int32_t* __restrict__ expert_offsets, int32_t* __restrict__ slot_pos, int32_t* __restrict__ copy_row,
    int32_t* __restrict__ recv_token, int splits, const uint32_t* __restrict__ coact_part,
    uint32_t* __restrict__ coact) {
    const int b = blockIdx.x;
    if (b < g.C)
        layout_scatter_block(g, idx, keep, mask, er, el, ws, send_counts, send_offsets, recv_offsets, expert_counts,
                             expert_offsets, slot_pos, copy_row, recv_token, b);
    else
        coact_reduce_block(g.E, splits, 0, coact_part, coact, b - g.C);
}

struct Front {
    Geom g;
    Workspace ws;
    uint32_t* coact_part;
    size_t bytes;
};

Front front_carve(const cap_topology* tp, void* base) {
    Front f;
    f.g = make_geom(tp, kParts);
    size_t lay = 0;
    f.ws = carve(f.g, base, &lay);
    lay = align256(lay);
    f.coact_part = reinterpret_cast<uint32_t*>(static_cast<char*>(base) + lay);
    f.bytes = lay + coact_part_bytes(tp->T, tp->E);
    return f;
}

template <int V, int K>
void launch_rc(const Front& f, const cap_topology* tp, const float* logits, float p, bool vec, int32_t* idx,
               float* w, uint8_t* keep, uint64_t* mask, uint8_t* vol, hipStream_t st) {
    if (vec)
        route_count_kernel<V, K, true><<<f.g.Cs, kRcThreads, 0, st>>>(
            f.g, logits, tp->inter_node_cost, p, tp->expert_rank, tp->expert_local, idx, w, keep, mask, f.ws, vol);
    else
        route_count_kernel<V, K, false><<<f.g.Cs, kRcThreads, 0, st>>>(
            f.g, logits, tp->inter_node_cost, p, tp->expert_rank, tp->expert_local, idx, w, keep, mask, f.ws, vol);
}

template <int V>
void launch_rc_k(const Front& f, const cap_topology* tp, const float* logits, float p, bool vec, int32_t* idx,
                 float* w, uint8_t* keep, uint64_t* mask, uint8_t* vol, hipStream_t st) {
    switch (tp->k) {
        case 1: launch_rc<V, 1>(f, tp, logits, p, vec, idx, w, keep, mask, vol, st); break;
        case 2: launch_rc<V, 2>(f, tp, logits, p, vec, idx, w, keep, mask, vol, st); break;
        case 3: launch_rc<V, 3>(f, tp, logits, p, vec, idx, w, keep, mask, vol, st); break;
        case 4: launch_rc<V, 4>(f, tp, logits, p, vec, idx, w, keep, mask, vol, st); break;
        case 5: launch_rc<V, 5>(f, tp, logits, p, vec, idx, w, keep, mask, vol, st); break;
        case 6: launch_rc<V, 6>(f, tp, logits, p, vec, idx, w, keep, mask, vol, st); break;
        case 7: launch_rc<V, 7>(f, tp, logits, p, vec, idx, w, keep, mask, vol, st); break;
        default: launch_rc<V, 8>(f, tp, logits, p, vec, idx, w, keep, mask, vol, st); break;
    }
}

}  // namespace

size_t front_end_workspace_bytes(const cap_topology* tp) { return front_carve(tp, nullptr).bytes; }

cap_status front_end_launch(const cap_topology* tp, const float* logits, float p, int32_t* idx, float* w,
                            uint8_t* keep, uint64_t* mask, const cap_layout* o, uint32_t* coact, void* wsp,
                            hipStream_t st) {
    const Front f = front_carve(tp, wsp);
    int V = 1;
    while (kGroup * V < tp->E) V <<= 1;
    const int CW = V < 4 ? V : 4;
    const bool vec = (tp->E == kGroup * V) && (reinterpret_cast<uintptr_t>(logits) % (4 * CW) == 0);
    switch (V) {
        case 1: launch_rc_k<1>(f, tp, logits, p, vec, idx, w, keep, mask, o->vol, st); break;
        case 2: launch_rc_k<2>(f, tp, logits, p, vec, idx, w, keep, mask, o->vol, st); break;
        case 4: launch_rc_k<4>(f, tp, logits, p, vec, idx, w, keep, mask, o->vol, st); break;
        case 8: launch_rc_k<8>(f, tp, logits, p, vec, idx, w, keep, mask, o->vol, st); break;
        case 16: launch_rc_k<16>(f, tp, logits, p, vec, idx, w, keep, mask, o->vol, st); break;
        default: launch_rc_k<32>(f, tp, logits, p, vec, idx, w, keep, mask, o->vol, st); break;
    }
    CAP_LAUNCH_CHECK();
    const int per = coact_tokens_per_split(tp->T);
    const int splits = coact ? coact_splits(tp->T) : 0;
    front_scan_tile_kernel<<<f.g.W + 1 + splits, kTileThreads, 0, st>>>(f.g, f.ws, o->totals, idx, keep, per,
                                                                   f.coact_part);
    CAP_LAUNCH_CHECK();
    const int reduce_blocks = coact ? coact_reduce_blocks(tp->E) : 0;
    front_scatter_reduce_kernel<<<f.g.C + reduce_blocks, kChunk, 0, st>>>(
        f.g, idx, keep, mask, tp->expert_rank, tp->expert_local, f.ws, o->send_counts, o->send_offsets,
        o->recv_offsets, o->expert_counts, o->expert_offsets, o->slot_pos, o->copy_row, o->recv_token, splits,
        f.coact_part, coact);
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

}  // namespace cap
