// Device-centric all-to-all layout, expert-sorted layout and send volume.
//
// Sec. II-C: a token is sent once to every device that hosts one of its kept
// experts, and the experts of that device share the copy.  Eq. 3 classes a
// destination as the own device, another device of the same node, or a device
// on another node; the per-token counts of each class are the send volume.
//
// Three launches, no global atomics, deterministic:
//   1. count   one block per chunk of up to 512 tokens of one source rank:
//              per-chunk counts of kept rows per expert slot position and of
//              copies per destination device (LDS integer atomics, whose sum
//              does not depend on order), plus per-token volume and per-chunk
//              volume sums.
//   2. scan    one block: exclusive scans over chunks (per column), over slot
//              positions (expert offsets), over destinations (send offsets,
//              receive offsets); totals.
//   3. scatter one block per chunk: stable in-chunk ranks from per-wave
//              bitsets (LDS atomicOr, order independent) and popcounts, then
//              slot_pos, copy_row and recv_token.
// Workspace: [C][E+R] int32 chunk counts (turned into chunk bases in place)
//            followed by [C][4] int64 volume sums; C = R * ceil(T_loc / 512).
#include "cap_device.hpp"

namespace cap {
namespace {

constexpr int kChunk = 512;        // tokens per chunk = threads per block
constexpr int kWavesPerChunk = kChunk / kWave;

struct Geom {
    int T, E, k, R, rpn, tpr, E_loc, cpr, C;
};

__device__ __forceinline__ void chunk_range(const Geom& g, int c, int& t0, int& t1, int& src) {
    src = c / g.cpr;
    t0 = src * g.tpr + (c % g.cpr) * kChunk;
    t1 = min(t0 + kChunk, (src + 1) * g.tpr);
}

__device__ __forceinline__ int slot_position(const int32_t* er, const int32_t* el, int e, const Geom& g) {
    if (static_cast<unsigned>(e) >= static_cast<unsigned>(g.E)) return -1;
    const int r = er[e], l = el[e];
    if (static_cast<unsigned>(r) >= static_cast<unsigned>(g.R) ||
        static_cast<unsigned>(l) >= static_cast<unsigned>(g.E_loc))
        return -1;
    return r * g.E_loc + l;
}

__global__ __launch_bounds__(kChunk) void layout_count_kernel(
    Geom g, const int32_t* __restrict__ idx, const uint8_t* __restrict__ keep,
    const uint64_t* __restrict__ mask, const int32_t* __restrict__ er, const int32_t* __restrict__ el,
    int32_t* __restrict__ part, int64_t* __restrict__ volpart, uint8_t* __restrict__ vol) {
    __shared__ int cnt[kMaxE + kMaxR];
    __shared__ int pos_lds[kMaxE];
    __shared__ unsigned long long vsum[4];
    const int W = g.E + g.R;
    for (int i = threadIdx.x; i < W; i += blockDim.x) cnt[i] = 0;
    for (int e = threadIdx.x; e < g.E; e += blockDim.x) pos_lds[e] = slot_position(er, el, e, g);
    if (threadIdx.x < 4) vsum[threadIdx.x] = 0;
    __syncthreads();

    int t0, t1, src;
    chunk_range(g, blockIdx.x, t0, t1, src);
    const int t = t0 + threadIdx.x;
    if (t < t1) {
        for (int s = 0; s < g.k; ++s) {
            const size_t q = static_cast<size_t>(t) * g.k + s;
            if (!keep[q]) continue;
            const int e = idx[q];
            const int P = static_cast<unsigned>(e) < static_cast<unsigned>(g.E) ? pos_lds[e] : -1;
            if (P >= 0) atomicAdd(&cnt[P], 1);
        }
        const uint64_t m = mask[t];
        const int src_node = src / g.rpn;
        int n_dev = 0, n_intra = 0, n_inter = 0;
        uint64_t nodes = 0;
        for (int d = 0; d < g.R; ++d) {
            if (!((m >> d) & 1ull)) continue;
            atomicAdd(&cnt[g.E + d], 1);
            ++n_dev;
            const int nd = d / g.rpn;
            if (nd != src_node) ++n_inter;
            else if (d != src) ++n_intra;
            nodes |= 1ull << nd;
        }
        const int n_nodes = __popcll(nodes);
        const uint32_t packed = static_cast<uint32_t>(n_dev) | (static_cast<uint32_t>(n_intra) << 8) |
                                (static_cast<uint32_t>(n_inter) << 16) | (static_cast<uint32_t>(n_nodes) << 24);
        reinterpret_cast<uint32_t*>(vol)[t] = packed;
        atomicAdd(&vsum[0], static_cast<unsigned long long>(n_dev));
        atomicAdd(&vsum[1], static_cast<unsigned long long>(n_intra));
        atomicAdd(&vsum[2], static_cast<unsigned long long>(n_inter));
        atomicAdd(&vsum[3], static_cast<unsigned long long>(n_nodes));
    }
    __syncthreads();
    int32_t* out = part + static_cast<size_t>(blockIdx.x) * W;
    for (int i = threadIdx.x; i < W; i += blockDim.x) out[i] = cnt[i];
    if (threadIdx.x < 4) volpart[blockIdx.x * 4 + threadIdx.x] = static_cast<int64_t>(vsum[threadIdx.x]);
}

constexpr int kScanThreads = 1024;
constexpr int kScanRows = 32;      // chunks staged in LDS per pass

__global__ __launch_bounds__(kScanThreads) void layout_scan_kernel(
    Geom g, int32_t* __restrict__ part, const int64_t* __restrict__ volpart,
    int32_t* __restrict__ send_counts, int32_t* __restrict__ send_offsets,
    int32_t* __restrict__ recv_offsets, int32_t* __restrict__ expert_counts,
    int32_t* __restrict__ expert_offsets, int64_t* __restrict__ totals) {
    __shared__ int32_t stage[kScanRows * (kMaxE + kMaxR)];
    __shared__ int32_t carry[kMaxE + kMaxR];
    __shared__ int32_t rank_start[kMaxR + 1][kMaxR];   // dst prefix at each rank's first chunk
    __shared__ int32_t scan_buf[kMaxE];
    const int W = g.E + g.R;
    for (int i = threadIdx.x; i < W; i += blockDim.x) carry[i] = 0;
    __syncthreads();

    // Column-wise exclusive scan over chunks, in passes of kScanRows chunks.
    for (int c0 = 0; c0 < g.C; c0 += kScanRows) {
        const int rows = min(kScanRows, g.C - c0);
        for (int i = threadIdx.x; i < rows * W; i += blockDim.x)
            stage[i] = part[static_cast<size_t>(c0) * W + i];
        __syncthreads();
        if (threadIdx.x < W) {
            const int col = threadIdx.x;
            int run = carry[col];
            for (int r = 0; r < rows; ++r) {
                const int c = c0 + r;
                if (col >= g.E && (c % g.cpr) == 0) rank_start[c / g.cpr][col - g.E] = run;
                const int v = stage[r * W + col];
                stage[r * W + col] = run;
                run += v;
            }
            carry[col] = run;
        }
        __syncthreads();
        for (int i = threadIdx.x; i < rows * W; i += blockDim.x)
            part[static_cast<size_t>(c0) * W + i] = stage[i];
        __syncthreads();
    }
    if (threadIdx.x < g.R) rank_start[g.R][threadIdx.x] = carry[g.E + threadIdx.x];
    __syncthreads();

    // Expert totals and offsets in slot-position order (Hillis-Steele scan).
    if (threadIdx.x < g.E) {
        expert_counts[threadIdx.x] = carry[threadIdx.x];
        scan_buf[threadIdx.x] = carry[threadIdx.x];
    }
    __syncthreads();
    for (int off = 1; off < g.E; off <<= 1) {
        int v = 0;
        if (threadIdx.x < g.E && threadIdx.x >= off) v = scan_buf[threadIdx.x - off];
        __syncthreads();
        if (threadIdx.x < g.E) scan_buf[threadIdx.x] += v;
        __syncthreads();
    }
    if (threadIdx.x < g.E) expert_offsets[threadIdx.x + 1] = scan_buf[threadIdx.x];
    if (threadIdx.x == 0) expert_offsets[0] = 0;

    // send_counts[s][d] = prefix at rank s+1 start minus prefix at rank s start.
    for (int i = threadIdx.x; i < g.R * g.R; i += blockDim.x) {
        const int s = i / g.R, d = i % g.R;
        send_counts[i] = rank_start[s + 1][d] - rank_start[s][d];
    }
    if (threadIdx.x < g.R) {
        const int s = threadIdx.x;
        int run = 0;
        for (int d = 0; d < g.R; ++d) {
            send_offsets[s * g.R + d] = run;
            run += rank_start[s + 1][d] - rank_start[s][d];
        }
    }
    if (threadIdx.x == 0) {
        int run = 0;
        for (int d = 0; d < g.R; ++d) {
            recv_offsets[d] = run;
            run += carry[g.E + d];
        }
        recv_offsets[g.R] = run;
    }
    if (threadIdx.x < 4) {
        int64_t s = 0;
        for (int c = 0; c < g.C; ++c) s += volpart[c * 4 + threadIdx.x];
        totals[threadIdx.x] = s;
    }
}

__global__ __launch_bounds__(kChunk) void layout_scatter_kernel(
    Geom g, const int32_t* __restrict__ idx, const uint8_t* __restrict__ keep,
    const uint64_t* __restrict__ mask, const int32_t* __restrict__ er, const int32_t* __restrict__ el,
    const int32_t* __restrict__ base, const int32_t* __restrict__ expert_offsets,
    const int32_t* __restrict__ recv_offsets, int32_t* __restrict__ slot_pos,
    int32_t* __restrict__ copy_row, int32_t* __restrict__ recv_token) {
    __shared__ unsigned long long bits[kWavesPerChunk][kMaxE + kMaxR];
    __shared__ int32_t pre[kWavesPerChunk][kMaxE + kMaxR];
    __shared__ int pos_lds[kMaxE];
    __shared__ int32_t gbase[kMaxE + kMaxR];
    const int W = g.E + g.R;
    const int wave = threadIdx.x / kWave;
    for (int i = threadIdx.x; i < kWavesPerChunk * W; i += blockDim.x) bits[i / W][i % W] = 0ull;
    for (int e = threadIdx.x; e < g.E; e += blockDim.x) pos_lds[e] = slot_position(er, el, e, g);
    const int32_t* cb = base + static_cast<size_t>(blockIdx.x) * W;
    for (int i = threadIdx.x; i < W; i += blockDim.x)
        gbase[i] = cb[i] + (i < g.E ? expert_offsets[i] : 0);
    __syncthreads();

    int t0, t1, src;
    chunk_range(g, blockIdx.x, t0, t1, src);
    const int t = t0 + threadIdx.x;
    const bool live = t < t1;
    const unsigned long long me = 1ull << lane_id();
    int P[kMaxK];
    int D[kMaxK];
    uint64_t m = 0;
    if (live) {
        m = mask[t];
        for (int s = 0; s < g.k; ++s) {
            const size_t q = static_cast<size_t>(t) * g.k + s;
            const int e = idx[q];
            const bool ok = keep[q] && static_cast<unsigned>(e) < static_cast<unsigned>(g.E);
            P[s] = ok ? pos_lds[e] : -1;
            D[s] = P[s] >= 0 ? P[s] / g.E_loc : -1;
            if (P[s] >= 0) atomicOr(&bits[wave][P[s]], me);
        }
        for (int d = 0; d < g.R; ++d)
            if ((m >> d) & 1ull) atomicOr(&bits[wave][g.E + d], me);
    }
    __syncthreads();
    for (int col = threadIdx.x; col < W; col += blockDim.x) {
        int run = 0;
        for (int w = 0; w < kWavesPerChunk; ++w) {
            pre[w][col] = run;
            run += __popcll(bits[w][col]);
        }
    }
    __syncthreads();
    if (!live) return;
    const unsigned long long below = lanemask_lt();
    for (int s = 0; s < g.k; ++s) {
        const size_t q = static_cast<size_t>(t) * g.k + s;
        if (P[s] < 0) {
            slot_pos[q] = -1;
            copy_row[q] = -1;
            continue;
        }
        const int Pe = P[s];
        slot_pos[q] = gbase[Pe] + pre[wave][Pe] + __popcll(bits[wave][Pe] & below);
        const int d = D[s];
        const int col = g.E + d;
        copy_row[q] = ((m >> d) & 1ull) ? gbase[col] + pre[wave][col] + __popcll(bits[wave][col] & below) : -1;
    }
    for (int d = 0; d < g.R; ++d) {
        if (!((m >> d) & 1ull)) continue;
        const int col = g.E + d;
        const int row = gbase[col] + pre[wave][col] + __popcll(bits[wave][col] & below);
        const long long at = static_cast<long long>(recv_offsets[d]) + row;
        if (at < static_cast<long long>(g.T) * g.k) recv_token[at] = t;   // malformed masks stay in bounds
    }
}

Geom make_geom(const cap_topology* tp) {
    Geom g;
    g.T = tp->T; g.E = tp->E; g.k = tp->k; g.R = tp->R; g.rpn = tp->ranks_per_node;
    g.tpr = tp->tokens_per_rank; g.E_loc = tp->E / tp->R;
    g.cpr = (tp->tokens_per_rank + kChunk - 1) / kChunk;
    g.C = g.R * g.cpr;
    return g;
}

}  // namespace

size_t layout_workspace_bytes(const cap_topology* tp) {
    const Geom g = make_geom(tp);
    size_t a = static_cast<size_t>(g.C) * (g.E + g.R) * sizeof(int32_t);
    a = (a + 255) & ~static_cast<size_t>(255);
    return a + static_cast<size_t>(g.C) * 4 * sizeof(int64_t);
}

cap_status dispatch_layout_launch(const cap_topology* tp, const int32_t* idx, const uint8_t* keep,
                                  const uint64_t* mask, const cap_layout* o, void* ws, hipStream_t st) {
    const Geom g = make_geom(tp);
    size_t a = static_cast<size_t>(g.C) * (g.E + g.R) * sizeof(int32_t);
    a = (a + 255) & ~static_cast<size_t>(255);
    int32_t* part = static_cast<int32_t*>(ws);
    int64_t* volpart = reinterpret_cast<int64_t*>(static_cast<char*>(ws) + a);
    layout_count_kernel<<<g.C, kChunk, 0, st>>>(g, idx, keep, mask, tp->expert_rank, tp->expert_local,
                                                 part, volpart, o->vol);
    CAP_LAUNCH_CHECK();
    layout_scan_kernel<<<1, kScanThreads, 0, st>>>(g, part, volpart, o->send_counts, o->send_offsets,
                                                   o->recv_offsets, o->expert_counts, o->expert_offsets,
                                                   o->totals);
    CAP_LAUNCH_CHECK();
    layout_scatter_kernel<<<g.C, kChunk, 0, st>>>(g, idx, keep, mask, tp->expert_rank, tp->expert_local,
                                                   part, o->expert_offsets, o->recv_offsets, o->slot_pos,
                                                   o->copy_row, o->recv_token);
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

}  // namespace cap
