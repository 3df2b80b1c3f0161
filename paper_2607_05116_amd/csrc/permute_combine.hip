// Token permutation and weighted combine (Sec. II-C; Eq. 1).
//
// The index kernels (row source, row plan) write one int per expert-sorted
// row from one thread per (received token, slot).  The four row movers are
// HBM-bound and built the same way:
//   * one wave owns one row piece at a time (a token's row, or a contiguous
//     part of it when there are too few tokens to fill the chip);
//   * the token's k routing slots are read one slot per lane, so a token's
//     metadata costs one round of parallel loads; small per-launch tables
//     (expert -> device, receive offsets, send bases) sit in LDS;
//   * the wave compacts its valid slots into a uniform list with a ballot and
//     then issues every 16-byte load of a batch before it uses any, so each
//     lane keeps JB (x rows) loads in flight instead of one.
//
//   expert gather  (dest rank r)  read each received token once, write it to
//                  every kept expert row of r (device-centric: one copy per
//                  device, shared by that device's experts).
//   send pack      (source rank s) read each token of s once, write one row per
//                  kept destination device into the send buffer.
//   dest reduce    (rank r) per received token: sum of w'_s * Y over the token's
//                  kept experts on r (local aggregation before the return); a
//                  mode skips the tokens with one row on r, whose one-term
//                  sum the FFN's epilogue writes (row plan).
//   src reduce     (rank s) per token of s: sum of the rows every kept device
//                  returned (+ the shared experts' output).
// Accumulation is fp32 in a fixed order (slot order / ascending device).
//
// A kept slot's row in rank r's expert-sorted buffer is slot_pos - (first row
// of r); the slot is on r exactly when that difference falls inside r's row
// range (pruned slots hold -1), so gather and dest reduce need no expert ->
// device lookup.
#include "cap_device.hpp"

namespace cap {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;
constexpr int kTargetWaves = 8192;   // row pieces per launch worth splitting rows for

struct Topo {
    int T, E, k, R, tpr, E_loc;
};

// Piece p of a row of vpr 16-byte chunks cut into `pieces` near-equal parts.
struct Piece {
    int begin, end;
};
__device__ __forceinline__ Piece row_piece(int vpr, int pieces, int p) {
    const int per = (vpr + pieces - 1) / pieces;
    const int b = min(vpr, p * per);
    return Piece{b, min(vpr, b + per)};
}

// Uniform list of the rows held by the lanes whose `row` is >= 0, in lane
// (= slot) order; returns their count.  Lanes >= kMaxK never hold a row.
__device__ __forceinline__ int compact_rows(int row, int (&rows)[kMaxK]) {
    uint64_t vb = __ballot(row >= 0);
    const int n = __popcll(vb);
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
        rows[j] = -1;
        if (j < n) {
            const int s = __ffsll(static_cast<unsigned long long>(vb)) - 1;
            rows[j] = __builtin_amdgcn_readlane(row, s);
            vb &= vb - 1;
        }
    }
    return n;
}

__device__ __forceinline__ float lane_value(float v, int s) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), s));
}

// ---------------------------------------------------------------- row load / store helpers
struct Bf16Row {                              // 8 bf16 per chunk
    static constexpr int kElems = 8;
    __device__ static void load(const u32x4& v, float* f) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f[2 * i] = __uint_as_float(v[i] << 16);
            f[2 * i + 1] = __uint_as_float(v[i] & 0xFFFF0000u);
        }
    }
    __device__ static u32x4 store(const float* f) {
        u32x4 v;
        v[0] = pack_bf16x2(f[0], f[1]);
        v[1] = pack_bf16x2(f[2], f[3]);
        v[2] = pack_bf16x2(f[4], f[5]);
        v[3] = pack_bf16x2(f[6], f[7]);
        return v;
    }
};

struct F32Row {                               // 4 fp32 per chunk
    static constexpr int kElems = 4;
    __device__ static void load(const u32x4& v, float* f) {
#pragma unroll
        for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(v[i]);
    }
    __device__ static u32x4 store(const float* f) {
        u32x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = __float_as_uint(f[i]);
        return v;
    }
};

// Copy chunks [pc.begin, pc.end) of src to rows[0..n) of out.
template <int JB>
__device__ __forceinline__ void fan_out(const u32x4* __restrict__ src, u32x4* __restrict__ out, int vpr,
                                        Piece pc, int n, const int (&rows)[kMaxK]) {
    for (int c0 = pc.begin + lane_id(); c0 < pc.end; c0 += kWave * JB) {
        u32x4 v[JB];
#pragma unroll
        for (int j = 0; j < JB; ++j) {
            const int c = c0 + j * kWave;
            if (c < pc.end) v[j] = src[c];
        }
#pragma unroll
        for (int r = 0; r < kMaxK; ++r) {
            if (r >= n) break;
            u32x4* dst = out + static_cast<size_t>(rows[r]) * vpr;
#pragma unroll
            for (int j = 0; j < JB; ++j) {
                const int c = c0 + j * kWave;
                if (c < pc.end) dst[c] = v[j];
            }
        }
    }
}

// ---------------------------------------------------------------- expert gather
template <int JB>
__global__ __launch_bounds__(kThreads) void expert_gather_kernel(
    Topo g, int rank, int vpr, int pieces, const u32x4* __restrict__ x, const int32_t* __restrict__ slot_pos,
    const int32_t* __restrict__ expert_offsets, const int32_t* __restrict__ recv_offsets,
    const int32_t* __restrict__ recv_token, u32x4* __restrict__ out, int out_rows) {
    const int r0 = recv_offsets[rank];
    if (r0 < 0) return;
    const int U = min(recv_offsets[rank + 1] - r0, g.T * g.k - r0);
    const int base = expert_offsets[rank * g.E_loc];
    const int rows_r = min(expert_offsets[(rank + 1) * g.E_loc] - base, out_rows);
    const int items = U * pieces;
    const int lane = lane_id();
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int it = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; it < items; it += nwaves) {
        const int u = it / pieces;
        const int t = recv_token[r0 + u];
        if (static_cast<unsigned>(t) >= static_cast<unsigned>(g.T)) continue;
        int row = -1;
        if (lane < g.k) {
            const int rr = slot_pos[static_cast<size_t>(t) * g.k + lane] - base;
            row = static_cast<unsigned>(rr) < static_cast<unsigned>(rows_r) ? rr : -1;
        }
        int rows[kMaxK];
        const int n = compact_rows(row, rows);
        fan_out<JB>(x + static_cast<size_t>(t) * vpr, out, vpr, row_piece(vpr, pieces, it - u * pieces), n, rows);
    }
}

// ---------------------------------------------------------------- row source
// Index-only expert gather: one thread per (received token, slot) writes the
// token index into the slot's expert-sorted row.
__global__ __launch_bounds__(kThreads) void row_source_kernel(
    Topo g, int rank, const int32_t* __restrict__ slot_pos, const int32_t* __restrict__ expert_offsets,
    const int32_t* __restrict__ recv_offsets, const int32_t* __restrict__ recv_token, int32_t* __restrict__ out,
    int out_rows) {
    const int r0 = recv_offsets[rank];
    if (r0 < 0) return;
    const int U = min(recv_offsets[rank + 1] - r0, g.T * g.k - r0);
    const int base = expert_offsets[rank * g.E_loc];
    const int rows_r = min(expert_offsets[(rank + 1) * g.E_loc] - base, out_rows);
    const long long items = static_cast<long long>(U) * g.k;
    for (long long i = static_cast<long long>(blockIdx.x) * kThreads + threadIdx.x; i < items;
         i += static_cast<long long>(gridDim.x) * kThreads) {
        const int u = static_cast<int>(i / g.k);
        const int s = static_cast<int>(i - static_cast<long long>(u) * g.k);
        const int t = recv_token[r0 + u];
        if (static_cast<unsigned>(t) >= static_cast<unsigned>(g.T)) continue;
        const int rr = slot_pos[static_cast<size_t>(t) * g.k + s] - base;
        if (static_cast<unsigned>(rr) < static_cast<unsigned>(rows_r)) out[rr] = t;
    }
}

// Row plan for the FFN with the destination combine folded in: the row
// source, and for a row whose token has no other kept slot on the rank (one
// term in its destination reduce), the receive row the term goes to and its
// gate weight; -1 and 0 otherwise (also when the receive row is at or past
// parts_rows).  The count of a token's rows on the rank is the destination
// reduce's own (kept slots whose expert-sorted row lies in the rank's range).
__global__ __launch_bounds__(kThreads) void row_plan_kernel(
    Topo g, int rank, const float* __restrict__ w, const int32_t* __restrict__ slot_pos,
    const int32_t* __restrict__ expert_offsets, const int32_t* __restrict__ recv_offsets,
    const int32_t* __restrict__ recv_token, int32_t* __restrict__ row_src, int32_t* __restrict__ row_dst,
    float* __restrict__ row_w, int rows_cap, int parts_rows) {
    const int r0 = recv_offsets[rank];
    if (r0 < 0) return;
    const int U = min(recv_offsets[rank + 1] - r0, g.T * g.k - r0);
    const int base = expert_offsets[rank * g.E_loc];
    const int rows_r = min(expert_offsets[(rank + 1) * g.E_loc] - base, rows_cap);
    const long long items = static_cast<long long>(U) * g.k;
    for (long long i = static_cast<long long>(blockIdx.x) * kThreads + threadIdx.x; i < items;
         i += static_cast<long long>(gridDim.x) * kThreads) {
        const int u = static_cast<int>(i / g.k);
        const int s = static_cast<int>(i - static_cast<long long>(u) * g.k);
        const int t = recv_token[r0 + u];
        if (static_cast<unsigned>(t) >= static_cast<unsigned>(g.T)) continue;
        const size_t q0 = static_cast<size_t>(t) * g.k;
        const int rr = slot_pos[q0 + s] - base;
        if (static_cast<unsigned>(rr) >= static_cast<unsigned>(rows_r)) continue;
        int n = 0;
        for (int s2 = 0; s2 < g.k; ++s2)
            n += static_cast<unsigned>(slot_pos[q0 + s2] - base) < static_cast<unsigned>(rows_r) ? 1 : 0;
        const bool single = n == 1 && r0 + u < parts_rows;
        row_src[rr] = t;
        row_dst[rr] = single ? r0 + u : -1;
        row_w[rr] = single ? w[q0 + s] : 0.0f;
    }
}

// ---------------------------------------------------------------- send pack
template <int JB>
__global__ __launch_bounds__(kThreads) void send_pack_kernel(
    Topo g, int src_rank, int vpr, int pieces, const u32x4* __restrict__ x, const int32_t* __restrict__ idx,
    const uint8_t* __restrict__ keep, const int32_t* __restrict__ er, const uint64_t* __restrict__ mask,
    const int32_t* __restrict__ copy_row, const int32_t* __restrict__ send_counts,
    const int32_t* __restrict__ send_offsets, u32x4* __restrict__ out, int out_rows) {
    __shared__ int32_t dev_of[kMaxE];
    __shared__ int32_t row0[kMaxR];   // send_offsets[s][d] - (rows of d from sources < s)
    __shared__ int32_t total_lds;
    for (int e = threadIdx.x; e < g.E; e += kThreads) dev_of[e] = er[e];
    if (threadIdx.x < g.R) row0[threadIdx.x] = send_offsets[src_rank * g.R + threadIdx.x];
    if (threadIdx.x == 0) total_lds = 0;
    __syncthreads();
    for (int j = threadIdx.x; j < src_rank * g.R; j += kThreads) atomicSub(&row0[j % g.R], send_counts[j]);
    if (threadIdx.x < g.R) atomicAdd(&total_lds, send_counts[src_rank * g.R + threadIdx.x]);
    __syncthreads();
    const int total = min(total_lds, out_rows);
    const int lane = lane_id();
    const int items = g.tpr * pieces;
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int it = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; it < items; it += nwaves) {
        const int i = it / pieces;
        const int t = src_rank * g.tpr + i;
        const uint64_t m = mask[t];
        int d = -1, cr = -1;
        if (lane < g.k) {
            const size_t q = static_cast<size_t>(t) * g.k + lane;
            const int e = idx[q];
            if (keep[q] && static_cast<unsigned>(e) < static_cast<unsigned>(g.E)) d = dev_of[e];
            cr = copy_row[q];
            if (static_cast<unsigned>(d) >= static_cast<unsigned>(g.R) || !((m >> d) & 1ull)) d = -1;
        }
        // one row per device: the device's first kept slot writes it
        bool first = d >= 0;
#pragma unroll
        for (int s2 = 0; s2 < kMaxK; ++s2) {
            const int d2 = __shfl(d, s2);
            if (s2 < lane && d2 == d) first = false;
        }
        int row = -1;
        if (first) {
            const int rr = row0[d] + cr;
            row = static_cast<unsigned>(rr) < static_cast<unsigned>(total) ? rr : -1;
        }
        int rows[kMaxK];
        const int n = compact_rows(row, rows);
        fan_out<JB>(x + static_cast<size_t>(t) * vpr, out, vpr, row_piece(vpr, pieces, it - i * pieces), n, rows);
    }
}

// ---------------------------------------------------------------- dest reduce
template <typename RowT, int JB>
__global__ __launch_bounds__(kThreads) void dest_reduce_kernel(
    Topo g, int rank, int vpr, int pieces, const u32x4* __restrict__ Y, const float* __restrict__ w,
    const int32_t* __restrict__ slot_pos, const int32_t* __restrict__ expert_offsets,
    const int32_t* __restrict__ recv_offsets, const int32_t* __restrict__ recv_token,
    u32x4* __restrict__ out, int in_rows, int out_rows, int skip_single) {
    const int r0 = recv_offsets[rank];
    if (r0 < 0) return;
    const int U = min(min(recv_offsets[rank + 1] - r0, g.T * g.k - r0), out_rows - r0);
    const int base = expert_offsets[rank * g.E_loc];
    const int rows_r = min(expert_offsets[(rank + 1) * g.E_loc] - base, in_rows);
    const int items = U * pieces;
    const int lane = lane_id();
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int it = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; it < items; it += nwaves) {
        const int u = it / pieces;
        const int t = recv_token[r0 + u];
        int row = -1;
        float wl = 0.0f;
        if (lane < g.k && static_cast<unsigned>(t) < static_cast<unsigned>(g.T)) {
            const size_t q = static_cast<size_t>(t) * g.k + lane;
            const int rr = slot_pos[q] - base;
            if (static_cast<unsigned>(rr) < static_cast<unsigned>(rows_r)) {
                row = rr;
                wl = w[q];
            }
        }
        // slot-ordered list of (row, weight)
        uint64_t vb = __ballot(row >= 0);
        const int n = __popcll(vb);
        if (skip_single && n == 1) continue;       // written by the FFN's epilogue (wave-uniform)
        int rows[kMaxK];
        float wt[kMaxK];
#pragma unroll
        for (int j = 0; j < kMaxK; ++j) {
            rows[j] = 0;
            wt[j] = 0.0f;
            if (j < n) {
                const int s = __ffsll(static_cast<unsigned long long>(vb)) - 1;
                rows[j] = __builtin_amdgcn_readlane(row, s);
                wt[j] = lane_value(wl, s);
                vb &= vb - 1;
            }
        }
        const Piece pc = row_piece(vpr, pieces, it - u * pieces);
        u32x4* dst = out + static_cast<size_t>(r0 + u) * vpr;
        for (int c0 = pc.begin + lane; c0 < pc.end; c0 += kWave * JB) {
            u32x4 v[kMaxK][JB];
#pragma unroll
            for (int r = 0; r < kMaxK; ++r) {
                if (r >= n) break;
                const u32x4* src = Y + static_cast<size_t>(rows[r]) * vpr;
#pragma unroll
                for (int j = 0; j < JB; ++j) {
                    const int c = c0 + j * kWave;
                    if (c < pc.end) v[r][j] = src[c];
                }
            }
#pragma unroll
            for (int j = 0; j < JB; ++j) {
                const int c = c0 + j * kWave;
                float acc[RowT::kElems];
#pragma unroll
                for (int e = 0; e < RowT::kElems; ++e) acc[e] = 0.0f;
#pragma unroll
                for (int r = 0; r < kMaxK; ++r) {
                    if (r >= n) break;
                    float f[RowT::kElems];
                    RowT::load(v[r][j], f);
#pragma unroll
                    for (int e = 0; e < RowT::kElems; ++e) acc[e] = __builtin_fmaf(wt[r], f[e], acc[e]);
                }
                if (c < pc.end) dst[c] = RowT::store(acc);
            }
        }
    }
}

// ---------------------------------------------------------------- src reduce
template <typename RowT, int JB>
__global__ __launch_bounds__(kThreads) void src_reduce_kernel(
    Topo g, int src_rank, int vpr, int pieces, const u32x4* __restrict__ parts,
    const int32_t* __restrict__ idx, const uint8_t* __restrict__ keep, const int32_t* __restrict__ er,
    const uint64_t* __restrict__ mask, const int32_t* __restrict__ copy_row,
    const int32_t* __restrict__ recv_offsets, const u32x4* __restrict__ shared,
    u32x4* __restrict__ out, int in_rows) {
    __shared__ int32_t dev_of[kMaxE];
    __shared__ int32_t roff[kMaxR + 1];
    for (int e = threadIdx.x; e < g.E; e += kThreads) dev_of[e] = er[e];
    if (threadIdx.x <= g.R) roff[threadIdx.x] = recv_offsets[threadIdx.x];
    __syncthreads();
    const int total = min(roff[g.R], in_rows);
    const int lane = lane_id();
    const int items = g.tpr * pieces;
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int it = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; it < items; it += nwaves) {
        const int i = it / pieces;
        const int t = src_rank * g.tpr + i;
        const uint64_t m = mask[t];
        int d = -1, cr = -1;
        if (lane < g.k) {
            const size_t q = static_cast<size_t>(t) * g.k + lane;
            const int e = idx[q];
            cr = copy_row[q];
            if (keep[q] && static_cast<unsigned>(e) < static_cast<unsigned>(g.E)) d = dev_of[e];
            if (static_cast<unsigned>(d) >= static_cast<unsigned>(g.R) || !((m >> d) & 1ull) || cr < 0) d = -1;
        }
        // one returned row per kept device (its first kept slot), ascending device
        bool first = d >= 0;
#pragma unroll
        for (int s2 = 0; s2 < kMaxK; ++s2) {
            const int d2 = __shfl(d, s2);
            if (s2 < lane && d2 == d) first = false;
        }
        int row = -1;
        if (first) {
            const int rr = roff[d] + cr;
            row = (rr >= 0 && rr < total) ? rr : -1;
        }
        int ord = 0;   // place of this lane's device among the valid devices
#pragma unroll
        for (int s2 = 0; s2 < kMaxK; ++s2) {
            const int d2 = __shfl(d, s2);
            const int row2 = __shfl(row, s2);
            if (row2 >= 0 && d2 < d) ++ord;
        }
        const uint64_t valid = __ballot(row >= 0);
        const int n = __popcll(valid);
        int rows[kMaxK];
#pragma unroll
        for (int j = 0; j < kMaxK; ++j) {
            rows[j] = 0;
            if (j < n) {
                // ords of the valid lanes are distinct, so exactly one lane answers
                const uint64_t at = __ballot(row >= 0 && ord == j);
                rows[j] = at ? __builtin_amdgcn_readlane(row, __ffsll(static_cast<unsigned long long>(at)) - 1) : 0;
            }
        }
        const Piece pc = row_piece(vpr, pieces, it - i * pieces);
        const size_t orow = static_cast<size_t>(i) * vpr;
        for (int c0 = pc.begin + lane; c0 < pc.end; c0 += kWave * JB) {
            u32x4 v[kMaxK + 1][JB];
#pragma unroll
            for (int j = 0; j < JB; ++j) {
                const int c = c0 + j * kWave;
                if (shared && c < pc.end) v[kMaxK][j] = shared[orow + c];
            }
#pragma unroll
            for (int r = 0; r < kMaxK; ++r) {
                if (r >= n) break;
                const u32x4* src = parts + static_cast<size_t>(rows[r]) * vpr;
#pragma unroll
                for (int j = 0; j < JB; ++j) {
                    const int c = c0 + j * kWave;
                    if (c < pc.end) v[r][j] = src[c];
                }
            }
#pragma unroll
            for (int j = 0; j < JB; ++j) {
                const int c = c0 + j * kWave;
                float acc[RowT::kElems];
                if (shared) {
                    RowT::load(v[kMaxK][j], acc);
                } else {
#pragma unroll
                    for (int e = 0; e < RowT::kElems; ++e) acc[e] = 0.0f;
                }
#pragma unroll
                for (int r = 0; r < kMaxK; ++r) {
                    if (r >= n) break;
                    float f[RowT::kElems];
                    RowT::load(v[r][j], f);
#pragma unroll
                    for (int e = 0; e < RowT::kElems; ++e) acc[e] += f[e];
                }
                if (c < pc.end) out[orow + c] = RowT::store(acc);
            }
        }
    }
}

Topo make_topo(const cap_topology* tp) {
    Topo g;
    g.T = tp->T; g.E = tp->E; g.k = tp->k; g.R = tp->R; g.tpr = tp->tokens_per_rank;
    g.E_loc = tp->E / tp->R;
    return g;
}

// Pieces per row: split rows (in whole 64-lane chunk groups) only when the
// rows alone would leave the chip short of waves.
int row_pieces(long long rows_upper, int vpr) {
    int p = 1;
    while (p < 4 && rows_upper * p < kTargetWaves && vpr >= 2 * p * kWave) p *= 2;
    return p;
}

int row_grid(long long items_upper) {
    const long long need = (items_upper + kWavesPerBlock - 1) / kWavesPerBlock;
    const long long cap = static_cast<long long>(device_cu_count()) * 8;
    return static_cast<int>(need < 1 ? 1 : (need < cap ? need : cap));
}

}  // namespace

cap_status row_plan_launch(const cap_topology* tp, int rank, const float* w, const cap_layout* lay, int32_t* row_src,
                           int32_t* row_dst, float* row_w, int rows_cap, int parts_rows, hipStream_t st) {
    const Topo g = make_topo(tp);
    const long long items = static_cast<long long>(g.T) * g.k;
    long long grid = (items + kThreads - 1) / kThreads;
    const long long cap = static_cast<long long>(device_cu_count()) * 8;
    grid = grid < 1 ? 1 : (grid < cap ? grid : cap);
    row_plan_kernel<<<static_cast<int>(grid), kThreads, 0, st>>>(g, rank, w, lay->slot_pos, lay->expert_offsets,
                                                                 lay->recv_offsets, lay->recv_token, row_src,
                                                                 row_dst, row_w, rows_cap, parts_rows);
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

cap_status permute_launch(const cap_topology* tp, cap_permute_mode mode, int rank, cap_dtype dt, int d,
                          const void* x, const int32_t* idx, const uint8_t* keep, const uint64_t* mask,
                          const cap_layout* lay, void* out, int out_rows, hipStream_t st) {
    const Topo g = make_topo(tp);
    if (mode == CAP_PERMUTE_ROW_SOURCE) {
        const long long items = static_cast<long long>(g.T) * g.k;
        long long grid = (items + kThreads - 1) / kThreads;
        const long long cap = static_cast<long long>(device_cu_count()) * 8;
        grid = grid < 1 ? 1 : (grid < cap ? grid : cap);
        row_source_kernel<<<static_cast<int>(grid), kThreads, 0, st>>>(
            g, rank, lay->slot_pos, lay->expert_offsets, lay->recv_offsets, lay->recv_token,
            static_cast<int32_t*>(out), out_rows);
        CAP_LAUNCH_CHECK();
        return CAP_OK;
    }
    const int row_bytes = d * (dt == CAP_DTYPE_BF16 ? 2 : 4);
    const int vpr = row_bytes / 16;
    const u32x4* xv = static_cast<const u32x4*>(x);
    u32x4* ov = static_cast<u32x4*>(out);
    if (mode == CAP_PERMUTE_EXPERT_GATHER) {
        const int pieces = row_pieces(g.T, vpr);
        expert_gather_kernel<4><<<row_grid(static_cast<long long>(g.T) * pieces), kThreads, 0, st>>>(
            g, rank, vpr, pieces, xv, lay->slot_pos, lay->expert_offsets, lay->recv_offsets, lay->recv_token,
            ov, out_rows);
    } else {
        const int pieces = row_pieces(g.tpr, vpr);
        send_pack_kernel<4><<<row_grid(static_cast<long long>(g.tpr) * pieces), kThreads, 0, st>>>(
            g, rank, vpr, pieces, xv, idx, keep, tp->expert_rank, mask, lay->copy_row, lay->send_counts,
            lay->send_offsets, ov, out_rows);
    }
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

cap_status combine_launch(const cap_topology* tp, cap_combine_mode mode, int rank, cap_dtype dt, int d,
                          const void* in, int in_rows, const int32_t* idx, const float* w, const uint8_t* keep,
                          const uint64_t* mask, const cap_layout* lay, const void* shared_out, void* out,
                          int out_rows, hipStream_t st) {
    const Topo g = make_topo(tp);
    const int vpr = d * (dt == CAP_DTYPE_BF16 ? 2 : 4) / 16;
    const u32x4* iv = static_cast<const u32x4*>(in);
    const u32x4* sv = static_cast<const u32x4*>(shared_out);
    u32x4* ov = static_cast<u32x4*>(out);
    if (mode == CAP_COMBINE_DEST_REDUCE || mode == CAP_COMBINE_DEST_REDUCE_MULTI) {
        const int skip = mode == CAP_COMBINE_DEST_REDUCE_MULTI ? 1 : 0;
        const int pieces = row_pieces(g.T, vpr);
        const int grid = row_grid(static_cast<long long>(g.T) * pieces);
        if (dt == CAP_DTYPE_BF16)
            dest_reduce_kernel<Bf16Row, 2><<<grid, kThreads, 0, st>>>(
                g, rank, vpr, pieces, iv, w, lay->slot_pos, lay->expert_offsets, lay->recv_offsets,
                lay->recv_token, ov, in_rows, out_rows, skip);
        else
            dest_reduce_kernel<F32Row, 2><<<grid, kThreads, 0, st>>>(
                g, rank, vpr, pieces, iv, w, lay->slot_pos, lay->expert_offsets, lay->recv_offsets,
                lay->recv_token, ov, in_rows, out_rows, skip);
    } else {
        const int pieces = row_pieces(g.tpr, vpr);
        const int grid = row_grid(static_cast<long long>(g.tpr) * pieces);
        if (dt == CAP_DTYPE_BF16)
            src_reduce_kernel<Bf16Row, 2><<<grid, kThreads, 0, st>>>(
                g, rank, vpr, pieces, iv, idx, keep, tp->expert_rank, mask, lay->copy_row, lay->recv_offsets,
                sv, ov, in_rows);
        else
            src_reduce_kernel<F32Row, 2><<<grid, kThreads, 0, st>>>(
                g, rank, vpr, pieces, iv, idx, keep, tp->expert_rank, mask, lay->copy_row, lay->recv_offsets,
                sv, ov, in_rows);
    }
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

}  // namespace cap
