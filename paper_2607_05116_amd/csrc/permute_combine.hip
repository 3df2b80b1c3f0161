// Token permutation and weighted combine (Sec. II-C; Eq. 1).
//
// Both are HBM-bound row movers.  One wave owns one row at a time; each lane
// moves 16-byte pieces (8 bf16 or 4 fp32) so a wave touches 1 KiB per vector
// access, fully coalesced.  The grids are persistent (grid-stride over rows)
// and read the row counts from device memory, so nothing waits on the host.
//
//   expert gather  (dest rank r)  read each received token once, write it to
//                  every kept expert row of r (device-centric: one copy per
//                  device, shared by that device's experts).
//   send pack      (source rank s) read each token of s once, write one row per
//                  kept destination device into the send buffer.
//   dest reduce    (rank r) per received token: sum of w'_s * Y over the token's
//                  kept experts on r (local aggregation before the return).
//   src reduce     (rank s) per token of s: sum of the rows every kept device
//                  returned (+ the shared experts' output).
// Accumulation is fp32 in a fixed order (slot order / ascending device).
#include "cap_device.hpp"

namespace cap {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;

struct Topo {
    int T, E, k, R, tpr, E_loc;
};

__device__ __forceinline__ int expert_rank_of(const int32_t* er, int e, const Topo& g) {
    return static_cast<unsigned>(e) < static_cast<unsigned>(g.E) ? er[e] : -1;
}

// ---------------------------------------------------------------- expert gather
template <typename V>
__global__ __launch_bounds__(kThreads) void expert_gather_kernel(
    Topo g, int rank, int vec_per_row, const V* __restrict__ x, const int32_t* __restrict__ idx,
    const uint8_t* __restrict__ keep, const int32_t* __restrict__ er, const int32_t* __restrict__ slot_pos,
    const int32_t* __restrict__ expert_offsets, const int32_t* __restrict__ recv_offsets,
    const int32_t* __restrict__ recv_token, V* __restrict__ out, int out_rows) {
    const int r0 = recv_offsets[rank];
    const int U = min(recv_offsets[rank + 1] - r0, g.T * g.k - r0);
    const int base = expert_offsets[rank * g.E_loc];
    const int rows_r = min(expert_offsets[(rank + 1) * g.E_loc] - base, out_rows);
    if (r0 < 0) return;
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int u = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; u < U; u += nwaves) {
        const int t = recv_token[r0 + u];
        if (static_cast<unsigned>(t) >= static_cast<unsigned>(g.T)) continue;
        int dst[kMaxK];
#pragma unroll
        for (int s = 0; s < kMaxK; ++s) {
            dst[s] = -1;
            if (s < g.k) {
                const size_t q = static_cast<size_t>(t) * g.k + s;
                if (keep[q] && expert_rank_of(er, idx[q], g) == rank) {
                    const int row = slot_pos[q] - base;
                    dst[s] = (static_cast<unsigned>(row) < static_cast<unsigned>(rows_r)) ? row : -1;
                }
            }
        }
        const V* src = x + static_cast<size_t>(t) * vec_per_row;
        for (int c = lane_id(); c < vec_per_row; c += kWave) {
            const V v = src[c];
#pragma unroll
            for (int s = 0; s < kMaxK; ++s)
                if (dst[s] >= 0) out[static_cast<size_t>(dst[s]) * vec_per_row + c] = v;
        }
    }
}

// ---------------------------------------------------------------- send pack
template <typename V>
__global__ __launch_bounds__(kThreads) void send_pack_kernel(
    Topo g, int src_rank, int vec_per_row, const V* __restrict__ x, const int32_t* __restrict__ idx,
    const uint8_t* __restrict__ keep, const int32_t* __restrict__ er, const uint64_t* __restrict__ mask,
    const int32_t* __restrict__ copy_row, const int32_t* __restrict__ send_counts,
    const int32_t* __restrict__ send_offsets, V* __restrict__ out, int out_rows) {
    __shared__ int32_t row0[kMaxR];   // send_offsets[s][d] - (rows of d from sources < s)
    if (threadIdx.x < g.R) {
        const int d = threadIdx.x;
        int before = 0;
        for (int s2 = 0; s2 < src_rank; ++s2) before += send_counts[s2 * g.R + d];
        row0[d] = send_offsets[src_rank * g.R + d] - before;
    }
    __syncthreads();
    int total = 0;
    for (int d = 0; d < g.R; ++d) total += send_counts[src_rank * g.R + d];
    total = min(total, out_rows);
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int i = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; i < g.tpr; i += nwaves) {
        const int t = src_rank * g.tpr + i;
        const uint64_t m = mask[t];
        int dst[kMaxK];
#pragma unroll
        for (int s = 0; s < kMaxK; ++s) {
            dst[s] = -1;
            if (s < g.k) {
                const size_t q = static_cast<size_t>(t) * g.k + s;
                const int d = expert_rank_of(er, idx[q], g);
                if (keep[q] && d >= 0 && d < g.R && ((m >> d) & 1ull)) {
                    bool first = true;      // one row per device: the device's first kept slot writes it
                    for (int s2 = 0; s2 < s; ++s2) {
                        const size_t q2 = static_cast<size_t>(t) * g.k + s2;
                        if (keep[q2] && expert_rank_of(er, idx[q2], g) == d) first = false;
                    }
                    const int row = row0[d] + copy_row[q];
                    if (first && static_cast<unsigned>(row) < static_cast<unsigned>(total)) dst[s] = row;
                }
            }
        }
        const V* src = x + static_cast<size_t>(t) * vec_per_row;
        for (int c = lane_id(); c < vec_per_row; c += kWave) {
            const V v = src[c];
#pragma unroll
            for (int s = 0; s < kMaxK; ++s)
                if (dst[s] >= 0) out[static_cast<size_t>(dst[s]) * vec_per_row + c] = v;
        }
    }
}

// ---------------------------------------------------------------- row load / store helpers
struct Bf16Row {
    typedef uint4 V;                           // 8 bf16
    static constexpr int kElems = 8;
    __device__ static void load(const V& v, float* f) {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f[2 * i] = __uint_as_float(w[i] << 16);
            f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
        }
    }
    __device__ static V store(const float* f) {
        V v;
        v.x = pack_bf16x2(f[0], f[1]);
        v.y = pack_bf16x2(f[2], f[3]);
        v.z = pack_bf16x2(f[4], f[5]);
        v.w = pack_bf16x2(f[6], f[7]);
        return v;
    }
};

struct F32Row {
    typedef float4 V;
    static constexpr int kElems = 4;
    __device__ static void load(const V& v, float* f) { f[0] = v.x; f[1] = v.y; f[2] = v.z; f[3] = v.w; }
    __device__ static V store(const float* f) { return make_float4(f[0], f[1], f[2], f[3]); }
};

// ---------------------------------------------------------------- dest reduce
template <typename RowT>
__global__ __launch_bounds__(kThreads) void dest_reduce_kernel(
    Topo g, int rank, int vec_per_row, const typename RowT::V* __restrict__ Y,
    const int32_t* __restrict__ idx, const float* __restrict__ w, const uint8_t* __restrict__ keep,
    const int32_t* __restrict__ er, const int32_t* __restrict__ slot_pos,
    const int32_t* __restrict__ expert_offsets, const int32_t* __restrict__ recv_offsets,
    const int32_t* __restrict__ recv_token, typename RowT::V* __restrict__ out, int in_rows, int out_rows) {
    typedef typename RowT::V V;
    const int r0 = recv_offsets[rank];
    const int U = min(min(recv_offsets[rank + 1] - r0, g.T * g.k - r0), out_rows - r0);
    const int base = expert_offsets[rank * g.E_loc];
    const int rows_r = min(expert_offsets[(rank + 1) * g.E_loc] - base, in_rows);
    if (r0 < 0) return;
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int u = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; u < U; u += nwaves) {
        const int t = recv_token[r0 + u];
        int row[kMaxK];
        float wt[kMaxK];
#pragma unroll
        for (int s = 0; s < kMaxK; ++s) {
            row[s] = -1;
            wt[s] = 0.0f;
            if (s < g.k && static_cast<unsigned>(t) < static_cast<unsigned>(g.T)) {
                const size_t q = static_cast<size_t>(t) * g.k + s;
                if (keep[q] && expert_rank_of(er, idx[q], g) == rank) {
                    const int rr = slot_pos[q] - base;
                    if (static_cast<unsigned>(rr) < static_cast<unsigned>(rows_r)) { row[s] = rr; wt[s] = w[q]; }
                }
            }
        }
        V* dst = out + static_cast<size_t>(r0 + u) * vec_per_row;
        for (int c = lane_id(); c < vec_per_row; c += kWave) {
            float acc[RowT::kElems];
#pragma unroll
            for (int i = 0; i < RowT::kElems; ++i) acc[i] = 0.0f;
#pragma unroll
            for (int s = 0; s < kMaxK; ++s) {
                if (row[s] < 0) continue;
                float f[RowT::kElems];
                RowT::load(Y[static_cast<size_t>(row[s]) * vec_per_row + c], f);
#pragma unroll
                for (int i = 0; i < RowT::kElems; ++i) acc[i] = __builtin_fmaf(wt[s], f[i], acc[i]);
            }
            dst[c] = RowT::store(acc);
        }
    }
}

// ---------------------------------------------------------------- src reduce
template <typename RowT>
__global__ __launch_bounds__(kThreads) void src_reduce_kernel(
    Topo g, int src_rank, int vec_per_row, const typename RowT::V* __restrict__ parts,
    const int32_t* __restrict__ idx, const uint8_t* __restrict__ keep, const int32_t* __restrict__ er,
    const uint64_t* __restrict__ mask, const int32_t* __restrict__ copy_row,
    const int32_t* __restrict__ recv_offsets, const typename RowT::V* __restrict__ shared,
    typename RowT::V* __restrict__ out, int in_rows) {
    typedef typename RowT::V V;
    const int total = min(recv_offsets[g.R], in_rows);
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int i = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; i < g.tpr; i += nwaves) {
        const int t = src_rank * g.tpr + i;
        const uint64_t m = mask[t];
        // one returned row per kept device, ascending device id
        int rows[kMaxK];
        int n = 0;
        for (int d = 0; d < g.R && n < kMaxK; ++d) {
            if (!((m >> d) & 1ull)) continue;
            int cr = -1;
            for (int s = 0; s < g.k; ++s) {
                const size_t q = static_cast<size_t>(t) * g.k + s;
                if (cr < 0 && keep[q] && expert_rank_of(er, idx[q], g) == d) cr = copy_row[q];
            }
            const int row = recv_offsets[d] + cr;
            if (cr >= 0 && row >= 0 && row < total) rows[n++] = row;
        }
        V* dst = out + static_cast<size_t>(i) * vec_per_row;
        for (int c = lane_id(); c < vec_per_row; c += kWave) {
            float acc[RowT::kElems];
            if (shared) {
                RowT::load(shared[static_cast<size_t>(i) * vec_per_row + c], acc);
            } else {
#pragma unroll
                for (int j = 0; j < RowT::kElems; ++j) acc[j] = 0.0f;
            }
            for (int j = 0; j < n; ++j) {
                float f[RowT::kElems];
                RowT::load(parts[static_cast<size_t>(rows[j]) * vec_per_row + c], f);
#pragma unroll
                for (int e = 0; e < RowT::kElems; ++e) acc[e] += f[e];
            }
            dst[c] = RowT::store(acc);
        }
    }
}

Topo make_topo(const cap_topology* tp) {
    Topo g;
    g.T = tp->T; g.E = tp->E; g.k = tp->k; g.R = tp->R; g.tpr = tp->tokens_per_rank;
    g.E_loc = tp->E / tp->R;
    return g;
}

int row_grid(long long rows_upper) {
    const long long need = (rows_upper + kWavesPerBlock - 1) / kWavesPerBlock;
    const long long cap = static_cast<long long>(device_cu_count()) * 8;
    return static_cast<int>(need < 1 ? 1 : (need < cap ? need : cap));
}

}  // namespace

cap_status permute_launch(const cap_topology* tp, cap_permute_mode mode, int rank, cap_dtype dt, int d,
                          const void* x, const int32_t* idx, const uint8_t* keep, const uint64_t* mask,
                          const cap_layout* lay, void* out, int out_rows, hipStream_t st) {
    const Topo g = make_topo(tp);
    const int row_bytes = d * (dt == CAP_DTYPE_BF16 ? 2 : 4);
    const int vpr = row_bytes / 16;
    if (mode == CAP_PERMUTE_EXPERT_GATHER) {
        expert_gather_kernel<uint4><<<row_grid(g.T), kThreads, 0, st>>>(
            g, rank, vpr, static_cast<const uint4*>(x), idx, keep, tp->expert_rank, lay->slot_pos,
            lay->expert_offsets, lay->recv_offsets, lay->recv_token, static_cast<uint4*>(out), out_rows);
    } else {
        send_pack_kernel<uint4><<<row_grid(g.tpr), kThreads, 0, st>>>(
            g, rank, vpr, static_cast<const uint4*>(x), idx, keep, tp->expert_rank, mask, lay->copy_row,
            lay->send_counts, lay->send_offsets, static_cast<uint4*>(out), out_rows);
    }
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

cap_status combine_launch(const cap_topology* tp, cap_combine_mode mode, int rank, cap_dtype dt, int d,
                          const void* in, int in_rows, const int32_t* idx, const float* w, const uint8_t* keep,
                          const uint64_t* mask, const cap_layout* lay, const void* shared_out, void* out,
                          int out_rows, hipStream_t st) {
    const Topo g = make_topo(tp);
    if (mode == CAP_COMBINE_DEST_REDUCE) {
        if (dt == CAP_DTYPE_BF16) {
            dest_reduce_kernel<Bf16Row><<<row_grid(g.T), kThreads, 0, st>>>(
                g, rank, d / 8, static_cast<const uint4*>(in), idx, w, keep, tp->expert_rank, lay->slot_pos,
                lay->expert_offsets, lay->recv_offsets, lay->recv_token, static_cast<uint4*>(out), in_rows, out_rows);
        } else {
            dest_reduce_kernel<F32Row><<<row_grid(g.T), kThreads, 0, st>>>(
                g, rank, d / 4, static_cast<const float4*>(in), idx, w, keep, tp->expert_rank, lay->slot_pos,
                lay->expert_offsets, lay->recv_offsets, lay->recv_token, static_cast<float4*>(out), in_rows, out_rows);
        }
    } else {
        if (dt == CAP_DTYPE_BF16) {
            src_reduce_kernel<Bf16Row><<<row_grid(g.tpr), kThreads, 0, st>>>(
                g, rank, d / 8, static_cast<const uint4*>(in), idx, keep, tp->expert_rank, mask, lay->copy_row,
                lay->recv_offsets, static_cast<const uint4*>(shared_out), static_cast<uint4*>(out), in_rows);
        } else {
            src_reduce_kernel<F32Row><<<row_grid(g.tpr), kThreads, 0, st>>>(
                g, rank, d / 4, static_cast<const float4*>(in), idx, keep, tp->expert_rank, mask, lay->copy_row,
                lay->recv_offsets, static_cast<const float4*>(shared_out), static_cast<float4*>(out), in_rows);
        }
    }
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

}  // namespace cap
