// Expert co-activation counts on the pruned routing (Sec. IV-B: how often two
// experts are selected together; Sec. VII: placement runs on pruned traces).
//
// Two launches, no global atomics, deterministic (integer sums):
//   1. tile    block (row group of 16 experts, token split): an LDS tile
//              [16][E] of counts; each token adds 1 to (i, j) for every kept
//              expert i in the row group and every kept expert j (i == j gives
//              the diagonal N_i).  LDS integer atomics: the sum is order
//              independent.  The tile is written to its split's partial slab.
//   2. reduce  coact[i][j] = (accumulate ? coact[i][j] : 0) + sum over splits,
//              in split order.
// Workspace: [S][E][E] uint32 partials.
#include "cap_device.hpp"

namespace cap {
namespace {

constexpr int kRows = 16;
constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void coact_tile_kernel(
    int T, int k, int E, int tokens_per_split, const int32_t* __restrict__ idx,
    const uint8_t* __restrict__ keep, uint32_t* __restrict__ part) {
    __shared__ uint32_t tile[kRows * kMaxE];
    const int r0 = blockIdx.x * kRows;
    const int split = blockIdx.y;
    for (int i = threadIdx.x; i < kRows * E; i += kThreads) tile[i] = 0;
    __syncthreads();
    const int t_begin = split * tokens_per_split;
    const int t_end = min(T, t_begin + tokens_per_split);
    for (int t = t_begin + threadIdx.x; t < t_end; t += kThreads) {
        int e[kMaxK];
        int n = 0;
        for (int s = 0; s < k; ++s) {
            const size_t q = static_cast<size_t>(t) * k + s;
            const int x = idx[q];
            if (keep[q] && static_cast<unsigned>(x) < static_cast<unsigned>(E)) e[n++] = x;
        }
        for (int a = 0; a < n; ++a) {
            const int i = e[a] - r0;
            if (static_cast<unsigned>(i) >= static_cast<unsigned>(kRows)) continue;
            for (int b = 0; b < n; ++b) atomicAdd(&tile[i * E + e[b]], 1u);
        }
    }
    __syncthreads();
    const int rows = min(kRows, E - r0);
    uint32_t* out = part + (static_cast<size_t>(split) * E + r0) * E;
    for (int i = threadIdx.x; i < rows * E; i += kThreads) out[i] = tile[i];
}

__global__ __launch_bounds__(kThreads) void coact_reduce_kernel(
    int E, int splits, int accumulate, const uint32_t* __restrict__ part, uint32_t* __restrict__ coact) {
    const int n = E * E;
    for (int i = blockIdx.x * kThreads + threadIdx.x; i < n; i += gridDim.x * kThreads) {
        uint32_t v = accumulate ? coact[i] : 0u;
        for (int s = 0; s < splits; ++s) v += part[static_cast<size_t>(s) * n + i];
        coact[i] = v;
    }
}

int coact_splits(int T, int E) {
    const int row_groups = (E + kRows - 1) / kRows;
    int s = (512 + row_groups - 1) / row_groups;     // aim for ~512 tile blocks
    const int max_s = (T + 255) / 256;               // at least 256 tokens per split
    if (s > max_s) s = max_s;
    if (s > 64) s = 64;
    return s < 1 ? 1 : s;
}

}  // namespace

size_t coact_workspace_bytes(int T, int E) {
    return static_cast<size_t>(coact_splits(T, E)) * E * E * sizeof(uint32_t);
}

cap_status coactivation_launch(int T, int k, int E, const int32_t* idx, const uint8_t* keep, uint32_t* coact,
                               int accumulate, void* ws, hipStream_t st) {
    const int S = coact_splits(T, E);
    const int per = (T + S - 1) / S;
    dim3 grid((E + kRows - 1) / kRows, S);
    uint32_t* part = static_cast<uint32_t*>(ws);
    coact_tile_kernel<<<grid, kThreads, 0, st>>>(T, k, E, per, idx, keep, part);
    CAP_LAUNCH_CHECK();
    const int blocks = (E * E + kThreads - 1) / kThreads;
    coact_reduce_kernel<<<blocks, kThreads, 0, st>>>(E, S, accumulate, part, coact);
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

}  // namespace cap
