// Adjustment Approach of the communication-computation trade-off (Sec. V):
// starting from the communication-oriented placement, repeatedly swap one
// expert of the most loaded device with one of the least loaded device,
// choosing, among the swaps that lower the larger of the two loads, the one
// that raises the communication objective C (Eq. 2-3) least.  The placements
// after each swap form the placement spectrum; the load of a device is the
// number of rows it computes (Eq. 4: L_g = sum of N_e over its experts, with
// N_e the kept (token, expert) pairs of expert e, the diagonal of the
// co-activation counts).
//
// Readings where the paper is open (the same as the host implementation):
//   p_ij     C_ij / (N_i + N_j - C_ij) (0 when the denominator is 0);
//   devices  the most loaded (ties: lower id) and the least loaded (ties:
//            lower id); the spectrum ends when their loads are equal;
//   swaps    e on the former and f on the latter with N_e > N_f and
//            L_lo + N_e - N_f < L_hi (the larger load falls);
//   choice   the smallest increase of C, ties by lower e, then lower f; the
//            increase is summed over the pairs whose distance changes: for
//            every other expert j, ascending, p_ej (d(lo, pi_j) - d(hi, pi_j))
//            then p_fj (d(hi, pi_j) - d(lo, pi_j)), in fp64 without
//            contraction (d = 0 / 1 / c, Eq. 3; c is the fp32 argument);
//   e and f exchange devices and local slots.
//
// One launch computes p into the workspace with many workgroups; a second
// launch of ONE workgroup runs the whole swap sequence: per step, one thread
// per candidate (strided), each summing its increase sequentially; a
// fixed-order reduction picks the first minimum, so the sequence is
// deterministic.  Every loop is bounded (max_swaps steps).
#pragma clang fp contract(off)

#include "cap_device.hpp"

namespace cap {
namespace {

constexpr int kAdjThreads = 1024;

__global__ __launch_bounds__(256) void coact_probability_kernel(const uint32_t* __restrict__ C, int E,
                                                                double* __restrict__ P) {
    const int n = E * E;
    for (int x = blockIdx.x * blockDim.x + threadIdx.x; x < n; x += gridDim.x * blockDim.x) {
        const int i = x / E, j = x % E;
        double p = 0.0;
        if (i != j) {
            const double cij = static_cast<double>(C[x]);
            const double den = static_cast<double>(C[i * E + i]) + static_cast<double>(C[j * E + j]) - cij;
            p = den > 0.0 ? cij / den : 0.0;
        }
        P[x] = p;
    }
}

__device__ __forceinline__ double device_distance(int a, int b, int rpn, double c) {
    return a == b ? 0.0 : ((a / rpn == b / rpn) ? 1.0 : c);
}

__global__ __launch_bounds__(kAdjThreads) void adjustment_kernel(
    const uint32_t* __restrict__ C, const double* __restrict__ P, int E, int R, int rpn, float c_f,
    int32_t* __restrict__ expert_rank, int32_t* __restrict__ expert_local, int max_swaps,
    int32_t* __restrict__ swaps, double* __restrict__ deltas, int32_t* __restrict__ n_swaps) {
    __shared__ int er[kMaxE], el[kMaxE];
    __shared__ long long N[kMaxE];
    __shared__ long long L[kMaxR];
    __shared__ int es[kMaxE], fs[kMaxE];
    __shared__ int ctl[4];                       // hi, lo, |es|, |fs|
    __shared__ double best_d[kAdjThreads / kWave];
    __shared__ int best_k[kAdjThreads / kWave];
    const int tid = threadIdx.x;
    const double c = static_cast<double>(c_f);
    for (int e = tid; e < E; e += blockDim.x) {
        er[e] = expert_rank[e];
        el[e] = expert_local[e];
        N[e] = static_cast<long long>(C[e * E + e]);
    }
    __syncthreads();
    int done = 0;
    int step = 0;
    for (; step < max_swaps; ++step) {
        // device loads, each a sequential integer sum over ascending experts
        for (int g = tid; g < R; g += blockDim.x) {
            long long s = 0;
            for (int e = 0; e < E; ++e) s += (er[e] == g) ? N[e] : 0;
            L[g] = s;
        }
        __syncthreads();
        if (tid == 0) {
            int hi = 0, lo = 0;
            for (int g = 1; g < R; ++g) {
                if (L[g] > L[hi]) hi = g;
                if (L[g] < L[lo]) lo = g;
            }
            int ne = 0, nf = 0;
            for (int e = 0; e < E; ++e) {
                if (er[e] == hi) es[ne++] = e;
                if (er[e] == lo) fs[nf++] = e;
            }
            ctl[0] = hi;
            ctl[1] = lo;
            ctl[2] = ne;
            ctl[3] = (L[hi] == L[lo]) ? 0 : nf;  // no candidates once the loads are equal
        }
        __syncthreads();
        const int hi = ctl[0], lo = ctl[1], ne = ctl[2], nf = ctl[3];
        const long long Lhi = L[hi], Llo = L[lo];
        // this thread's first minimum over its candidates k = ie * nf + if
        double bd = 0.0;
        int bk = -1;
        for (int k = tid; k < ne * nf; k += blockDim.x) {
            const int e = es[k / nf], f = fs[k % nf];
            if (!(N[e] > N[f] && Llo + N[e] - N[f] < Lhi)) continue;
            const double* pe = P + static_cast<size_t>(e) * E;
            const double* pf = P + static_cast<size_t>(f) * E;
            double d = 0.0;
            for (int j = 0; j < E; ++j) {
                if (j == e || j == f) continue;
                const int g = er[j];
                const double a = device_distance(lo, g, rpn, c) - device_distance(hi, g, rpn, c);
                d = d + pe[j] * a;
                d = d + pf[j] * -a;
            }
            if (bk < 0 || d < bd) {
                bd = d;
                bk = k;
            }
        }
        // fixed-order reduction: smaller increase, then lower candidate index
        auto better = [](double d1, int k1, double d2, int k2) {
            if (k2 < 0) return true;
            if (k1 < 0) return false;
            return d1 < d2 || (d1 == d2 && k1 < k2);
        };
        for (int off = kWave / 2; off >= 1; off >>= 1) {
            const double od = __shfl_down(bd, off);
            const int ok = __shfl_down(bk, off);
            if (better(od, ok, bd, bk)) {
                bd = od;
                bk = ok;
            }
        }
        if (lane_id() == 0) {
            best_d[tid / kWave] = bd;
            best_k[tid / kWave] = bk;
        }
        __syncthreads();
        if (tid == 0) {
            double d = 0.0;
            int k = -1;
            for (int w = 0; w < static_cast<int>(blockDim.x) / kWave; ++w)
                if (better(best_d[w], best_k[w], d, k)) {
                    d = best_d[w];
                    k = best_k[w];
                }
            if (k < 0) {
                ctl[2] = -1;                     // no swap applies: the spectrum ends
            } else {
                const int e = es[k / nf], f = fs[k % nf];
                er[e] = lo;
                er[f] = hi;
                const int t = el[e];
                el[e] = el[f];
                el[f] = t;
                swaps[2 * step] = e;
                swaps[2 * step + 1] = f;
                if (deltas) deltas[step] = d;
            }
        }
        __syncthreads();
        done = ctl[2] < 0;
        __syncthreads();
        if (done) break;
    }
    for (int e = tid; e < E; e += blockDim.x) {
        expert_rank[e] = er[e];
        expert_local[e] = el[e];
    }
    if (tid == 0) *n_swaps = step;
}

}  // namespace

size_t adjustment_workspace_bytes(int E) { return static_cast<size_t>(E) * E * sizeof(double); }

cap_status adjustment_launch(const uint32_t* coact, int E, int R, int rpn, float c, int32_t* expert_rank,
                             int32_t* expert_local, int max_swaps, int32_t* swaps, double* deltas,
                             int32_t* n_swaps, void* ws, hipStream_t st) {
    double* P = static_cast<double*>(ws);
    const int blocks = (E * E + 255) / 256;
    coact_probability_kernel<<<blocks, 256, 0, st>>>(coact, E, P);
    CAP_LAUNCH_CHECK();
    adjustment_kernel<<<1, kAdjThreads, 0, st>>>(coact, P, E, R, rpn, c, expert_rank, expert_local, max_swaps,
                                                 swaps, deltas, n_swaps);
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

}  // namespace cap
