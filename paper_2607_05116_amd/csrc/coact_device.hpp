// Kernels of the expert co-activation counts, shared by the co-activation
// call and the fused front end (see coactivation.hip for the method).
#pragma once

#include <math.h>

#include "cap_device.hpp"

namespace cap {
namespace {


constexpr int kThreads = 256;
constexpr int kMaxSplitTokens = 512;   // <= 512 tokens x k^2 pairs stays below 2^16
constexpr int kMaxSplits = 2048;
constexpr int kTriWordsMax = (kMaxE * (kMaxE + 1) / 2 + 1) / 2;
constexpr int kReduceWords = 32;                       // words per reduce block
constexpr int kReduceGroups = kThreads / kReduceWords; // split groups per reduce block

__host__ __device__ inline int tri_size(int E) { return E * (E + 1) / 2; }
__host__ __device__ inline int tri_words(int E) { return (tri_size(E) + 1) / 2; }
__device__ __forceinline__ int row_start(int i, int E) { return i * E - i * (i - 1) / 2; }
__device__ __forceinline__ int tri_index(int i, int j, int E) { return row_start(i, E) + (j - i); }

// Split bid: tokens [bid * tokens_per_split, ...) -> packed partial triangle.
__device__ __forceinline__ void coact_tile_block(int T, int k, int E, int tokens_per_split,
                                                 const int32_t* __restrict__ idx, const uint8_t* __restrict__ keep,
                                                 uint32_t* __restrict__ part, int bid) {
    __shared__ uint32_t tri[kTriWordsMax];
    const int TW = tri_words(E);
    for (int i = threadIdx.x; i < TW; i += kThreads) tri[i] = 0;
    __syncthreads();
    const int t_begin = bid * tokens_per_split;
    const int t_end = min(T, t_begin + tokens_per_split);
    for (int t = t_begin + threadIdx.x; t < t_end; t += kThreads) {
        int e[kMaxK];
        bool kp[kMaxK];
        const size_t q0 = static_cast<size_t>(t) * k;
#pragma unroll
        for (int s = 0; s < kMaxK; ++s) {
            e[s] = 0;
            kp[s] = false;
            if (s < k) {
                e[s] = idx[q0 + s];
                kp[s] = keep[q0 + s] != 0;
            }
        }
#pragma unroll
        for (int s = 0; s < kMaxK; ++s) kp[s] = kp[s] && static_cast<unsigned>(e[s]) < static_cast<unsigned>(E);
#pragma unroll
        for (int a = 0; a < kMaxK; ++a) {
#pragma unroll
            for (int b = a; b < kMaxK; ++b) {
                if (kp[a] && kp[b]) {
                    const int i = min(e[a], e[b]), j = max(e[a], e[b]);
                    const int x = tri_index(i, j, E);
                    const uint32_t inc = (a != b && i == j) ? 2u : 1u;
                    atomicAdd(&tri[x >> 1], inc << ((x & 1) * 16));
                }
            }
        }
    }
    __syncthreads();
    uint32_t* out = part + static_cast<size_t>(bid) * TW;
    for (int i = threadIdx.x; i < TW; i += kThreads) out[i] = tri[i];
}

__global__ __launch_bounds__(kThreads) void coact_tile_kernel(
    int T, int k, int E, int tokens_per_split, const int32_t* __restrict__ idx,
    const uint8_t* __restrict__ keep, uint32_t* __restrict__ part) {
    coact_tile_block(T, k, E, tokens_per_split, idx, keep, part, blockIdx.x);
}

// (i, j) of triangle entry x (row-major upper triangle of an E x E matrix).
__device__ __forceinline__ void tri_coords(int x, int E, int& i, int& j) {
    const double b = 2.0 * E + 1.0;
    int r = static_cast<int>((b - sqrt(b * b - 8.0 * x)) * 0.5);
    r = max(0, min(E - 1, r));
    if (r + 1 < E && row_start(r + 1, E) <= x) ++r;
    if (r > 0 && row_start(r, E) > x) --r;
    i = r;
    j = r + (x - row_start(r, E));
}

// Reduce block bid: packed words [bid * kReduceWords, ...) over every split.
__device__ __forceinline__ void coact_reduce_block(int E, int splits, int accumulate,
                                                   const uint32_t* __restrict__ part, uint32_t* __restrict__ coact,
                                                   int bid) {
    __shared__ uint32_t lo_s[kReduceGroups][kReduceWords];
    __shared__ uint32_t hi_s[kReduceGroups][kReduceWords];
    const int TW = tri_words(E);
    const int wl = threadIdx.x % kReduceWords;
    const int grp = threadIdx.x / kReduceWords;
    const int w = bid * kReduceWords + wl;
    uint32_t lo = 0, hi = 0;
    if (w < TW) {
        for (int s0 = grp * 8; s0 < splits; s0 += kReduceGroups * 8) {
            uint32_t v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = (s0 + u < splits) ? part[static_cast<size_t>(s0 + u) * TW + w] : 0u;
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                lo += v[u] & 0xFFFFu;
                hi += v[u] >> 16;
            }
        }
    }
    lo_s[grp][wl] = lo;
    hi_s[grp][wl] = hi;
    __syncthreads();
    if (grp < 2 && w < TW) {
        uint32_t sum = 0;
#pragma unroll
        for (int g2 = 0; g2 < kReduceGroups; ++g2) sum += grp == 0 ? lo_s[g2][wl] : hi_s[g2][wl];
        const int x = 2 * w + grp;
        if (x < tri_size(E)) {
            int i, j;
            tri_coords(x, E, i, j);
            const size_t ij = static_cast<size_t>(i) * E + j;
            const size_t ji = static_cast<size_t>(j) * E + i;
            coact[ij] = (accumulate ? coact[ij] : 0u) + sum;
            if (i != j) coact[ji] = (accumulate ? coact[ji] : 0u) + sum;
        }
    }
}

__global__ __launch_bounds__(kThreads) void coact_reduce_kernel(
    int E, int splits, int accumulate, const uint32_t* __restrict__ part, uint32_t* __restrict__ coact) {
    coact_reduce_block(E, splits, accumulate, part, coact, blockIdx.x);
}

inline int coact_tokens_per_split(int T) {
    int per = 256;
    while (per < kMaxSplitTokens && (T + per - 1) / per > kMaxSplits) per *= 2;
    return per;
}

inline int coact_splits(int T) {
    const int per = coact_tokens_per_split(T);
    return (T + per - 1) / per;
}

inline int coact_reduce_blocks(int E) { return (tri_words(E) + kReduceWords - 1) / kReduceWords; }

}  // namespace
}  // namespace cap
