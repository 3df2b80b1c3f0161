// Kernels of the expert co-activation counts, shared by the co-activation
// call and the fused front end (see coactivation.hip for the method).
#pragma once

#include <math.h>

#include "cap_device.hpp"

namespace cap {
namespace {


constexpr int kThreads = 256;          // reduce blocks
constexpr int kTileThreads = 256;      // tile blocks: one token per thread
constexpr int kSplitTokens = 256;      // tokens per split (up to 512 keep k^2 x tokens below 2^16)
static_assert(kSplitTokens == kTileThreads && kSplitTokens <= 512, "one token per tile thread");
constexpr int kTriWordsMax = (kMaxE * (kMaxE + 1) / 2 + 1) / 2;
constexpr int kTriQuadsMax = (kTriWordsMax + 3) / 4;
constexpr int kReduceQuads = 32;                       // 16-byte columns per reduce block
constexpr int kReduceGroups = kThreads / kReduceQuads; // split groups per reduce block
static_assert(kReduceQuads * 8 == kThreads, "one triangle entry per reduce thread");

__host__ __device__ inline int tri_size(int E) { return E * (E + 1) / 2; }
__host__ __device__ inline int tri_words(int E) { return (tri_size(E) + 1) / 2; }
// A split's slab is padded to whole 16-byte quads (the padding stays zero).
__host__ __device__ inline int tri_quads(int E) { return (tri_words(E) + 3) / 4; }
__device__ __forceinline__ int row_start(int i, int E) {
    return static_cast<int>(__umul24(i, E) - (__umul24(i, i - 1) >> 1));   // i < 2^12, so 24-bit products
}
__device__ __forceinline__ int tri_index(int i, int j, int E) { return row_start(i, E) + (j - i); }

// Split bid: tokens [bid * tokens_per_split, ...) -> packed partial triangle.
__device__ __forceinline__ void coact_tile_block(int T, int k, int E, int tokens_per_split,
                                                 const int32_t* __restrict__ idx, const uint8_t* __restrict__ keep,
                                                 uint32_t* __restrict__ part, int bid) {
    __shared__ uint4 tri4[kTriQuadsMax];
    uint32_t* tri = reinterpret_cast<uint32_t*>(tri4);
    const int TQ = tri_quads(E);
    for (int i = threadIdx.x; i < TQ; i += kTileThreads) tri4[i] = make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();
    const int t_begin = bid * tokens_per_split;
    const int t_end = min(T, t_begin + tokens_per_split);
    for (int t = t_begin + threadIdx.x; t < t_end; t += kTileThreads) {
        int e[kMaxK];
        bool kp[kMaxK];
        // every slot loaded unconditionally (slots past k reload slot k - 1 and
        // are dropped below), so all the loads go out before the first wait
        const size_t q0 = static_cast<size_t>(t) * k;
#pragma unroll
        for (int s = 0; s < kMaxK; ++s) {
            const size_t q = q0 + min(s, k - 1);
            e[s] = idx[q];
            kp[s] = keep[q] != 0;
        }
#pragma unroll
        for (int s = 0; s < kMaxK; ++s)
            kp[s] = kp[s] && s < k && static_cast<unsigned>(e[s]) < static_cast<unsigned>(E);
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
    // the slab out in 16-byte pieces, four LDS reads in flight per thread
    // (indices past the end are clamped to the last quad, which is then
    // written more than once with the same value: no branch, no early wait)
    uint4* out = reinterpret_cast<uint4*>(part) + static_cast<size_t>(bid) * TQ;
    for (int i0 = threadIdx.x; i0 < TQ; i0 += 4 * kTileThreads) {
        uint4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = tri4[min(i0 + u * kTileThreads, TQ - 1)];
#pragma unroll
        for (int u = 0; u < 4; ++u) out[min(i0 + u * kTileThreads, TQ - 1)] = v[u];
    }
}

__global__ __launch_bounds__(kTileThreads) void coact_tile_kernel(
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

// Reduce block bid: packed quads [bid * kReduceQuads, ...) over every split
// (8 split groups of 32 threads, each thread one 16-byte column), then thread
// i owns triangle entry bid * 256 + i: the groups' sums in a fixed order.
__device__ __forceinline__ void coact_reduce_block(int E, int splits, int accumulate,
                                                   const uint32_t* __restrict__ part, uint32_t* __restrict__ coact,
                                                   int bid) {
    __shared__ uint32_t acc_s[kReduceGroups][kReduceQuads * 8];
    const int TQ = tri_quads(E);
    const int ql = threadIdx.x % kReduceQuads;
    const int grp = threadIdx.x / kReduceQuads;
    const int q = bid * kReduceQuads + ql;
    uint32_t lo[4] = {0u, 0u, 0u, 0u}, hi[4] = {0u, 0u, 0u, 0u};
    if (q < TQ) {
        const uint4* src = reinterpret_cast<const uint4*>(part) + q;
        for (int s0 = grp * 8; s0 < splits; s0 += kReduceGroups * 8) {
            uint4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                v[u] = src[static_cast<size_t>(min(s0 + u, splits - 1)) * TQ];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const uint32_t m = (s0 + u < splits) ? ~0u : 0u;   // splits past the end count 0
                v[u].x &= m; v[u].y &= m; v[u].z &= m; v[u].w &= m;
                lo[0] += v[u].x & 0xFFFFu; hi[0] += v[u].x >> 16;
                lo[1] += v[u].y & 0xFFFFu; hi[1] += v[u].y >> 16;
                lo[2] += v[u].z & 0xFFFFu; hi[2] += v[u].z >> 16;
                lo[3] += v[u].w & 0xFFFFu; hi[3] += v[u].w >> 16;
            }
        }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        acc_s[grp][8 * ql + 2 * c] = lo[c];
        acc_s[grp][8 * ql + 2 * c + 1] = hi[c];
    }
    __syncthreads();
    uint32_t sum = 0;
#pragma unroll
    for (int g2 = 0; g2 < kReduceGroups; ++g2) sum += acc_s[g2][threadIdx.x];
    const int x = bid * (kReduceQuads * 8) + threadIdx.x;
    if (x < tri_size(E)) {
        int i, j;
        tri_coords(x, E, i, j);
        const size_t ij = static_cast<size_t>(i) * E + j;
        const size_t ji = static_cast<size_t>(j) * E + i;
        coact[ij] = (accumulate ? coact[ij] : 0u) + sum;
        if (i != j) coact[ji] = (accumulate ? coact[ji] : 0u) + sum;
    }
}

__global__ __launch_bounds__(kThreads) void coact_reduce_kernel(
    int E, int splits, int accumulate, const uint32_t* __restrict__ part, uint32_t* __restrict__ coact) {
    coact_reduce_block(E, splits, accumulate, part, coact, blockIdx.x);
}

inline int coact_tokens_per_split(int) { return kSplitTokens; }

inline int coact_splits(int T) {
    const int per = coact_tokens_per_split(T);
    return (T + per - 1) / per;
}

inline int coact_reduce_blocks(int E) { return (tri_quads(E) + kReduceQuads - 1) / kReduceQuads; }
inline size_t coact_part_bytes(int T, int E) {
    return static_cast<size_t>(coact_splits(T)) * tri_quads(E) * 16;
}

}  // namespace
}  // namespace cap
