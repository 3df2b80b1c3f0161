// Per-token top-k routing, gates and communication-aware device pruning
// (Sec. II-A, Eq. 1; Sec. VI, Eq. 6 and its greedy), shared by the kernel that
// reads router logits from memory and the one that computes them in LDS.  The
// arithmetic and the packed-key networks are described in route_prune.hip.
#pragma once
#pragma clang fp contract(off)

#include <math.h>

#include "cap_device.hpp"

namespace cap {
namespace {

constexpr int kGroup = 8;              // lanes per token
constexpr int kTokensPerBlock = 32;    // 256 threads
constexpr double kNoKey = -1.0;        // below every packed key

// Gate exponential: Cody & Waite argument reduction with ln2 split as
// LN2_HI (ln 2 to 16 significant bits, exact products n*LN2_HI for |n| < 2^8)
// plus LN2_LO (fp32 nearest to ln2 - LN2_HI); Taylor polynomial of degree 7
// with fp32(1/j!) coefficients by Horner with fused multiply-add; scaled by
// 2^n.  Inputs below -87.33 give 0, so results are never subnormal.
__device__ __forceinline__ float gate_exp(float z) {
    const float n = __builtin_rintf(z * 1.44269504088896340736f);
    float r = __builtin_fmaf(-n, 0.693145751953125f, z);
    r = __builtin_fmaf(-n, 1.42860682030941723212e-6f, r);
    float q = (float)(1.0 / 5040.0);
    q = __builtin_fmaf(q, r, (float)(1.0 / 720.0));
    q = __builtin_fmaf(q, r, (float)(1.0 / 120.0));
    q = __builtin_fmaf(q, r, (float)(1.0 / 24.0));
    q = __builtin_fmaf(q, r, (float)(1.0 / 6.0));
    q = __builtin_fmaf(q, r, 0.5f);
    q = __builtin_fmaf(q, r, 1.0f);
    q = __builtin_fmaf(q, r, 1.0f);
    const float e = __builtin_ldexpf(q, static_cast<int>(n));
    return (z >= -87.33f) ? e : 0.0f;
}

// Order-preserving image of a float (total order on non-NaN values).
__device__ __forceinline__ uint32_t ordered_bits(float x) {
    const uint32_t b = __float_as_uint(x + 0.0f);   // -0.0 -> +0.0
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float from_ordered_bits(uint32_t u) {
    return __uint_as_float((u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u);
}

__device__ __forceinline__ double pack_key(float x, int e) {
    const uint64_t k = (static_cast<uint64_t>(ordered_bits(x)) << 30) | static_cast<uint64_t>(255 - e);
    return __longlong_as_double(static_cast<long long>(k));
}
__device__ __forceinline__ int key_expert(double k) {
    return 255 - static_cast<int>(static_cast<uint64_t>(__double_as_longlong(k)) & 255u);
}
__device__ __forceinline__ float key_logit(double k) {
    return from_ordered_bits(static_cast<uint32_t>(static_cast<uint64_t>(__double_as_longlong(k)) >> 30));
}

// Descending compare-exchange.
__device__ __forceinline__ void cx(double& a, double& b) {
    const double hi = __builtin_fmax(a, b);
    const double lo = __builtin_fmin(a, b);
    a = hi;
    b = lo;
}

// Bitonic sort (descending) of N = 2^m keys.
template <int N>
__device__ __forceinline__ void bitonic_sort(double (&v)[N]) {
#pragma unroll
    for (int size = 2; size <= N; size <<= 1) {
#pragma unroll
        for (int stride = size / 2; stride >= 1; stride >>= 1) {
#pragma unroll
            for (int i = 0; i < N; ++i) {
                const int j = i ^ stride;
                if (j > i) {
                    // descending within blocks whose (i & size) == 0, ascending otherwise
                    if ((i & size) == 0) cx(v[i], v[j]);
                    else cx(v[j], v[i]);
                }
            }
        }
    }
}

// a := top N of (a, b), both sorted descending; result sorted descending.
template <int N>
__device__ __forceinline__ void merge_top(double (&a)[N], const double (&b)[N]) {
#pragma unroll
    for (int s = 0; s < N; ++s) a[s] = __builtin_fmax(a[s], b[N - 1 - s]);   // bitonic
#pragma unroll
    for (int stride = N / 2; stride >= 1; stride >>= 1)
#pragma unroll
        for (int i = 0; i < N; ++i)
            if ((i & stride) == 0) cx(a[i], a[i + stride]);
}

// Lane swaps inside a group of 8 lanes (DPP): xor 1, xor 2 (quad permutes)
// and the mirror i <-> 7 - i (the third merge only needs each lane of one
// half paired with a lane of the other half).
template <int CTRL>
__device__ __forceinline__ double dpp_swap(double v) {
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(b), CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, static_cast<int>(b >> 32), CTRL, 0xF, 0xF, false);
    return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<uint32_t>(lo));
}
constexpr int kDppXor1 = 0xB1;          // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;          // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;   // row_half_mirror

template <int CTRL, int N>
__device__ __forceinline__ void merge_with_partner(double (&a)[N]) {
    double b[N];
#pragma unroll
    for (int s = 0; s < N; ++s) b[s] = dpp_swap<CTRL>(a[s]);
    merge_top<N>(a, b);
}

constexpr int pow2_at_least(int k) { return k <= 1 ? 1 : k <= 2 ? 2 : k <= 4 ? 4 : 8; }

// Value of lane s of the caller's 8-lane group (ds_swizzle, bit-mask mode:
// lane = (lane & 0b11000) | s within each 32-lane half).
template <int S>
__device__ __forceinline__ int group_lane(int v) {
    return __builtin_amdgcn_ds_swizzle(v, 0x18 | (S << 5));
}
template <int S>
__device__ __forceinline__ float group_lane(float v) {
    return __int_as_float(group_lane<S>(__float_as_int(v)));
}

// One step of a descending sort across the 8 lanes: the lane that is `lower`
// in its pair keeps the larger (key, a), the other keeps the smaller.
template <int CTRL>
__device__ __forceinline__ void lane_cx(double& key, float& a, bool lower) {
    const double pk = dpp_swap<CTRL>(key);
    const float pa = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(a), CTRL, 0xF, 0xF, false));
    const bool take = lower ? (pk > key) : (pk < key);
    key = take ? pk : key;
    a = take ? pa : a;
}
constexpr int kDppMirror4 = 0x1B;       // quad_perm [3,2,1,0]

// What a lane knows of its token after the decision: the expert of its slot
// (lane g < K), whether that slot is kept, and the token's device mask.
struct RouteResult {
    int e;
    bool has_slot, keep;
    uint64_t mask;
};

// The whole decision for one token, from its logits: lane g (of the token's
// 8-lane group) holds vals[c * CW + i] = logit of expert c * (8 * CW) + g * CW
// + i, CW = min(V, 4).  er_lds[e] is the rank of expert e (LDS, ready).
// Writes idx / w' / keep for slot g (g < K) and the device mask (lane 0), and
// returns the lane's part of the result.
template <int V, int K, bool VEC, bool NAIVE>
__device__ __forceinline__ RouteResult route_token(const float (&vals)[V], int g, int t, bool live, int E, int R,
                                                   int ranks_per_node, int tokens_per_rank, float inter_node_cost,
                                                   float p, const int* er_lds, int32_t* __restrict__ out_idx,
                                                   float* __restrict__ out_w, uint8_t* __restrict__ out_keep,
                                                   uint64_t* __restrict__ out_mask) {
    constexpr int KP = pow2_at_least(K);
    constexpr int CW = V < 4 ? V : 4;
    double keys[V];
#pragma unroll
    for (int c = 0; c < V / CW; ++c)
#pragma unroll
        for (int i = 0; i < CW; ++i) {
            const int e = c * (kGroup * CW) + g * CW + i;
            keys[c * CW + i] = (VEC || e < E) ? pack_key(vals[c * CW + i], e) : kNoKey;
        }

    // ---- lane-local top KP: sort blocks of KP keys, merge them
    double top[KP];
    {
        constexpr int B = V < KP ? V : KP;     // keys per block
#pragma unroll
        for (int s = 0; s < KP; ++s) top[s] = s < B ? keys[s] : kNoKey;
        bitonic_sort<KP>(top);
#pragma unroll
        for (int b0 = KP; b0 < V; b0 += KP) {
            double blk[KP];
#pragma unroll
            for (int s = 0; s < KP; ++s) blk[s] = keys[b0 + s];
            bitonic_sort<KP>(blk);
            merge_top<KP>(top, blk);
        }
    }
    // ---- merge across the 8 lanes of the token
    merge_with_partner<kDppXor1, KP>(top);
    merge_with_partner<kDppXor2, KP>(top);
    merge_with_partner<kDppHalfMirror, KP>(top);

    // ---- lane g owns slot g (lanes g >= K own nothing)
    double mine = top[0];
#pragma unroll
    for (int s = 1; s < KP; ++s) mine = (g == s) ? top[s] : mine;
    const bool has_slot = g < K;
    const int my_e = key_expert(mine);
    const int my_dev = has_slot ? er_lds[my_e < E ? my_e : 0] : -1;

    // gates: q_g = gate_exp(l_g - l_0); S = ((q_0 + q_1) + ...) in slot order
    const float q = has_slot ? gate_exp(key_logit(mine) - key_logit(top[0])) : 0.0f;
    float qs[K];
    int devs[K];
#define CAP_GATHER_SLOT(S_)                                  \
    if constexpr (S_ < K) {                                  \
        qs[S_] = group_lane<S_>(q);                          \
        devs[S_] = group_lane<S_>(my_dev);                   \
    }
    CAP_GATHER_SLOT(0) CAP_GATHER_SLOT(1) CAP_GATHER_SLOT(2) CAP_GATHER_SLOT(3)
    CAP_GATHER_SLOT(4) CAP_GATHER_SLOT(5) CAP_GATHER_SLOT(6) CAP_GATHER_SLOT(7)
#undef CAP_GATHER_SLOT
    float S = 0.0f;
#pragma unroll
    for (int s = 0; s < K; ++s) S = S + qs[s];
    float ws[K];                               // every slot's gate, on every lane
#pragma unroll
    for (int s = 0; s < K; ++s) ws[s] = qs[s] / S;

    // ---- pruning
    const float target = 1.0f - p;
    const bool keep_all = (p == 0.0f);
    uint64_t mask = 0;
    float Sk = 0.0f;
    int n_keep = K;                         // naive: slots kept (a prefix)
    if constexpr (NAIVE) {
        // expert level: the shortest slot prefix whose running score reaches 1 - p
        float cum = 0.0f;
#pragma unroll
        for (int s = 0; s < K; ++s) {
            cum = cum + ws[s];
            if (!keep_all && n_keep == K && cum >= target) n_keep = s + 1;
        }
#pragma unroll
        for (int s = 0; s < K; ++s) {
            if (s < n_keep) mask |= 1ull << devs[s];
            Sk = Sk + ((s < n_keep) ? ws[s] : 0.0f);
        }
    } else {
        const int src = (live ? t : 0) / tokens_per_rank;
        const int src_node = src / ranks_per_node;
        // lane g is a candidate if slot g is the first slot of its device;
        // a = that device's score summed in slot order
        bool cand = has_slot;
        float a = 0.0f;
#pragma unroll
        for (int s = 0; s < K; ++s) {
            const bool same = devs[s] == my_dev;
            if (s < g) cand = cand && !same;
            a = a + ((s >= g && same) ? ws[s] : 0.0f);
        }
        float ratio = a;
        if (my_dev == src) ratio = INFINITY;
        else if (R > ranks_per_node && my_dev / ranks_per_node != src_node) ratio = a / inter_node_cost;
        const uint64_t kbits = (1ull << 61) | (static_cast<uint64_t>(__float_as_uint(ratio)) << 30) |
                               (static_cast<uint64_t>(63 - (my_dev & 63)) << 3);
        double ck = cand ? __longlong_as_double(static_cast<long long>(kbits)) : kNoKey;
        float ca = a;
        // descending sort across the group (bitonic, mirrored first step per stage)
        lane_cx<kDppXor1>(ck, ca, (g & 1) == 0);
        lane_cx<kDppMirror4>(ck, ca, (g & 3) < 2);
        lane_cx<kDppXor1>(ck, ca, (g & 1) == 0);
        lane_cx<kDppHalfMirror>(ck, ca, g < 4);
        lane_cx<kDppXor2>(ck, ca, (g & 2) == 0);
        lane_cx<kDppXor1>(ck, ca, (g & 1) == 0);
        // greedy retention in key order, replayed by every lane
        const uint32_t ck_hi = static_cast<uint32_t>(static_cast<uint64_t>(__double_as_longlong(ck)) >> 32);
        const int ck_lo = static_cast<int>(static_cast<uint64_t>(__double_as_longlong(ck)));
        float cum = 0.0f;
        bool done = false;
#define CAP_GREEDY_STEP(S_)                                                          \
        if constexpr (S_ < K) {                                                          \
            const bool c2 = (group_lane<S_>(static_cast<int>(ck_hi)) >> 29) == 1;        \
            const float a2 = group_lane<S_>(ca);                                         \
            const int d2 = 63 - ((group_lane<S_>(ck_lo) >> 3) & 63);                     \
            if (c2 && (keep_all || !done)) mask |= 1ull << d2;                           \
            cum = cum + (c2 ? a2 : 0.0f);                                                \
            done = done || (c2 && cum >= target);                                        \
        }
        CAP_GREEDY_STEP(0) CAP_GREEDY_STEP(1) CAP_GREEDY_STEP(2) CAP_GREEDY_STEP(3)
        CAP_GREEDY_STEP(4) CAP_GREEDY_STEP(5) CAP_GREEDY_STEP(6) CAP_GREEDY_STEP(7)
#undef CAP_GREEDY_STEP
#pragma unroll
        for (int s = 0; s < K; ++s) Sk = Sk + (((mask >> devs[s]) & 1ull) ? ws[s] : 0.0f);
    }

    // ---- lane g writes slot g
    const bool my_keep = has_slot && (NAIVE ? (g < n_keep) : ((mask >> (my_dev & 63)) & 1ull));
    if (live && has_slot) {
        float my_w = ws[0];
#pragma unroll
        for (int s = 1; s < K; ++s) my_w = (g == s) ? ws[s] : my_w;
        const size_t qi = static_cast<size_t>(t) * K + g;
        out_idx[qi] = my_e;
        out_w[qi] = my_keep ? my_w / Sk : 0.0f;
        out_keep[qi] = my_keep ? 1 : 0;
        if (g == 0) out_mask[t] = mask;
    }
    return RouteResult{my_e, has_slot, my_keep, mask};
}

}  // namespace
}  // namespace cap
