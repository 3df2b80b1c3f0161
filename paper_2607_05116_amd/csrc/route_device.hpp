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
constexpr double kNoKey = -__builtin_inf();   // below every packed key

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

// Selection key of (logit x, expert e): the fp64 whose high word is the bits
// of x (with -0.0 folded to +0.0) and whose low word is 255 - e, with all 32
// bits of the low word complemented when x is negative.  fp64 order on such keys is the selection
// order: sign and magnitude of the high word order the logits as fp32 order
// does, and within one logit the low word puts the lower expert first on
// either side of zero (complementing reverses the order of the magnitudes of
// negative keys).  No key is NaN or infinite for finite logits; keys of 0.0
// and of tiny subnormal logits are fp64 subnormals, compared exactly because
// fp64 denormals are not flushed.
__device__ __forceinline__ double pack_key(float x, uint32_t tie_g, uint32_t tie_c) {
    const uint32_t hi = __float_as_uint(x + 0.0f);
    uint32_t lo;
    // lo = sign mask ^ tie_g ^ tie_c in one three-input bit op (truth table 0x96)
    asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(lo) : "v"(static_cast<int32_t>(hi) >> 31), "v"(tie_g), "s"(tie_c));
    return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}
__device__ __forceinline__ int key_expert(double k) {
    const uint64_t b = static_cast<uint64_t>(__double_as_longlong(k));
    const uint32_t lo = static_cast<uint32_t>(b) ^ static_cast<uint32_t>(static_cast<int32_t>(b >> 32) >> 31);
    return 255 - static_cast<int>(lo & 255u);
}
__device__ __forceinline__ float key_logit(double k) {
    return __uint_as_float(static_cast<uint32_t>(static_cast<uint64_t>(__double_as_longlong(k)) >> 32));
}

// Descending compare-exchange.
__device__ __forceinline__ void cx(double& a, double& b) {
    const double hi = __builtin_fmax(a, b);
    const double lo = __builtin_fmin(a, b);
    a = hi;
    b = lo;
}

// Descending sort of N = 2^m keys by Batcher's odd-even merge sort (Knuth,
// TAOCP vol. 3, Sec. 5.3.4): runs of length 2p are merged from sorted halves,
// comparing at distance k = p, p/2, ..., 1 only inside each run; 19
// compare-exchanges for N = 8, against 24 for the bitonic sorter.
template <int N>
__device__ __forceinline__ void sort_desc(double (&v)[N]) {
#pragma unroll
    for (int p = 1; p < N; p <<= 1)
#pragma unroll
        for (int k = p; k >= 1; k >>= 1)
#pragma unroll
            for (int j = k % p; j + k < N; j += 2 * k)
#pragma unroll
                for (int i = 0; i < k; ++i)
                    if (i + j + k < N && (i + j) / (2 * p) == (i + j + k) / (2 * p)) cx(v[i + j], v[i + j + k]);
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
    const int lo = __builtin_amdgcn_mov_dpp(static_cast<int>(b), CTRL, 0xF, 0xF, true);
    const int hi = __builtin_amdgcn_mov_dpp(static_cast<int>(b >> 32), CTRL, 0xF, 0xF, true);
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
// in its pair keeps the larger (key, a), the other keeps the smaller.  Keys
// are distinct except kNoKey, whose a is never read.
template <int CTRL>
__device__ __forceinline__ void lane_cx(double& key, float& a, bool lower) {
    const double pk = dpp_swap<CTRL>(key);
    const float pa = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(a), CTRL, 0xF, 0xF, true));
    const double nk = lower ? __builtin_fmax(key, pk) : __builtin_fmin(key, pk);
    a = (nk == key) ? a : pa;
    key = nk;
}
template <int CTRL>
__device__ __forceinline__ uint64_t dpp_swap_u64(uint64_t v) {
    return static_cast<uint64_t>(__double_as_longlong(dpp_swap<CTRL>(__longlong_as_double(static_cast<long long>(v)))));
}

// Lanes of a wave whose position g in their 8-lane group is above s.
__device__ __forceinline__ constexpr uint64_t lanes_after_slot(int s) {
    return 0x0101010101010101ull * ((0xFFull << (s + 1)) & 0xFFull);
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
    // 255 - e = 255 ^ e, and e = c * 8 * CW + g * CW + i sums disjoint bit
    // fields, so the tie word is a lane term xor a constant
    const uint32_t tie_g = 255u ^ static_cast<uint32_t>(g * CW);
    double keys[V];
#pragma unroll
    for (int c = 0; c < V / CW; ++c)
#pragma unroll
        for (int i = 0; i < CW; ++i) {
            const int e = c * (kGroup * CW) + g * CW + i;
            keys[c * CW + i] = (VEC || e < E) ? pack_key(vals[c * CW + i], tie_g, static_cast<uint32_t>(c * (kGroup * CW) + i))
                                              : kNoKey;
        }

    // ---- lane-local top KP: sort blocks of KP keys, merge them
    double top[KP];
    {
        constexpr int B = V < KP ? V : KP;     // keys per block
#pragma unroll
        for (int s = 0; s < KP; ++s) top[s] = s < B ? keys[s] : kNoKey;
        sort_desc<KP>(top);
#pragma unroll
        for (int b0 = KP; b0 < V; b0 += KP) {
            double blk[KP];
#pragma unroll
            for (int s = 0; s < KP; ++s) blk[s] = keys[b0 + s];
            sort_desc<KP>(blk);
            merge_top<KP>(top, blk);
        }
    }
    // ---- merge across the 8 lanes of the token
    merge_with_partner<kDppXor1, KP>(top);
    merge_with_partner<kDppXor2, KP>(top);
    merge_with_partner<kDppHalfMirror, KP>(top);

    // ---- lane g owns slot g (lanes g >= K own nothing): top[g mod KP] by a
    // select on each bit of g
    double sel[KP];
#pragma unroll
    for (int s = 0; s < KP; ++s) sel[s] = top[s];
#pragma unroll
    for (int half = KP / 2, bit = 0; half >= 1; half >>= 1, ++bit)
#pragma unroll
        for (int i = 0; i < half; ++i) sel[i] = ((g >> bit) & 1) ? sel[2 * i + 1] : sel[2 * i];
    const double mine = sel[0];
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
    float S = qs[0];
#pragma unroll
    for (int s = 1; s < K; ++s) S = S + qs[s];
    // lane g divides for its own slot; every lane then takes every slot's gate
    const float my_w = q / S;
    float ws[K];
#define CAP_GATHER_GATE(S_) \
    if constexpr (S_ < K) ws[S_] = group_lane<S_>(my_w);
    CAP_GATHER_GATE(0) CAP_GATHER_GATE(1) CAP_GATHER_GATE(2) CAP_GATHER_GATE(3)
    CAP_GATHER_GATE(4) CAP_GATHER_GATE(5) CAP_GATHER_GATE(6) CAP_GATHER_GATE(7)
#undef CAP_GATHER_GATE

    // ---- pruning: a prefix of a ranked list is kept; each lane sets the bit of
    // the device it ranks, and the group ORs the bits together
    const float target = 1.0f - p;
    const bool keep_all = (p == 0.0f);
    bool rank_kept;                         // the device this lane ranks is kept
    int rank_dev;
    bool slot_kept = false;                 // naive: slot g is in the kept prefix
    if constexpr (NAIVE) {
        // expert level: the shortest slot prefix whose running score reaches 1 - p
        float cum = ws[0];
        int n_keep = (!keep_all && cum >= target) ? 1 : K;
#pragma unroll
        for (int s = 1; s < K; ++s) {
            cum = cum + ws[s];
            n_keep = (n_keep == K && !keep_all && cum >= target) ? s + 1 : n_keep;
        }
        rank_kept = has_slot && g < n_keep;
        slot_kept = rank_kept;
        rank_dev = my_dev & 63;
    } else {
        const int src = small_quotient(live ? t : 0, tokens_per_rank);
        // lane g is a candidate if slot g is the first slot of its device
        // (no earlier slot on the same device: a lane mask built from ballots);
        // a = that device's score summed in slot order (earlier slots add +0)
        uint64_t repeat = 0;
        float a = 0.0f;
#pragma unroll
        for (int s = 0; s < K; ++s) {
            const bool same = devs[s] == my_dev;
            a = a + (same ? ws[s] : 0.0f);
            repeat |= __builtin_amdgcn_ballot_w64(same) & lanes_after_slot(s);
        }
        const bool cand = has_slot && !__builtin_amdgcn_inverse_ballot_w64(repeat);
        float ratio = a;
        if (my_dev == src) ratio = INFINITY;
        else if (R > ranks_per_node &&
                 small_quotient(my_dev, ranks_per_node) != small_quotient(src, ranks_per_node))
            ratio = a / inter_node_cost;
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
        // greedy retention in key order, replayed by every lane: the running
        // sum over the ranked candidates (non-candidates rank last and add +0,
        // so they can neither change the sum nor be the first to reach 1 - p)
        const uint64_t ckb = static_cast<uint64_t>(__double_as_longlong(ck));
        const bool ranked = (static_cast<uint32_t>(ckb >> 32) >> 29) == 1u;
        // The sum never decreases, so the first rank at which it reaches 1 - p
        // is the number of earlier ranks at which it was still below.
        const float ra = ranked ? ca : 0.0f;
        float cum = group_lane<0>(ra);
        int below = (cum < target) ? 1 : 0;
#define CAP_GREEDY_STEP(S_)                                                   \
        if constexpr (S_ > 0 && S_ < K - 1) {                                     \
            cum = cum + group_lane<S_>(ra);                                       \
            below += (cum < target) ? 1 : 0;                                      \
        }
        CAP_GREEDY_STEP(1) CAP_GREEDY_STEP(2) CAP_GREEDY_STEP(3)
        CAP_GREEDY_STEP(4) CAP_GREEDY_STEP(5) CAP_GREEDY_STEP(6)
#undef CAP_GREEDY_STEP
        rank_kept = ranked && (keep_all || g <= below);   // ranks 0 .. first reaching rank
        rank_dev = 63 - static_cast<int>((ckb >> 3) & 63u);
    }
    uint64_t mask = rank_kept ? (1ull << rank_dev) : 0ull;
    mask |= dpp_swap_u64<kDppXor1>(mask);
    mask |= dpp_swap_u64<kDppXor2>(mask);
    mask |= dpp_swap_u64<kDppHalfMirror>(mask);

    // ---- S' = kept gates summed in slot order; lane g writes slot g
    const bool my_keep = NAIVE ? slot_kept : has_slot && ((mask >> (my_dev & 63)) & 1ull);
    const float kw = my_keep ? my_w : 0.0f;
    float Sk = group_lane<0>(kw);
#define CAP_KEPT_SUM(S_) \
    if constexpr (S_ > 0 && S_ < K) Sk = Sk + group_lane<S_>(kw);
    CAP_KEPT_SUM(1) CAP_KEPT_SUM(2) CAP_KEPT_SUM(3) CAP_KEPT_SUM(4) CAP_KEPT_SUM(5) CAP_KEPT_SUM(6) CAP_KEPT_SUM(7)
#undef CAP_KEPT_SUM
    if (live && has_slot) {
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
