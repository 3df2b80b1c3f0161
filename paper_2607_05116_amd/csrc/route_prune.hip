// Top-k routing, normalised gates and communication-aware device pruning.
//
// Top-k and gates: Sec. II-A, Eq. 1 (Gate_i is the normalised routing weight
// of the i-th selected expert).  Pruning: Sec. VI, Eq. 6 and the greedy that
// follows it (keep devices in descending a_d / c_d until the kept score sum
// reaches 1 - p).
//
// Every floating-point step that decides a kept device is fp32 in a fixed
// order, with no contraction, so the decision is reproducible bit for bit:
//   gates  w_s = q_s / S, q_s = gate_exp(l_s - l_0), S = ((q_0 + q_1) + ...)
//   a_d    = sum of w_s on device d in slot order
//   key_d  = +inf (own device), a_d / 1 (same node), a_d / c (other node)
//   greedy running sum in key order (ties: lower device id), stop at >= 1 - p
//   w'_s   = w_s / S' over kept slots (S' summed in slot order).
//
// Layout: 8 lanes cooperate on one token (8 tokens per wave).  Lane j of a
// group holds V logits of the row, loaded as 16-byte vectors so a group reads
// the row in contiguous 128-byte pieces.  Each lane keeps a sorted top-KI list
// of its own values (stable: it scans its values in ascending expert order and
// inserts only on strictly greater), then three butterfly steps (xor 1, 2, 4)
// merge partner lists with a bitonic network under the total order
// (value desc, index asc).  After the merge all 8 lanes hold the token's
// top-KI list, compute the gates and the pruning redundantly (uniform work, no
// divergence) and lane j writes slot j.
#pragma clang fp contract(off)

#include <math.h>

#include "cap_device.hpp"

namespace cap {
namespace {

constexpr int kGroup = 8;              // lanes per token
constexpr int kTokensPerBlock = 32;    // 256 threads

// Gate exponential: Cody & Waite argument reduction with ln2 split as
// LN2_HI (ln 2 to 16 significant bits, exact products n*LN2_HI for |n| < 2^8)
// plus LN2_LO (fp32 nearest to ln2 - LN2_HI); Taylor polynomial of degree 7
// with fp32(1/j!) coefficients by Horner with fused multiply-add; scaled by
// 2^n.  Inputs below -87.33 give 0, so results are never subnormal.
__device__ __forceinline__ float gate_exp(float z) {
    if (!(z >= -87.33f)) return 0.0f;
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
    return __builtin_ldexpf(q, static_cast<int>(n));
}

// (value desc, index asc): true if (av, ai) ranks before (bv, bi).
__device__ __forceinline__ bool ranks_before(float av, int ai, float bv, int bi) {
    return av > bv || (av == bv && ai < bi);
}

template <int V, int KI>
__global__ __launch_bounds__(256) void route_prune_kernel(
    const float* __restrict__ logits, int T, int E, int k, int R, int ranks_per_node,
    int tokens_per_rank, float inter_node_cost, float p, int vec_ok,
    const int32_t* __restrict__ expert_rank, int32_t* __restrict__ out_idx,
    float* __restrict__ out_w, uint8_t* __restrict__ out_keep, uint64_t* __restrict__ out_mask) {
    __shared__ int er_lds[kMaxE];
    for (int e = threadIdx.x; e < E; e += blockDim.x) er_lds[e] = expert_rank[e] & 63;
    __syncthreads();

    const int g = threadIdx.x & (kGroup - 1);
    const int t = blockIdx.x * kTokensPerBlock + (threadIdx.x >> 3);
    const bool live = t < T;
    const float* row = logits + static_cast<size_t>(live ? t : T - 1) * E;

    // ---- load this lane's V values; element order ascending within the lane
    constexpr int CW = V < 4 ? V : 4;          // vector width
    float vals[V];
    int ids[V];
#pragma unroll
    for (int c = 0; c < V / CW; ++c) {
        const int e0 = c * (kGroup * CW) + g * CW;
        if (vec_ok) {
            if constexpr (CW == 4) {
                const float4 v = *reinterpret_cast<const float4*>(row + e0);
                vals[c * 4 + 0] = v.x; vals[c * 4 + 1] = v.y; vals[c * 4 + 2] = v.z; vals[c * 4 + 3] = v.w;
            } else if constexpr (CW == 2) {
                const float2 v = *reinterpret_cast<const float2*>(row + e0);
                vals[c * 2 + 0] = v.x; vals[c * 2 + 1] = v.y;
            } else {
                vals[c] = row[e0];
            }
        } else {
#pragma unroll
            for (int i = 0; i < CW; ++i) vals[c * CW + i] = (e0 + i < E) ? row[e0 + i] : -INFINITY;
        }
#pragma unroll
        for (int i = 0; i < CW; ++i) ids[c * CW + i] = e0 + i;
    }

    // ---- lane-local sorted top-KI (stable insertion on strictly greater)
    float lv[KI];
    int li[KI];
#pragma unroll
    for (int s = 0; s < KI; ++s) { lv[s] = -INFINITY; li[s] = 0x7fffffff; }
#pragma unroll
    for (int i = 0; i < V; ++i) {
        const float x = vals[i];
        const int xe = ids[i];
        bool gt[KI];
#pragma unroll
        for (int s = 0; s < KI; ++s) gt[s] = x > lv[s];
#pragma unroll
        for (int s = KI - 1; s >= 1; --s) {
            lv[s] = gt[s - 1] ? lv[s - 1] : (gt[s] ? x : lv[s]);
            li[s] = gt[s - 1] ? li[s - 1] : (gt[s] ? xe : li[s]);
        }
        lv[0] = gt[0] ? x : lv[0];
        li[0] = gt[0] ? xe : li[0];
    }

    // ---- butterfly merge of the 8 lane lists (bitonic, total order)
#pragma unroll
    for (int m = 1; m < kGroup; m <<= 1) {
        float ov[KI];
        int oi[KI];
#pragma unroll
        for (int s = 0; s < KI; ++s) {
            ov[s] = __shfl_xor(lv[s], m);
            oi[s] = __shfl_xor(li[s], m);
        }
        float cv[KI];
        int ci[KI];
#pragma unroll
        for (int s = 0; s < KI; ++s) {
            const bool mine = ranks_before(lv[s], li[s], ov[KI - 1 - s], oi[KI - 1 - s]);
            cv[s] = mine ? lv[s] : ov[KI - 1 - s];
            ci[s] = mine ? li[s] : oi[KI - 1 - s];
        }
#pragma unroll
        for (int h = KI / 2; h >= 1; h >>= 1) {
#pragma unroll
            for (int s = 0; s < KI; ++s) {
                if ((s & h) == 0) {
                    const bool swap = ranks_before(cv[s + h], ci[s + h], cv[s], ci[s]);
                    const float tv = cv[s];
                    const int ti = ci[s];
                    cv[s] = swap ? cv[s + h] : cv[s];
                    ci[s] = swap ? ci[s + h] : ci[s];
                    cv[s + h] = swap ? tv : cv[s + h];
                    ci[s + h] = swap ? ti : ci[s + h];
                }
            }
        }
#pragma unroll
        for (int s = 0; s < KI; ++s) { lv[s] = cv[s]; li[s] = ci[s]; }
    }

    // ---- normalised gates (softmax over the k selected logits)
    float w[KI];
    float S = 0.0f;
#pragma unroll
    for (int s = 0; s < KI; ++s) {
        w[s] = 0.0f;
        if (s < k) {
            w[s] = gate_exp(lv[s] - lv[0]);
            S = S + w[s];
        }
    }
#pragma unroll
    for (int s = 0; s < KI; ++s) w[s] = (s < k) ? w[s] / S : 0.0f;

    // ---- device-level pruning
    const int src = (live ? t : 0) / tokens_per_rank;
    const int src_node = src / ranks_per_node;
    int dev[KI];
    int first[KI];
#pragma unroll
    for (int s = 0; s < KI; ++s) {
        dev[s] = (s < k) ? er_lds[li[s] < E ? li[s] : 0] : -1;
        first[s] = s;
    }
#pragma unroll
    for (int s = 1; s < KI; ++s)
#pragma unroll
        for (int s2 = s - 1; s2 >= 0; --s2)
            if (s < k && dev[s2] == dev[s]) first[s] = s2;

    float a[KI];
#pragma unroll
    for (int j = 0; j < KI; ++j) a[j] = 0.0f;
#pragma unroll
    for (int s = 0; s < KI; ++s)
#pragma unroll
        for (int j = 0; j <= s; ++j)
            if (s < k && first[s] == j) a[j] = a[j] + w[s];

    bool cand[KI];
    float key[KI];
#pragma unroll
    for (int j = 0; j < KI; ++j) {
        cand[j] = (j < k) && first[j] == j;
        const int d = dev[j];
        if (d == src)
            key[j] = INFINITY;
        else if (d / ranks_per_node == src_node)
            key[j] = a[j] / 1.0f;
        else
            key[j] = a[j] / inter_node_cost;
    }
    int rank[KI];
#pragma unroll
    for (int j = 0; j < KI; ++j) {
        int r = 0;
#pragma unroll
        for (int j2 = 0; j2 < KI; ++j2)
            if (cand[j2] && j2 != j &&
                (key[j2] > key[j] || (key[j2] == key[j] && dev[j2] < dev[j])))
                ++r;
        rank[j] = r;
    }
    int stop_rank = KI;                  // keep every candidate unless the target is met earlier
    if (p != 0.0f) {
        const float target = 1.0f - p;
        float cum = 0.0f;
        bool done = false;
#pragma unroll
        for (int r = 0; r < KI; ++r) {
#pragma unroll
            for (int j = 0; j < KI; ++j) {
                if (!done && cand[j] && rank[j] == r) {
                    cum = cum + a[j];
                    if (cum >= target) { stop_rank = r; done = true; }
                }
            }
        }
    }
    uint64_t mask = 0;
    bool keep[KI];
#pragma unroll
    for (int j = 0; j < KI; ++j)
        if (cand[j] && rank[j] <= stop_rank) mask |= 1ull << dev[j];
    float Sk = 0.0f;
#pragma unroll
    for (int s = 0; s < KI; ++s) {
        keep[s] = (s < k) && ((mask >> dev[s]) & 1ull);
        if (keep[s]) Sk = Sk + w[s];
    }

    // ---- lane g writes slot g
    if (live) {
        int my_idx = 0;
        float my_w = 0.0f;
        uint8_t my_keep = 0;
#pragma unroll
        for (int s = 0; s < KI; ++s) {
            if (s == g) {
                my_idx = li[s];
                my_w = keep[s] ? w[s] / Sk : 0.0f;
                my_keep = keep[s] ? 1 : 0;
            }
        }
        if (g < k) {
            const size_t q = static_cast<size_t>(t) * k + g;
            out_idx[q] = my_idx;
            out_w[q] = my_w;
            out_keep[q] = my_keep;
        }
        if (g == 0) out_mask[t] = mask;
    }
}

template <int V, int KI>
void launch_route(const cap_topology* tp, const float* logits, float p, int vec_ok,
                  int32_t* idx, float* w, uint8_t* keep, uint64_t* mask, hipStream_t st) {
    const int blocks = (tp->T + kTokensPerBlock - 1) / kTokensPerBlock;
    route_prune_kernel<V, KI><<<blocks, 256, 0, st>>>(
        logits, tp->T, tp->E, tp->k, tp->R, tp->ranks_per_node, tp->tokens_per_rank,
        tp->inter_node_cost, p, vec_ok, tp->expert_rank, idx, w, keep, mask);
}

template <int V>
void launch_route_k(const cap_topology* tp, const float* logits, float p, int vec_ok,
                    int32_t* idx, float* w, uint8_t* keep, uint64_t* mask, hipStream_t st) {
    if (tp->k <= 1) launch_route<V, 1>(tp, logits, p, vec_ok, idx, w, keep, mask, st);
    else if (tp->k <= 2) launch_route<V, 2>(tp, logits, p, vec_ok, idx, w, keep, mask, st);
    else if (tp->k <= 4) launch_route<V, 4>(tp, logits, p, vec_ok, idx, w, keep, mask, st);
    else launch_route<V, 8>(tp, logits, p, vec_ok, idx, w, keep, mask, st);
}

}  // namespace

cap_status route_prune_launch(const cap_topology* tp, const float* logits, float p, int32_t* idx,
                              float* w, uint8_t* keep, uint64_t* mask, hipStream_t st) {
    int V = 1;
    while (kGroup * V < tp->E) V <<= 1;
    const int CW = V < 4 ? V : 4;
    // Vector loads cover exactly 8*V columns: only when that is the row length
    // (every other E takes the bounds-checked scalar path).
    const int vec_ok = (tp->E == kGroup * V) && (reinterpret_cast<uintptr_t>(logits) % (4 * CW) == 0);
    switch (V) {
        case 1: launch_route_k<1>(tp, logits, p, vec_ok, idx, w, keep, mask, st); break;
        case 2: launch_route_k<2>(tp, logits, p, vec_ok, idx, w, keep, mask, st); break;
        case 4: launch_route_k<4>(tp, logits, p, vec_ok, idx, w, keep, mask, st); break;
        case 8: launch_route_k<8>(tp, logits, p, vec_ok, idx, w, keep, mask, st); break;
        case 16: launch_route_k<16>(tp, logits, p, vec_ok, idx, w, keep, mask, st); break;
        default: launch_route_k<32>(tp, logits, p, vec_ok, idx, w, keep, mask, st); break;
    }
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

}  // namespace cap
