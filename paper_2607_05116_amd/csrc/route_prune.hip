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
//   key_d  = +inf (own device), a_d (same node), a_d / c (other node)
//   greedy running sum in key order (ties: lower device id), stop at >= 1 - p
//   w'_s   = w_s / S' over kept slots (S' summed in slot order).
//
// Selection keys.  A (logit, expert) pair is packed into one fp64 whose order
// is the selection order (logit descending, then expert id ascending): the
// high word is the logit's own bits, so fp64 sign-magnitude order matches fp32
// order, and the low word is 255 - expert, complemented for negative logits
// (whose fp64 magnitudes order in reverse).  Such a double is never NaN or
// infinite; zero and tiny logits give fp64 subnormals, which are not flushed,
// so v_max_f64 / v_min_f64 compare every key exactly and a compare-exchange is
// two branch-free instructions.  -0.0 is folded to +0.0 first, because the two
// compare equal as logits (the tie then goes to the lower expert id, as for
// any other equal pair).
//
// Layout: 8 lanes cooperate on one token (8 tokens per wave).  Lane j holds V
// logits of the row (loaded as 16-byte vectors, so a group reads the row in
// contiguous 128-byte pieces), sorts them in blocks of KP = pow2 >= k with
// Batcher's odd-even merge sort and keeps the top KP (bitonic merges of the
// sorted blocks); three butterfly merges across the group (DPP lane swaps)
// leave every lane with the token's sorted top KP.  From there lane j owns
// slot j: it computes its own gate exponential and gate division and takes
// the slot-ordered sums (S, a_d, S') from the group's lanes through
// ds_swizzle broadcasts, so every sum keeps its sequential order.  The
// candidate devices (one lane each) are sorted across the group with the same
// kind of packed-double keys; every lane replays the greedy's running sum over
// the ranked list, which fixes how many of the ranked devices are kept, and
// the group ORs the kept devices' bits into the mask.  Rows of 64, 128 or 256
// logits take the four-lane form below (route_prune4_kernel), which computes
// the same bits with all of a token's cross-lane traffic inside one quad.
#pragma clang fp contract(off)

#include <math.h>

#include "route_device.hpp"

namespace cap {
namespace {



// ---------------------------------------------------------------------------
// Four lanes per token (16 tokens per wave), for rows of E = 4 V4 logits with
// V4 = 16, 32 or 64: the same decision as route_token with the group's
// cross-lane traffic inside a quad, where DPP quad permutes broadcast any lane
// (no LDS swizzle), and two butterfly merges instead of three.  Lane h holds
// logits c * 16 + h * 4 + [0, 4) and owns slots h and h + 4; every sum keeps
// the slot (or rank) order of route_token, so the two agree bit for bit.
constexpr int kQuad = 4;
constexpr int kQuadTokensPerBlock = 64;     // 256 threads

template <int S>
__device__ __forceinline__ int quad_lane(int v) {
    return __builtin_amdgcn_mov_dpp(v, S | (S << 2) | (S << 4) | (S << 6), 0xF, 0xF, true);
}
template <int S>
__device__ __forceinline__ float quad_lane(float v) {
    return __int_as_float(quad_lane<S>(__float_as_int(v)));
}

// Lanes of a wave whose slot h + 4 u in their quad comes after slot s.
__device__ __forceinline__ constexpr uint64_t quad_lanes_after(int u, int s) {
    return 0x1111111111111111ull *
           (s - 4 * u < 0 ? 0xFull : s - 4 * u >= 3 ? 0ull : ((0xFull << (s - 4 * u + 1)) & 0xFull));
}

// One across-the-quad step (stride 1 or 2) of a bitonic sort stage of the given
// size, for keys i = h + 4 u: i keeps the larger of its pair when it is the
// lower index of a descending block or the upper index of an ascending one.
template <int CTRL>
__device__ __forceinline__ void quad_cx(double (&ck)[2], float (&ca)[2], int h, int stride, int size) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const bool desc = ((h + 4 * u) & size) == 0;
        const bool lower = (h & stride) == 0;
        lane_cx<CTRL>(ck[u], ca[u], lower == desc);
    }
}

template <int V4, int K, bool NAIVE>
__device__ __forceinline__ void route_token4(const float (&vals)[V4], int h, int t, bool live, int E, int R,
                                             int ranks_per_node, int tokens_per_rank, float inter_node_cost,
                                             float p, const int* er_lds, int32_t* __restrict__ out_idx,
                                             float* __restrict__ out_w, uint8_t* __restrict__ out_keep,
                                             uint64_t* __restrict__ out_mask) {
    constexpr int KP = pow2_at_least(K);
    constexpr int NS = (K + kQuad - 1) / kQuad;     // slots per lane
    static_assert(V4 >= KP && V4 % KP == 0 && V4 % 4 == 0, "whole blocks of KP keys per lane");

    // keys: expert c * 16 + h * 4 + i; 255 - e = 255 ^ e over disjoint bit fields
    const uint32_t tie_h = 255u ^ static_cast<uint32_t>(h * 4);
    double keys[V4];
#pragma unroll
    for (int c = 0; c < V4 / 4; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i)
            keys[c * 4 + i] = pack_key(vals[c * 4 + i], tie_h, static_cast<uint32_t>(c * 16 + i));

    // lane-local top KP, then the quad's
    double top[KP];
#pragma unroll
    for (int s = 0; s < KP; ++s) top[s] = keys[s];
    sort_desc<KP>(top);
#pragma unroll
    for (int b0 = KP; b0 < V4; b0 += KP) {
        double blk[KP];
#pragma unroll
        for (int s = 0; s < KP; ++s) blk[s] = keys[b0 + s];
        sort_desc<KP>(blk);
        merge_top<KP>(top, blk);
    }
    merge_with_partner<kDppXor1, KP>(top);
    merge_with_partner<kDppXor2, KP>(top);

    // the lane's slots h + 4 u
    bool has[NS];
    int my_e[NS], my_dev[NS];
    float q[NS];
#pragma unroll
    for (int u = 0; u < NS; ++u) {
        double m = top[0];
#pragma unroll
        for (int s = 1; s < kQuad && 4 * u + s < KP; ++s) m = (h == s) ? top[4 * u + s] : m;
        if (4 * u > 0) m = (h == 0) ? top[4 * u] : m;
        has[u] = h + 4 * u < K;
        my_e[u] = key_expert(m);
        my_dev[u] = has[u] ? er_lds[my_e[u] < E ? my_e[u] : 0] : -1;
        q[u] = has[u] ? gate_exp(key_logit(m) - key_logit(top[0])) : 0.0f;
    }
    float qs[K];
    int devs[K];
#define CAP_QUAD_GATHER(S_)                                  \
    if constexpr (S_ < K) {                                  \
        qs[S_] = quad_lane<S_ % 4>(q[S_ / 4]);               \
        devs[S_] = quad_lane<S_ % 4>(my_dev[S_ / 4]);        \
    }
    CAP_QUAD_GATHER(0) CAP_QUAD_GATHER(1) CAP_QUAD_GATHER(2) CAP_QUAD_GATHER(3)
    CAP_QUAD_GATHER(4) CAP_QUAD_GATHER(5) CAP_QUAD_GATHER(6) CAP_QUAD_GATHER(7)
#undef CAP_QUAD_GATHER
    float S = qs[0];
#pragma unroll
    for (int s = 1; s < K; ++s) S = S + qs[s];
    float my_w[NS];
#pragma unroll
    for (int u = 0; u < NS; ++u) my_w[u] = q[u] / S;
    float ws[K];
#define CAP_QUAD_GATE(S_) \
    if constexpr (S_ < K) ws[S_] = quad_lane<S_ % 4>(my_w[S_ / 4]);
    CAP_QUAD_GATE(0) CAP_QUAD_GATE(1) CAP_QUAD_GATE(2) CAP_QUAD_GATE(3)
    CAP_QUAD_GATE(4) CAP_QUAD_GATE(5) CAP_QUAD_GATE(6) CAP_QUAD_GATE(7)
#undef CAP_QUAD_GATE

    const float target = 1.0f - p;
    const bool keep_all = (p == 0.0f);
    uint64_t bits = 0;                              // devices this lane keeps
    bool slot_kept[NS];
#pragma unroll
    for (int u = 0; u < NS; ++u) slot_kept[u] = false;
    if constexpr (NAIVE) {
        float cum = ws[0];
        int n_keep = (!keep_all && cum >= target) ? 1 : K;
#pragma unroll
        for (int s = 1; s < K; ++s) {
            cum = cum + ws[s];
            n_keep = (n_keep == K && !keep_all && cum >= target) ? s + 1 : n_keep;
        }
#pragma unroll
        for (int u = 0; u < NS; ++u) {
            slot_kept[u] = has[u] && h + 4 * u < n_keep;
            bits |= slot_kept[u] ? (1ull << (my_dev[u] & 63)) : 0ull;
        }
    } else {
        const int src = small_quotient(live ? t : 0, tokens_per_rank);
        const int src_node = small_quotient(src, ranks_per_node);
        double ck[2];
        float ca[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            ck[u] = kNoKey;
            ca[u] = 0.0f;
        }
#pragma unroll
        for (int u = 0; u < NS; ++u) {
            // candidate: no earlier slot on the same device; a = that device's
            // score in slot order (earlier slots add +0)
            uint64_t repeat = 0;
            float a = 0.0f;
#pragma unroll
            for (int s = 0; s < K; ++s) {
                const bool same = devs[s] == my_dev[u];
                a = a + (same ? ws[s] : 0.0f);
                repeat |= __builtin_amdgcn_ballot_w64(same) & quad_lanes_after(u, s);
            }
            const bool cand = has[u] && !__builtin_amdgcn_inverse_ballot_w64(repeat);
            float ratio = a;
            if (my_dev[u] == src) ratio = INFINITY;
            else if (R > ranks_per_node && small_quotient(my_dev[u], ranks_per_node) != src_node)
                ratio = a / inter_node_cost;
            const uint64_t kbits = (1ull << 61) | (static_cast<uint64_t>(__float_as_uint(ratio)) << 30) |
                                   (static_cast<uint64_t>(63 - (my_dev[u] & 63)) << 3);
            ck[u] = cand ? __longlong_as_double(static_cast<long long>(kbits)) : kNoKey;
            ca[u] = a;
        }
        // descending bitonic sort of the 8 candidate keys, key i = h + 4 u at
        // lane h, register u: strides 1 and 2 across the quad, stride 4 in-lane
        quad_cx<kDppXor1>(ck, ca, h, 1, 2);
        quad_cx<kDppXor2>(ck, ca, h, 2, 4);
        quad_cx<kDppXor1>(ck, ca, h, 1, 4);
        {                                           // stride 4 of the size-8 stage (descending)
            const double hi = __builtin_fmax(ck[0], ck[1]);
            const double lo = __builtin_fmin(ck[0], ck[1]);
            const bool first = hi == ck[0];
            const float a_hi = first ? ca[0] : ca[1];
            const float a_lo = first ? ca[1] : ca[0];
            ck[0] = hi;
            ck[1] = lo;
            ca[0] = a_hi;
            ca[1] = a_lo;
        }
        quad_cx<kDppXor2>(ck, ca, h, 2, 8);
        quad_cx<kDppXor1>(ck, ca, h, 1, 8);
        // greedy retention in rank order, replayed by every lane (see route_token)
        float ra[2];
        bool ranked[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            ranked[u] = (static_cast<uint32_t>(static_cast<uint64_t>(__double_as_longlong(ck[u])) >> 32) >> 29) == 1u;
            ra[u] = ranked[u] ? ca[u] : 0.0f;
        }
        float cum = quad_lane<0>(ra[0]);
        int below = (cum < target) ? 1 : 0;
#define CAP_QUAD_GREEDY(S_)                                                   \
        if constexpr (S_ > 0 && S_ < K - 1) {                                     \
            cum = cum + quad_lane<S_ % 4>(ra[S_ / 4]);                            \
            below += (cum < target) ? 1 : 0;                                      \
        }
        CAP_QUAD_GREEDY(1) CAP_QUAD_GREEDY(2) CAP_QUAD_GREEDY(3)
        CAP_QUAD_GREEDY(4) CAP_QUAD_GREEDY(5) CAP_QUAD_GREEDY(6)
#undef CAP_QUAD_GREEDY
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const bool kept = ranked[u] && (keep_all || h + 4 * u <= below);
            const int dev = 63 - static_cast<int>((static_cast<uint64_t>(__double_as_longlong(ck[u])) >> 3) & 63u);
            bits |= kept ? (1ull << dev) : 0ull;
        }
    }
    uint64_t mask = bits;
    mask |= dpp_swap_u64<kDppXor1>(mask);
    mask |= dpp_swap_u64<kDppXor2>(mask);

    // S' = kept gates summed in slot order; lane h writes its slots
    bool my_keep[NS];
    float kw[NS];
#pragma unroll
    for (int u = 0; u < NS; ++u) {
        my_keep[u] = NAIVE ? slot_kept[u] : has[u] && ((mask >> (my_dev[u] & 63)) & 1ull);
        kw[u] = my_keep[u] ? my_w[u] : 0.0f;
    }
    float Sk = quad_lane<0>(kw[0]);
#define CAP_QUAD_KEPT(S_) \
    if constexpr (S_ > 0 && S_ < K) Sk = Sk + quad_lane<S_ % 4>(kw[S_ / 4]);
    CAP_QUAD_KEPT(1) CAP_QUAD_KEPT(2) CAP_QUAD_KEPT(3) CAP_QUAD_KEPT(4) CAP_QUAD_KEPT(5) CAP_QUAD_KEPT(6)
    CAP_QUAD_KEPT(7)
#undef CAP_QUAD_KEPT
    if (live) {
#pragma unroll
        for (int u = 0; u < NS; ++u) {
            if (!has[u]) continue;
            const size_t qi = static_cast<size_t>(t) * K + h + 4 * u;
            out_idx[qi] = my_e[u];
            out_w[qi] = my_keep[u] ? my_w[u] / Sk : 0.0f;
            out_keep[qi] = my_keep[u] ? 1 : 0;
        }
        if (h == 0) out_mask[t] = mask;
    }
}

template <int V4, int K, bool NAIVE>
__global__ __launch_bounds__(256) void route_prune4_kernel(
    const float* __restrict__ logits, int T, int E, int R, int ranks_per_node,
    int tokens_per_rank, float inter_node_cost, float p,
    const int32_t* __restrict__ expert_rank, int32_t* __restrict__ out_idx,
    float* __restrict__ out_w, uint8_t* __restrict__ out_keep, uint64_t* __restrict__ out_mask) {
    static_assert(kMaxE <= 256, "one table entry per thread");
    __shared__ int er_lds[kMaxE];
    const int er_v = expert_rank[min(static_cast<int>(threadIdx.x), E - 1)];   // no branch: no early wait

    const int h = threadIdx.x & (kQuad - 1);
    const int t = blockIdx.x * kQuadTokensPerBlock + (threadIdx.x >> 2);
    const bool live = t < T;
    const float* row = logits + static_cast<size_t>(live ? t : T - 1) * E;
    float vals[V4];
#pragma unroll
    for (int c = 0; c < V4 / 4; ++c) {
        const float4 v = *reinterpret_cast<const float4*>(row + c * 16 + h * 4);
        vals[c * 4 + 0] = v.x; vals[c * 4 + 1] = v.y; vals[c * 4 + 2] = v.z; vals[c * 4 + 3] = v.w;
    }
    er_lds[threadIdx.x] = er_v & 63;           // entries past E are never read
    __syncthreads();                           // er_lds ready
    route_token4<V4, K, NAIVE>(vals, h, t, live, E, R, ranks_per_node, tokens_per_rank, inter_node_cost, p,
                               er_lds, out_idx, out_w, out_keep, out_mask);
}

template <int V, int K, bool VEC, bool NAIVE>
__global__ __launch_bounds__(256) void route_prune_kernel(
    const float* __restrict__ logits, int T, int E, int R, int ranks_per_node,
    int tokens_per_rank, float inter_node_cost, float p,
    const int32_t* __restrict__ expert_rank, int32_t* __restrict__ out_idx,
    float* __restrict__ out_w, uint8_t* __restrict__ out_keep, uint64_t* __restrict__ out_mask) {
    // expert -> rank table in LDS, one entry per thread; its load is issued
    // together with the logit loads so that neither waits for the other
    static_assert(kMaxE <= kTokensPerBlock * kGroup, "one table entry per thread");
    __shared__ int er_lds[kMaxE];
    const int er_v = expert_rank[min(static_cast<int>(threadIdx.x), E - 1)];   // no branch: no early wait

    const int g = threadIdx.x & (kGroup - 1);
    const int t = blockIdx.x * kTokensPerBlock + (threadIdx.x >> 3);
    const bool live = t < T;
    const float* row = logits + static_cast<size_t>(live ? t : T - 1) * E;

    // ---- this lane's V logits; lane g owns columns c*(8*CW) + g*CW + [0, CW)
    constexpr int CW = V < 4 ? V : 4;          // vector width
    float vals[V];
    if constexpr (VEC) {
#pragma unroll
        for (int c = 0; c < V / CW; ++c) {
            const int e0 = c * (kGroup * CW) + g * CW;
            if constexpr (CW == 4) {
                const float4 q = *reinterpret_cast<const float4*>(row + e0);
                vals[c * 4 + 0] = q.x; vals[c * 4 + 1] = q.y; vals[c * 4 + 2] = q.z; vals[c * 4 + 3] = q.w;
            } else if constexpr (CW == 2) {
                const float2 q = *reinterpret_cast<const float2*>(row + e0);
                vals[c * 2 + 0] = q.x; vals[c * 2 + 1] = q.y;
            } else {
                vals[c] = row[e0];
            }
        }
    } else {
#pragma unroll
        for (int c = 0; c < V / CW; ++c)
#pragma unroll
            for (int i = 0; i < CW; ++i) {
                const int e = c * (kGroup * CW) + g * CW + i;
                vals[c * CW + i] = row[e < E ? e : E - 1];
            }
    }
    er_lds[threadIdx.x] = er_v & 63;           // entries past E are never read
    __syncthreads();                           // er_lds ready
    route_token<V, K, VEC, NAIVE>(vals, g, t, live, E, R, ranks_per_node, tokens_per_rank, inter_node_cost, p,
                                  er_lds, out_idx, out_w, out_keep, out_mask);
}

template <int V, int K, bool NAIVE>
void launch_route_mode(const cap_topology* tp, const float* logits, float p, int vec_ok,
                       int32_t* idx, float* w, uint8_t* keep, uint64_t* mask, hipStream_t st) {
    if constexpr (V >= 8) {
        if (vec_ok) {                           // E = 64, 128, 256: four lanes per token
            const int blocks4 = (tp->T + kQuadTokensPerBlock - 1) / kQuadTokensPerBlock;
            route_prune4_kernel<2 * V, K, NAIVE><<<blocks4, 256, 0, st>>>(
                logits, tp->T, tp->E, tp->R, tp->ranks_per_node, tp->tokens_per_rank, tp->inter_node_cost, p,
                tp->expert_rank, idx, w, keep, mask);
            return;
        }
    }
    const int blocks = (tp->T + kTokensPerBlock - 1) / kTokensPerBlock;
    if constexpr (V < 8) {                      // the vector-load eight-lane form only where no quad form exists
        if (vec_ok) {
            route_prune_kernel<V, K, true, NAIVE><<<blocks, 256, 0, st>>>(
                logits, tp->T, tp->E, tp->R, tp->ranks_per_node, tp->tokens_per_rank,
                tp->inter_node_cost, p, tp->expert_rank, idx, w, keep, mask);
            return;
        }
    }
    route_prune_kernel<V, K, false, NAIVE><<<blocks, 256, 0, st>>>(
        logits, tp->T, tp->E, tp->R, tp->ranks_per_node, tp->tokens_per_rank,
        tp->inter_node_cost, p, tp->expert_rank, idx, w, keep, mask);
}

template <int V, int K>
void launch_route(const cap_topology* tp, const float* logits, float p, bool naive, int vec_ok,
                  int32_t* idx, float* w, uint8_t* keep, uint64_t* mask, hipStream_t st) {
    if (naive) launch_route_mode<V, K, true>(tp, logits, p, vec_ok, idx, w, keep, mask, st);
    else launch_route_mode<V, K, false>(tp, logits, p, vec_ok, idx, w, keep, mask, st);
}

template <int V>
void launch_route_k(const cap_topology* tp, const float* logits, float p, bool naive, int vec_ok,
                    int32_t* idx, float* w, uint8_t* keep, uint64_t* mask, hipStream_t st) {
    switch (tp->k) {
        case 1: launch_route<V, 1>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
        case 2: launch_route<V, 2>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
        case 3: launch_route<V, 3>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
        case 4: launch_route<V, 4>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
        case 5: launch_route<V, 5>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
        case 6: launch_route<V, 6>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
        case 7: launch_route<V, 7>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
        default: launch_route<V, 8>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
    }
}

}  // namespace

cap_status route_prune_launch(const cap_topology* tp, const float* logits, float p, bool naive, int32_t* idx,
                              float* w, uint8_t* keep, uint64_t* mask, hipStream_t st) {
    int V = 1;
    while (kGroup * V < tp->E) V <<= 1;
    const int CW = V < 4 ? V : 4;
    // Vector loads cover exactly 8*V columns: only when that is the row length
    // (every other E takes the bounds-checked scalar path).
    const int vec_ok = (tp->E == kGroup * V) && (reinterpret_cast<uintptr_t>(logits) % (4 * CW) == 0);
    switch (V) {
        case 1: launch_route_k<1>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
        case 2: launch_route_k<2>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
        case 4: launch_route_k<4>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
        case 8: launch_route_k<8>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
        case 16: launch_route_k<16>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
        default: launch_route_k<32>(tp, logits, p, naive, vec_ok, idx, w, keep, mask, st); break;
    }
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

}  // namespace cap
