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
// the group ORs the kept devices' bits into the mask.
#pragma clang fp contract(off)

#include <math.h>

#include "route_device.hpp"

namespace cap {
namespace {



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
    const int blocks = (tp->T + kTokensPerBlock - 1) / kTokensPerBlock;
    if (vec_ok)
        route_prune_kernel<V, K, true, NAIVE><<<blocks, 256, 0, st>>>(
            logits, tp->T, tp->E, tp->R, tp->ranks_per_node, tp->tokens_per_rank,
            tp->inter_node_cost, p, tp->expert_rank, idx, w, keep, mask);
    else
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
