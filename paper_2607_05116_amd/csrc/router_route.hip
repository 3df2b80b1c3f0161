// Router GEMM fused with top-k routing and communication-aware pruning
// (Eq. 1: the gate takes the top k of the router logits x W_g^T; Sec. VI,
// Eq. 6 pruning).  Each block computes the fp32 logits of 64 or 128 tokens on the
// matrix cores into LDS and routes those tokens from there, so the logits
// never go through HBM.  The routing itself is route_token, the same code the
// logits-in kernel runs, so the two agree bit for bit on the same logits.
//
// GEMM: logits[t][e] = sum_k x[t][k] * W_g[e][k], bf16 operands, fp32
// accumulation in K order per 16-wide MFMA step.  K = d in stages of 64
// (one 128-byte line per operand row) filled by direct-to-LDS loads into a
// ring of three buffers, two stages in flight.  A block holds BT = 128 or 64
// tokens (128 when E > 128, halving the router-weight reads, which then
// dominate the loads); each of its four waves
// owns 32 tokens and all (BT = 128) or half (BT = 64) of the expert columns
// (v_mfma_f32_32x32x16_bf16 with the W_g fragment first, so a lane holds one
// token's logits for 16 experts per 32-expert block).  The expert dimension is
// padded to EP = max(32, 8 V) columns (rows past E repeat row E - 1 and are
// never routed on).
#include "route_device.hpp"

namespace cap {
namespace {

constexpr int kRtK = 64;           // K per stage
constexpr int kRtStages = 3;       // stage buffers in LDS (two stages in flight)
constexpr int kRtRowB = kRtK * 2;  // bytes per LDS row (one 128-byte line)

typedef __attribute__((address_space(3))) void rt_lds_void;

// 16-byte chunk c of stage row r sits at physical chunk c ^ rt_swz(r), so the
// fragment reads (32 rows, one chunk) spread over the banks.
__device__ __forceinline__ int rt_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Wave-wide direct-to-LDS copy: lane i reads 16 bytes at p_i and they land at
// LDS byte M0 + 16 i.  Inline assembly so the compiler's wait-count pass does
// not drain it before every LDS read; the kernel waits explicitly.  s_nop 4
// covers the wait states the hardware needs after the M0 write.
__device__ __forceinline__ void rt_lds_dma16(const void* p, uint32_t lds_addr) {
    asm volatile("s_nop 4\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(p), "{m0}"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory");
}

// Workgroup barrier without a memory fence (a fence would drain the stage
// loads in flight); the empty asm keeps memory accesses on their side.
__device__ __forceinline__ void rt_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <int V, int K, int EP, int BT, bool VEC>
__global__ __launch_bounds__(256) void router_route_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wg, int d, int T, int E, int R,
    int ranks_per_node, int tokens_per_rank, float inter_node_cost, float p,
    const int32_t* __restrict__ expert_rank, int32_t* __restrict__ out_idx, float* __restrict__ out_w,
    uint8_t* __restrict__ out_keep, uint64_t* __restrict__ out_mask, float* __restrict__ logits_out) {
    constexpr int NR = BT + EP;                             // stage rows: tokens, then experts
    constexpr int STAGE_B = NR * kRtRowB;
    constexpr int LPITCH = EP + 4;                          // logits row pitch (floats), padded
    constexpr int TILE_B = BT * LPITCH * 4;
    constexpr int LDS_B = kRtStages * STAGE_B > TILE_B ? kRtStages * STAGE_B : TILE_B;
    constexpr int WE = 4 / (BT / 32);                       // waves sharing a 32-token group
    constexpr int NJ = EP / 32 / WE;                        // 32-expert MFMA blocks per wave
    constexpr int LOADS = NR / 8;                           // 1 KB direct loads per stage
    constexpr int LOADS_PER_WAVE = (LOADS + 3) / 4;
    constexpr int LOADS_MIN_WAVE = LOADS / 4;               // loads of a stage every wave has issued
    static_assert(BT == 64 || BT == 128, "four waves of 32 tokens, or two per token group");
    static_assert(EP % 32 == 0 && EP >= 8 * V && (EP / 32) % WE == 0, "padded expert columns");
    static_assert(LDS_B + kMaxE * 4 <= 160 * 1024, "LDS");

    __shared__ __attribute__((aligned(1024))) uint8_t lds[LDS_B];
    __shared__ int er_lds[kMaxE];
    for (int e = threadIdx.x; e < E; e += 256) er_lds[e] = expert_rank[e] & 63;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int t0 = blockIdx.x * BT;
    const int wt = wave / WE, we = wave - wt * WE;           // token group, expert part
    const uint32_t lds_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((rt_lds_void*)lds));
    const int KT = d / kRtK;
    const size_t pitch = static_cast<size_t>(d) * 2;

    // Load i of a stage covers stage rows 8 i .. 8 i + 7 (lane l: row 8 i + l / 8,
    // physical chunk l % 8); rows < BT are tokens (clamped to T - 1), the rest
    // experts (clamped to E - 1).  i < BT / 8 exactly when the rows are tokens.
    auto issue_stage = [&](int kt, int buf) {
#pragma unroll
        for (int ii = 0; ii < LOADS_PER_WAVE; ++ii) {
            const int i = ii * 4 + wave;
            if (LOADS % 4 != 0 && i >= LOADS) break;        // wave-uniform
            const int r = 8 * i + (lane >> 3);
            const int chunk = (lane & 7) ^ rt_swz(r);
            const char* row = (i < BT / 8)
                                  ? reinterpret_cast<const char*>(x) + static_cast<size_t>(min(t0 + r, T - 1)) * pitch
                                  : reinterpret_cast<const char*>(wg) +
                                        static_cast<size_t>(min(r - BT, E - 1)) * pitch;
            rt_lds_dma16(row + static_cast<size_t>(kt) * kRtRowB + chunk * 16,
                         lds_base + static_cast<uint32_t>(buf * STAGE_B + i * 1024));
        }
    };

    f32x16 acc[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[j][r] = 0.0f;

    const int fr_row = lane & 31;
    const int fr_swz = rt_swz(fr_row);          // = rt_swz of the fragment's stage row
    const int fr_half = lane >> 5;
    // Ring of kRtStages buffers, two stages in flight, and the fragments one
    // K step ahead of the MFMAs.  A stage's last K step reads its fragments,
    // then the wave waits until only the loads of the stage after next (at
    // least LOADS_MIN_WAVE of its own) can still be pending, so the next stage
    // has landed; after the barrier every wave is done reading the current
    // stage, whose buffer takes the stage three ahead, and the next stage's
    // first fragments are read while the current MFMAs run.
    constexpr int KS = kRtK / 16;                            // K steps per stage
    static_assert(KS % 2 == 0, "the fragment sets alternate within a stage");
    auto read_frags = [&](int stage_buf, int ks, bf16x8& fx, bf16x8 (&fw)[NJ]) {
        const uint8_t* sx = lds + stage_buf * STAGE_B;       // token rows
        const uint8_t* sw = sx + BT * kRtRowB + we * NJ * 32 * kRtRowB;   // this wave's expert rows
        const int pc = ((2 * ks + fr_half) ^ fr_swz) << 4;
        fx = *reinterpret_cast<const bf16x8*>(sx + (wt * 32 + fr_row) * kRtRowB + pc);
#pragma unroll
        for (int j = 0; j < NJ; ++j) fw[j] = *reinterpret_cast<const bf16x8*>(sw + (j * 32 + fr_row) * kRtRowB + pc);
    };
    issue_stage(0, 0);
    if (KT > 1) issue_stage(1, 1);
    if (KT > 1) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LOADS_MIN_WAVE) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    rt_barrier();                                            // stage 0 complete in every wave
    if (KT > 2) issue_stage(2, 2);
    bf16x8 fx[2], fw[2][NJ];
    read_frags(0, 0, fx[0], fw[0]);
    int buf = 0;                                             // buffer of stage kt
    for (int kt = 0; kt < KT; ++kt) {
        const int nbuf = (buf + 1 == kRtStages) ? 0 : buf + 1;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int cur = ks & 1, nxt = cur ^ 1;
            if (ks + 1 < KS) {
                read_frags(buf, ks + 1, fx[nxt], fw[nxt]);
            } else if (kt + 1 < KT) {
                if (kt + 2 < KT) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LOADS_MIN_WAVE) : "memory");
                else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                // this wave's reads of stage kt have returned before its buffer
                // can be handed to the loads of stage kt + 3
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                rt_barrier();                                // stage kt + 1 complete; stage kt read by all
                if (kt + 3 < KT) issue_stage(kt + 3, buf);
                read_frags(nbuf, 0, fx[nxt], fw[nxt]);
            }
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[cur][j], fx[cur], acc[j], 0, 0, 0);
        }
        buf = nbuf;
    }

    // Logits tile [BT][EP] in LDS over the stage buffers: lane l holds token
    // wt * 32 + l % 32, experts 32 (we * NJ + j) + 8 q + 4 (l / 32) + 0..3 in
    // register group q of block j.
    __syncthreads();                                         // every wave is done with the stages
    float* tile = reinterpret_cast<float*>(lds);
    {
        float* trow = tile + (wt * 32 + fr_row) * LPITCH + we * NJ * 32;
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                f32x4 v;
                v[0] = acc[j][4 * q]; v[1] = acc[j][4 * q + 1]; v[2] = acc[j][4 * q + 2]; v[3] = acc[j][4 * q + 3];
                *reinterpret_cast<f32x4*>(trow + 32 * j + 8 * q + 4 * fr_half) = v;
            }
    }
    __syncthreads();
    if (logits_out) {
        const int n = min(BT, T - t0) * E;
        for (int i = threadIdx.x; i < n; i += 256) {
            const int tl = i / E, e = i - tl * E;
            logits_out[static_cast<size_t>(t0 + tl) * E + e] = tile[tl * LPITCH + e];
        }
    }

    // Routing: 8 lanes per token, 32 tokens per pass.
    constexpr int CW = V < 4 ? V : 4;
    const int g = threadIdx.x & (kGroup - 1);
#pragma unroll 1
    for (int pass = 0; pass < BT / kTokensPerBlock; ++pass) {
        const int tl = pass * kTokensPerBlock + (threadIdx.x >> 3);
        const int t = t0 + tl;
        const bool live = t < T;
        const float* row = tile + tl * LPITCH;
        float vals[V];
#pragma unroll
        for (int c = 0; c < V / CW; ++c) {
            const int e0 = c * (kGroup * CW) + g * CW;
            if constexpr (CW == 4) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(row + e0);
                vals[c * 4 + 0] = v[0]; vals[c * 4 + 1] = v[1]; vals[c * 4 + 2] = v[2]; vals[c * 4 + 3] = v[3];
            } else {
#pragma unroll
                for (int i = 0; i < CW; ++i) vals[c * CW + i] = row[e0 + i];
            }
        }
        route_token<V, K, VEC, false>(vals, g, t, live, E, R, ranks_per_node, tokens_per_rank, inter_node_cost,
                                      p, er_lds, out_idx, out_w, out_keep, out_mask);
    }
}

template <int V, int K>
void launch_router_route(const cap_topology* tp, int d, const uint16_t* x, const uint16_t* wg, float p,
                         int32_t* idx, float* w, uint8_t* keep, uint64_t* mask, float* logits, hipStream_t st) {
    constexpr int EP = 8 * V > 32 ? 8 * V : 32;
    // 128-token blocks halve the router-weight reads per token where they
    // dominate (E > 128); with fewer experts 64-token blocks give more blocks
    constexpr int BT = (EP > 128 || EP < 64) ? 128 : 64;
    const int blocks = (tp->T + BT - 1) / BT;
    if (tp->E == 8 * V)
        router_route_kernel<V, K, EP, BT, true><<<blocks, 256, 0, st>>>(
            x, wg, d, tp->T, tp->E, tp->R, tp->ranks_per_node, tp->tokens_per_rank, tp->inter_node_cost, p,
            tp->expert_rank, idx, w, keep, mask, logits);
    else
        router_route_kernel<V, K, EP, BT, false><<<blocks, 256, 0, st>>>(
            x, wg, d, tp->T, tp->E, tp->R, tp->ranks_per_node, tp->tokens_per_rank, tp->inter_node_cost, p,
            tp->expert_rank, idx, w, keep, mask, logits);
}

template <int V>
void launch_router_route_k(const cap_topology* tp, int d, const uint16_t* x, const uint16_t* wg, float p,
                           int32_t* idx, float* w, uint8_t* keep, uint64_t* mask, float* logits, hipStream_t st) {
    switch (tp->k) {
        case 1: launch_router_route<V, 1>(tp, d, x, wg, p, idx, w, keep, mask, logits, st); break;
        case 2: launch_router_route<V, 2>(tp, d, x, wg, p, idx, w, keep, mask, logits, st); break;
        case 3: launch_router_route<V, 3>(tp, d, x, wg, p, idx, w, keep, mask, logits, st); break;
        case 4: launch_router_route<V, 4>(tp, d, x, wg, p, idx, w, keep, mask, logits, st); break;
        case 5: launch_router_route<V, 5>(tp, d, x, wg, p, idx, w, keep, mask, logits, st); break;
        case 6: launch_router_route<V, 6>(tp, d, x, wg, p, idx, w, keep, mask, logits, st); break;
        case 7: launch_router_route<V, 7>(tp, d, x, wg, p, idx, w, keep, mask, logits, st); break;
        default: launch_router_route<V, 8>(tp, d, x, wg, p, idx, w, keep, mask, logits, st); break;
    }
}

}  // namespace

bool router_route_supported(const cap_topology* tp, int d) {
    return tp->E > 16 && tp->E <= kMaxE && d >= kRtK && d % kRtK == 0;
}

cap_status router_route_launch(const cap_topology* tp, int d, const void* x, const void* wg, float p, int32_t* idx,
                               float* w, uint8_t* keep, uint64_t* mask, float* logits, hipStream_t st) {
    const auto* xb = static_cast<const uint16_t*>(x);
    const auto* wb = static_cast<const uint16_t*>(wg);
    int V = 4;
    while (kGroup * V < tp->E) V <<= 1;
    switch (V) {
        case 4: launch_router_route_k<4>(tp, d, xb, wb, p, idx, w, keep, mask, logits, st); break;
        case 8: launch_router_route_k<8>(tp, d, xb, wb, p, idx, w, keep, mask, logits, st); break;
        case 16: launch_router_route_k<16>(tp, d, xb, wb, p, idx, w, keep, mask, logits, st); break;
        default: launch_router_route_k<32>(tp, d, xb, wb, p, idx, w, keep, mask, logits, st); break;
    }
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

}  // namespace cap
