// Grouped SwiGLU expert FFN over one rank's experts (Eq. 1, Expert_i(x); the
// experts are SwiGLU FFNs: y = W2 (silu(W1 x) * (W3 x))).
//
// Two grouped GEMMs per call over the ragged experts (row offsets are read on
// the device):
//   gate/up   H[m][j] = silu(X W1^T)[m][j] * (X W3^T)[m][j]   (K = d)
//   down      Y[m][o] = (H W2^T)[m][o]                         (K = inter)
//
// bf16 path (gfx950 MFMA v_mfma_f32_16x16x32_bf16, fp32 accumulation):
//   * Block tile 256 x 256, eight waves (two per SIMD) of 64 x 128 each.
//   * Operands are both K-contiguous (token rows of X / H; weight rows of W).
//     gfx950 direct-to-LDS loads (global_load_lds_dwordx4) fill a double
//     buffer of K = 64 stages: every operand row of a stage is one whole
//     128-byte line, which the direct-to-LDS path moves at about twice the
//     rate of half lines.  One barrier per stage.
//   * Half of the waves issue all the stage loads and the other half all the
//     output stores, so no wave's in-order memory counter mixes the two (a
//     wait for a stage never waits for a tile's worth of stores to drain).
//   * Each wave reads its LDS fragments one MFMA K step ahead of its MFMAs
//     (16 x 16 x 32 MFMAs: half the accumulator reads and writes per flop of
//     the 32 x 32 x 16 form, measured 3-4 % faster on whole calls).
//   * Calls of many m-tiles run both GEMMs in one persistent kernel with a
//     tile queue per XCD (ffn_fused_bf16_kernel); calls of few m-tiles run one
//     persistent kernel per GEMM (ffn_gemm_bf16_kernel).  Every output element
//     takes the same arithmetic in both, so the two give identical bits.
//   * Optionally (a combine plan) the down GEMM's epilogue writes the rows of
//     tokens with a single kept expert on the rank, scaled by their gate
//     weight, into the receive-side buffer instead of Y (Sec. II-C local
//     aggregation of a one-term sum).
// fp32 path: a plain LDS-tiled FMA kernel (small shapes only).
#include "cap_device.hpp"

#include <type_traits>

namespace cap {
namespace {

constexpr int kMaxExpertsLocal = kMaxE;

// Compile-time loop: f(std::integral_constant<int, 0>) ... f(<N - 1>).
template <int N, int I = 0, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<N, I + 1>(f);
    }
}

// ------------------------------------------------------------------ tile scheduler
// Fills mt_prefix[0..E_loc] (m-tiles before each expert) and row bounds.
template <int BM>
__device__ void build_schedule(const int32_t* row_offsets, int E_loc, int max_rows, int* mt_prefix,
                               int* row_begin, int* row_end) {
    const int base = row_offsets[0];
    for (int l = threadIdx.x; l < E_loc; l += blockDim.x) {
        int b = row_offsets[l] - base, e = row_offsets[l + 1] - base;
        b = max(0, min(b, max_rows));
        e = max(b, min(e, max_rows));
        row_begin[l] = b;
        row_end[l] = e;
        mt_prefix[l + 1] = (e - b + BM - 1) / BM;
    }
    if (threadIdx.x == 0) mt_prefix[0] = 0;
    __syncthreads();
    for (int off = 1; off < E_loc; off <<= 1) {
        int v = 0;
        const int i = threadIdx.x + 1;
        if (i <= E_loc && i > off) v = mt_prefix[i - off];
        __syncthreads();
        if (i <= E_loc) mt_prefix[i] += v;
        __syncthreads();
    }
}

__device__ __forceinline__ int find_expert(const int* mt_prefix, int E_loc, int m_tile) {
    int lo = 0, hi = E_loc - 1;           // largest l with mt_prefix[l] <= m_tile
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (mt_prefix[mid] <= m_tile) lo = mid; else hi = mid - 1;
    }
    return lo;
}

__device__ __forceinline__ int worker_id() {
    const int G = gridDim.x, b = blockIdx.x;
    return (G % 8 == 0) ? (b % 8) * (G / 8) + b / 8 : b;
}

// silu(g) = g * sigmoid(g); hardware exp2 and reciprocal (about 1 ulp each),
// far inside the bf16 rounding that H then takes.
__device__ __forceinline__ float silu(float g) { return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)); }

// Scalar base of a direct load: uniform by construction; readfirstlane keeps it
// in scalar registers (widening through uint32_t so the low word is never
// sign-extended).
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
    const uint64_t b = reinterpret_cast<uint64_t>(p);
    const uint64_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b)));
    const uint64_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b >> 32)));
    return reinterpret_cast<const void*>((hi << 32) | lo);
}

// Wave-wide copies global -> LDS (gfx950 global_load_lds_dwordx4): lane i
// reads 16 bytes at base + voff_i and they land at LDS byte M0 + 16 * i; base
// is a scalar register pair, voff a 32-bit per-lane byte offset, and the
// instruction's immediate offset stays 0 (it would shift the LDS address too).
// They are inline assembly so that the compiler's wait-count pass does not
// treat every later LDS read as aliasing them (it would drain all in-flight
// stages); the kernel waits on them explicitly with wait_loads().  Because the
// compiler does not see the instruction, it also does not insert the wait
// states the hardware needs before it: a VALU write of an SGPR (v_readfirstlane
// of the base) needs 5 wait states before a vector-memory instruction reads it,
// and an SALU write of M0 needs 1 before an LDS DMA; the s_nop 4 inside each
// statement provides 5.
//
// Direct load of row block I: byte offset lane_off + I * blk_bytes, formed
// inside the statement (v_mad_u32_u24; both factors stay below 2^24) so the
// compiler keeps no per-block offset registers alive across the K loop.
template <int I>
__device__ __forceinline__ void lds_dma16_blk(const void* base, uint32_t lane_off, uint32_t blk_bytes,
                                              uint32_t lds_addr) {
    uint32_t off;
    asm volatile("v_mad_u32_u24 %0, %1, %2, %3\n\ts_nop 4\n\tglobal_load_lds_dwordx4 %0, %4"
                 : "=&v"(off)
                 : "n"(I), "s"(blk_bytes), "v"(lane_off), "s"(uniform_ptr(base)),
                   "{m0}"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory");
}

// Direct load of rows first + ld_row, clamped to last (rows past an expert's
// end repeat its last row): offset min(first + ld_row, last) * pitch + col_b.
__device__ __forceinline__ void lds_dma16_clamped(const void* base, uint32_t ld_row, int first, int last,
                                                  uint32_t pitch, uint32_t col_b, uint32_t lds_addr) {
    uint32_t off;
    asm volatile("v_add_u32 %0, %1, %2\n\tv_min_i32 %0, %3, %0\n\tv_mad_u32_u24 %0, %0, %4, %5\n\t"
                 "s_nop 4\n\tglobal_load_lds_dwordx4 %0, %6"
                 : "=&v"(off)
                 : "s"(first), "v"(ld_row), "s"(last), "s"(pitch), "v"(col_b), "s"(uniform_ptr(base)),
                   "{m0}"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory");
}

// Direct load of one 16-byte chunk per lane at base + off + add (a gathered
// row: off is the lane's row offset plus its chunk, add the stage's K offset).
__device__ __forceinline__ void lds_dma16_at(const void* base, uint32_t off, uint32_t add, uint32_t lds_addr) {
    uint32_t v;
    asm volatile("v_add_u32 %0, %1, %2\n\ts_nop 4\n\tglobal_load_lds_dwordx4 %0, %3"
                 : "=&v"(v)
                 : "v"(off), "s"(add), "s"(uniform_ptr(base)), "{m0}"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory");
}

// ------------------------------------------------------------------ bf16 MFMA GEMM
// LDS holds kStages stages; a stage is the A tile [BM][64] and the B tile
// [BN][64] (bf16, 128-byte rows).  A stage row is one whole 128-byte line of
// the K-contiguous operand: the direct-to-LDS path moves full lines at about
// twice the rate of half lines, which is what sets the stage depth to K = 64.
// 16-byte chunk c of row r sits at physical chunk c ^ lds_swz(r); fragment
// reads (16 consecutive rows, one chunk) then hit distinct banks for both 128-
// and 256-byte bank windows.
constexpr int kStageK = 64;                 // K per stage
constexpr int kStages = 2;                  // double buffer: prefetch distance 1
constexpr int kRowB = kStageK * 2;          // bytes per LDS row
constexpr int kChunks = kRowB / 16;         // 16-byte chunks per row

__device__ __forceinline__ int lds_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Workgroup barrier without the memory fence that __syncthreads() carries (the
// fence would drain every in-flight prefetch).  LDS visibility is ensured by
// explicit waits: vmcnt for the direct-to-LDS loads, and lgkmcnt(0) before a
// barrier that publishes ds_write data (staged outputs, broadcast values); the
// empty asm statements keep memory accesses from being moved across the
// barrier.
__device__ __forceinline__ void block_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Wait until every vector-memory operation of this wave has completed: its
// direct-to-LDS loads have landed in LDS (the compiler does not see them, so
// it inserts no wait of its own).
__device__ __forceinline__ void wait_loads() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

typedef __attribute__((address_space(3))) void lds_void;


// ------------------------------------------------------------------ shared tile pieces
// Block tile 256 x 256, eight waves in a 4 x 2 grid, each wave 64 x 128.
constexpr int kBM = 256, kBN = 256, kWavesM = 4, kWavesN = 2;
constexpr int kNW = kWavesM * kWavesN;
constexpr int kNL = kNW / 2;                          // loader waves; the rest are storers
constexpr int kWM = kBM / kWavesM, kWN = kBN / kWavesN;
constexpr int kMI = kWM / 16, kNJ = kWN / 16;         // 16 x 16 MFMA blocks per wave
constexpr int kRowsPerLoad = 1024 / kRowB;            // rows one wave-wide 16-byte load covers
constexpr int kALd = kBM / kRowsPerLoad / kNL;        // direct loads per loader wave per stage
constexpr int kBLd = kBN / kRowsPerLoad / kNL;
constexpr int kBRun = kBLd / 2;                       // a loader's B rows: two runs of 32
constexpr int kStageBytes = (kBM + kBN) * kRowB;
static_assert(kNL % 4 == 0, "one loader and one storer wave per SIMD");
static_assert(kBM % (kRowsPerLoad * kNL) == 0 && kBN % (kRowsPerLoad * kNL) == 0, "load split");
static_assert(kALd + kBLd <= 60, "loads per stage must fit the vmcnt field");
static_assert(kWN % 64 == 0, "gate/up pairs need 64-column wave tiles");
static_assert(kBRun * kRowsPerLoad == 32, "a gate/up loader covers one 32-row W1/W3 pair");
static_assert(kALd * kRowsPerLoad == kWM, "loader wave w loads the A rows that waves of row w read");
static_assert(kStageK == 64, "a stage is two MFMA K steps of 32");
static_assert(kNJ >= kMI, "the next step's A fragments are read after the first kMI B blocks");
static_assert(kStages == 2, "staging lives in stage buffer 1");

// Per-lane constants of the direct loads and the fragment reads.
struct LaneMap {
    int ld_row;          // direct loads: lane l writes row l / 8 of its 1 KiB block ...
    uint32_t col_b[2];   // ... at physical chunk l % 8, fetching logical chunk (l % 8) ^ swz(row):
                         // the swizzle of row (8 * blk + l / 8) is swz(l / 8) ^ (blk & 1)
    int fr_row, fr_swz, fr_kc;     // fragment reads: row r = ... + lane % 16, K chunk kc(lane / 16)
};
__device__ __forceinline__ LaneMap lane_map(int lane) {
    LaneMap m;
    m.ld_row = lane >> 3;
    const int pc = lane & (kChunks - 1);
    m.col_b[0] = static_cast<uint32_t>((pc ^ lds_swz(m.ld_row)) * 16);
    m.col_b[1] = static_cast<uint32_t>((pc ^ lds_swz(kRowsPerLoad + m.ld_row)) * 16);
    m.fr_row = lane & 15;
    m.fr_swz = lds_swz(m.fr_row);
    // K chunk of lane group g = lane / 16 within a K step: 0, 2, 1, 3, so
    // that lanes l and l + 32 (read in one LDS pass) take chunks of opposite
    // parity and, under the row swizzle, distinct banks
    m.fr_kc = ((lane >> 3) & 2) | (lane >> 5);
    return m;
}

// Fragments and MFMAs.  One MFMA K step is K = 32 (two per stage).  Lane
// (r, g) = (lane % 16, lane / 16) reads row r of each 16-row block at 16-byte
// chunk 4 ks + kc(g) of K step ks, kc = (0, 2, 1, 3) (8 consecutive K; A and
// B take the same K positions, so the contraction pairs them correctly
// whatever order the hardware sums them in).  The MFMA takes the weight fragment as its first
// operand, so a lane's 4 accumulators of block (i, j) hold output columns
// 16 j + 4 q + 0..3 of tile row 16 i + r.
__device__ __forceinline__ const bf16x8& frag_at(const uint8_t* p) { return *reinterpret_cast<const bf16x8*>(p); }

// One K step of a wave's 64 x 128 block: its kMI x kNJ MFMAs, B block outer.
// With rd, the fragments of the next K step (K step nks of the stage at nst)
// are read between them: B fragment j into b[j] right after the last MFMA
// that uses it, and the A fragments into the other set an (after the first
// kMI B blocks), so one step's MFMAs cover the next step's LDS latency with
// 64 fragment registers per lane.
__device__ __forceinline__ void k_step(const bf16x8 (&ac)[kMI], bf16x8 (&an)[kMI], bf16x8 (&b)[kNJ],
                                       f32x4 (&acc)[kMI][kNJ], const uint8_t* nst, int nks, int wm, int wn,
                                       const LaneMap& lm, bool rd) {
    const int pc = ((4 * nks + lm.fr_kc) ^ lm.fr_swz) << 4;
    const uint8_t* sa = nst + (wm * kWM + lm.fr_row) * kRowB + pc;
    const uint8_t* sb = nst + (kBM + wn * kWN + lm.fr_row) * kRowB + pc;
#pragma unroll
    for (int j = 0; j < kNJ; ++j) {
#pragma unroll
        for (int i = 0; i < kMI; ++i)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[j], ac[i], acc[i][j], 0, 0, 0);
        if (rd) {
            if (j < kMI) an[j] = frag_at(sa + j * 16 * kRowB);
            b[j] = frag_at(sb + j * 16 * kRowB);
        }
    }
    static_for<kNJ>([&](auto J) {
        constexpr int j = decltype(J)::value;
        __builtin_amdgcn_sched_group_barrier(0x008, kMI, 0);                 // block j's MFMAs
        __builtin_amdgcn_sched_group_barrier(0x100, j < kMI ? 2 : 1, 0);     // its fragment reads
    });
}

// The K loop of one tile: KT stages of K = 64 (two K steps each).
// sync(kt) makes stage kt visible and issues the loads of stage kt + 1 (the
// loaders' wait for their own loads, the workgroup barrier, the next issue and
// any per-stage bookkeeping of the caller).  A wave's fragment reads run one K
// step ahead of its MFMAs; the barrier of stage kt + 1 comes after the reads of
// stage kt's second K step have returned (so the loads issued after it may
// overwrite stage kt's buffer) and before that step's MFMAs.  A wave whose
// 64 rows all lie past the tile's valid rows (active = false) computes
// nothing: its accumulators stay zero and are never stored.
template <typename Sync>
__device__ __forceinline__ void k_loop(int KT, const uint8_t* lds, int wm, int wn, const LaneMap& lm, bool active,
                                       f32x4 (&acc)[kMI][kNJ], Sync&& sync) {
    bf16x8 a0[kMI], a1[kMI], b[kNJ];
    sync(0);
    if (active) {
        const int pc = (lm.fr_kc ^ lm.fr_swz) << 4;
#pragma unroll
        for (int i = 0; i < kMI; ++i) a0[i] = frag_at(lds + (wm * kWM + i * 16 + lm.fr_row) * kRowB + pc);
#pragma unroll
        for (int j = 0; j < kNJ; ++j) b[j] = frag_at(lds + (kBM + wn * kWN + j * 16 + lm.fr_row) * kRowB + pc);
    }
    for (int kt = 0; kt < KT; ++kt) {
        if (active) k_step(a0, a1, b, acc, lds + (kt % kStages) * kStageBytes, 1, wm, wn, lm, true);
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");       // stage kt fully read
        // stage kt + 1 visible (after the last stage: a plain barrier; the
        // fragments read after it are never used)
        sync(kt + 1);
        if (active) k_step(a1, a0, b, acc, lds + ((kt + 1) % kStages) * kStageBytes, 0, wm, wn, lm, true);
    }
}

// Destination combine folded into the down GEMM's epilogue (Sec. II-C local
// aggregation, Eq. 1): row i of the call whose token has no other kept expert
// on the rank goes to row dst[i] of the receive-side buffer, scaled by its
// gate weight, instead of to Y.  The storer waves load the plan of a down
// tile's rows during its K loop into an LDS table (dst, w per row of the tile).
struct CombinePlan {
    const int32_t* dst;      // [max_rows] receive row, or -1: write Y (nullptr: no combine)
    const float* w;          // [max_rows] gate weight w'
    uint16_t* parts;         // [parts_rows][d] receive-side rows
    int parts_rows;
};

// One 16-byte chunk (8 bf16 of a Y row) scaled by w the way the destination
// reduce does it for a single term: fp32 fmaf(w, y, 0), then bf16 rounded to
// nearest even (the hardware conversion gives the reduce's bits for finite
// values).
__device__ __forceinline__ u32x4 scale_chunk(const u32x4& v, float w) {
    u32x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float lo = __builtin_fmaf(w, __uint_as_float(v[i] << 16), 0.0f);
        const float hi = __builtin_fmaf(w, __uint_as_float(v[i] & 0xFFFF0000u), 0.0f);
        o[i] = pack_bf16x2_rne(lo, hi);
    }
    return o;
}

// Epilogue of a tile of rows [row0, row0 + rows) and block column nt.
// Lane (r, q) = (lane % 16, lane / 16) holds columns 4 q + 0..3 of row r of
// each 16 x 16 block.  For a pair of adjacent blocks (32 output columns) the
// 16-lane rows of the wave swap (permlane16_swap: odd rows of the first
// operand with even rows of the second) so that each lane holds 8 consecutive
// columns: lane (r, q) gets columns 8 (q / 2) + 0..7 of block q % 2 of the
// pair, one 16-byte piece.  Gate/up: the B tile interleaves 32-row blocks of
// W1 and W3, so blocks 4p + {0, 1} and 4p + {2, 3} are the gate and up sums of
// the same 32 outputs; SiLU-and-multiply happens in registers and H is
// rounded to bf16 once.  Loader waves write their pieces to the staging area
// (stage buffer 1), storer waves to the output; after a barrier the storers
// also write the staged rows.  Storers never wait for their stores here.
// Down GEMM with a combine plan (plan_dst != nullptr): a row whose plan entry
// names a receive row in [0, parts_rows) is scaled (by the wave that holds
// its accumulators, before staging) and written there, every other row to
// the output.
template <bool GUP>
__device__ __forceinline__ void store_tile(const f32x4 (&acc)[kMI][kNJ], uint16_t* __restrict__ out, int N_out,
                                           int row0, int rows, int nt, int wave, int lane, uint8_t* staging,
                                           const int* plan_dst = nullptr, const float* plan_w = nullptr,
                                           uint16_t* __restrict__ parts = nullptr, int parts_rows = 0) {
    constexpr int OUT_C = GUP ? kWN / 2 : kWN;        // output columns of a wave tile
    constexpr int OUT_RB = OUT_C * 2;                 // bytes per staged output row
    constexpr int OUT_CH = OUT_RB / 16;               // 16-byte chunks per staged row
    constexpr int OUT_RPW = 256 / OUT_RB;             // staged rows per 256-byte bank window
    constexpr int STG_B = kWM * OUT_RB;               // staging bytes per loader wave
    constexpr int NP = OUT_C / 32;                    // 32-column block pairs of a wave's output
    static_assert(kNL * STG_B <= kStageBytes, "staging fits in stage buffer 1");
    static_assert(OUT_RB == 128 || OUT_RB == 256, "staged row layout");
    // staged output rows: 16-byte chunk c of row r at physical chunk
    // c ^ ((r / OUT_RPW) % OUT_CH), conflict-free for column writes (8
    // consecutive rows, one chunk) and row reads
    auto stg_swz = [](int r) { return (r / OUT_RPW) & (OUT_CH - 1); };
    const bool loader = wave < kNL;
    const int wm = wave / kWavesN, wn = wave % kWavesN;
    // the lane index is made opaque so that lane-derived addresses are formed
    // here, per tile, and not kept live across the K loop
    int ep_lane = lane;
    asm volatile("" : "+v"(ep_lane));
    const int ep_row = ep_lane & 15, ep_q = ep_lane >> 4;
    const int ep_c = 2 * (ep_q & 1) + (ep_q >> 1);     // this lane's chunk within a pair's four
    uint8_t* my_stg = staging + (loader ? wave : 0) * STG_B;
    const int out_c0 = (GUP ? nt * (kBN / 2) : nt * kBN) + wn * OUT_C;
#pragma unroll
    for (int i = 0; i < kMI; ++i) {
        if (!loader && wm * kWM + i * 16 >= rows) continue;            // wave-uniform
        const int r = i * 16 + ep_row;                                 // row within the wave tile
        const bool row_ok = wm * kWM + r < rows;
        uint16_t* crow = out + static_cast<size_t>(row0 + wm * kWM + r) * N_out + out_c0;
        int dst = -1;
        float dw = 0.0f;
        if (!GUP && plan_dst && row_ok) {
            dst = plan_dst[wm * kWM + r];
            dw = plan_w[wm * kWM + r];
            if (static_cast<unsigned>(dst) >= static_cast<unsigned>(parts_rows)) dst = -1;
            else if (!loader) crow = parts + static_cast<size_t>(dst) * N_out + out_c0;
        }
#pragma unroll
        for (int pr = 0; pr < NP; ++pr) {
            float v0[4], v1[4];                        // the pair's two output blocks
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if constexpr (GUP) {
                    v0[e] = silu(acc[i][4 * pr + 0][e]) * acc[i][4 * pr + 2][e];
                    v1[e] = silu(acc[i][4 * pr + 1][e]) * acc[i][4 * pr + 3][e];
                } else {
                    v0[e] = acc[i][2 * pr + 0][e];
                    v1[e] = acc[i][2 * pr + 1][e];
                }
            }
            const uint32_t x0 = pack_bf16x2_rne(v0[0], v0[1]);
            const uint32_t x1 = pack_bf16x2_rne(v0[2], v0[3]);
            const uint32_t y0 = pack_bf16x2_rne(v1[0], v1[1]);
            const uint32_t y1 = pack_bf16x2_rne(v1[2], v1[3]);
            const auto ra = __builtin_amdgcn_permlane16_swap(x0, y0, false, false);
            const auto rb = __builtin_amdgcn_permlane16_swap(x1, y1, false, false);
            u32x4 o;
            o[0] = ra[0]; o[1] = rb[0]; o[2] = ra[1]; o[3] = rb[1];
            const int c = 4 * pr + ep_c;                               // 8-column chunk in the wave tile
            if (dst >= 0) o = scale_chunk(o, dw);
            if (loader) {
                *reinterpret_cast<u32x4*>(my_stg + r * OUT_RB + 16 * (c ^ stg_swz(r))) = o;
            } else if (row_ok) {
                *reinterpret_cast<u32x4*>(crow + 8 * c) = o;
            }
        }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    block_barrier();                                                   // staging written
    if (!loader) {
        // storer wave w writes the staged tile of loader wave w - kNL
        const int lw = wave - kNL;
        const int lwm = lw / kWavesN, lwn = lw % kWavesN;
        const uint8_t* stg = staging + lw * STG_B;
        const int l_c0 = (GUP ? nt * (kBN / 2) : nt * kBN) + lwn * OUT_C;
        constexpr int ROWS_PER_READ = 1024 / OUT_RB;
#pragma unroll
        for (int r0 = 0; r0 < kWM; r0 += ROWS_PER_READ) {
            if (lwm * kWM + r0 >= rows) break;                          // wave-uniform
            const int r = r0 + ep_lane / OUT_CH;
            const int c = ep_lane % OUT_CH;
            const u32x4 vv = *reinterpret_cast<const u32x4*>(stg + r * OUT_RB + 16 * (c ^ stg_swz(r)));
            if (lwm * kWM + r < rows) {
                uint16_t* orow = out + static_cast<size_t>(row0 + lwm * kWM + r) * N_out;
                if (!GUP && plan_dst) {   // the loader wave scaled the row when it staged it
                    const int dst = plan_dst[lwm * kWM + r];
                    if (static_cast<unsigned>(dst) < static_cast<unsigned>(parts_rows))
                        orow = parts + static_cast<size_t>(dst) * N_out;
                }
                *reinterpret_cast<u32x4*>(orow + l_c0 + 8 * c) = vv;
            }
        }
    }
}

// Operand sources of one tile for one loader wave: A rows (or, gathered, the
// base of x) and the wave's two 32-row B runs; pitch = bytes per operand row.
struct TileSrc {
    const char* a;
    const char* b[2];
    uint32_t pitch, blk;                 // row pitch; bytes per 8-row block
    int rows;                            // valid A rows (past them: the last row again)
};

// Issues one stage's direct-to-LDS loads of a loader wave into stage buffer
// kt % 2: A rows wave * 64 .. + 63 and the wave's 64 B rows.  a_off holds the
// per-lane byte offsets of gathered A rows (gathered = true).
__device__ __forceinline__ void issue_stage(const TileSrc& s, int kt, int wave, const LaneMap& lm,
                                            const uint32_t (&lane_off)[2], bool gathered,
                                            const uint32_t* a_off, uint32_t lds_base) {
    const uint32_t st = lds_base + static_cast<uint32_t>((kt % kStages) * kStageBytes);
    const uint32_t kb = static_cast<uint32_t>(kt) * kStageK * 2;
    const uint32_t a_lds = st + wave * kALd * 1024;
    const int a_first = wave * kALd * kRowsPerLoad;
    if (a_first >= s.rows) {
        // no valid row in this wave's 64 A rows: the waves that would read them
        // compute nothing (k_loop's active flag), so they are not loaded
    } else if (gathered) {
        static_for<kALd>([&](auto I) { lds_dma16_at(s.a, a_off[I.value], kb, a_lds + I.value * 1024); });
    } else if (a_first + kALd * kRowsPerLoad <= s.rows) {                 // wave-uniform
        const char* a_base = s.a + kb + static_cast<size_t>(wave * kALd) * s.blk;
        static_for<kALd>([&](auto I) {
            lds_dma16_blk<I.value>(a_base, lane_off[(wave * kALd + I.value) & 1], s.blk, a_lds + I.value * 1024);
        });
    } else {
        // the last tile of an expert: rows past its end repeat its last row
        static_for<kALd>([&](auto I) {
            lds_dma16_clamped(s.a + kb, lm.ld_row, a_first + I.value * kRowsPerLoad, s.rows - 1, s.pitch,
                              lm.col_b[(wave * kALd + I.value) & 1], a_lds + I.value * 1024);
        });
    }
    const uint32_t b_lds = st + kBM * kRowB + wave * kBLd * 1024;
    static_for<kBLd>([&](auto I) {
        constexpr int i = decltype(I)::value;
        lds_dma16_blk<i % kBRun>(s.b[i / kBRun] + kb, lane_off[(wave * kBLd + i) & 1], s.blk, b_lds + i * 1024);
    });
}

// Sources of tile (expert l, rows [row0, row0 + rows), block column nt) for
// loader wave lw.  Gate/up: A = x (K = d), B runs = W1 and W3 rows
// nt * 128 + lw * 32 .. + 31 (the B tile interleaves 32-row blocks of W1 and
// W3); down: A = H (K = inter), B runs = W2 rows nt * 256 + lw * 64 .. + 63.
__device__ __forceinline__ TileSrc tile_src(bool gu, bool gathered, const uint16_t* A, const uint16_t* B0,
                                            const uint16_t* B1, int l, int row0, int rows, int nt, int lw, int K,
                                            int N_out) {
    TileSrc s;
    s.pitch = static_cast<uint32_t>(K) * 2u;
    s.blk = static_cast<uint32_t>(kRowsPerLoad) * s.pitch;
    s.rows = rows;
    s.a = gathered ? reinterpret_cast<const char*>(A) : reinterpret_cast<const char*>(A + static_cast<size_t>(row0) * K);
    if (gu) {
        const size_t row = static_cast<size_t>(l) * N_out + nt * (kBN / 2) + lw * 32;
        s.b[0] = reinterpret_cast<const char*>(B0 + row * K);
        s.b[1] = reinterpret_cast<const char*>(B1 + row * K);
    } else {
        const size_t row = static_cast<size_t>(l) * N_out + nt * kBN + lw * kBLd * kRowsPerLoad;
        s.b[0] = reinterpret_cast<const char*>(B0 + row * K);
        s.b[1] = reinterpret_cast<const char*>(B0 + (row + 32) * K);
    }
    return s;
}

// Lane byte offsets of the current tile's loads (pitch-dependent) and, for
// gathered A, of each A row this lane loads (x row row_src[row0 + r],
// clamped into [0, x_rows)).
__device__ __forceinline__ void lane_offsets(const TileSrc& s, const LaneMap& lm, uint32_t (&lane_off)[2]) {
    lane_off[0] = lm.ld_row * s.pitch + lm.col_b[0];
    lane_off[1] = lm.ld_row * s.pitch + lm.col_b[1];
}
__device__ __forceinline__ void gather_offsets(const TileSrc& s, const LaneMap& lm, int wave, int row0,
                                               const int32_t* __restrict__ row_src, int x_rows,
                                               uint32_t (&a_off)[kALd]) {
#pragma unroll
    for (int i = 0; i < kALd; ++i) {
        const int r = min(wave * kALd * kRowsPerLoad + i * kRowsPerLoad + lm.ld_row, s.rows - 1);
        int tok = row_src[row0 + r];
        tok = min(max(tok, 0), x_rows - 1);
        a_off[i] = static_cast<uint32_t>(tok) * s.pitch + lm.col_b[(wave * kALd + i) & 1];
    }
}

// ------------------------------------------------------------------ two-kernel bf16 path
// One persistent kernel per GEMM (used for calls of few m-tiles).  Roles:
// loads and stores share one in-order completion counter per wave, so a wave
// that stores its outputs and then waits for a stage would also wait for
// every store to drain (a whole tile of outputs per CU, all CUs at once).  The
// loader waves therefore issue every direct-to-LDS stage load and never store
// to global memory (they stage their outputs in LDS); the storer waves issue
// no loads, write their own and the staged outputs, and never wait for
// stores.  The staging area is stage buffer 1, free from the end of a tile's K
// loop until the next tile fills its stage 1 (one barrier later).
// Tiles are ordered expert, m-tile, n-tile (n fastest: neighbours share the A
// rows); block b runs on XCD b % 8, so the block -> worker map gives each XCD
// a contiguous run of tiles and their operands share that XCD's L2.
// GATHER: row i of A is A[row_src[i]] (A has x_rows rows).
template <bool GATEUP, bool GATHER>
__global__ __launch_bounds__(kNW * kWave, 1) void ffn_gemm_bf16_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ B0, const uint16_t* __restrict__ B1,
    uint16_t* __restrict__ C, const int32_t* __restrict__ row_offsets, int E_loc, int max_rows, int K,
    int N_out, const int32_t* __restrict__ row_src, int x_rows, CombinePlan cp) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[kStages * kStageBytes];
    __shared__ int plan_dst[kBM];
    __shared__ float plan_w[kBM];
    __shared__ int mt_prefix[kMaxExpertsLocal + 1];
    __shared__ int row_begin[kMaxExpertsLocal];
    __shared__ int row_end[kMaxExpertsLocal];

    build_schedule<kBM>(row_offsets, E_loc, max_rows, mt_prefix, row_begin, row_end);
    const int n_tiles = GATEUP ? N_out / (kBN / 2) : N_out / kBN;
    const int total = mt_prefix[E_loc] * n_tiles;
    const int KT = K / kStageK;
    const int lane = threadIdx.x % kWave;
    const int wave = static_cast<int>(__builtin_amdgcn_readfirstlane(threadIdx.x / kWave));
    const bool loader = wave < kNL;
    const int wm = wave / kWavesN, wn = wave % kWavesN;
    const uint32_t lds_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void*)lds));
    const LaneMap lm = lane_map(lane);
    // combine plan of a down tile: each storer lane loads one row's entry at
    // the third stage (after the second, where the fused kernel's storers
    // wait for their previous stores to drain) and writes it to the LDS table
    // at the last; the epilogue reads the table after the K loop's final
    // barrier
    const bool comb = !GATEUP && cp.dst != nullptr;
    int pl_d = -1;
    float pl_w = 0.0f;
    auto load_plan = [&](int kt, int KTn, int r0, int nrows) {
        const int q = (wave - kNL) * kWave + lane;
        if (kt == min(2, KTn - 1)) {
            pl_d = -1;
            pl_w = 0.0f;
            if (q < nrows) {
                pl_d = cp.dst[r0 + q];
                pl_w = cp.w[r0 + q];
            }
        }
        if (kt == KTn - 1) {
            plan_dst[q] = pl_d;
            plan_w[q] = pl_w;
        }
    };

    int row0 = 0, rows = 0, nt = 0;
    TileSrc src;
    uint32_t lane_off[2] = {0, 0};
    uint32_t a_off[kALd];
    auto start_tile = [&](int tile) {
        const int m_tile = tile / n_tiles;
        nt = tile % n_tiles;
        // wave-uniform: keep them in scalar registers
        const int l = __builtin_amdgcn_readfirstlane(find_expert(mt_prefix, E_loc, m_tile));
        row0 = __builtin_amdgcn_readfirstlane(row_begin[l] + (m_tile - mt_prefix[l]) * kBM);
        rows = __builtin_amdgcn_readfirstlane(min(kBM, row_end[l] - row0));
        if (!loader) return;
        src = tile_src(GATEUP, GATHER, A, B0, B1, l, row0, rows, nt, wave, K, N_out);
        lane_offsets(src, lm, lane_off);
        if constexpr (GATHER) gather_offsets(src, lm, wave, row0, row_src, x_rows, a_off);
        issue_stage(src, 0, wave, lm, lane_off, GATHER, a_off, lds_base);
    };

    int tile = worker_id();
    if (tile < total) start_tile(tile);
    while (tile < total) {
        f32x4 acc[kMI][kNJ];
#pragma unroll
        for (int i = 0; i < kMI; ++i)
#pragma unroll
            for (int j = 0; j < kNJ; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r) acc[i][j][r] = 0.0f;

        k_loop(KT, lds, wm, wn, lm, wm * kWM < rows, acc, [&](int kt) {
            if (loader) wait_loads();              // this wave's part of stage kt has landed
            block_barrier();                       // stage kt visible; the other buffer is free
            if (loader && kt + 1 < KT) issue_stage(src, kt + 1, wave, lm, lane_off, GATHER, a_off, lds_base);
            if (comb && !loader) load_plan(kt, KT, row0, rows);
        });

        // every wave is done with this tile's LDS: loaders start the next
        // tile's stage 0 (buffer 0), buffer 1 becomes the staging area
        block_barrier();
        const int cur_row0 = row0, cur_rows = rows, cur_nt = nt;
        const int next = tile + gridDim.x;
        if (next < total) start_tile(next);
        store_tile<GATEUP>(acc, C, N_out, cur_row0, cur_rows, cur_nt, wave, lane, lds + kStageBytes,
                           comb ? plan_dst : nullptr, plan_w, cp.parts, cp.parts_rows);
        tile = next;
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// ------------------------------------------------------------------ fused bf16 FFN
// Both GEMMs in one persistent kernel (calls of many m-tiles).  The m-tiles
// (256 expert-sorted rows) are split into one contiguous range per XCD; a
// workgroup reads its XCD from the XCC_ID hardware register.  Each XCD has a
// queue: the gate/up tiles of its m-tiles, then their down tiles, claimed one
// at a time through an atomic counter.  A down tile reads the H rows of its
// m-tile, which gate/up tiles of the same XCD wrote: those stores are in that
// XCD's L2, which its loads read.  Each storer wave adds 1 to its m-tile's
// ready counter once its store counter has drained after a gate/up tile; a
// down tile starts when that counter reaches (gate/up n-tiles) x (storer
// waves).  The gate/up tail thereby overlaps the first down tiles, and each
// XCD reads the weights of only the experts its rows belong to.
//
// The next queue entry is claimed during a tile's first stage, published at
// its second and, for a down tile, its readiness polled two stages before the
// end; a ready tile's first stage is issued before the epilogue, as in the
// two-kernel path.  Counts of this tile's stores are delivered during the next
// tile's second stage, or before any wait.
//
// No wait can deadlock: a workgroup waits (before a down tile) only once every
// gate/up tile of its XCD's queue has been claimed; a gate/up tile is claimed
// only by a running workgroup and never waits, and a workgroup delivers its own
// pending counts before it waits.  Each wait is also bounded (spin_limit
// polls): past it the kernel adds 1 to *wait_err (the caller's counter, or a
// word of the workspace when the caller passes none) and goes on, so a wait
// that gave up is visible to the caller.  A queue no workgroup touched (an XCD
// that ran none of them) is run by the last workgroup to finish, so every tile
// is computed whatever the dispatch.  target_bias is 0; a caller testing the
// give-up path passes 1, which makes every wait's target unreachable, so each
// down tile waits once and gives up after spin_limit polls.
//
// sync (ints, zero at launch): the queue counter of XCD x at
// x * kSyncQueueStride, the workspace error word, the finished-workgroup
// count, then one ready counter per m-tile.
constexpr int kSyncQueueStride = 32;                 // one 128-byte line per queue counter
constexpr int kMaxXcc = 8;
constexpr int kSyncErr = kMaxXcc * kSyncQueueStride;
constexpr int kSyncDone = kSyncErr + 1;
constexpr int kSyncReady = kSyncErr + kSyncQueueStride;
constexpr int kGroupM = 4;                 // m-tiles per group of the queue order
constexpr int kSpinLimit = 1 << 20;        // default polls before a wait gives up

__device__ __forceinline__ int xcc_register() {
    int x;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
    return x;
}

__device__ __forceinline__ int atomic_add_agent(int* p, int v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <bool GATHER>
__global__ __launch_bounds__(kNW * kWave, 1) void ffn_fused_bf16_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W1, const uint16_t* __restrict__ W3,
    const uint16_t* __restrict__ W2, uint16_t* __restrict__ H, uint16_t* __restrict__ Y,
    const int32_t* __restrict__ row_offsets, int E_loc, int max_rows, int d, int inter,
    const int32_t* __restrict__ row_src, int x_rows, int n_xcc, int* __restrict__ sync,
    int* __restrict__ wait_err, int spin_limit, int target_bias, CombinePlan cp) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[kStages * kStageBytes];
    __shared__ int plan_dst[kBM];
    __shared__ float plan_w[kBM];
    __shared__ int mt_prefix[kMaxExpertsLocal + 1];
    __shared__ int row_begin[kMaxExpertsLocal];
    __shared__ int row_end[kMaxExpertsLocal];
    // LDS broadcasts, one slot per value: each is written by one wave before a
    // barrier and read after it, and not written again before another barrier
    __shared__ int bcast[4];                // next entry; may it start early; finished count; untouched queue

    build_schedule<kBM>(row_offsets, E_loc, max_rows, mt_prefix, row_begin, row_end);
    const int MT = mt_prefix[E_loc];
    const int n_gu = inter / (kBN / 2), n_dn = d / kBN;
    const int target = n_gu * (kNW - kNL) + target_bias;
    int* const ready = sync + kSyncReady;
    const int lane = threadIdx.x % kWave;
    const int wave = static_cast<int>(__builtin_amdgcn_readfirstlane(threadIdx.x / kWave));
    const bool loader = wave < kNL;
    const int wm = wave / kWavesN, wn = wave % kWavesN;
    const uint32_t lds_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void*)lds));
    const LaneMap lm = lane_map(lane);
    // combine plan of a down tile (as in the two-kernel path)
    const bool comb = cp.dst != nullptr;
    int pl_d = -1;
    float pl_w = 0.0f;
    auto load_plan = [&](int kt, int KTn, int r0, int nrows) {
        const int q = (wave - kNL) * kWave + lane;
        if (kt == min(2, KTn - 1)) {
            pl_d = -1;
            pl_w = 0.0f;
            if (q < nrows) {
                pl_d = cp.dst[r0 + q];
                pl_w = cp.w[r0 + q];
            }
        }
        if (kt == KTn - 1) {
            plan_dst[q] = pl_d;
            plan_w[q] = pl_w;
        }
    };

    // queue of XCD slot x: m-tiles [mb, mb + MX); gate/up entries [0, GU), down [GU, Q)
    int x = xcc_register() % n_xcc;
    int mb = 0, MX = 0, GU = 0, Q = 0;
    int* queue = sync;
    auto set_queue = [&](int xs) {
        mb = (xs * MT) / n_xcc;
        MX = ((xs + 1) * MT) / n_xcc - mb;
        GU = MX * n_gu;
        Q = GU + MX * n_dn;
        queue = sync + xs * kSyncQueueStride;
    };
    // Entry u of a GEMM with nn n-tiles -> (m-tile offset, n-tile): the m-tiles
    // go in groups of kGroupM; within a group the n-tile is the outer index.
    // The workgroups of an XCD then run a block of about kGroupM m-tiles x
    // (CUs / kGroupM) n-tiles at a time, so each operand stream (an m-tile's
    // rows, an n-tile's weight rows) is shared by several running tiles and
    // the expert's weights are streamed into the XCD once per group of
    // m-tiles instead of once per one or two m-tiles.
    auto entry_tile = [&](int u, int nn, int& m_off, int& nt) {
        const int g = u / (kGroupM * nn);
        const int v = u - g * (kGroupM * nn);
        const int gm = min(kGroupM, MX - g * kGroupM);
        m_off = g * kGroupM + v % gm;
        nt = v / gm;
    };

    struct Tile { int gu, m, nt, row0, rows, KT; };
    Tile T{};
    TileSrc src;
    uint32_t lane_off[2] = {0, 0};
    uint32_t a_off[kALd];
    auto decode = [&](int t) {
        Tile D;
        D.gu = t < GU ? 1 : 0;
        const int u = D.gu ? t : t - GU;
        int m_off, nt;
        entry_tile(u, D.gu ? n_gu : n_dn, m_off, nt);
        D.m = __builtin_amdgcn_readfirstlane(mb + m_off);
        D.nt = __builtin_amdgcn_readfirstlane(nt);
        D.KT = (D.gu ? d : inter) / kStageK;
        const int l = __builtin_amdgcn_readfirstlane(find_expert(mt_prefix, E_loc, D.m));
        D.row0 = __builtin_amdgcn_readfirstlane(row_begin[l] + (D.m - mt_prefix[l]) * kBM);
        D.rows = __builtin_amdgcn_readfirstlane(min(kBM, row_end[l] - D.row0));
        if (loader) {
            src = D.gu ? tile_src(true, GATHER, X, W1, W3, l, D.row0, D.rows, D.nt, wave, d, inter)
                       : tile_src(false, false, H, W2, nullptr, l, D.row0, D.rows, D.nt, wave, inter, d);
            lane_offsets(src, lm, lane_off);
            if (GATHER && D.gu) gather_offsets(src, lm, wave, D.row0, row_src, x_rows, a_off);
        }
        return D;
    };
    auto issue = [&](int kt) {
        if (loader) issue_stage(src, kt, wave, lm, lane_off, GATHER && T.gu, a_off, lds_base);
    };
    // wave 0 waits until m-tile m's H rows are complete, then the workgroup goes on
    auto wait_ready = [&](int m) {
        if (wave == 0 && lane == 0) {
            int polls = 0;
            while (atomic_add_agent(ready + m, 0) < target) {
                if (++polls > spin_limit) {
                    atomic_add_agent(wait_err, 1);
                    break;
                }
                __builtin_amdgcn_s_sleep(4);
            }
        }
        block_barrier();
    };
    // a storer wave counts its drained gate/up stores on the m-tile's counter
    int pending = -1;
    auto deliver = [&]() {
        if (!loader && pending >= 0) {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            if (lane == 0) atomic_add_agent(ready + pending, 1);
            pending = -1;
        }
    };
    auto claim_blocking = [&]() {
        if (wave == kNL && lane == 0) bcast[0] = atomic_add_agent(queue, 1);
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        block_barrier();
        return __builtin_amdgcn_readfirstlane(bcast[0]);
    };

    bool checked_others = false;
    set_queue(x);
    for (;;) {
        int t = claim_blocking();
        if (t < Q) {
            T = decode(t);
            if (!T.gu) wait_ready(T.m);
            issue(0);
        }
        while (t < Q) {
            f32x4 acc[kMI][kNJ];
#pragma unroll
            for (int i = 0; i < kMI; ++i)
#pragma unroll
                for (int j = 0; j < kNJ; ++j)
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc[i][j][r] = 0.0f;

            const int KT = T.KT;
            const bool ahead = KT >= 4;            // claim, publish and poll inside the K loop
            int claim = 0, poll = 0;
            k_loop(KT, lds, wm, wn, lm, wm * kWM < T.rows, acc, [&](int kt) {
                if (loader) wait_loads();
                block_barrier();
                if (kt + 1 < KT) issue(kt + 1);
                if (comb && !T.gu && !loader) load_plan(kt, KT, T.row0, T.rows);
                if (ahead) {
                    if (kt == 0 && wave == kNL && lane == 0) claim = atomic_add_agent(queue, 1);
                    if (kt == 1) {
                        deliver();
                        if (wave == kNL) {
                            if (lane == 0) bcast[0] = claim;
                            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // visible at the next barrier
                        }
                    }
                    if (kt == KT - 2 && wave == 0) {
                        const int nx = bcast[0];
                        if (nx >= GU && nx < Q && lane == 0) {
                            int m_off, nt;
                            entry_tile(nx - GU, n_dn, m_off, nt);
                            poll = atomic_add_agent(ready + mb + m_off, 0);
                        }
                    }
                }
            });
            if (ahead && wave == 0 && lane == 0) {
                const int nx = bcast[0];
                bcast[1] = (nx < GU || nx >= Q || poll >= target) ? 1 : 0;
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            block_barrier();                       // every wave is done with this tile's LDS
            if (!ahead) {
                deliver();
                if (wave == kNL && lane == 0) {
                    bcast[0] = atomic_add_agent(queue, 1);
                    bcast[1] = 0;
                }
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                block_barrier();
            }
            const int nx = __builtin_amdgcn_readfirstlane(bcast[0]);
            const int early = __builtin_amdgcn_readfirstlane(bcast[1]) | (nx < GU ? 1 : 0);
            const Tile C = T;
            if (nx < Q) {
                T = decode(nx);
                if (early) issue(0);
            }
            if (C.gu) store_tile<true>(acc, H, inter, C.row0, C.rows, C.nt, wave, lane, lds + kStageBytes);
            else store_tile<false>(acc, Y, d, C.row0, C.rows, C.nt, wave, lane, lds + kStageBytes,
                                   comb ? plan_dst : nullptr, plan_w, cp.parts, cp.parts_rows);
            if (C.gu) pending = C.m;
            if (nx < Q && !early) {
                deliver();                         // the next tile may need this tile's rows
                wait_ready(T.m);
                issue(0);
            }
            t = nx;
        }
        deliver();
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        // The last workgroup to finish runs any queue that none touched.
        if (!checked_others) {
            checked_others = true;
            if (wave == 0 && lane == 0) bcast[2] = atomic_add_agent(sync + kSyncDone, 1);
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            block_barrier();
            if (__builtin_amdgcn_readfirstlane(bcast[2]) != static_cast<int>(gridDim.x) - 1) break;
        }
        if (wave == 0 && lane == 0) {
            int found = -1;
            for (int xs = 0; xs < n_xcc && found < 0; ++xs)
                if (atomic_add_agent(sync + xs * kSyncQueueStride, 0) == 0) found = xs;
            bcast[3] = found;
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        block_barrier();
        x = __builtin_amdgcn_readfirstlane(bcast[3]);
        if (x < 0) break;
        set_queue(x);
    }
}

// Zeroes the fused kernel's counters (a kernel rather than a memset, so that
// captured graphs hold no memset node).
__global__ __launch_bounds__(256) void zero_ints_kernel(int* __restrict__ p, int n) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0;
}

// ------------------------------------------------------------------ fp32 SIMT GEMM (small shapes)
constexpr int kF32Tile = 64;
constexpr int kF32K = 16;

template <bool GATEUP>
__global__ __launch_bounds__(256) void ffn_gemm_f32_kernel(
    const float* __restrict__ A, const float* __restrict__ B0, const float* __restrict__ B1,
    float* __restrict__ C, const int32_t* __restrict__ row_offsets, int E_loc, int max_rows, int K, int N_out,
    const int32_t* __restrict__ row_src, int x_rows) {
    __shared__ float sa[kF32K][kF32Tile + 1];
    __shared__ float sb0[kF32K][kF32Tile + 1];
    __shared__ float sb1[kF32K][kF32Tile + 1];
    __shared__ int mt_prefix[kMaxExpertsLocal + 1];
    __shared__ int row_begin[kMaxExpertsLocal];
    __shared__ int row_end[kMaxExpertsLocal];
    build_schedule<kF32Tile>(row_offsets, E_loc, max_rows, mt_prefix, row_begin, row_end);
    const int n_tiles = (N_out + kF32Tile - 1) / kF32Tile;
    const int total = mt_prefix[E_loc] * n_tiles;
    const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
    for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
        const int m_tile = tile / n_tiles, nt = tile % n_tiles;
        const int l = find_expert(mt_prefix, E_loc, m_tile);
        const int row0 = row_begin[l] + (m_tile - mt_prefix[l]) * kF32Tile;
        const int rows_valid = min(kF32Tile, row_end[l] - row0);
        const float* W0 = B0 + static_cast<size_t>(l) * N_out * K;
        const float* W1 = GATEUP ? B1 + static_cast<size_t>(l) * N_out * K : nullptr;
        float acc0[4][4] = {}, acc1[4][4] = {};
        for (int k0 = 0; k0 < K; k0 += kF32K) {
            for (int i = threadIdx.x; i < kF32K * kF32Tile; i += 256) {
                const int r = i / kF32K, kk = i % kF32K;
                const int gk = k0 + kk;
                int gr = row0 + min(r, rows_valid - 1);
                if (row_src) gr = min(max(row_src[gr], 0), x_rows - 1);
                const int gn = nt * kF32Tile + r;
                sa[kk][r] = gk < K ? A[static_cast<size_t>(gr) * K + gk] : 0.0f;
                sb0[kk][r] = (gk < K && gn < N_out) ? W0[static_cast<size_t>(gn) * K + gk] : 0.0f;
                if (GATEUP) sb1[kk][r] = (gk < K && gn < N_out) ? W1[static_cast<size_t>(gn) * K + gk] : 0.0f;
            }
            __syncthreads();
#pragma unroll
            for (int kk = 0; kk < kF32K; ++kk) {
                float a[4], b0[4], b1[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    a[i] = sa[kk][ty * 4 + i];
                    b0[i] = sb0[kk][tx * 4 + i];
                    b1[i] = GATEUP ? sb1[kk][tx * 4 + i] : 0.0f;
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        acc0[i][j] = __builtin_fmaf(a[i], b0[j], acc0[i][j]);
                        if (GATEUP) acc1[i][j] = __builtin_fmaf(a[i], b1[j], acc1[i][j]);
                    }
            }
            __syncthreads();
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = ty * 4 + i;
            if (r >= rows_valid) continue;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int n = nt * kF32Tile + tx * 4 + j;
                if (n >= N_out) continue;
                C[static_cast<size_t>(row0 + r) * N_out + n] =
                    GATEUP ? silu(acc0[i][j]) * acc1[i][j] : acc0[i][j];
            }
        }
    }
}

int persistent_grid(long long tiles_upper) {
    const long long cus = device_cu_count();
    long long g = tiles_upper < cus ? tiles_upper : cus;
    if (g >= 8) g -= g % 8;          // whole XCD rounds
    return static_cast<int>(g < 1 ? 1 : g);
}

// Row capacity from which a bf16 call runs the fused kernel: 32 m-tiles, so
// that every XCD gets several; below it the two-kernel path spreads the few
// m-tiles' n-tiles over all CUs.
constexpr int kFusedMinRows = 32 * kBM;

int fused_sync_ints(int max_rows) { return kSyncReady + (max_rows + kBM - 1) / kBM + kMaxExpertsLocal + 1; }

size_t ffn_h_bytes(int max_rows, int inter, cap_dtype dt) {
    const size_t h = static_cast<size_t>(max_rows) * inter * (dt == CAP_DTYPE_BF16 ? 2 : 4);
    return (h + 255) & ~static_cast<size_t>(255);
}

}  // namespace

// Workspace: H [max_rows][inter], then (bf16) the fused kernel's counters.
size_t ffn_workspace_bytes(int max_rows, int inter, cap_dtype dt) {
    return ffn_h_bytes(max_rows, inter, dt) + (dt == CAP_DTYPE_BF16 ? sizeof(int) * fused_sync_ints(max_rows) : 0);
}

// bf16: the direct loads form 8-row block offsets (16 K bytes) with 24-bit
// multiplies, so K = d or inter stays below 2^20 (2^19 here).
cap_status ffn_supported(cap_dtype dt, int d, int inter) {
    if (dt == CAP_DTYPE_BF16)
        return (d % kBN == 0 && inter % (kBN / 2) == 0 && d <= (1 << 19) && inter <= (1 << 19)) ? CAP_OK
                                                                                              : CAP_ERR_UNSUPPORTED;
    return (d % 4 == 0) ? CAP_OK : CAP_ERR_UNSUPPORTED;
}

// row_src == nullptr: xs holds the expert-sorted rows; otherwise row i is
// xs[row_src[i]] and xs has x_rows rows.  row_dst != nullptr (bf16 only): the
// destination combine of single-expert tokens goes into the down GEMM's
// epilogue (row_dst, row_w, parts, parts_rows: CombinePlan).
cap_status expert_ffn_launch(cap_dtype dt, int E_loc, int d, int inter, int max_rows, const void* xs, int x_rows,
                             const int32_t* row_src, const int32_t* row_offsets, const void* w1, const void* w3,
                             const void* w2, void* y, void* ws, const cap_ffn_options* opt, hipStream_t st,
                             const int32_t* row_dst, const float* row_w, void* parts, int parts_rows) {
    const CombinePlan cp{row_dst, row_w, static_cast<uint16_t*>(parts), parts_rows};
    const CombinePlan none{nullptr, nullptr, nullptr, 0};
    if (dt == CAP_DTYPE_BF16) {
        const auto* a = static_cast<const uint16_t*>(xs);
        const auto* b1 = static_cast<const uint16_t*>(w1);
        const auto* b3 = static_cast<const uint16_t*>(w3);
        const auto* b2 = static_cast<const uint16_t*>(w2);
        auto* h = static_cast<uint16_t*>(ws);
        auto* out = static_cast<uint16_t*>(y);
        // The fused kernel maps XCC_ID % n_xcc to a queue: with 8 XCCs the ids
        // are 0..7 (one per XCD); with one XCC all CUs share one L2.  Other
        // partitions take the two-kernel path, which needs no such mapping.
        const int n_xcc = device_xcc_count();
        if (max_rows >= kFusedMinRows && (n_xcc == kMaxXcc || n_xcc == 1)) {
            int* sync = reinterpret_cast<int*>(static_cast<char*>(ws) + ffn_h_bytes(max_rows, inter, dt));
            zero_ints_kernel<<<1, 256, 0, st>>>(sync, fused_sync_ints(max_rows));
            CAP_LAUNCH_CHECK();
            int g = persistent_grid(1ll << 30);
            // a caller's cap on the grid (with fewer workgroups than XCDs
            // the last one runs the untouched queues)
            if (opt && opt->max_workgroups > 0 && opt->max_workgroups < g) g = opt->max_workgroups;
            int* err = (opt && opt->wait_errors) ? opt->wait_errors : sync + kSyncErr;
            const int spin = (opt && opt->spin_limit > 0) ? opt->spin_limit : kSpinLimit;
            const int bias = (opt && opt->force_wait_timeout) ? 1 : 0;
            if (row_src)
                ffn_fused_bf16_kernel<true><<<g, kNW * kWave, 0, st>>>(a, b1, b3, b2, h, out, row_offsets, E_loc,
                                                                       max_rows, d, inter, row_src, x_rows, n_xcc, sync,
                                                                       err, spin, bias, cp);
            else
                ffn_fused_bf16_kernel<false><<<g, kNW * kWave, 0, st>>>(a, b1, b3, b2, h, out, row_offsets, E_loc,
                                                                        max_rows, d, inter, nullptr, 0, n_xcc, sync,
                                                                        err, spin, bias, cp);
            CAP_LAUNCH_CHECK();
            return CAP_OK;
        }
        const long long mt_upper = (static_cast<long long>(max_rows) + kBM - 1) / kBM + E_loc;
        const int g1 = persistent_grid(mt_upper * (inter / (kBN / 2)));
        if (row_src)
            ffn_gemm_bf16_kernel<true, true><<<g1, kNW * kWave, 0, st>>>(a, b1, b3, h, row_offsets, E_loc, max_rows, d,
                                                                         inter, row_src, x_rows, none);
        else
            ffn_gemm_bf16_kernel<true, false><<<g1, kNW * kWave, 0, st>>>(a, b1, b3, h, row_offsets, E_loc, max_rows, d,
                                                                          inter, nullptr, 0, none);
        CAP_LAUNCH_CHECK();
        const int g2 = persistent_grid(mt_upper * (d / kBN));
        ffn_gemm_bf16_kernel<false, false><<<g2, kNW * kWave, 0, st>>>(h, b2, nullptr, out, row_offsets, E_loc,
                                                                       max_rows, inter, d, nullptr, 0, cp);
        CAP_LAUNCH_CHECK();
    } else {
        const long long mt_upper = (static_cast<long long>(max_rows) + kF32Tile - 1) / kF32Tile + E_loc;
        const int g1 = persistent_grid(mt_upper * ((inter + kF32Tile - 1) / kF32Tile)) * 4;
        ffn_gemm_f32_kernel<true><<<g1, 256, 0, st>>>(
            static_cast<const float*>(xs), static_cast<const float*>(w1), static_cast<const float*>(w3),
            static_cast<float*>(ws), row_offsets, E_loc, max_rows, d, inter, row_src, x_rows);
        CAP_LAUNCH_CHECK();
        const int g2 = persistent_grid(mt_upper * ((d + kF32Tile - 1) / kF32Tile)) * 4;
        ffn_gemm_f32_kernel<false><<<g2, 256, 0, st>>>(
            static_cast<const float*>(ws), static_cast<const float*>(w2), nullptr, static_cast<float*>(y),
            row_offsets, E_loc, max_rows, inter, d, nullptr, 0);
        CAP_LAUNCH_CHECK();
    }
    return CAP_OK;
}

}  // namespace cap
