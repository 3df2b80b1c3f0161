// Grouped SwiGLU expert FFN over one rank's experts (Eq. 1, Expert_i(x); the
// experts are SwiGLU FFNs: y = W2 (silu(W1 x) * (W3 x))).
//
// Two grouped GEMMs per call, each a persistent kernel with a device-side tile
// scheduler over the ragged experts (row offsets are read on the device):
//   gate/up   H[m][j] = silu(X W1^T)[m][j] * (X W3^T)[m][j]   (K = d)
//   down      Y[m][o] = (H W2^T)[m][o]                         (K = inter)
//
// bf16 path (gfx950 MFMA v_mfma_f32_32x32x16_bf16, fp32 accumulation):
//   * Block tile 256 x 256, eight waves (two per SIMD) of 64 x 128 each.
//   * Operands are both K-contiguous (token rows of X / H; weight rows of W).
//     gfx950 direct-to-LDS loads (global_load_lds_dwordx4) fill a double
//     buffer of K = 64 stages: every operand row of a stage is one whole
//     128-byte line, which the direct-to-LDS path moves at about twice the
//     rate of half lines.  One barrier per stage.
//   * Half of the waves issue all the stage loads and the other half all the
//     output stores, so no wave's in-order memory counter mixes the two (a
//     wait for a stage never waits for a tile's worth of stores to drain).
//   * The MFMA is issued with the weight fragment as its first operand, so a
//     lane's 16 accumulators hold 4 consecutive output columns per register
//     group; lanes r and r + 32 exchange halves so each stores 16 bytes.
//   * Gate/up: the B tile interleaves 32-row blocks of W1 and W3 (W1 rows j..j+31,
//     then W3 rows j..j+31, ...), so the gate and up accumulators of one output
//     element sit in the same lane and register; SiLU-and-multiply happens in
//     registers and H is rounded to bf16 once.
//   * Tiles are ordered expert, m-tile, n-tile (n fastest: neighbours share the
//     X rows); block b runs on XCD b % 8, so the block -> worker map gives each
//     XCD a contiguous run of tiles and their operands share that XCD's L2.
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
struct Sched {
    int n_tiles;        // tiles along N
    int total;          // total tiles
};

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
// stages); the kernel waits on them explicitly with wait_vmem().  Because the
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
// explicit vmcnt waits on the direct-to-LDS loads and the compiler's lgkmcnt
// waits on ds_read; the empty asm statements keep memory accesses from being
// moved across the barrier.
__device__ __forceinline__ void block_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Wait until at most n of this wave's vector-memory operations are in flight
// (n rounded down to a multiple of 4, at most 60).  Vector-memory operations
// complete in issue order, so with n = (operations issued after the stage we
// need) that stage has landed in LDS; waiting for fewer is only stricter.
__device__ __forceinline__ void wait_vmem(int n) {
    switch (n >= 60 ? 15 : n >> 2) {
        case 15: asm volatile("s_waitcnt vmcnt(60)" ::: "memory"); break;
        case 14: asm volatile("s_waitcnt vmcnt(56)" ::: "memory"); break;
        case 13: asm volatile("s_waitcnt vmcnt(52)" ::: "memory"); break;
        case 12: asm volatile("s_waitcnt vmcnt(48)" ::: "memory"); break;
        case 11: asm volatile("s_waitcnt vmcnt(44)" ::: "memory"); break;
        case 10: asm volatile("s_waitcnt vmcnt(40)" ::: "memory"); break;
        case 9: asm volatile("s_waitcnt vmcnt(36)" ::: "memory"); break;
        case 8: asm volatile("s_waitcnt vmcnt(32)" ::: "memory"); break;
        case 7: asm volatile("s_waitcnt vmcnt(28)" ::: "memory"); break;
        case 6: asm volatile("s_waitcnt vmcnt(24)" ::: "memory"); break;
        case 5: asm volatile("s_waitcnt vmcnt(20)" ::: "memory"); break;
        case 4: asm volatile("s_waitcnt vmcnt(16)" ::: "memory"); break;
        case 3: asm volatile("s_waitcnt vmcnt(12)" ::: "memory"); break;
        case 2: asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); break;
        case 1: asm volatile("s_waitcnt vmcnt(4)" ::: "memory"); break;
        default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    }
}

typedef __attribute__((address_space(3))) void lds_void;


// Roles.  Loads and stores share one in-order completion counter per wave,
// so a wave that stores its outputs and then waits for a stage would also
// wait for every store to drain (a whole tile of outputs per CU, all CUs at
// once).  The first half of the waves ("loaders") therefore issue every
// direct-to-LDS stage load and never store to global memory: they leave their
// outputs in an LDS staging area.  The other half ("storers") issue no loads;
// they write their own outputs and the staged ones, and never wait for
// stores.  The staging area is stage buffer 1, free from the end of a tile's K
// loop until the next tile fills its stage 1 (one barrier later).
//
// GATHER: row i of A is A[row_src[i]] (A has x_rows rows): each loader lane
// keeps the byte offsets of the rows it loads for the current tile.
template <int BM, int BN, int WAVES_M, int WAVES_N, bool GATEUP, bool GATHER>
__global__ __launch_bounds__(WAVES_M * WAVES_N * kWave, 1) void ffn_gemm_bf16_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ B0, const uint16_t* __restrict__ B1,
    uint16_t* __restrict__ C, const int32_t* __restrict__ row_offsets, int E_loc, int max_rows, int K,
    int N_out, const int32_t* __restrict__ row_src, int x_rows) {
    constexpr int NW = WAVES_M * WAVES_N;
    constexpr int NL = NW / 2;                             // loader waves
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int MI = WM / 32, NJ = WN / 32;
    constexpr int KS = kStageK / 16;                       // MFMA K steps per stage
    constexpr int ROWS_PER_LOAD = 1024 / kRowB;            // rows one wave-wide 16-byte load covers
    constexpr int A_LD = BM / ROWS_PER_LOAD / NL;          // direct loads per loader wave per stage
    constexpr int B_LD = BN / ROWS_PER_LOAD / NL;
    constexpr int STAGE_B = (BM + BN) * kRowB;
    constexpr int OUT_C = GATEUP ? WN / 2 : WN;            // output columns of a wave tile
    constexpr int OUT_RB = OUT_C * 2;                      // bytes per staged output row
    constexpr int OUT_CH = OUT_RB / 16;                    // 16-byte chunks per staged row
    constexpr int OUT_RPW = 256 / OUT_RB;                  // staged rows per 256-byte bank window
    constexpr int STG_B = WM * OUT_RB;                     // staging bytes per loader wave
    static_assert(NW % 2 == 0 && NL % 4 == 0, "one loader and one storer wave per SIMD");
    static_assert(BM % (ROWS_PER_LOAD * NL) == 0 && BN % (ROWS_PER_LOAD * NL) == 0, "load split");
    static_assert(A_LD + B_LD <= 60, "loads per stage must fit the vmcnt field");
    static_assert(!GATEUP || (WN % 64 == 0), "gate/up pairs need 64-column wave tiles");
    static_assert(32 % ROWS_PER_LOAD == 0, "a direct load must stay inside one W1/W3 block");
    static_assert(KS % 2 == 0, "fragments are read two K steps at a time");
    static_assert(kStages == 2 && NL * STG_B <= STAGE_B, "staging lives in stage buffer 1");
    static_assert(OUT_RB == 128 || OUT_RB == 256, "staged row layout");

    __shared__ __attribute__((aligned(1024))) uint8_t lds[kStages * STAGE_B];
    __shared__ int mt_prefix[kMaxExpertsLocal + 1];
    __shared__ int row_begin[kMaxExpertsLocal];
    __shared__ int row_end[kMaxExpertsLocal];

    build_schedule<BM>(row_offsets, E_loc, max_rows, mt_prefix, row_begin, row_end);
    const int n_tiles = GATEUP ? N_out / (BN / 2) : N_out / BN;
    const int total = mt_prefix[E_loc] * n_tiles;
    const int KT = K / kStageK;
    const int lane = threadIdx.x % kWave;
    const uint32_t wave_u = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wave = static_cast<int>(wave_u);
    const bool loader = wave < NL;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const uint32_t lds_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void*)lds));
    uint8_t* const staging = lds + STAGE_B;                // stage buffer 1

    // direct-load lane mapping: lane l writes row (l >> 3) of its 1 KiB block
    // at physical chunk (l & 7), so it fetches logical chunk (l & 7) ^ swz(row)
    // (the swizzle of a tile row depends on the block parity too).
    const int ld_row = lane >> 3;
    const int ld_pc = lane & (kChunks - 1);
    // fragment lane mapping (row r = ... + (lane & 31); swz depends on lane & 31 only)
    const int fr_row = lane & 31;
    const int fr_swz = lds_swz(fr_row);
    const int fr_half = lane >> 5;
    // staged output rows: 16-byte chunk c of row r at physical chunk
    // c ^ ((r / OUT_RPW) % OUT_CH), conflict-free for column writes and row reads
    auto stg_swz = [&](int r) { return (r / OUT_RPW) & (OUT_CH - 1); };

    // Per-tile load sources (loader waves): wave-uniform byte bases.  A rows
    // past the expert's end are clamped to its last row (never stored).
    // A loader's B rows are one contiguous run (down) or two (gate/up: its
    // W1 rows, then the matching W3 rows), so two scalar bases cover them.
    constexpr int B_RUN = GATEUP ? B_LD / 2 : B_LD;        // loads per contiguous B run
    static_assert(!GATEUP || B_RUN * ROWS_PER_LOAD == 32, "a gate/up loader covers one 32-row W1/W3 pair");
    struct TileSrc {
        const char* a;              // A + row0 * K (GATHER: A)
        int a_last;                 // last valid row of the tile
        const char* b[2];           // first row of each B run
    };
    auto tile_sources = [&](int tile, int& row0, int& rows_valid, int& nt) {
        TileSrc src;
        const int m_tile = tile / n_tiles;
        nt = tile % n_tiles;
        // wave-uniform: keep them in scalar registers
        const int l = __builtin_amdgcn_readfirstlane(find_expert(mt_prefix, E_loc, m_tile));
        row0 = __builtin_amdgcn_readfirstlane(row_begin[l] + (m_tile - mt_prefix[l]) * BM);
        rows_valid = __builtin_amdgcn_readfirstlane(min(BM, row_end[l] - row0));
        src.a = GATHER ? reinterpret_cast<const char*>(A)
                       : reinterpret_cast<const char*>(A + static_cast<size_t>(row0) * K);
        src.a_last = rows_valid - 1;
        const int lw = loader ? wave : 0;
        if constexpr (GATEUP) {
            const size_t row = static_cast<size_t>(l) * N_out + nt * (BN / 2) + lw * 32;
            src.b[0] = reinterpret_cast<const char*>(B0 + row * K);
            src.b[1] = reinterpret_cast<const char*>(B1 + row * K);
        } else {
            const size_t row = static_cast<size_t>(l) * N_out + nt * BN + lw * B_LD * ROWS_PER_LOAD;
            src.b[0] = src.b[1] = reinterpret_cast<const char*>(B0 + row * K);
        }
        return src;
    };
    // Lane byte offsets of a direct load within its 8-row block: the swizzle
    // of row (blk * 8 + ld_row) is ld_row ^ (blk & 1), so two values cover
    // every block; the block's own row offset is added inside the load.
    const uint32_t col_b[2] = {static_cast<uint32_t>((ld_pc ^ lds_swz(ld_row)) * 16),
                               static_cast<uint32_t>((ld_pc ^ lds_swz(ROWS_PER_LOAD + ld_row)) * 16)};
    const uint32_t pitch = static_cast<uint32_t>(K) * 2u;                 // bytes per operand row
    const uint32_t lane_off[2] = {ld_row * pitch + col_b[0], ld_row * pitch + col_b[1]};
    const uint32_t blk_bytes = static_cast<uint32_t>(ROWS_PER_LOAD) * pitch;
    // GATHER: byte offset (row and chunk) of each A row this loader lane loads
    uint32_t a_off[GATHER ? A_LD : 1];
    auto gather_offsets = [&](int tile_row0, int a_last) {
        if constexpr (GATHER) {
            if (!loader) return;
#pragma unroll
            for (int i = 0; i < A_LD; ++i) {
                const int r = min(wave * A_LD * ROWS_PER_LOAD + i * ROWS_PER_LOAD + ld_row, a_last);
                int tok = row_src[tile_row0 + r];
                tok = min(max(tok, 0), x_rows - 1);
                a_off[i] = static_cast<uint32_t>(tok) * pitch + col_b[(wave * A_LD + i) & 1];
            }
        }
    };
    auto issue_stage = [&](const TileSrc& src, int kt) {
        if (!loader) return;
        const uint32_t st = lds_base + static_cast<uint32_t>((kt % kStages) * STAGE_B);
        const size_t kb = static_cast<size_t>(kt) * kStageK * 2;
        const char* a_base = src.a + kb + static_cast<size_t>(wave * A_LD) * blk_bytes;
        const uint32_t a_lds = st + wave * A_LD * 1024;
        const int a_first = wave * A_LD * ROWS_PER_LOAD;
        if constexpr (GATHER) {
            static_for<A_LD>([&](auto I) {
                lds_dma16_at(src.a, a_off[I.value], static_cast<uint32_t>(kb), a_lds + I.value * 1024);
            });
        } else if (a_first + A_LD * ROWS_PER_LOAD - 1 <= src.a_last) {           // wave-uniform
            static_for<A_LD>([&](auto I) {
                lds_dma16_blk<I.value>(a_base, lane_off[(wave * A_LD + I.value) & 1], blk_bytes, a_lds + I.value * 1024);
            });
        } else {
            // the last tile of an expert: rows past its end repeat its last row
            static_for<A_LD>([&](auto I) {
                lds_dma16_clamped(src.a + kb, ld_row, a_first + I.value * ROWS_PER_LOAD, src.a_last, pitch,
                                  col_b[(wave * A_LD + I.value) & 1], a_lds + I.value * 1024);
            });
        }
        const uint32_t b_lds = st + BM * kRowB + wave * B_LD * 1024;
        static_for<B_LD>([&](auto I) {
            constexpr int i = decltype(I)::value;
            lds_dma16_blk<i % B_RUN>(src.b[i / B_RUN] + kb, lane_off[(wave * B_LD + i) & 1], blk_bytes,
                                     b_lds + i * 1024);
        });
    };

    int tile = worker_id();
    int row0 = 0, rows_valid = 0, nt = 0;
    TileSrc src;
    if (tile < total) {
        src = tile_sources(tile, row0, rows_valid, nt);
        gather_offsets(row0, src.a_last);
        issue_stage(src, 0);
    }
    while (tile < total) {
        f32x16 acc[MI][NJ];
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

        for (int kt = 0; kt < KT; ++kt) {
            if (loader) wait_vmem(0);              // this wave's part of stage kt has landed
            block_barrier();                       // stage kt visible; the other buffer is free
            if (kt + 1 < KT) issue_stage(src, kt + 1);
            const uint8_t* sa = lds + (kt % kStages) * STAGE_B;
            const uint8_t* sb = sa + BM * kRowB;
#pragma unroll
            for (int k2 = 0; k2 < KS; k2 += 2) {
                bf16x8 fa[2][MI], fb[2][NJ];
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const int pc = ((2 * (k2 + ks) + fr_half) ^ fr_swz) << 4;
#pragma unroll
                    for (int i = 0; i < MI; ++i)
                        fa[ks][i] = *reinterpret_cast<const bf16x8*>(sa + (wm * WM + i * 32 + fr_row) * kRowB + pc);
#pragma unroll
                    for (int j = 0; j < NJ; ++j)
                        fb[ks][j] = *reinterpret_cast<const bf16x8*>(sb + (wn * WN + j * 32 + fr_row) * kRowB + pc);
                }
#pragma unroll
                for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                    for (int i = 0; i < MI; ++i)
#pragma unroll
                        for (int j = 0; j < NJ; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[ks][j], fa[ks][i], acc[i][j], 0, 0, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 2 * (MI + NJ), 0);   // DS reads
                __builtin_amdgcn_sched_group_barrier(0x008, 2 * MI * NJ, 0);     // MFMA
            }
        }

        // every wave is done with this tile's LDS: loaders start the next
        // tile's stage 0 (buffer 0), buffer 1 becomes the staging area
        block_barrier();
        const int cur_row0 = row0, cur_rows = rows_valid, cur_nt = nt;
        const int next = tile + gridDim.x;
        if (next < total) {
            src = tile_sources(next, row0, rows_valid, nt);
            gather_offsets(row0, src.a_last);
            issue_stage(src, 0);
        }

        // Epilogue.  Lane (r, h) = (lane % 32, lane / 32) holds, for register
        // group g, columns 8g + 4h + 0..3 of row r of each 32x32 block.  Lanes
        // r and r + 32 swap halves (permlane32_swap) so that each holds 8
        // consecutive columns: groups (0, 1) -> lane r columns 0..7, lane r + 32
        // columns 8..15; groups (2, 3) likewise at 16 and 24.  Loaders write
        // those 16 bytes to staging, storers to the output.
        uint8_t* my_stg = staging + (loader ? wave : 0) * STG_B;
        const int out_c0 = GATEUP ? cur_nt * (BN / 2) + wn * (WN / 2) : cur_nt * BN + wn * WN;
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            if (!loader && wm * WM + i * 32 >= cur_rows) continue;      // wave-uniform
            const int r = i * 32 + fr_row;                              // row within the wave tile
            const bool row_ok = wm * WM + r < cur_rows;
            uint16_t* crow = C + static_cast<size_t>(cur_row0 + wm * WM + r) * N_out + out_c0;
            constexpr int NB = GATEUP ? NJ / 2 : NJ;                    // 32-column output blocks
#pragma unroll
            for (int jb = 0; jb < NB; ++jb) {
                float v[16];
                if constexpr (GATEUP) {
#pragma unroll
                    for (int e = 0; e < 16; ++e) v[e] = silu(acc[i][2 * jb][e]) * acc[i][2 * jb + 1][e];
                } else {
#pragma unroll
                    for (int e = 0; e < 16; ++e) v[e] = acc[i][jb][e];
                }
#pragma unroll
                for (int gp = 0; gp < 4; gp += 2) {
                    const uint32_t x0 = pack_bf16x2_rne(v[4 * gp + 0], v[4 * gp + 1]);
                    const uint32_t x1 = pack_bf16x2_rne(v[4 * gp + 2], v[4 * gp + 3]);
                    const uint32_t y0 = pack_bf16x2_rne(v[4 * gp + 4], v[4 * gp + 5]);
                    const uint32_t y1 = pack_bf16x2_rne(v[4 * gp + 6], v[4 * gp + 7]);
                    const auto ra = __builtin_amdgcn_permlane32_swap(x0, y0, false, false);
                    const auto rb = __builtin_amdgcn_permlane32_swap(x1, y1, false, false);
                    u32x4 out;
                    out[0] = ra[0]; out[1] = rb[0]; out[2] = ra[1]; out[3] = rb[1];
                    const int c = jb * 4 + gp + fr_half;                // 8-column chunk in the wave tile
                    if (loader) {
                        *reinterpret_cast<u32x4*>(my_stg + r * OUT_RB + 16 * (c ^ stg_swz(r))) = out;
                    } else if (row_ok) {
                        *reinterpret_cast<u32x4*>(crow + 8 * c) = out;
                    }
                }
            }
        }
        block_barrier();                                                // staging written
        if (!loader) {
            // storer wave w writes the staged tile of loader wave w - NL
            const int lw = wave - NL;
            const int lwm = lw / WAVES_N, lwn = lw % WAVES_N;
            const uint8_t* stg = staging + lw * STG_B;
            const int l_c0 = GATEUP ? cur_nt * (BN / 2) + lwn * (WN / 2) : cur_nt * BN + lwn * WN;
            constexpr int ROWS_PER_READ = 1024 / OUT_RB;
#pragma unroll
            for (int r0 = 0; r0 < WM; r0 += ROWS_PER_READ) {
                if (lwm * WM + r0 >= cur_rows) break;                   // wave-uniform
                const int r = r0 + lane / OUT_CH;
                const int c = lane % OUT_CH;
                const u32x4 vv = *reinterpret_cast<const u32x4*>(stg + r * OUT_RB + 16 * (c ^ stg_swz(r)));
                if (lwm * WM + r < cur_rows)
                    *reinterpret_cast<u32x4*>(C + static_cast<size_t>(cur_row0 + lwm * WM + r) * N_out + l_c0 + 8 * c) = vv;
            }
        }
        tile = next;
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
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

// Tile configurations (bf16).
constexpr int kBM = 256, kBN = 256, kWavesM = 4, kWavesN = 2;

int persistent_grid(long long tiles_upper) {
    const long long cus = device_cu_count();
    long long g = tiles_upper < cus ? tiles_upper : cus;
    if (g >= 8) g -= g % 8;          // whole XCD rounds
    return static_cast<int>(g < 1 ? 1 : g);
}

}  // namespace

size_t ffn_workspace_bytes(int max_rows, int inter, cap_dtype dt) {
    return static_cast<size_t>(max_rows) * inter * (dt == CAP_DTYPE_BF16 ? 2 : 4);
}

cap_status ffn_supported(cap_dtype dt, int d, int inter) {
    if (dt == CAP_DTYPE_BF16) return (d % kBN == 0 && inter % (kBN / 2) == 0) ? CAP_OK : CAP_ERR_UNSUPPORTED;
    return (d % 4 == 0) ? CAP_OK : CAP_ERR_UNSUPPORTED;
}

// row_src == nullptr: xs holds the expert-sorted rows; otherwise row i is
// xs[row_src[i]] and xs has x_rows rows.
cap_status expert_ffn_launch(cap_dtype dt, int E_loc, int d, int inter, int max_rows, const void* xs, int x_rows,
                             const int32_t* row_src, const int32_t* row_offsets, const void* w1, const void* w3,
                             const void* w2, void* y, void* ws, hipStream_t st) {
    if (dt == CAP_DTYPE_BF16) {
        const long long mt_upper = (static_cast<long long>(max_rows) + kBM - 1) / kBM + E_loc;
        const int g1 = persistent_grid(mt_upper * (inter / (kBN / 2)));
        const auto* a = static_cast<const uint16_t*>(xs);
        if (row_src)
            ffn_gemm_bf16_kernel<kBM, kBN, kWavesM, kWavesN, true, true><<<g1, kWavesM * kWavesN * kWave, 0, st>>>(
                a, static_cast<const uint16_t*>(w1), static_cast<const uint16_t*>(w3), static_cast<uint16_t*>(ws),
                row_offsets, E_loc, max_rows, d, inter, row_src, x_rows);
        else
            ffn_gemm_bf16_kernel<kBM, kBN, kWavesM, kWavesN, true, false><<<g1, kWavesM * kWavesN * kWave, 0, st>>>(
                a, static_cast<const uint16_t*>(w1), static_cast<const uint16_t*>(w3), static_cast<uint16_t*>(ws),
                row_offsets, E_loc, max_rows, d, inter, nullptr, 0);
        CAP_LAUNCH_CHECK();
        const int g2 = persistent_grid(mt_upper * (d / kBN));
        ffn_gemm_bf16_kernel<kBM, kBN, kWavesM, kWavesN, false, false><<<g2, kWavesM * kWavesN * kWave, 0, st>>>(
            static_cast<const uint16_t*>(ws), static_cast<const uint16_t*>(w2), nullptr,
            static_cast<uint16_t*>(y), row_offsets, E_loc, max_rows, inter, d, nullptr, 0);
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
