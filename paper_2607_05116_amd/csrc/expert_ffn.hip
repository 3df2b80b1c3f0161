// Grouped SwiGLU expert FFN over one rank's experts (Eq. 1, Expert_i(x); the
// experts are SwiGLU FFNs: y = W2 (silu(W1 x) * (W3 x))).
//
// Two grouped GEMMs per call, each a persistent kernel with a device-side tile
// scheduler over the ragged experts (row offsets are read on the device):
//   gate/up   H[m][j] = silu(X W1^T)[m][j] * (X W3^T)[m][j]   (K = d)
//   down      Y[m][o] = (H W2^T)[m][o]                         (K = inter)
//
// bf16 path (gfx950 MFMA v_mfma_f32_32x32x16_bf16, fp32 accumulation):
//   * Block tile BM x BN x 64, waves arranged WAVES_M x WAVES_N, each wave a
//     (BM/WAVES_M) x (BN/WAVES_N) sub-tile of 32x32 MFMA blocks.
//   * Operands are both K-contiguous (token rows of X / H; weight rows of W).
//     Global -> registers -> LDS, double-buffered, one barrier per K step.
//     LDS rows are 128 B (64 bf16); the 16-byte chunk c of row r is stored at
//     chunk c ^ (r & 7) so the MFMA fragment reads (8 consecutive rows, same
//     chunk) hit distinct banks.
//   * The MFMA is issued with the weight fragment as its first operand, so a
//     lane's 16 accumulators hold 4 consecutive output columns per register
//     group and the epilogue stores 8 bytes at a time.
//   * Gate/up: the B tile interleaves 32-row blocks of W1 and W3 (W1 rows j..j+31,
//     then W3 rows j..j+31, ...), so the gate and up accumulators of one output
//     element sit in the same lane and register; SiLU-and-multiply happens in
//     registers and H is rounded to bf16 once.
//   * Tiles are ordered expert, m-tile, n-tile (n fastest: neighbours share the
//     X rows); block b runs on XCD b % 8, so the block -> worker map gives each
//     XCD a contiguous run of tiles and their operands share that XCD's L2.
// fp32 path: a plain LDS-tiled FMA kernel (small shapes only).
#include "cap_device.hpp"

namespace cap {
namespace {

constexpr int kBK = 64;           // K per LDS stage (bf16): one 128-byte row
constexpr int kMaxExpertsLocal = kMaxE;

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

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// ------------------------------------------------------------------ bf16 MFMA GEMM
template <int BM, int BN, int WAVES_M, int WAVES_N, bool GATEUP>
__global__ __launch_bounds__(WAVES_M * WAVES_N * kWave, 1) void ffn_gemm_bf16_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ B0, const uint16_t* __restrict__ B1,
    uint16_t* __restrict__ C, const int32_t* __restrict__ row_offsets, int E_loc, int max_rows, int K,
    int N_out) {
    constexpr int NT = WAVES_M * WAVES_N * kWave;
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int MI = WM / 32, NJ = WN / 32;
    constexpr int A_LD = BM * 8 / NT;      // 16-byte chunks per thread per stage
    constexpr int B_LD = BN * 8 / NT;
    static_assert(BM * 8 % NT == 0 && BN * 8 % NT == 0, "tile / thread mismatch");
    static_assert(!GATEUP || (WN % 64 == 0), "gate/up pairs need 64-column wave tiles");

    __shared__ __attribute__((aligned(16))) uint8_t lds[2][(BM + BN) * 128];
    __shared__ int mt_prefix[kMaxExpertsLocal + 1];
    __shared__ int row_begin[kMaxExpertsLocal];
    __shared__ int row_end[kMaxExpertsLocal];

    build_schedule<BM>(row_offsets, E_loc, max_rows, mt_prefix, row_begin, row_end);
    const int n_tiles = GATEUP ? N_out / (BN / 2) : N_out / BN;
    const int total = mt_prefix[E_loc] * n_tiles;
    const int KT = K / kBK;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;

    for (int tile = worker_id(); tile < total; tile += gridDim.x) {
        const int m_tile = tile / n_tiles;
        const int nt = tile % n_tiles;
        const int l = find_expert(mt_prefix, E_loc, m_tile);
        const int row0 = row_begin[l] + (m_tile - mt_prefix[l]) * BM;
        const int rows_valid = min(BM, row_end[l] - row0);

        // This thread's 16-byte chunks: column kc, rows rbase + (NT/8)*i.  In LDS
        // they sit at a_off0 + i*(NT/8)*128 (the XOR key r & 7 is the same for
        // every i).  A rows are clamped into the expert; B rows are a fixed
        // stride apart.
        static_assert(NT / 8 >= 32 && (NT / 8) % 32 == 0, "chunk rows must keep the 32-row blocks");
        const int kc = tid & 7, rbase = tid >> 3;
        const int swz = (kc ^ (rbase & 7)) << 4;
        const int a_off0 = rbase * 128 + swz;
        const int b_off0 = BM * 128 + rbase * 128 + swz;
        int a_row[A_LD];
#pragma unroll
        for (int i = 0; i < A_LD; ++i) a_row[i] = row0 + min(rbase + (NT / 8) * i, rows_valid - 1);
        const uint16_t* Acol = A + kc * 8;
        // B chunk i covers tile row rbase + (NT/8)*i.
        //   gate/up: 32-row block q = ((NT/8)*i + rbase) / 32 alternates W1 / W3
        //   down:    row n = nt*BN + rbase + (NT/8)*i of W2
        const uint16_t* b0;
        const uint16_t* b1;
        if constexpr (GATEUP) {
            const size_t off = (static_cast<size_t>(l) * N_out + nt * (BN / 2) + (rbase & 31)) * K + kc * 8;
            b0 = B0 + off;
            b1 = B1 + off;
        } else {
            b0 = B0 + (static_cast<size_t>(l) * N_out + nt * BN + rbase) * K + kc * 8;
            b1 = b0;
        }
        // B chunk i: source row offset (in elements) from b0 / b1.
#define CAP_B_PTR(i)                                                                               \
    (GATEUP ? ((((((NT / 8) * (i) + rbase) >> 5) & 1) ? b1 : b0) +                                  \
               static_cast<size_t>((((NT / 8) * (i) + rbase) >> 5) >> 1) * 32 * K)                  \
            : (b0 + static_cast<size_t>((NT / 8) * (i)) * K))

        f32x16 acc[MI][NJ];
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

        u32x4 ra[A_LD], rb[B_LD];
#pragma unroll
        for (int i = 0; i < A_LD; ++i)
            ra[i] = *reinterpret_cast<const u32x4*>(Acol + static_cast<size_t>(a_row[i]) * K);
#pragma unroll
        for (int i = 0; i < B_LD; ++i) rb[i] = *reinterpret_cast<const u32x4*>(CAP_B_PTR(i));
#pragma unroll
        for (int i = 0; i < A_LD; ++i) *reinterpret_cast<u32x4*>(&lds[0][a_off0 + i * (NT / 8) * 128]) = ra[i];
#pragma unroll
        for (int i = 0; i < B_LD; ++i) *reinterpret_cast<u32x4*>(&lds[0][b_off0 + i * (NT / 8) * 128]) = rb[i];
        __syncthreads();

        for (int kt = 0; kt < KT; ++kt) {
            const int cur = kt & 1;
            if (kt + 1 < KT) {
                const int koff = (kt + 1) * kBK;
#pragma unroll
                for (int i = 0; i < A_LD; ++i)
                    ra[i] = *reinterpret_cast<const u32x4*>(Acol + static_cast<size_t>(a_row[i]) * K + koff);
#pragma unroll
                for (int i = 0; i < B_LD; ++i) rb[i] = *reinterpret_cast<const u32x4*>(CAP_B_PTR(i) + koff);
            }
            const uint8_t* sa = lds[cur];
            const uint8_t* sb = lds[cur] + BM * 128;
#pragma unroll
            for (int ks = 0; ks < kBK / 16; ++ks) {
                const int kc = 2 * ks + (lane >> 5);
                bf16x8 fa[MI], fb[NJ];
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    const int r = wm * WM + i * 32 + (lane & 31);
                    fa[i] = *reinterpret_cast<const bf16x8*>(sa + r * 128 + ((kc ^ (r & 7)) << 4));
                }
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    const int r = wn * WN + j * 32 + (lane & 31);
                    fb[j] = *reinterpret_cast<const bf16x8*>(sb + r * 128 + ((kc ^ (r & 7)) << 4));
                }
#pragma unroll
                for (int i = 0; i < MI; ++i)
#pragma unroll
                    for (int j = 0; j < NJ; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
            }
            if (kt + 1 < KT) {
                uint8_t* dst = lds[cur ^ 1];
#pragma unroll
                for (int i = 0; i < A_LD; ++i) *reinterpret_cast<u32x4*>(&dst[a_off0 + i * (NT / 8) * 128]) = ra[i];
#pragma unroll
                for (int i = 0; i < B_LD; ++i) *reinterpret_cast<u32x4*>(&dst[b_off0 + i * (NT / 8) * 128]) = rb[i];
            }
            __syncthreads();
        }

        // epilogue: lane holds token row m = lane % 32 of each 32-row block and,
        // per register group g, output columns 8g + 4*(lane/32) + 0..3 of each
        // 32-column block.
        const int m_lane = lane & 31;
        const int n_sub = (lane >> 5) * 4;
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            const int mr = wm * WM + i * 32 + m_lane;
            if (mr >= rows_valid) continue;
            uint16_t* crow = C + static_cast<size_t>(row0 + mr) * N_out;
            if constexpr (GATEUP) {
#pragma unroll
                for (int jp = 0; jp < NJ / 2; ++jp) {
                    const int j0 = nt * (BN / 2) + (wn * WN / 64 + jp) * 32;
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        float h[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            h[e] = silu(acc[i][2 * jp][4 * g + e]) * acc[i][2 * jp + 1][4 * g + e];
                        uint2 v;
                        v.x = pack_bf16x2(h[0], h[1]);
                        v.y = pack_bf16x2(h[2], h[3]);
                        *reinterpret_cast<uint2*>(crow + j0 + 8 * g + n_sub) = v;
                    }
                }
            } else {
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    const int c0 = nt * BN + wn * WN + j * 32;
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        uint2 v;
                        v.x = pack_bf16x2(acc[i][j][4 * g + 0], acc[i][j][4 * g + 1]);
                        v.y = pack_bf16x2(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
                        *reinterpret_cast<uint2*>(crow + c0 + 8 * g + n_sub) = v;
                    }
                }
            }
        }
    }
}

// ------------------------------------------------------------------ fp32 SIMT GEMM (small shapes)
constexpr int kF32Tile = 64;
constexpr int kF32K = 16;

template <bool GATEUP>
__global__ __launch_bounds__(256) void ffn_gemm_f32_kernel(
    const float* __restrict__ A, const float* __restrict__ B0, const float* __restrict__ B1,
    float* __restrict__ C, const int32_t* __restrict__ row_offsets, int E_loc, int max_rows, int K, int N_out) {
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
                const int gr = row0 + min(r, rows_valid - 1);
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
constexpr int kBM = 256, kBN = 256, kWavesM = 2, kWavesN = 2;

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

cap_status expert_ffn_launch(cap_dtype dt, int E_loc, int d, int inter, int max_rows, const void* xs,
                             const int32_t* row_offsets, const void* w1, const void* w3, const void* w2,
                             void* y, void* ws, hipStream_t st) {
    if (dt == CAP_DTYPE_BF16) {
        const long long mt_upper = (static_cast<long long>(max_rows) + kBM - 1) / kBM + E_loc;
        const int g1 = persistent_grid(mt_upper * (inter / (kBN / 2)));
        ffn_gemm_bf16_kernel<kBM, kBN, kWavesM, kWavesN, true><<<g1, kWavesM * kWavesN * kWave, 0, st>>>(
            static_cast<const uint16_t*>(xs), static_cast<const uint16_t*>(w1), static_cast<const uint16_t*>(w3),
            static_cast<uint16_t*>(ws), row_offsets, E_loc, max_rows, d, inter);
        CAP_LAUNCH_CHECK();
        const int g2 = persistent_grid(mt_upper * (d / kBN));
        ffn_gemm_bf16_kernel<kBM, kBN, kWavesM, kWavesN, false><<<g2, kWavesM * kWavesN * kWave, 0, st>>>(
            static_cast<const uint16_t*>(ws), static_cast<const uint16_t*>(w2), nullptr,
            static_cast<uint16_t*>(y), row_offsets, E_loc, max_rows, inter, d);
        CAP_LAUNCH_CHECK();
    } else {
        const long long mt_upper = (static_cast<long long>(max_rows) + kF32Tile - 1) / kF32Tile + E_loc;
        const int g1 = persistent_grid(mt_upper * ((inter + kF32Tile - 1) / kF32Tile)) * 4;
        ffn_gemm_f32_kernel<true><<<g1, 256, 0, st>>>(
            static_cast<const float*>(xs), static_cast<const float*>(w1), static_cast<const float*>(w3),
            static_cast<float*>(ws), row_offsets, E_loc, max_rows, d, inter);
        CAP_LAUNCH_CHECK();
        const int g2 = persistent_grid(mt_upper * ((d + kF32Tile - 1) / kF32Tile)) * 4;
        ffn_gemm_f32_kernel<false><<<g2, 256, 0, st>>>(
            static_cast<const float*>(ws), static_cast<const float*>(w2), nullptr, static_cast<float*>(y),
            row_offsets, E_loc, max_rows, inter, d);
        CAP_LAUNCH_CHECK();
    }
    return CAP_OK;
}

}  // namespace cap
