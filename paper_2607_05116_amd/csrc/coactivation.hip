// Expert co-activation counts on the pruned routing (Sec. IV-B: how often two
// experts are selected together; Sec. VII: placement runs on pruned traces).
//
// C[i][j] counts, over tokens, the ordered pairs of kept slots (s, s') with
// experts (i, j); s == s' gives the diagonal N_i.  C is symmetric, so only the
// upper triangle i <= j is accumulated (row-major, E(E+1)/2 entries); a pair
// of distinct slots adds 1 to (min, max), or 2 when both slots name the same
// expert (both orders land on the diagonal).
//
// Two launches, no global atomics, deterministic (integer sums):
//   1. tile    one block per split of consecutive tokens: the whole triangle
//              in LDS as packed 16-bit counters (two per 32-bit word; a split
//              holds at most 512 tokens and a token adds at most k^2 = 64 to
//              one counter, so none reaches 2^16), LDS integer atomics (order
//              independent), written to the split's partial slab.
//   2. reduce  every packed word summed over the splits (split groups in
//              parallel, then a fixed-order LDS sum), unpacked and written to
//              (i, j) and (j, i), added to C when accumulating.
// Workspace: [S][4 * ceil(ceil(E(E+1)/4) / 4)] uint32 packed partials (each
// split's slab padded to whole 16-byte quads).
#include "coact_device.hpp"

namespace cap {

size_t coact_workspace_bytes(int T, int E) {
    return coact_part_bytes(T, E);
}

cap_status coactivation_launch(int T, int k, int E, const int32_t* idx, const uint8_t* keep, uint32_t* coact,
                               int accumulate, void* ws, hipStream_t st) {
    const int per = coact_tokens_per_split(T);
    const int S = coact_splits(T);
    uint32_t* part = static_cast<uint32_t*>(ws);
    coact_tile_kernel<<<S, kTileThreads, 0, st>>>(T, k, E, per, idx, keep, part);
    CAP_LAUNCH_CHECK();
    coact_reduce_kernel<<<coact_reduce_blocks(E), kThreads, 0, st>>>(E, S, accumulate, part, coact);
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

}  // namespace cap
