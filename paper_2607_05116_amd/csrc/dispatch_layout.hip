// Device-centric all-to-all layout, expert-sorted layout and send volume.
//
// Sec. II-C: a token is sent once to every device that hosts one of its kept
// experts, and the experts of that device share the copy.  Eq. 3 classes a
// destination as the own device, another device of the same node, or a device
// on another node; the per-token counts of each class are the send volume.
//
// The layout is a stable counting sort of the kept slots into E expert
// buckets (slot-position order) and of the (token, kept device) copies into R
// device buckets, with W = E + R columns.  Three launches, no global atomics,
// deterministic:
//   1. count    one block per chunk of up to 256 tokens of one source rank:
//               per-chunk column counts (LDS integer atomics, whose sum does
//               not depend on order), per-token volume, per-chunk volume sums.
//   2. colscan  one block per column: exclusive scan of the column over the
//               chunks (in place) and the column total; one more block sums
//               the volumes.
//   3. scatter  one block per chunk: every block scans the column totals
//               itself (expert offsets, receive offsets; block 0 also writes
//               them out with the send counts and offsets), then stable
//               in-chunk ranks from per-wave bitsets (LDS atomicOr, order
//               independent) and popcounts give slot_pos, copy_row and
//               recv_token.
// Workspace: [C][W] int32 chunk counts (turned into chunk bases in place),
//            [W] int32 column totals, [C][4] int64 volume sums;
//            C = R * ceil(T_loc / 256).
#include "layout_device.hpp"

#include <mutex>

// Workspace of cap_dispatch_layout_static, for callers that cannot allocate:
// one copy per GPU, held until the process ends.  Host code never uses this
// name as an address (in host code it is only a stand-in for the symbol); it
// takes the device address from hipGetSymbolAddress, per device.
static __device__ __align__(256) unsigned char scratch[cap::kLayoutScratchBytes];

namespace cap {

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept; nullptr if the runtime refuses.
void* layout_scratch_ptr() {
    static std::mutex mu;
    static void* ptrs[kMaxDevices] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(mu);
    if (!ptrs[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
        ptrs[dev] = p;
    }
    return ptrs[dev];
}

size_t layout_workspace_bytes(const cap_topology* tp) {
    size_t b = 0;
    carve(make_geom(tp, 1), nullptr, &b);
    return b;
}

cap_status dispatch_layout_launch(const cap_topology* tp, const int32_t* idx, const uint8_t* keep,
                                  const uint64_t* mask, const cap_layout* o, void* wsp, hipStream_t st) {
    const Geom g = make_geom(tp, 1);
    const Workspace ws = carve(g, wsp, nullptr);
    layout_count_kernel<<<g.C, kChunk, 0, st>>>(g, idx, keep, mask, tp->expert_rank, tp->expert_local, ws, o->vol);
    CAP_LAUNCH_CHECK();
    layout_colscan_kernel<<<g.W + 1, kChunk, 0, st>>>(g, ws, o->totals);
    CAP_LAUNCH_CHECK();
    layout_scatter_kernel<<<g.C, kChunk, 0, st>>>(g, idx, keep, mask, tp->expert_rank, tp->expert_local, ws,
                                                   o->send_counts, o->send_offsets, o->recv_offsets,
                                                   o->expert_counts, o->expert_offsets, o->slot_pos,
                                                   o->copy_row, o->recv_token);
    CAP_LAUNCH_CHECK();
    return CAP_OK;
}

}  // namespace cap
