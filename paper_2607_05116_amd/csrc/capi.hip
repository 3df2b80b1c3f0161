// C ABI entry points: host-side validation, workspace sizing, launches.
#include <hip/hip_runtime.h>

#include <atomic>

#include "cap_device.hpp"

namespace cap {

cap_status route_prune_launch(const cap_topology*, const float*, float, bool, int32_t*, float*, uint8_t*, uint64_t*,
                              hipStream_t);
bool router_route_supported(const cap_topology*, int);
cap_status router_route_launch(const cap_topology*, int, const void*, const void*, float, int32_t*, float*, uint8_t*,
                               uint64_t*, float*, hipStream_t);
size_t layout_workspace_bytes(const cap_topology*);
void* layout_scratch_ptr();
cap_status dispatch_layout_launch(const cap_topology*, const int32_t*, const uint8_t*, const uint64_t*,
                                  const cap_layout*, void*, hipStream_t);
cap_status permute_launch(const cap_topology*, cap_permute_mode, int, cap_dtype, int, const void*, const int32_t*,
                          const uint8_t*, const uint64_t*, const cap_layout*, void*, int, hipStream_t);
cap_status combine_launch(const cap_topology*, cap_combine_mode, int, cap_dtype, int, const void*, int,
                          const int32_t*, const float*, const uint8_t*, const uint64_t*, const cap_layout*,
                          const void*, void*, int, hipStream_t);
size_t ffn_workspace_bytes(int, int, cap_dtype);
cap_status ffn_supported(cap_dtype, int, int);
cap_status expert_ffn_launch(cap_dtype, int, int, int, int, const void*, int, const int32_t*, const int32_t*,
                             const void*, const void*, const void*, void*, void*, const cap_ffn_options*,
                             hipStream_t, const int32_t*, const float*, void*, int);
cap_status row_plan_launch(const cap_topology*, int, const float*, const cap_layout*, int32_t*, int32_t*, float*,
                           int, int, hipStream_t);
size_t coact_workspace_bytes(int, int);
size_t adjustment_workspace_bytes(int);
size_t front_end_workspace_bytes(const cap_topology*);
cap_status front_end_launch(const cap_topology*, const float*, float, int32_t*, float*, uint8_t*, uint64_t*,
                            const cap_layout*, uint32_t*, void*, hipStream_t);
cap_status adjustment_launch(const uint32_t*, int, int, int, float, int32_t*, int32_t*, int, int32_t*, double*,
                             int32_t*, void*, hipStream_t);
cap_status coactivation_launch(int, int, int, const int32_t*, const uint8_t*, uint32_t*, int, void*,
                               hipStream_t);

// Compute-unit count of the current device, cached per device.
int device_cu_count() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cache[dev].store(n, std::memory_order_relaxed);
    return n;
}

// XCD (XCC) count of the current device, cached per device; 0 when the
// runtime cannot tell (callers then take paths that do not depend on it).
int device_xcc_count() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess || n <= 0) return 0;
    cache[dev].store(n, std::memory_order_relaxed);
    return n;
}

namespace {

bool topo_ok(const cap_topology* t) {
    if (!t || !t->expert_rank || !t->expert_local) return false;
    if (t->k < 1 || t->k > kMaxK) return false;
    if (t->E < 1 || t->E > kMaxE || t->k > t->E) return false;
    if (t->R < 1 || t->R > kMaxR || t->E % t->R != 0) return false;
    if (t->ranks_per_node < 1 || t->R % t->ranks_per_node != 0) return false;
    if (t->T < 1 || t->T % t->R != 0 || t->tokens_per_rank != t->T / t->R) return false;
    if (static_cast<long long>(t->T) * t->k >= (1ll << 31)) return false;
    if (!(t->inter_node_cost >= 1.0f) || !(t->inter_node_cost < INFINITY)) return false;
    return true;
}

bool layout_ok(const cap_layout* l) {
    return l && l->send_counts && l->send_offsets && l->recv_offsets && l->recv_token && l->expert_counts &&
           l->expert_offsets && l->slot_pos && l->copy_row && l->vol && l->totals;
}

bool row_dtype_ok(cap_dtype dt, int d) {
    if (d < 1) return false;
    if (dt == CAP_DTYPE_BF16) return d % 8 == 0;
    if (dt == CAP_DTYPE_F32) return d % 4 == 0;
    return false;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

}  // namespace
}  // namespace cap

using namespace cap;

extern "C" {

const char* cap_status_string(cap_status s) {
    switch (s) {
        case CAP_OK: return "CAP_OK";
        case CAP_ERR_INVALID_ARG: return "CAP_ERR_INVALID_ARG: invalid argument";
        case CAP_ERR_UNSUPPORTED: return "CAP_ERR_UNSUPPORTED: dtype/mode/shape not supported";
        case CAP_ERR_WORKSPACE: return "CAP_ERR_WORKSPACE: workspace too small";
        case CAP_ERR_HIP: return "CAP_ERR_HIP: kernel launch failed";
    }
    return "CAP_ERR_UNKNOWN";
}

int32_t cap_version(void) { return 100; }

size_t cap_workspace_size(cap_op op, const cap_topology* topo, int32_t d, int32_t inter, int32_t max_rows,
                          cap_dtype dtype) {
    switch (op) {
        case CAP_OP_DISPATCH_LAYOUT:
            return topo_ok(topo) ? layout_workspace_bytes(topo) : 0;
        case CAP_OP_EXPERT_FFN:
            if (max_rows < 0 || inter < 1) return 0;
            return ffn_workspace_bytes(max_rows, inter, dtype);
        case CAP_OP_COACTIVATION:
            if (!topo || topo->T < 1 || topo->E < 1 || topo->E > kMaxE) return 0;
            return coact_workspace_bytes(topo->T, topo->E);
        case CAP_OP_ROUTE_LAYOUT:
            return topo_ok(topo) ? front_end_workspace_bytes(topo) : 0;
        case CAP_OP_ADJUSTMENT:
            if (!topo || topo->E < 1 || topo->E > kMaxE) return 0;
            return adjustment_workspace_bytes(topo->E);
        default:
            return 0;
    }
}

cap_status cap_route_prune(const cap_topology* topo, const float* logits, float p, int32_t* idx, float* w,
                           uint8_t* keep, uint64_t* dst_mask, void* stream) {
    if (!topo_ok(topo) || !logits || !idx || !w || !keep || !dst_mask) return CAP_ERR_INVALID_ARG;
    if (!(p >= 0.0f) || !(p < 1.0f)) return CAP_ERR_INVALID_ARG;
    return route_prune_launch(topo, logits, p, false, idx, w, keep, dst_mask, as_stream(stream));
}

cap_status cap_route_prune_naive(const cap_topology* topo, const float* logits, float p, int32_t* idx, float* w,
                                 uint8_t* keep, uint64_t* dst_mask, void* stream) {
    if (!topo_ok(topo) || !logits || !idx || !w || !keep || !dst_mask) return CAP_ERR_INVALID_ARG;
    if (!(p >= 0.0f) || !(p < 1.0f)) return CAP_ERR_INVALID_ARG;
    return route_prune_launch(topo, logits, p, true, idx, w, keep, dst_mask, as_stream(stream));
}

cap_status cap_router_route_prune(const cap_topology* topo, cap_dtype dtype, int32_t d, const void* x,
                                  const void* w_gate, float p, int32_t* idx, float* w, uint8_t* keep,
                                  uint64_t* dst_mask, float* logits, void* stream) {
    if (!topo_ok(topo) || !x || !w_gate || !idx || !w || !keep || !dst_mask) return CAP_ERR_INVALID_ARG;
    if (!(p >= 0.0f) || !(p < 1.0f) || d < 1) return CAP_ERR_INVALID_ARG;
    if (dtype != CAP_DTYPE_BF16 || !router_route_supported(topo, d)) return CAP_ERR_UNSUPPORTED;
    if (!aligned16(x) || !aligned16(w_gate) || (reinterpret_cast<uintptr_t>(logits) & 3) != 0)
        return CAP_ERR_INVALID_ARG;
    return router_route_launch(topo, d, x, w_gate, p, idx, w, keep, dst_mask, logits, as_stream(stream));
}

cap_status cap_dispatch_layout(const cap_topology* topo, const int32_t* idx, const uint8_t* keep,
                               const uint64_t* dst_mask, const cap_layout* out, void* ws, size_t ws_bytes,
                               void* stream) {
    if (!topo_ok(topo) || !idx || !keep || !dst_mask || !layout_ok(out)) return CAP_ERR_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(out->vol) & 3) != 0) return CAP_ERR_INVALID_ARG;
    const size_t need = layout_workspace_bytes(topo);
    if (!ws || ws_bytes < need || (reinterpret_cast<uintptr_t>(ws) & 255) != 0) return CAP_ERR_WORKSPACE;
    return dispatch_layout_launch(topo, idx, keep, dst_mask, out, ws, as_stream(stream));
}

cap_status cap_route_layout(const cap_topology* topo, const float* logits, float p, int32_t* idx, float* w,
                            uint8_t* keep, uint64_t* dst_mask, const cap_layout* out, uint32_t* coact, void* ws,
                            size_t ws_bytes, void* stream) {
    if (!topo_ok(topo) || !logits || !idx || !w || !keep || !dst_mask || !layout_ok(out)) return CAP_ERR_INVALID_ARG;
    if (!(p >= 0.0f) || !(p < 1.0f)) return CAP_ERR_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(out->vol) & 3) != 0) return CAP_ERR_INVALID_ARG;
    if (!ws || ws_bytes < front_end_workspace_bytes(topo) || (reinterpret_cast<uintptr_t>(ws) & 255) != 0)
        return CAP_ERR_WORKSPACE;
    return front_end_launch(topo, logits, p, idx, w, keep, dst_mask, out, coact, ws, as_stream(stream));
}

cap_status cap_dispatch_layout_static(const cap_topology* topo, const int32_t* idx, const uint8_t* keep,
                                      const uint64_t* dst_mask, const cap_layout* out, void* stream) {
    if (!topo_ok(topo) || !idx || !keep || !dst_mask || !layout_ok(out)) return CAP_ERR_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(out->vol) & 3) != 0) return CAP_ERR_INVALID_ARG;
    if (layout_workspace_bytes(topo) > kLayoutScratchBytes) return CAP_ERR_WORKSPACE;
    void* ws = layout_scratch_ptr();
    if (!ws) return CAP_ERR_HIP;
    return dispatch_layout_launch(topo, idx, keep, dst_mask, out, ws, as_stream(stream));
}

size_t cap_dispatch_layout_static_max_bytes(void) { return kLayoutScratchBytes; }

cap_status cap_permute(const cap_topology* topo, cap_permute_mode mode, int32_t rank, cap_dtype dtype,
                       int32_t d, const void* x, const int32_t* idx, const uint8_t* keep, const uint64_t* dst_mask,
                       const cap_layout* lay, void* out, int32_t out_rows, void* stream) {
    if (!topo_ok(topo) || !idx || !keep || !dst_mask || !layout_ok(lay) || !out) return CAP_ERR_INVALID_ARG;
    if (rank < 0 || rank >= topo->R || out_rows < 0) return CAP_ERR_INVALID_ARG;
    if (mode == CAP_PERMUTE_ROW_SOURCE) {
        if ((reinterpret_cast<uintptr_t>(out) & 3) != 0) return CAP_ERR_INVALID_ARG;
        return permute_launch(topo, mode, rank, dtype, d, x, idx, keep, dst_mask, lay, out, out_rows,
                              as_stream(stream));
    }
    if (mode != CAP_PERMUTE_EXPERT_GATHER && mode != CAP_PERMUTE_SEND_PACK) return CAP_ERR_UNSUPPORTED;
    if (!x || !row_dtype_ok(dtype, d)) return CAP_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(out)) return CAP_ERR_INVALID_ARG;
    return permute_launch(topo, mode, rank, dtype, d, x, idx, keep, dst_mask, lay, out, out_rows,
                          as_stream(stream));
}

}  // extern "C"

namespace {

// Validation shared by the FFN entry points (CAP_OK when the call may launch).
cap_status ffn_check(cap_dtype dtype, int32_t E_loc, int32_t d, int32_t inter, int32_t max_rows, const void* x,
                     int32_t x_rows, const int32_t* row_src, const int32_t* row_offsets, const void* w1,
                     const void* w3, const void* w2, void* y, void* ws, size_t ws_bytes,
                     const cap_ffn_options* opt) {
    if (!x || !row_offsets || !w1 || !w3 || !w2 || !y) return CAP_ERR_INVALID_ARG;
    if (E_loc < 1 || E_loc > kMaxE || d < 1 || inter < 1 || max_rows < 0) return CAP_ERR_INVALID_ARG;
    if (row_src && x_rows < 1) return CAP_ERR_INVALID_ARG;
    if (opt && (opt->max_workgroups < 0 || opt->spin_limit < 0)) return CAP_ERR_INVALID_ARG;
    if (opt && opt->wait_errors && (reinterpret_cast<uintptr_t>(opt->wait_errors) & 3) != 0)
        return CAP_ERR_INVALID_ARG;
    if (dtype != CAP_DTYPE_BF16 && dtype != CAP_DTYPE_F32) return CAP_ERR_UNSUPPORTED;
    const cap_status sup = ffn_supported(dtype, d, inter);
    if (sup != CAP_OK) return sup;
    if (row_src) {
        // gathered row offsets are 32-bit byte offsets from x
        const unsigned long long x_bytes =
            static_cast<unsigned long long>(x_rows) * d * (dtype == CAP_DTYPE_BF16 ? 2u : 4u);
        if (x_bytes >= (1ull << 32)) return CAP_ERR_UNSUPPORTED;
    }
    if (!aligned16(x) || !aligned16(y) || !aligned16(w1) || !aligned16(w3) || !aligned16(w2))
        return CAP_ERR_INVALID_ARG;
    if (!ws || ws_bytes < ffn_workspace_bytes(max_rows, inter, dtype) || !aligned16(ws)) return CAP_ERR_WORKSPACE;
    return CAP_OK;
}

}  // namespace

extern "C" {

cap_status cap_expert_ffn_ex(cap_dtype dtype, int32_t E_loc, int32_t d, int32_t inter, int32_t max_rows,
                             const void* x, int32_t x_rows, const int32_t* row_src, const int32_t* row_offsets,
                             const void* w1, const void* w3, const void* w2, void* y, void* ws, size_t ws_bytes,
                             const cap_ffn_options* opt, void* stream) {
    const cap_status st = ffn_check(dtype, E_loc, d, inter, max_rows, x, x_rows, row_src, row_offsets, w1, w3, w2,
                                    y, ws, ws_bytes, opt);
    if (st != CAP_OK || max_rows == 0) return st;
    return expert_ffn_launch(dtype, E_loc, d, inter, max_rows, x, row_src ? x_rows : 0, row_src, row_offsets, w1,
                             w3, w2, y, ws, opt, as_stream(stream), nullptr, nullptr, nullptr, 0);
}

cap_status cap_expert_ffn_combine(cap_dtype dtype, int32_t E_loc, int32_t d, int32_t inter, int32_t max_rows,
                                  const void* x, int32_t x_rows, const int32_t* row_src, const int32_t* row_offsets,
                                  const void* w1, const void* w3, const void* w2, void* y, const int32_t* row_dst,
                                  const float* row_w, void* parts, int32_t parts_rows, void* ws, size_t ws_bytes,
                                  const cap_ffn_options* opt, void* stream) {
    const cap_status st = ffn_check(dtype, E_loc, d, inter, max_rows, x, x_rows, row_src, row_offsets, w1, w3, w2,
                                    y, ws, ws_bytes, opt);
    if (st != CAP_OK) return st;
    if (dtype != CAP_DTYPE_BF16) return CAP_ERR_UNSUPPORTED;
    if (!row_dst || !row_w || !parts || parts_rows < 0) return CAP_ERR_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(row_dst) & 3) != 0 || (reinterpret_cast<uintptr_t>(row_w) & 3) != 0 ||
        !aligned16(parts))
        return CAP_ERR_INVALID_ARG;
    if (max_rows == 0) return CAP_OK;
    return expert_ffn_launch(dtype, E_loc, d, inter, max_rows, x, row_src ? x_rows : 0, row_src, row_offsets, w1,
                             w3, w2, y, ws, opt, as_stream(stream), row_dst, row_w, parts, parts_rows);
}

cap_status cap_row_plan(const cap_topology* topo, int32_t rank, const float* w, const cap_layout* lay,
                        int32_t* row_src, int32_t* row_dst, float* row_w, int32_t rows_cap, int32_t parts_rows,
                        void* stream) {
    if (!topo_ok(topo) || !w || !layout_ok(lay) || !row_src || !row_dst || !row_w) return CAP_ERR_INVALID_ARG;
    if (rank < 0 || rank >= topo->R || rows_cap < 0 || parts_rows < 0) return CAP_ERR_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(row_src) & 3) != 0 || (reinterpret_cast<uintptr_t>(row_dst) & 3) != 0 ||
        (reinterpret_cast<uintptr_t>(row_w) & 3) != 0)
        return CAP_ERR_INVALID_ARG;
    return row_plan_launch(topo, rank, w, lay, row_src, row_dst, row_w, rows_cap, parts_rows, as_stream(stream));
}

cap_status cap_expert_ffn(cap_dtype dtype, int32_t E_loc, int32_t d, int32_t inter, int32_t max_rows,
                          const void* xs, const int32_t* row_offsets, const void* w1, const void* w3, const void* w2,
                          void* y, void* ws, size_t ws_bytes, void* stream) {
    return cap_expert_ffn_ex(dtype, E_loc, d, inter, max_rows, xs, 0, nullptr, row_offsets, w1, w3, w2, y, ws,
                             ws_bytes, nullptr, stream);
}

cap_status cap_expert_ffn_gather(cap_dtype dtype, int32_t E_loc, int32_t d, int32_t inter, int32_t max_rows,
                                 const void* x, int32_t x_rows, const int32_t* row_src, const int32_t* row_offsets,
                                 const void* w1, const void* w3, const void* w2, void* y, void* ws,
                                 size_t ws_bytes, void* stream) {
    if (!row_src) return CAP_ERR_INVALID_ARG;
    return cap_expert_ffn_ex(dtype, E_loc, d, inter, max_rows, x, x_rows, row_src, row_offsets, w1, w3, w2, y, ws,
                             ws_bytes, nullptr, stream);
}

cap_status cap_combine(const cap_topology* topo, cap_combine_mode mode, int32_t rank, cap_dtype dtype, int32_t d,
                       const void* in, int32_t in_rows, const int32_t* idx, const float* w, const uint8_t* keep,
                       const uint64_t* dst_mask, const cap_layout* lay, const void* shared_out, void* out,
                       int32_t out_rows, void* stream) {
    if (!topo_ok(topo) || !in || !idx || !keep || !dst_mask || !layout_ok(lay) || !out) return CAP_ERR_INVALID_ARG;
    if (rank < 0 || rank >= topo->R || in_rows < 0 || out_rows < 0) return CAP_ERR_INVALID_ARG;
    if (!row_dtype_ok(dtype, d)) return CAP_ERR_INVALID_ARG;
    if (!aligned16(in) || !aligned16(out) || (shared_out && !aligned16(shared_out))) return CAP_ERR_INVALID_ARG;
    if (mode == CAP_COMBINE_DEST_REDUCE || mode == CAP_COMBINE_DEST_REDUCE_MULTI) {
        if (!w) return CAP_ERR_INVALID_ARG;
    } else if (mode == CAP_COMBINE_SRC_REDUCE) {
        if (out_rows < topo->tokens_per_rank) return CAP_ERR_INVALID_ARG;
    } else {
        return CAP_ERR_UNSUPPORTED;
    }
    return combine_launch(topo, mode, rank, dtype, d, in, in_rows, idx, w, keep, dst_mask, lay, shared_out, out,
                          out_rows, as_stream(stream));
}

cap_status cap_coactivation(int32_t T, int32_t k, int32_t E, const int32_t* idx, const uint8_t* keep,
                            uint32_t* coact, int32_t accumulate, void* ws, size_t ws_bytes, void* stream) {
    if (!idx || !keep || !coact) return CAP_ERR_INVALID_ARG;
    if (T < 1 || k < 1 || k > kMaxK || E < 1 || E > kMaxE || static_cast<long long>(T) * k >= (1ll << 31))
        return CAP_ERR_INVALID_ARG;
    if (!ws || ws_bytes < coact_workspace_bytes(T, E) || (reinterpret_cast<uintptr_t>(ws) & 15) != 0)
        return CAP_ERR_WORKSPACE;
    return coactivation_launch(T, k, E, idx, keep, coact, accumulate, ws, as_stream(stream));
}

cap_status cap_adjustment_spectrum(const uint32_t* coact, int32_t E, int32_t R, int32_t ranks_per_node,
                                   float inter_node_cost, int32_t* expert_rank, int32_t* expert_local,
                                   int32_t max_swaps, int32_t* swaps, double* deltas, int32_t* n_swaps, void* ws,
                                   size_t ws_bytes, void* stream) {
    if (!coact || !expert_rank || !expert_local || !swaps || !n_swaps) return CAP_ERR_INVALID_ARG;
    if (E < 1 || E > kMaxE || R < 1 || R > kMaxR || E % R != 0) return CAP_ERR_INVALID_ARG;
    if (ranks_per_node < 1 || R % ranks_per_node != 0 || max_swaps < 0) return CAP_ERR_INVALID_ARG;
    if (!(inter_node_cost >= 1.0f) || !(inter_node_cost < INFINITY)) return CAP_ERR_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(deltas) & 7) != 0) return CAP_ERR_INVALID_ARG;
    if (!ws || ws_bytes < adjustment_workspace_bytes(E) || (reinterpret_cast<uintptr_t>(ws) & 7) != 0)
        return CAP_ERR_WORKSPACE;
    return adjustment_launch(coact, E, R, ranks_per_node, inter_node_cost, expert_rank, expert_local, max_swaps,
                             swaps, deltas, n_swaps, ws, as_stream(stream));
}

}  // extern "C"
