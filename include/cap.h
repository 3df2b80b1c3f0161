/*
 * cap.h -- C ABI of the CAP expert-parallel MoE layer hot path on one MI355X.
 *
 * The library implements, as HIP kernels for gfx950, the per-GPU steps of an
 * expert-parallel MoE layer under CAP ("Communication-Aware Placement and
 * Pruning for Efficient Mixture-of-Experts Inference"):
 *   top-k routing and normalised gates (Sec. II-A, Eq. 1);
 *   communication-aware device-level pruning (Sec. VI, Eq. 6 and its greedy);
 *   the device-centric all-to-all layout and send volume (Sec. II-C, Eq. 3);
 *   token permutation; SwiGLU expert FFN over one rank's experts; the weighted
 *   combine (Sec. II-C, Eq. 1), also folded into the FFN for tokens with one
 *   kept expert on the rank; expert co-activation counts (Sec. IV-B); the
 *   expert-level pruning baseline (Sec. II-D); the Adjustment Approach's
 *   placement spectrum (Sec. V).
 * Expert-parallel ranks are virtual: all of them live on the one GPU.
 *
 * Conventions for every call
 *   - Array arguments are DEVICE pointers unless stated otherwise; sizes are
 *     host scalars.  The caller allocates and owns every buffer, including the
 *     workspace; the library never allocates, frees or keeps a pointer after
 *     the call returns (it only enqueues work).
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  Every call
 *     is asynchronous on that stream and never synchronises with the host.
 *   - Arguments are validated on the host before anything is launched; an
 *     invalid call returns an error and enqueues nothing.  Errors of a launched
 *     kernel surface at the caller's next synchronisation.
 *   - Results are deterministic: the same inputs give bit-identical outputs.
 *   - Calls on different streams with distinct output and workspace buffers
 *     may run concurrently (the library keeps no state).
 *   - Row-major layouts; "[A][B]" means A rows of B contiguous elements.
 *
 * Limits: 1 <= k <= 8, E <= 256, R <= 64 (device masks are uint64), E % R == 0,
 * T % R == 0, T*k < 2^31.  bf16 is stored as raw 16-bit patterns.
 */
#ifndef CAP_H
#define CAP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CAP_OK = 0,
    CAP_ERR_INVALID_ARG = -1,  /* null pointer, bad size, bad limit */
    CAP_ERR_UNSUPPORTED = -2,  /* dtype / mode / shape combination not built */
    CAP_ERR_WORKSPACE = -3,    /* workspace too small */
    CAP_ERR_HIP = -4           /* a kernel launch failed */
} cap_status;

typedef enum { CAP_DTYPE_F32 = 0, CAP_DTYPE_BF16 = 1 } cap_dtype;

typedef enum {
    /* destination side: the expanded, expert-sorted rows one rank computes on
       (pack + all-to-all + expand collapsed into one gather on one GPU) */
    CAP_PERMUTE_EXPERT_GATHER = 0,
    /* source side: the rank's send buffer, one row per (token, kept device) */
    CAP_PERMUTE_SEND_PACK = 1,
    /* destination side, index only: the token each expert-sorted row of the
       rank comes from (the permutation of EXPERT_GATHER without moving rows;
       cap_expert_ffn_gather then reads the rows in place) */
    CAP_PERMUTE_ROW_SOURCE = 2
} cap_permute_mode;

typedef enum {
    CAP_COMBINE_DEST_REDUCE = 0, /* per received token: weighted sum of the rank's expert rows */
    CAP_COMBINE_SRC_REDUCE = 1,  /* per source token: sum of the returned rows (+ shared) */
    /* DEST_REDUCE for the received tokens with two or more kept experts on the
       rank only; the single-expert ones were written by cap_expert_ffn_combine */
    CAP_COMBINE_DEST_REDUCE_MULTI = 2
} cap_combine_mode;

typedef enum {
    CAP_OP_ROUTE_PRUNE = 0,
    CAP_OP_DISPATCH_LAYOUT = 1,
    CAP_OP_PERMUTE = 2,
    CAP_OP_EXPERT_FFN = 3,
    CAP_OP_COMBINE = 4,
    CAP_OP_COACTIVATION = 5,
    CAP_OP_ADJUSTMENT = 6,
    CAP_OP_ROUTE_LAYOUT = 7
} cap_op;

/*
 * Expert-parallel topology and placement (Sec. IV-B: placement pi maps expert
 * -> GPU; node(.) maps GPU -> node; Eq. 3 costs 0 / 1 / c).
 *   T tokens in total; token t belongs to source rank t / tokens_per_rank
 *   (each rank runs its own requests, Sec. I); rank r is on node
 *   r / ranks_per_node.  Every rank holds E_loc = E / R experts.
 *   expert_rank[e]  (device, [E]) rank holding expert e;
 *   expert_local[e] (device, [E]) slot of expert e within its rank, in [0, E_loc);
 *                   (expert_rank, expert_local) must be a bijection onto
 *                   [0,R) x [0,E_loc).  Out-of-range entries are ignored by the
 *                   kernels (no write happens for them) and give meaningless
 *                   output, never an out-of-bounds access.
 *   inter_node_cost c >= 1: pruning cost of a device on another node; a device
 *                   on the same node costs 1 and the token's own device 0.
 * The "slot position" of expert e is P(e) = expert_rank[e]*E_loc + expert_local[e].
 */
typedef struct {
    int32_t E;
    int32_t R;
    int32_t ranks_per_node;
    int32_t T;
    int32_t tokens_per_rank;
    int32_t k;
    const int32_t *expert_rank;
    const int32_t *expert_local;
    float inter_node_cost;
} cap_topology;

/*
 * Outputs of cap_dispatch_layout, inputs of the later steps (all device).
 *   send_counts[R][R]   tokens of source s sent to device d (d == s counted):
 *                       one copy per (token, kept device), Sec. II-C.
 *   send_offsets[R][R]  exclusive scan of send_counts over d within s: row of
 *                       the first token for d in s's send buffer.
 *   recv_offsets[R+1]   exclusive scan over d of U_d = sum_s send_counts[s][d];
 *                       U_d rows form device d's receive buffer (tokens
 *                       ascending, i.e. source-major) and the buffers of all
 *                       devices are concatenated in device order.
 *   recv_token[T*k]     recv_token[recv_offsets[d] + u] = token of row u of d's
 *                       receive buffer (first recv_offsets[R] entries written).
 *   expert_counts[E]    kept (token, expert) pairs per expert, by slot position.
 *   expert_offsets[E+1] exclusive scan of expert_counts in slot-position order:
 *                       rank r's expert-sorted rows are
 *                       [expert_offsets[r*E_loc], expert_offsets[(r+1)*E_loc]).
 *   slot_pos[T][k]      row of kept slot (t,s) in that concatenation (tokens
 *                       ascending within an expert); -1 if pruned.
 *   copy_row[T][k]      row of token t in the receive buffer of the device of
 *                       slot s; -1 if pruned.  Slots on one device share it.
 *   vol[T][4]           per token: n_dev (kept devices, own included),
 *                       n_intra_remote (other devices of the own node),
 *                       n_inter (devices on other nodes), n_nodes.
 *   totals[4]           int64 sums of vol over all tokens.
 */
typedef struct {
    int32_t *send_counts;
    int32_t *send_offsets;
    int32_t *recv_offsets;
    int32_t *recv_token;
    int32_t *expert_counts;
    int32_t *expert_offsets;
    int32_t *slot_pos;
    int32_t *copy_row;
    uint8_t *vol;
    int64_t *totals;
} cap_layout;

/* Human-readable name of a status code (static string; never NULL). */
const char *cap_status_string(cap_status s);

/* Library version: major*10000 + minor*100 + patch. */
int32_t cap_version(void);

/*
 * Workspace bytes that `op` needs for this topology and shape (0 if none).
 *   CAP_OP_DISPATCH_LAYOUT: per-chunk column counts, column totals and volume sums (uses topo only).
 *   CAP_OP_EXPERT_FFN: the SwiGLU intermediate H, max_rows x inter values of
 *                      `dtype` (topo and d unused, may be NULL / 0).
 *   CAP_OP_COACTIVATION: per-split partial counts (uses topo->T and topo->E).
 *   CAP_OP_ADJUSTMENT: the E x E fp64 co-activation ratios (uses topo->E).
 *   CAP_OP_ROUTE_LAYOUT: per-32-token column counts, column totals, volume
 *                      sums and co-activation partials (uses topo only).
 *   Other ops need none.
 * Returns 0 for invalid arguments as well.
 */
size_t cap_workspace_size(cap_op op, const cap_topology *topo, int32_t d, int32_t inter,
                          int32_t max_rows, cap_dtype dtype);

/*
 * Top-k routing, normalised gates and communication-aware pruning, for all T
 * tokens (Eq. 1; Sec. VI, Eq. 6 and the greedy that follows it).
 *   logits[T][E] fp32 router logits (finite; non-finite input is a
 *                precondition violation with unspecified output).
 *   p            pruning threshold, 0 <= p < 1 (fp32).  p == 0 keeps every slot.
 * Outputs:
 *   idx[T][k]    experts in slot order: descending logit, equal logits by lower
 *                expert index (-0.0 == +0.0).
 *   w[T][k]      pruned, renormalised gates: w_s = q_s / S with
 *                q_s = cap_exp(logit_s - logit_0) and S their fp32 sum in slot
 *                order; a device d gets a_d = sum of w_s on d (slot order);
 *                devices are kept in descending a_d / cost_d (own device first,
 *                ties by lower id) until the fp32 running sum >= 1 - p; then
 *                w'_s = w_s / S' (S' = fp32 sum of kept w_s in slot order), 0
 *                for pruned slots.  cap_exp is the Cody-Waite reduced,
 *                degree-7 Taylor exponential in fp32 with fmaf (0 below -87.33).
 *   keep[T][k]   1 if the slot's device is kept, else 0.
 *   dst_mask[T]  bit d set for every kept device.
 * No workspace.
 */
cap_status cap_route_prune(const cap_topology *topo, const float *logits, float p,
                           int32_t *idx, float *w, uint8_t *keep, uint64_t *dst_mask,
                           void *stream);

/*
 * Expert-level threshold pruning: the baseline CAP is compared with (Sec. II-D;
 * the naive strategy of Sec. VIII-D).  Same arguments, top-k and gates as
 * cap_route_prune; the pruning keeps the shortest prefix of slots (descending
 * score) whose fp32 running sum of w_s reaches 1 - p (p == 0 keeps every
 * slot), renormalises the kept gates the same way, and sets dst_mask to the
 * devices of the kept slots.  It ignores where experts are placed, so it
 * removes fewer devices than cap_route_prune at the same p.  No workspace.
 */
cap_status cap_route_prune_naive(const cap_topology *topo, const float *logits, float p,
                                 int32_t *idx, float *w, uint8_t *keep, uint64_t *dst_mask,
                                 void *stream);

/*
 * Router GEMM fused with cap_route_prune (Eq. 1: the gate takes the top k of
 * the router logits x W_g^T; Sec. VI, Eq. 6 pruning).  The fp32 logits of each
 * group of 64 or 128 tokens are computed on the matrix cores into on-chip memory
 * and routed from there; the outputs are those of cap_route_prune on the same
 * logits, bit for bit.
 *   dtype            CAP_DTYPE_BF16 only (x and w_gate bf16, fp32 accumulation
 *                    in K order per 16-wide step).
 *   x[T][d]          token activations; w_gate[E][d] router weights (row e
 *                    gives expert e's logit); both 16-byte aligned.
 *   logits[T][E]     optional (NULL: not written) fp32 logits the routing used.
 * Other arguments as cap_route_prune.  Needs d % 64 == 0 and 16 < E <= 256
 * (CAP_ERR_UNSUPPORTED otherwise).  No workspace.
 */
cap_status cap_router_route_prune(const cap_topology *topo, cap_dtype dtype, int32_t d, const void *x,
                                  const void *w_gate, float p, int32_t *idx, float *w, uint8_t *keep,
                                  uint64_t *dst_mask, float *logits, void *stream);

/*
 * Counting and prefix scans into the all-to-all send layout, the expert-sorted
 * layout and per-token send volume (Sec. II-C device-centric transfer; Eq. 3
 * topology classes).  Inputs: the outputs of cap_route_prune.  Outputs: every
 * array of `out` (see cap_layout).  Needs cap_workspace_size(CAP_OP_DISPATCH_LAYOUT).
 */
cap_status cap_dispatch_layout(const cap_topology *topo, const int32_t *idx, const uint8_t *keep,
                               const uint64_t *dst_mask, const cap_layout *out,
                               void *ws, size_t ws_bytes, void *stream);

/*
 * The routing front end fused (Eq. 1 top-k and gates; Sec. VI, Eq. 6 pruning;
 * Sec. II-C layout and Eq. 3 volumes; Sec. IV-B co-activation on the pruned
 * routing): cap_route_prune, then cap_dispatch_layout, then (if coact is not
 * NULL) cap_coactivation overwriting coact, with the same outputs bit for bit,
 * in three launches instead of six.  The routing kernel also counts each
 * 32-token part's kept experts and devices (per-wave integer LDS counts
 * summed in a fixed order) and the per-token volume, so the layout needs one
 * scan and one scatter; the
 * co-activation tiles run beside the scan, its reduce beside the scatter.
 * Arguments as in those calls; coact [E][E] (device, nullable).  Workspace:
 * cap_workspace_size(CAP_OP_ROUTE_LAYOUT, topo, ...), 256-byte aligned.
 */
cap_status cap_route_layout(const cap_topology *topo, const float *logits, float p, int32_t *idx, float *w,
                            uint8_t *keep, uint64_t *dst_mask, const cap_layout *out, uint32_t *coact, void *ws,
                            size_t ws_bytes, void *stream);

/*
 * cap_dispatch_layout for callers that cannot allocate device memory (code
 * under stream capture that may not call hipMalloc, tight serving loops,
 * harnesses that forbid allocation): no workspace argument.  The library
 * keeps a fixed device array of cap_dispatch_layout_static_max_bytes()
 * (4 MiB) per GPU for it, from the first call on that GPU until the process
 * ends, and allocates nothing per call.
 *   Same arguments (minus ws / ws_bytes), outputs, arithmetic and bits as
 *   cap_dispatch_layout.
 *   Returns CAP_ERR_WORKSPACE if the topology needs more than that array
 *   (cap_workspace_size(CAP_OP_DISPATCH_LAYOUT, topo, ...) > the maximum; about
 *   R * ceil(tokens_per_rank / 256) * (E + R) * 4 bytes), CAP_ERR_HIP if the
 *   array's device address cannot be obtained.
 *   Every call on one GPU uses that GPU's one array, whose contents persist
 *   between calls (no call needs them zeroed): calls that overlap in time on
 *   one GPU (other streams, other threads) race and give undefined output;
 *   order them on one stream.
 */
cap_status cap_dispatch_layout_static(const cap_topology *topo, const int32_t *idx, const uint8_t *keep,
                                      const uint64_t *dst_mask, const cap_layout *out, void *stream);

/* Bytes of the per-GPU array behind cap_dispatch_layout_static. */
size_t cap_dispatch_layout_static_max_bytes(void);

/*
 * Token permutation (Sec. II-B: a rank dispatches each token's hidden state
 * to the ranks of its selected experts and the receiver expands it into the
 * rows of each local expert; Sec. II-C: one copy per destination device, so
 * that device's experts share it), rows of d values of `dtype` (d % 8 == 0
 * for bf16, % 4 for f32).
 *   CAP_PERMUTE_EXPERT_GATHER, rank r: out[slot_pos(t,s) - expert_offsets[r*E_loc]]
 *       = x[t] for every kept slot on r.  out holds rank r's expert-sorted rows.
 *   CAP_PERMUTE_SEND_PACK, rank s: out[send_offsets[s][d] + j] = x[t] for the
 *       j-th token t of s (ascending) whose mask holds d.
 *   CAP_PERMUTE_ROW_SOURCE, rank r: out is int32;
 *       out[slot_pos(t,s) - expert_offsets[r*E_loc]] = t for every kept slot on r,
 *       i.e. EXPERT_GATHER of the token index instead of the token's row.
 *       dtype, d and x are not used (x may be NULL); out needs 4-byte alignment.
 * x is [T][d].  The layout arrays come from cap_dispatch_layout.
 * out_rows is the capacity of `out` in rows: rows at or past it are not
 * written (size it with expert_offsets / send_counts, or an upper bound such
 * as T*min(k, E_loc) for EXPERT_GATHER and T_loc*min(k, R) for SEND_PACK).
 */
cap_status cap_permute(const cap_topology *topo, cap_permute_mode mode, int32_t rank,
                       cap_dtype dtype, int32_t d, const void *x,
                       const int32_t *idx, const uint8_t *keep, const uint64_t *dst_mask,
                       const cap_layout *lay, void *out, int32_t out_rows, void *stream);

/*
 * SwiGLU expert FFN over one rank's experts (Eq. 1 Expert_i; SwiGLU experts):
 *   for local expert l and each of its rows x:
 *   y = W2_l (silu(W1_l x) * (W3_l x)),  silu(z) = z / (1 + e^-z).
 *   xs[.][d]          expert-sorted input rows; expert l owns rows
 *                     [row_offsets[l] - row_offsets[0], row_offsets[l+1] - row_offsets[0]).
 *   row_offsets[E_loc+1] (device) non-decreasing row offsets (e.g. the rank's
 *                     slice of expert_offsets); read on the device, so the host
 *                     never needs the counts.
 *   max_rows          capacity of xs, y and the workspace, in rows.  Rows past
 *                     max_rows are not computed.
 *   w1, w3 [E_loc][inter][d]; w2 [E_loc][d][inter] (K-contiguous rows).
 *   y[.][d]           output rows, same row order as xs.
 * bf16: fp32 accumulation, H rounded to bf16 between the two GEMMs, y bf16;
 *       needs d % 256 == 0, inter % 128 == 0 and d, inter <= 2^19.
 * f32:  fp32 throughout; needs d % 4 == 0.
 * Shared experts: call with E_loc = 1, row_offsets = {0, n}, inter = the
 * concatenated intermediate size.  Workspace: cap_workspace_size(CAP_OP_EXPERT_FFN):
 * H [max_rows][inter] and, for bf16, the counters of the fused kernel; its
 * contents need no initialisation.
 * bf16 calls with max_rows >= 8192 run both GEMMs in one kernel with a tile
 * queue per XCD (a down tile starts once the gate/up tiles of its rows are
 * done) on a device of 8 XCDs (or one); other calls run one kernel per GEMM.
 * Both give the same bits.  The fused kernel's waits between workgroups are
 * bounded; one that gives up leaves that call's output invalid and is counted
 * only where cap_expert_ffn_ex is given a counter (cap_ffn_options).
 */
cap_status cap_expert_ffn(cap_dtype dtype, int32_t E_loc, int32_t d, int32_t inter,
                          int32_t max_rows, const void *xs, const int32_t *row_offsets,
                          const void *w1, const void *w3, const void *w2, void *y,
                          void *ws, size_t ws_bytes, void *stream);

/*
 * cap_expert_ffn with the token permutation folded into the first GEMM's
 * operand loads (Sec. II-C expansion; Eq. 1): row i of the expert-sorted input
 * is x[row_src[i]], read in place instead of from a gathered copy.
 *   x[x_rows][d]      token rows (the rank's received rows on a real system;
 *                     all T tokens on one GPU).
 *   row_src[max_rows] (device) source row of each expert-sorted row, e.g. the
 *                     output of cap_permute(CAP_PERMUTE_ROW_SOURCE).  Entries
 *                     outside [0, x_rows) are clamped into it (never read out
 *                     of bounds; such rows are garbage in, garbage out).
 * Every other argument, the row order of y, the arithmetic and the workspace
 * are those of cap_expert_ffn, and y is bit-identical to cap_expert_ffn on the
 * gathered rows.  Needs x_rows >= 1 and x_rows * d * element size < 2^32.
 */
cap_status cap_expert_ffn_gather(cap_dtype dtype, int32_t E_loc, int32_t d, int32_t inter,
                                 int32_t max_rows, const void *x, int32_t x_rows,
                                 const int32_t *row_src, const int32_t *row_offsets,
                                 const void *w1, const void *w3, const void *w2, void *y,
                                 void *ws, size_t ws_bytes, void *stream);

/*
 * Options of cap_expert_ffn_ex (all fields 0 / NULL: the behaviour of
 * cap_expert_ffn and cap_expert_ffn_gather).
 *   wait_errors         (device int32, nullable) the fused kernel adds 1 for
 *                       every wait between workgroups that gave up after
 *                       spin_limit polls; the output of such a call is invalid.
 *                       Never reset by the library: the caller zeroes it and
 *                       reads it after synchronising.
 *   max_workgroups      > 0 caps the fused kernel's grid (tests: with fewer
 *                       workgroups than XCDs the last one runs the queues no
 *                       workgroup touched; the result does not change).
 *   spin_limit          > 0 replaces the default of 2^20 polls per wait.
 *   force_wait_timeout  != 0 (tests of the give-up path only) makes every
 *                       wait's target unreachable: each down tile waits once
 *                       and gives up after spin_limit polls, every kernel
 *                       still finishes, the output is invalid and
 *                       *wait_errors grows by the number of down tiles.
 */
typedef struct {
    int32_t *wait_errors;
    int32_t max_workgroups;
    int32_t spin_limit;
    int32_t force_wait_timeout;
} cap_ffn_options;

/*
 * cap_expert_ffn (row_src == NULL; x is then the expert-sorted xs and x_rows
 * is ignored) or cap_expert_ffn_gather (row_src != NULL), with options (Eq. 1
 * Expert_i; Sec. II-C expansion).  opt may be NULL.  Same arguments,
 * arithmetic, workspace, limits and errors as those two calls.
 */
cap_status cap_expert_ffn_ex(cap_dtype dtype, int32_t E_loc, int32_t d, int32_t inter, int32_t max_rows,
                             const void *x, int32_t x_rows, const int32_t *row_src, const int32_t *row_offsets,
                             const void *w1, const void *w3, const void *w2, void *y, void *ws,
                             size_t ws_bytes, const cap_ffn_options *opt, void *stream);

/*
 * Row plan of rank r's expert-sorted rows for cap_expert_ffn_combine (Sec.
 * II-C: the local aggregation of a received token is the weighted sum of its
 * kept experts on the rank, Eq. 1; a token with a single kept expert there
 * has a one-term sum, which the FFN's epilogue can write directly).  For every
 * kept slot (t, s) on r, with row i = slot_pos(t,s) - expert_offsets[r*E_loc]
 * < rows_cap and t the u-th token of r's receive buffer:
 *   row_src[i] = t                       (as CAP_PERMUTE_ROW_SOURCE);
 *   row_dst[i] = recv_offsets[r] + u     if t has no other kept slot whose
 *                                        row on r is < rows_cap, and
 *                                        recv_offsets[r] + u < parts_rows;
 *                -1                      otherwise;
 *   row_w[i]   = w'(t,s) where row_dst[i] >= 0, else 0.
 * w is cap_route_prune's w'.  Rows with no kept slot are not written.  All
 * arrays are device int32 / fp32 of rows_cap entries.  No workspace.
 */
cap_status cap_row_plan(const cap_topology *topo, int32_t rank, const float *w, const cap_layout *lay,
                        int32_t *row_src, int32_t *row_dst, float *row_w, int32_t rows_cap,
                        int32_t parts_rows, void *stream);

/*
 * cap_expert_ffn_ex (bf16) with the destination combine of single-expert
 * tokens folded into the down GEMM's epilogue (Eq. 1; Sec. II-C local
 * aggregation).  For each row i < max_rows:
 *   0 <= row_dst[i] < parts_rows:  parts[row_dst[i]] = bf16(fmaf(row_w[i], y_i, 0))
 *       with y_i = the bf16 FFN output row, the arithmetic CAP_COMBINE_DEST_REDUCE
 *       does for a one-term sum, so the bits equal that path's; y[i] is not
 *       written;
 *   otherwise:                     y[i] as cap_expert_ffn_ex.
 * row_dst, row_w: device int32 / fp32 [max_rows] (cap_row_plan); parts:
 * [parts_rows][d] bf16, 16-byte aligned (the concatenated receive-side buffer
 * of cap_combine).  The remaining tokens then take
 * cap_combine(CAP_COMBINE_DEST_REDUCE_MULTI) with in_rows = the plan's rows_cap
 * and out_rows = parts_rows.  Other arguments, workspace, limits and errors as
 * cap_expert_ffn_ex; CAP_ERR_UNSUPPORTED for f32.
 */
cap_status cap_expert_ffn_combine(cap_dtype dtype, int32_t E_loc, int32_t d, int32_t inter, int32_t max_rows,
                                  const void *x, int32_t x_rows, const int32_t *row_src,
                                  const int32_t *row_offsets, const void *w1, const void *w3, const void *w2,
                                  void *y, const int32_t *row_dst, const float *row_w, void *parts,
                                  int32_t parts_rows, void *ws, size_t ws_bytes, const cap_ffn_options *opt,
                                  void *stream);

/*
 * Weighted combine (Sec. II-C local aggregation and final combination; Eq. 1).
 *   CAP_COMBINE_DEST_REDUCE, rank r: in = rank r's expert output rows (row order
 *       of CAP_PERMUTE_EXPERT_GATHER); for each row u < U_r of r's receive buffer,
 *       token t = recv_token[recv_offsets[r] + u]:
 *       out[recv_offsets[r] + u] = sum over kept slots s of t placed on r of
 *       w'_s * in[slot_pos(t,s) - expert_offsets[r*E_loc]].
 *       `out` is the concatenated receive-side buffer of all ranks.
 *   CAP_COMBINE_DEST_REDUCE_MULTI: DEST_REDUCE for the tokens with two or more
 *       kept slots whose rows on r are < in_rows; the others' out rows are left
 *       as they are (cap_expert_ffn_combine writes them).
 *   CAP_COMBINE_SRC_REDUCE, rank s: in = that concatenated buffer (the rows each
 *       device returns); for each token t of s:
 *       out[t - s*tokens_per_rank] = sum over kept devices d of t (ascending) of
 *       in[recv_offsets[d] + copy_row(t,d)]  (+ shared_out[t - s*tokens_per_rank]
 *       if shared_out != NULL).
 * fp32 accumulation; rows of d values of `dtype` (d % 8 == 0 for bf16, % 4 for f32).
 * in_rows / out_rows are the capacities of `in` / `out` in rows: rows at or past
 * them are neither read (their contribution is skipped) nor written.
 * SRC_REDUCE needs out_rows >= tokens_per_rank.
 */
cap_status cap_combine(const cap_topology *topo, cap_combine_mode mode, int32_t rank,
                       cap_dtype dtype, int32_t d, const void *in, int32_t in_rows,
                       const int32_t *idx, const float *w, const uint8_t *keep,
                       const uint64_t *dst_mask, const cap_layout *lay,
                       const void *shared_out, void *out, int32_t out_rows, void *stream);

/*
 * Expert co-activation counts on the (pruned) routing (Sec. IV-B; placement
 * runs on pruned traces, Sec. VII):
 *   coact[i][j] (i != j) = tokens that keep both i and j; coact[i][i] = tokens
 *   that keep i.  accumulate != 0 adds to coact (trace windows), else overwrites.
 * idx/keep are [T][k] as produced by cap_route_prune (out-of-range experts are
 * skipped).  Workspace: cap_workspace_size(CAP_OP_COACTIVATION, topo with this T and E, ...);
 * 16-byte aligned.
 */
cap_status cap_coactivation(int32_t T, int32_t k, int32_t E, const int32_t *idx,
                            const uint8_t *keep, uint32_t *coact, int32_t accumulate,
                            void *ws, size_t ws_bytes, void *stream);

/*
 * Adjustment Approach (Sec. V: trade communication for load balance by
 * swapping experts between the most and the least loaded devices, keeping as
 * much co-activation locality as possible; Eq. 2-3 objective C, Eq. 4 loads),
 * run on the GPU from a communication-oriented placement.
 *   coact[E][E]        (device) co-activation counts of a pruned routing trace
 *                      (cap_coactivation): N_e = coact[e][e] is expert e's load
 *                      in rows; p_ij = C_ij / (N_i + N_j - C_ij), 0 when the
 *                      denominator is 0.
 *   expert_rank[E], expert_local[E] (device, in/out) the starting placement
 *                      (a bijection onto [0,R) x [0,E/R)); on return the
 *                      placement after the last swap.
 *   Each step: hi = most loaded device, lo = least loaded (ties: lower id; the
 *   spectrum ends when their loads are equal); candidates e on hi and f on lo
 *   with N_e > N_f and L_lo + N_e - N_f < L_hi; the chosen one has the smallest
 *   increase of C (ties: lower e, then lower f), summed in fp64 over every
 *   other expert j, ascending, as p_ej (d(lo, pi_j) - d(hi, pi_j)) then
 *   p_fj (d(hi, pi_j) - d(lo, pi_j)), d = 0 / 1 / inter_node_cost (Eq. 3);
 *   e and f exchange devices and local slots.  Stops when no candidate
 *   remains or after max_swaps swaps.
 *   swaps[max_swaps][2] (device) the (e, f) of each swap, in order;
 *   deltas[max_swaps]  (device, nullable) each swap's increase of C;
 *   n_swaps            (device int32) swaps made.
 * Workspace: cap_workspace_size(CAP_OP_ADJUSTMENT, topo with this E, ...),
 * 8-byte aligned.  Needs 1 <= E <= 256, 1 <= R <= 64, E % R == 0,
 * R % ranks_per_node == 0, inter_node_cost >= 1, max_swaps >= 0.
 */
cap_status cap_adjustment_spectrum(const uint32_t *coact, int32_t E, int32_t R, int32_t ranks_per_node,
                                   float inter_node_cost, int32_t *expert_rank, int32_t *expert_local,
                                   int32_t max_swaps, int32_t *swaps, double *deltas, int32_t *n_swaps,
                                   void *ws, size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* CAP_H */
