/*
 * CPU oracle of the CAP expert-parallel MoE layer hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
 * the benchmark's CPU-baseline leg may load or call this code.  The GPU product
 * path never links, loads or falls back to it, and the two share no code.
 *
 * It is written to be checked by eye against the paper ("Communication-Aware
 * Placement and Pruning for Efficient Mixture-of-Experts Inference"): plain
 * loops, no blocking, no fusion, one step per function.
 *
 * Precision: routing decisions (top-k, gates, pruning) run in fp32 exactly as
 * specified below, because a floating-point value decides an integer there
 * (which device is kept) and both implementations must decide it in the same
 * precision.  Expert FFN and combine accumulate in fp64 and store fp32.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fopenmp -shared -fPIC
 *
 * Parity unpinned: none of the functions below is unpinned; each has pins in the
 * test suite (closed forms, brute force, invariants, worked examples).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------------------
 * Gate exponential (the paper is silent on how exp is evaluated; a fixed,
 * fully specified evaluation makes the fp32 gate weights reproducible bit for
 * bit across implementations).
 *
 * Method: Cody & Waite (1980) argument reduction plus a Taylor polynomial.
 *   exp(z) = 2^n * exp(r),  n = round_to_nearest_even(z * log2(e)),
 *   r = z - n*ln2 computed as two fused steps with ln2 = LN2_HI + LN2_LO,
 *   exp(r) ~ sum_{j=0..7} r^j / j!  evaluated by Horner's rule with fmaf.
 * LN2_HI is ln 2 rounded to 16 significant bits (0x3F317200): n*LN2_HI is exact
 * for |n| < 2^8.  LN2_LO is the fp32 value nearest to ln2 - LN2_HI.
 * For z < -87.33 the result is 0 (exp(-87.33) is just above FLT_MIN, so every
 * returned value is a normal number).  Callers pass z <= 0.
 * ------------------------------------------------------------------------- */
#define ORC_LOG2E   1.44269504088896340736f
#define ORC_LN2_HI  0.693145751953125f
#define ORC_LN2_LO  1.42860682030941723212e-6f
#define ORC_EXP_MIN (-87.33f)

float orc_exp(float z)
{
    if (!(z >= ORC_EXP_MIN))
        return 0.0f;
    float n = rintf(z * ORC_LOG2E);
    float r = fmaf(-n, ORC_LN2_HI, z);
    r = fmaf(-n, ORC_LN2_LO, r);
    /* Horner: c7 r^7 + ... + c1 r + c0 with c_j = fp32(1/j!) */
    float q = (float)(1.0 / 5040.0);
    q = fmaf(q, r, (float)(1.0 / 720.0));
    q = fmaf(q, r, (float)(1.0 / 120.0));
    q = fmaf(q, r, (float)(1.0 / 24.0));
    q = fmaf(q, r, (float)(1.0 / 6.0));
    q = fmaf(q, r, 0.5f);
    q = fmaf(q, r, 1.0f);
    q = fmaf(q, r, 1.0f);
    return ldexpf(q, (int)n);
}

/* ---------------------------------------------------------------------------
 * Step O1 -- top-k routing (Sec. II-A, Eq. 1: the gating network selects the
 * top-k experts of each token).
 * Slot j holds the j-th largest logit; equal logits are ordered by the lower
 * expert index (float equality, so -0.0 == +0.0).  Plain selection: for each
 * slot, scan all experts and keep the best one not yet chosen.
 * ------------------------------------------------------------------------- */
void orc_topk(int T, int E, int k, const float *logits, int32_t *idx)
{
    for (int t = 0; t < T; ++t) {
        const float *L = logits + (size_t)t * E;
        int32_t *out = idx + (size_t)t * k;
        for (int j = 0; j < k; ++j) {
            int best = -1;
            for (int e = 0; e < E; ++e) {
                int taken = 0;
                for (int i = 0; i < j; ++i)
                    if (out[i] == e) taken = 1;
                if (taken) continue;
                if (best < 0 || L[e] > L[best])   /* strict: ties keep the lower index */
                    best = e;
            }
            out[j] = best;
        }
    }
}

/* ---------------------------------------------------------------------------
 * Step O2 -- normalised gate weights (Sec. II-A, Eq. 1: Gate_i(x) is the
 * normalised routing weight of the i-th selected expert).  Softmax over the k
 * selected logits, which equals softmax over all experts followed by
 * renormalisation over the top k.
 *   m = L[idx_0];  q_s = exp(L[idx_s] - m);  S = ((q_0 + q_1) + q_2) + ...;
 *   w_s = q_s / S   (fp32, IEEE division).
 * ------------------------------------------------------------------------- */
void orc_gates(int T, int E, int k, const float *logits, const int32_t *idx, float *w)
{
    float q[64];
    for (int t = 0; t < T; ++t) {
        const float *L = logits + (size_t)t * E;
        const int32_t *id = idx + (size_t)t * k;
        float m = L[id[0]];
        float S = 0.0f;
        for (int s = 0; s < k; ++s) {
            q[s] = orc_exp(L[id[s]] - m);
            S = S + q[s];
        }
        for (int s = 0; s < k; ++s)
            w[(size_t)t * k + s] = q[s] / S;
    }
}

/* ---------------------------------------------------------------------------
 * Steps O3-O4 -- communication-aware device-level pruning (Sec. VI, Eq. 6 and
 * the greedy solver that follows it).
 *   a_d  = sum of the token's gate weights over its selected experts placed on
 *          device d (fp32, added in slot order);
 *   c_d  = 0 for the token's own device, 1 for another device of the same node,
 *          c (inter_node_cost) for a device on another node;
 *   keep devices in descending a_d / c_d (own device first: ratio +inf; ties by
 *   lower device id) until the kept sum reaches 1 - p (fp32 running sum,
 *   compared with >=).  p == 0 keeps every device.
 * Slots on dropped devices are pruned; kept weights are renormalised:
 *   w'_s = w_s / S' with S' the fp32 sum of kept w_s in slot order; w'_s = 0
 *   when pruned.  mask bit d is set for every kept device.
 * ------------------------------------------------------------------------- */
void orc_prune(int T, int k, int ranks_per_node, int tokens_per_rank, float c, float p,
               const int32_t *expert_rank, const int32_t *idx, const float *w,
               uint8_t *keep, float *wp, uint64_t *mask)
{
    for (int t = 0; t < T; ++t) {
        const int32_t *id = idx + (size_t)t * k;
        const float *ws = w + (size_t)t * k;
        int src = t / tokens_per_rank;
        int src_node = src / ranks_per_node;

        /* candidate devices in order of first appearance, with a_d */
        int nd = 0;
        int dev[64];
        float a[64];
        for (int s = 0; s < k; ++s) {
            int d = expert_rank[id[s]];
            int j = 0;
            while (j < nd && dev[j] != d) ++j;
            if (j == nd) { dev[nd] = d; a[nd] = 0.0f; ++nd; }
            a[j] = a[j] + ws[s];
        }

        /* ratio key of each candidate */
        float key[64];
        for (int j = 0; j < nd; ++j) {
            int d = dev[j];
            if (d == src)
                key[j] = INFINITY;
            else if (d / ranks_per_node == src_node)
                key[j] = a[j] / 1.0f;
            else
                key[j] = a[j] / c;
        }

        /* order: key descending, then device id ascending (selection sort) */
        int order[64], used[64] = {0};
        for (int i = 0; i < nd; ++i) {
            int b = -1;
            for (int j = 0; j < nd; ++j) {
                if (used[j]) continue;
                if (b < 0 || key[j] > key[b] || (key[j] == key[b] && dev[j] < dev[b]))
                    b = j;
            }
            used[b] = 1;
            order[i] = b;
        }

        /* greedy retention */
        int kept[64] = {0};
        if (p == 0.0f) {
            for (int j = 0; j < nd; ++j) kept[j] = 1;
        } else {
            float target = 1.0f - p;
            float cum = 0.0f;
            for (int i = 0; i < nd; ++i) {
                int j = order[i];
                kept[j] = 1;
                cum = cum + a[j];
                if (cum >= target) break;
            }
        }

        uint64_t m = 0;
        for (int j = 0; j < nd; ++j)
            if (kept[j]) m |= (uint64_t)1 << dev[j];
        mask[t] = m;

        float S = 0.0f;
        for (int s = 0; s < k; ++s) {
            int d = expert_rank[id[s]];
            uint8_t kp = (uint8_t)((m >> d) & 1u);
            keep[(size_t)t * k + s] = kp;
            if (kp) S = S + ws[s];
        }
        for (int s = 0; s < k; ++s)
            wp[(size_t)t * k + s] = keep[(size_t)t * k + s] ? ws[s] / S : 0.0f;
    }
}

/* Naive expert-level threshold pruning (Sec. II-D, Sec. VIII-D): keep the
 * smallest prefix of the slots (descending score) whose cumulative score
 * reaches 1 - p; renormalise like orc_prune.  mask = devices of kept slots. */
void orc_prune_naive(int T, int k, const int32_t *expert_rank, float p,
                     const int32_t *idx, const float *w, uint8_t *keep, float *wp, uint64_t *mask)
{
    for (int t = 0; t < T; ++t) {
        const int32_t *id = idx + (size_t)t * k;
        const float *ws = w + (size_t)t * k;
        int n = k;
        if (p != 0.0f) {
            float target = 1.0f - p, cum = 0.0f;
            for (int s = 0; s < k; ++s) {
                cum = cum + ws[s];
                if (cum >= target) { n = s + 1; break; }
            }
        }
        uint64_t m = 0;
        float S = 0.0f;
        for (int s = 0; s < k; ++s) {
            uint8_t kp = (uint8_t)(s < n);
            keep[(size_t)t * k + s] = kp;
            if (kp) { S = S + ws[s]; m |= (uint64_t)1 << expert_rank[id[s]]; }
        }
        mask[t] = m;
        for (int s = 0; s < k; ++s)
            wp[(size_t)t * k + s] = keep[(size_t)t * k + s] ? ws[s] / S : 0.0f;
    }
}

/* ---------------------------------------------------------------------------
 * Step O5 -- device-centric all-to-all layout and send volume (Sec. II-C:
 * each token is sent once to every device that hosts one of its kept experts;
 * experts on that device share the copy; Eq. 3 distinguishes same-device,
 * same-node and cross-node destinations).
 * Written by direct enumeration:
 *   slot position of expert e: P(e) = expert_rank[e]*E_loc + expert_local[e];
 *   expert_counts[P], expert_offsets[P] (exclusive scan in slot order, E+1);
 *   slot_pos[t][s]  row of kept (t,s) in the concatenation of every rank's
 *                   expert-sorted buffer (experts in slot order, tokens
 *                   ascending within an expert); -1 if pruned;
 *   send_counts[s][d] tokens of source s sent to d (d == s included);
 *   send_offsets[s][d] exclusive scan over d within s;
 *   recv_offsets[d] exclusive scan of U_d = sum_s send_counts[s][d], R+1;
 *   copy_row[t][s]  row of token t in the receive buffer of the device of
 *                   slot s (tokens ascending); -1 if pruned;
 *   recv_token[recv_offsets[d] + row] = t;
 *   vol[t] = {n_dev, n_intra_remote, n_inter, n_nodes}; totals = sums.
 * ------------------------------------------------------------------------- */
void orc_dispatch_layout(int T, int E, int k, int R, int ranks_per_node, int tokens_per_rank,
                         const int32_t *expert_rank, const int32_t *expert_local,
                         const int32_t *idx, const uint8_t *keep, const uint64_t *mask,
                         int32_t *send_counts, int32_t *send_offsets,
                         int32_t *recv_offsets, int32_t *recv_token,
                         int32_t *expert_counts, int32_t *expert_offsets,
                         int32_t *slot_pos, int32_t *copy_row,
                         uint8_t *vol, int64_t *totals)
{
    int E_loc = E / R;
    for (size_t i = 0; i < (size_t)T * k; ++i) { slot_pos[i] = -1; copy_row[i] = -1; }

    /* expert-sorted rows */
    int32_t row = 0;
    for (int r = 0; r < R; ++r) {
        for (int l = 0; l < E_loc; ++l) {
            int P = r * E_loc + l;
            int e = -1;
            for (int x = 0; x < E; ++x)
                if (expert_rank[x] == r && expert_local[x] == l) e = x;
            expert_offsets[P] = row;
            int32_t cnt = 0;
            for (int t = 0; t < T; ++t)
                for (int s = 0; s < k; ++s) {
                    size_t q = (size_t)t * k + s;
                    if (keep[q] && idx[q] == e) { slot_pos[q] = row++; ++cnt; }
                }
            expert_counts[P] = cnt;
        }
    }
    expert_offsets[E] = row;

    /* send counts and offsets */
    for (int i = 0; i < R * R; ++i) send_counts[i] = 0;
    for (int t = 0; t < T; ++t) {
        int s = t / tokens_per_rank;
        for (int d = 0; d < R; ++d)
            if ((mask[t] >> d) & 1u) send_counts[s * R + d] += 1;
    }
    for (int s = 0; s < R; ++s) {
        int32_t acc = 0;
        for (int d = 0; d < R; ++d) { send_offsets[s * R + d] = acc; acc += send_counts[s * R + d]; }
    }

    /* receive buffers */
    int32_t acc = 0;
    for (int d = 0; d < R; ++d) {
        recv_offsets[d] = acc;
        for (int s = 0; s < R; ++s) acc += send_counts[s * R + d];
    }
    recv_offsets[R] = acc;
    for (int d = 0; d < R; ++d) {
        int32_t n = 0;
        for (int t = 0; t < T; ++t) {
            if (!((mask[t] >> d) & 1u)) continue;
            for (int s = 0; s < k; ++s) {
                size_t q = (size_t)t * k + s;
                if (keep[q] && expert_rank[idx[q]] == d) copy_row[q] = n;
            }
            recv_token[recv_offsets[d] + n] = t;
            ++n;
        }
    }

    /* per-token volume */
    for (int i = 0; i < 4; ++i) totals[i] = 0;
    for (int t = 0; t < T; ++t) {
        int src = t / tokens_per_rank;
        int src_node = src / ranks_per_node;
        int n_dev = 0, n_intra = 0, n_inter = 0, n_nodes = 0;
        int node_seen[64] = {0};
        for (int d = 0; d < R; ++d) {
            if (!((mask[t] >> d) & 1u)) continue;
            ++n_dev;
            int nd = d / ranks_per_node;
            if (nd != src_node) ++n_inter;
            else if (d != src) ++n_intra;
            if (!node_seen[nd]) { node_seen[nd] = 1; ++n_nodes; }
        }
        uint8_t *v = vol + (size_t)t * 4;
        v[0] = (uint8_t)n_dev; v[1] = (uint8_t)n_intra; v[2] = (uint8_t)n_inter; v[3] = (uint8_t)n_nodes;
        totals[0] += n_dev; totals[1] += n_intra; totals[2] += n_inter; totals[3] += n_nodes;
    }
}

/* ---------------------------------------------------------------------------
 * Token permutation (Sec. II-C, Fig. "Expert parallelism combined with data
 * parallelism"): the dispatch all-to-all and the expansion into per-expert rows.
 * expert_gather: for destination rank r, row (slot_pos - base_r) of its
 *   expert-sorted buffer is a copy of x[t], base_r = expert_offsets[r*E_loc].
 * send_pack: for source rank s, row send_offsets[s][d] + j of its send buffer
 *   is the j-th token of s (ascending) whose mask holds d.
 * Rows are copied byte for byte (row_bytes each).
 * ------------------------------------------------------------------------- */
void orc_expert_gather(int T, int k, int E, int R, int rank, size_t row_bytes,
                       const int32_t *expert_rank, const int32_t *idx, const uint8_t *keep,
                       const int32_t *slot_pos, const int32_t *expert_offsets,
                       const void *x, void *out)
{
    int E_loc = E / R;
    int32_t base = expert_offsets[rank * E_loc];
    for (int t = 0; t < T; ++t)
        for (int s = 0; s < k; ++s) {
            size_t q = (size_t)t * k + s;
            if (keep[q] && expert_rank[idx[q]] == rank)
                memcpy((char *)out + (size_t)(slot_pos[q] - base) * row_bytes,
                       (const char *)x + (size_t)t * row_bytes, row_bytes);
        }
}

void orc_send_pack(int R, int tokens_per_rank, int src, size_t row_bytes,
                   const uint64_t *mask, const int32_t *send_offsets, const void *x, void *out)
{
    for (int d = 0; d < R; ++d) {
        int32_t j = 0;
        for (int t = src * tokens_per_rank; t < (src + 1) * tokens_per_rank; ++t) {
            if (!((mask[t] >> d) & 1u)) continue;
            memcpy((char *)out + (size_t)(send_offsets[src * R + d] + j) * row_bytes,
                   (const char *)x + (size_t)t * row_bytes, row_bytes);
            ++j;
        }
    }
}

/* ---------------------------------------------------------------------------
 * Expert FFN (Eq. 1, Expert_i(x); the paper does not fix expert internals, the
 * workloads use SwiGLU experts):
 *   h_j = silu(W1[j] . x) * (W3[j] . x),  silu(z) = z / (1 + exp(-z)),
 *   y_o = W2[o] . h
 * fp64 accumulation throughout; h is not rounded.  Rows are independent and
 * each is computed in a fixed order, so the result does not depend on the
 * OpenMP thread count.
 * ------------------------------------------------------------------------- */
void orc_swiglu_rows(int n, int d, int inter, const float *X, const float *W1, const float *W3,
                     const float *W2, double *Y, int nthreads)
{
    if (nthreads < 1) nthreads = 1;
    #pragma omp parallel for num_threads(nthreads) schedule(dynamic, 1)
    for (int i = 0; i < n; ++i) {
        const float *x = X + (size_t)i * d;
        double *h = (double *)malloc(sizeof(double) * (size_t)inter);
        for (int j = 0; j < inter; ++j) {
            double g = 0.0, u = 0.0;
            const float *w1 = W1 + (size_t)j * d, *w3 = W3 + (size_t)j * d;
            for (int c = 0; c < d; ++c) {
                g += (double)w1[c] * (double)x[c];
                u += (double)w3[c] * (double)x[c];
            }
            h[j] = g / (1.0 + exp(-g)) * u;
        }
        for (int o = 0; o < d; ++o) {
            const float *w2 = W2 + (size_t)o * inter;
            double y = 0.0;
            for (int j = 0; j < inter; ++j) y += (double)w2[j] * h[j];
            Y[(size_t)i * d + o] = y;
        }
        free(h);
    }
}

/* ---------------------------------------------------------------------------
 * Weighted combine (Sec. II-C: outputs of experts on one device are
 * aggregated locally by a weighted sum; the aggregated row is returned and the
 * final combination happens at the token's source; Eq. 1).
 * dest_reduce on rank r: part[u] = sum over kept slots s of token
 *   t = recv_token[recv_offsets[r] + u] placed on r of w'_s * Y[slot_pos - base_r].
 * src_reduce on rank s: y[t - s*T_loc] = sum over devices d in mask(t), d
 *   ascending, of parts[recv_offsets[d] + copy_row(t,d)], plus shared[t] if given.
 * fp64 accumulation, fp32 store.
 * ------------------------------------------------------------------------- */
void orc_dest_reduce(int k, int E, int R, int rank, int d,
                     const int32_t *expert_rank, const int32_t *idx, const float *wp,
                     const uint8_t *keep, const int32_t *slot_pos, const int32_t *expert_offsets,
                     const int32_t *recv_offsets, const int32_t *recv_token,
                     const float *Y, float *part)
{
    int E_loc = E / R;
    int32_t base = expert_offsets[rank * E_loc];
    int32_t U = recv_offsets[rank + 1] - recv_offsets[rank];
    double *acc = (double *)malloc(sizeof(double) * (size_t)d);
    for (int32_t u = 0; u < U; ++u) {
        int t = recv_token[recv_offsets[rank] + u];
        for (int c = 0; c < d; ++c) acc[c] = 0.0;
        for (int s = 0; s < k; ++s) {
            size_t q = (size_t)t * k + s;
            if (!keep[q] || expert_rank[idx[q]] != rank) continue;
            const float *yr = Y + (size_t)(slot_pos[q] - base) * d;
            for (int c = 0; c < d; ++c) acc[c] += (double)wp[q] * (double)yr[c];
        }
        for (int c = 0; c < d; ++c) part[(size_t)u * d + c] = (float)acc[c];
    }
    free(acc);
}

void orc_src_reduce(int k, int R, int tokens_per_rank, int src, int d,
                    const int32_t *expert_rank, const int32_t *idx, const uint8_t *keep,
                    const uint64_t *mask, const int32_t *copy_row, const int32_t *recv_offsets,
                    const float *parts, const float *shared, float *y)
{
    double *acc = (double *)malloc(sizeof(double) * (size_t)d);
    for (int i = 0; i < tokens_per_rank; ++i) {
        int t = src * tokens_per_rank + i;
        for (int c = 0; c < d; ++c) acc[c] = shared ? (double)shared[(size_t)i * d + c] : 0.0;
        for (int dv = 0; dv < R; ++dv) {
            if (!((mask[t] >> dv) & 1u)) continue;
            int32_t cr = -1;
            for (int s = 0; s < k; ++s) {
                size_t q = (size_t)t * k + s;
                if (keep[q] && expert_rank[idx[q]] == dv) cr = copy_row[q];
            }
            const float *pr = parts + (size_t)(recv_offsets[dv] + cr) * d;
            for (int c = 0; c < d; ++c) acc[c] += (double)pr[c];
        }
        for (int c = 0; c < d; ++c) y[(size_t)i * d + c] = (float)acc[c];
    }
    free(acc);
}

/* ---------------------------------------------------------------------------
 * Step O6 -- expert co-activation counts on the pruned routing (Sec. IV-B:
 * how often two experts are selected together; Sec. VII: placement runs on
 * pruned traces).  C[i][j] (i != j) = tokens keeping both i and j;
 * C[i][i] = tokens keeping i.  accumulate != 0 adds to C instead of
 * overwriting it.
 * ------------------------------------------------------------------------- */
void orc_coactivation(int T, int k, int E, const int32_t *idx, const uint8_t *keep,
                      uint32_t *C, int accumulate)
{
    if (!accumulate)
        for (size_t i = 0; i < (size_t)E * E; ++i) C[i] = 0;
    for (int t = 0; t < T; ++t)
        for (int s = 0; s < k; ++s) {
            size_t q = (size_t)t * k + s;
            if (!keep[q]) continue;
            int i = idx[q];
            for (int s2 = 0; s2 < k; ++s2) {
                size_t q2 = (size_t)t * k + s2;
                if (keep[q2]) C[(size_t)i * E + idx[q2]] += 1;   /* s2 == s gives C[i][i] */
            }
        }
}

/* Element-wise orc_exp over an array (test convenience). */
void orc_exp_array(int64_t n, const float *z, float *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = orc_exp(z[i]);
}
