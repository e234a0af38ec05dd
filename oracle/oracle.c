/*
 * CPU oracle for the message-passing aggregation path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this code; the device library never
 * links, calls or includes it, and it includes nothing from the device
 * library.
 *
 * Everything here is the plain definition, written for a reader to check by
 * eye against the paper (PyG 2.0, arXiv 2507.16991):
 *
 *  - Eq. (1): h_v' = f(h_v, AGG{ g(h_w, e_wv, h_v) : w in N(v) }).  This path
 *    is the AGGREGATION step with message g = e_wv * h_w (a scalar edge
 *    weight, or no weight) and f left to the caller.  The aggregator is one of
 *    the permutation-invariant set functions named next to Eq. (1): sum, mean,
 *    max (the max also reports which edge attains it).
 *  - Sec. 2.2 "Accelerated Message Passing": the COO edge_index is converted
 *    to a compressed sparse format sorted by node, so that aggregation becomes
 *    a segmented reduction.  Rows here are destinations v (Eq. (1) aggregates
 *    at v over incoming edges (w, v)); within a row, edges keep their original
 *    COO order (a stable sort).
 *  - Sec. 2.2 "Heterogeneous Message Passing": the nested version of Eq. (1)
 *    adds a sum over the incoming edge types of each destination node type.
 *
 * Precision: all sums in fp64.  A weighted message is the fp32 product
 * fl32(w * x) (the product of two fp32 values is exact in fp64, so rounding it
 * once to fp32 gives the correctly rounded fp32 message).  An unweighted
 * message is x itself (bf16 features widen exactly to fp32).
 *
 * Readings where the paper is silent: empty rows aggregate to 0 (and argmax
 * -1); max keeps the first edge (lowest CSR position) among equal values,
 * comparing with '>' so that -0.0 and +0.0 tie; mean is sum / in-degree.
 *
 * More aggregators (Sec. 2.2 "Aggregations as a First-Class Principle":
 * besides sum, mean and max, advanced ones such as variance and standard
 * deviation, stacked together, in message passing and in global readouts):
 * min (with the first edge attaining it), the population variance of a row's
 * messages, sum of (m - mean)^2 / deg, and its square root.  A global readout
 * is the same aggregation over contiguous segments of nodes (col = identity).
 *
 * Segment matmul (Sec. 2.2, heterogeneous GNNs: the projections
 * {H_T W_T} over node types, with a three-dimensional weight W of shape
 * [|T|, F, F'], and their gradients with respect to H_T and W): rows of X are
 * grouped by type in contiguous segments; each segment is multiplied by its
 * own weight matrix.
 *
 * Backward (Sec. 2.2: the backward pass of an aggregation runs over the
 * transposed adjacency, which is why CSR and CSC are both cached): the
 * derivatives of the aggregation above with respect to the features x and the
 * edge weights w, given the gradient g of its output.  The fp32 rounding of a
 * weighted message is not differentiated (the message is taken as w * x).
 * The max routes each output element's gradient to the one edge the forward
 * pass reported for it (argmax), and nowhere for an empty row.
 *
 * Explanation mode (Sec. 2.4, with the PyG 1 materialization recalled in
 * Sec. 2.2): messages materialized as an E x F table, edited by a callback c,
 * then aggregated; and the gradients of that pipeline (with respect to each
 * message, to x, and to a per-edge factor such as an edge mask).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---- COO -> CSR (stable counting sort by destination) ------------------ */

/* rowptr[N+1] (int64), col[E] = src of the p-th edge in destination order,
 * perm[E] = its COO edge id, val_out[E] = val_in[perm] (if both given).
 * Returns 0, or -1 when an index is out of range. */
int oracle_coo_to_csr(int64_t E, int64_t N_dst, int64_t N_src, const int32_t* src,
                      const int32_t* dst, const float* val_in, int64_t* rowptr,
                      int32_t* col, int64_t* perm, float* val_out) {
    for (int64_t e = 0; e < E; ++e)
        if (dst[e] < 0 || dst[e] >= N_dst || src[e] < 0 || src[e] >= N_src) return -1;

    /* in-degree of every destination */
    for (int64_t v = 0; v <= N_dst; ++v) rowptr[v] = 0;
    for (int64_t e = 0; e < E; ++e) rowptr[dst[e] + 1] += 1;
    /* rowptr[v+1] = rowptr[v] + deg(v) */
    for (int64_t v = 0; v < N_dst; ++v) rowptr[v + 1] += rowptr[v];

    /* place edges in COO order: each destination's edges stay in order */
    int64_t* cursor = (int64_t*)malloc(sizeof(int64_t) * (size_t)(N_dst > 0 ? N_dst : 1));
    if (!cursor) return -2;
    for (int64_t v = 0; v < N_dst; ++v) cursor[v] = rowptr[v];
    for (int64_t e = 0; e < E; ++e) {
        int64_t p = cursor[dst[e]]++;
        if (col) col[p] = src[e];
        if (perm) perm[p] = e;
        if (val_in && val_out) val_out[p] = val_in[e];
    }
    free(cursor);
    return 0;
}

/* ---- messages --------------------------------------------------------- */

static inline float widen_bf16(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* feature x[row, f] widened to fp32 */
static inline float feature(const void* x, int x_is_bf16, int64_t F, int64_t row,
                            int64_t f) {
    if (x_is_bf16) return widen_bf16(((const uint16_t*)x)[row * F + f]);
    return ((const float*)x)[row * F + f];
}

/* message of edge p for feature f: x (unweighted) or fl32(w * x) */
static inline float message(const void* x, int x_is_bf16, int64_t F, int64_t row,
                            int64_t f, const float* w, int64_t p) {
    float xv = feature(x, x_is_bf16, F, row, f);
    if (!w) return xv;
    return (float)((double)w[p] * (double)xv);
}

/* ---- aggregation over CSR ---------------------------------------------- */

/* For each listed row i (rows == NULL: rows 0..n_rows-1) and each feature f,
 * over the CSR edges p in [rowptr[i], rowptr[i+1]):
 *   out_sum[k,f]  = sum_p m_p                      (fp64)
 *   out_mean[k,f] = out_sum[k,f] / deg_i            (0 if deg_i = 0)
 *   out_max[k,f]  = m_arg, argout[k,f] = arg, where arg is the first p with
 *                   the largest m_p ('>' scan; -1 and 0.0 for an empty row)
 *   scale[k,f]    = sum_p |m_p|                     (error scale of the sum)
 * k indexes the output rows in list order.  Any output may be NULL.
 * Rows are independent; nthreads > 0 splits them over OpenMP threads.
 * Returns 0, or -1 for an out-of-range column or row. */
int oracle_spmm(int64_t n_rows, const int64_t* rows, int64_t N_dst, int64_t N_src,
                const int64_t* rowptr, const int32_t* col, const float* w, const void* x,
                int x_is_bf16, int64_t F, double* out_sum, double* out_mean,
                float* out_max, int64_t* argout, double* scale, int nthreads) {
    int bad = 0;
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : 1) reduction(| : bad)
    for (int64_t k = 0; k < n_rows; ++k) {
        int64_t i = rows ? rows[k] : k;
        if (i < 0 || i >= N_dst) {
            bad = 1;
            continue;
        }
        int64_t p0 = rowptr[i], p1 = rowptr[i + 1];
        for (int64_t p = p0; p < p1; ++p)
            if (col[p] < 0 || col[p] >= N_src) bad = 1;
        if (bad) continue;
        int64_t deg = p1 - p0;
        for (int64_t f = 0; f < F; ++f) {
            double s = 0.0, a = 0.0;
            float best = 0.0f;
            int64_t arg = -1;
            for (int64_t p = p0; p < p1; ++p) {
                float m = message(x, x_is_bf16, F, col[p], f, w, p);
                s += (double)m;
                a += fabs((double)m);
                if (arg < 0 || m > best) {
                    best = m;
                    arg = p;
                }
            }
            if (out_sum) out_sum[k * F + f] = s;
            if (out_mean) out_mean[k * F + f] = deg > 0 ? s / (double)deg : 0.0;
            if (out_max) out_max[k * F + f] = arg < 0 ? 0.0f : best;
            if (argout) argout[k * F + f] = arg;
            if (scale) scale[k * F + f] = a;
        }
    }
    return bad ? -1 : 0;
}

/* ---- listed-row lookup ------------------------------------------------- */

/* Membership of row ids in a list, as a bit array over [0, N) plus the list
 * sorted by id (with each id's position in the original list), so that a
 * pass over E edges costs one bit test per edge and a binary search only for
 * edges of listed rows. */
typedef struct {
    uint64_t* bits;
    int64_t* sorted;  /* listed ids, ascending */
    int64_t* where;   /* where[j] = position in the caller's list of sorted[j] */
    int64_t n;
} row_set;

static int cmp_pair(const void* a, const void* b) {
    const int64_t* x = (const int64_t*)a;
    const int64_t* y = (const int64_t*)b;
    return x[0] < y[0] ? -1 : (x[0] > y[0] ? 1 : 0);
}

static void row_set_free(row_set* s) {
    free(s->bits);
    free(s->sorted);
    free(s->where);
}

/* 0, -1 (id out of range) or -2 (allocation) */
static int row_set_make(row_set* s, int64_t N, int64_t n, const int64_t* rows) {
    s->n = n;
    s->bits = (uint64_t*)calloc((size_t)((N + 63) / 64 + 1), sizeof(uint64_t));
    s->sorted = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    s->where = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t* pairs = (int64_t*)malloc(sizeof(int64_t) * 2 * (size_t)(n > 0 ? n : 1));
    if (!s->bits || !s->sorted || !s->where || !pairs) {
        free(pairs);
        row_set_free(s);
        return -2;
    }
    for (int64_t k = 0; k < n; ++k) {
        if (rows[k] < 0 || rows[k] >= N) {
            free(pairs);
            row_set_free(s);
            return -1;
        }
        pairs[2 * k] = rows[k];
        pairs[2 * k + 1] = k;
        s->bits[rows[k] >> 6] |= 1ull << (rows[k] & 63);
    }
    qsort(pairs, (size_t)n, 2 * sizeof(int64_t), cmp_pair);
    for (int64_t k = 0; k < n; ++k) {
        s->sorted[k] = pairs[2 * k];
        s->where[k] = pairs[2 * k + 1];
    }
    free(pairs);
    return 0;
}

/* position in the caller's list of row v, or -1 if v is not listed */
static inline int64_t row_set_find(const row_set* s, int64_t v) {
    if (!((s->bits[v >> 6] >> (v & 63)) & 1ull)) return -1;
    int64_t lo = 0, hi = s->n - 1;
    while (lo < hi) {
        int64_t mid = (lo + hi) >> 1;
        if (s->sorted[mid] < v) lo = mid + 1; else hi = mid;
    }
    return s->where[lo];
}

/* ---- aggregation of listed rows straight from COO ----------------------- */

/* Same outputs as oracle_spmm for the listed (distinct) rows, computed from
 * the COO arrays without building the CSR: one pass over the edges in COO
 * order, so each row sees its edges in the order of the stable CSR, and the
 * CSR position of edge e is rowptr[dst_e] + (number of earlier edges with the
 * same destination).  rowptr of the listed rows is taken from row_start when
 * given (row_start[k] = number of edges whose destination is below rows[k]),
 * else counted here.  `w` is in COO order.  Meant for graphs too large to
 * convert on the host; one thread.  Returns 0, -1 on a bad index, -2 on
 * allocation failure. */
int oracle_spmm_coo_rows(int64_t E, int64_t N_dst, int64_t N_src, const int32_t* src,
                         const int32_t* dst, const float* w_coo, const void* x,
                         int x_is_bf16, int64_t F, int64_t n_rows, const int64_t* rows,
                         const int64_t* row_start, double* out_sum, double* out_mean,
                         float* out_max, int64_t* argout, double* scale) {
    row_set set;
    int rc = row_set_make(&set, N_dst, n_rows, rows);
    if (rc != 0) return rc;
    int64_t* start = (int64_t*)calloc((size_t)(n_rows > 0 ? n_rows : 1), sizeof(int64_t));
    int64_t* seen = (int64_t*)calloc((size_t)(n_rows > 0 ? n_rows : 1), sizeof(int64_t));
    double* acc = (double*)calloc((size_t)((n_rows > 0 ? n_rows : 1) * (F > 0 ? F : 1)),
                                  sizeof(double));
    if (!start || !seen || !acc) {
        free(start); free(seen); free(acc); row_set_free(&set);
        return -2;
    }
    for (int64_t e = 0; e < E; ++e)
        if (dst[e] < 0 || dst[e] >= N_dst || src[e] < 0 || src[e] >= N_src) {
            free(start); free(seen); free(acc); row_set_free(&set);
            return -1;
        }
    if (row_start) {
        for (int64_t k = 0; k < n_rows; ++k) start[k] = row_start[k];
    } else {
        /* start[k] = number of edges whose destination is below rows[k] */
        for (int64_t e = 0; e < E; ++e) {
            int64_t v = dst[e];
            /* count listed rows above v: binary search in the sorted ids */
            int64_t lo = 0, hi = set.n;
            while (lo < hi) {
                int64_t mid = (lo + hi) >> 1;
                if (set.sorted[mid] <= v) lo = mid + 1; else hi = mid;
            }
            if (lo < set.n) start[lo] += 1; /* counted for sorted[lo] and all above */
        }
        /* prefix over the sorted list, then map back to list positions */
        int64_t run = 0;
        int64_t* tmp = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n_rows > 0 ? n_rows : 1));
        if (!tmp) {
            free(start); free(seen); free(acc); row_set_free(&set);
            return -2;
        }
        for (int64_t j = 0; j < set.n; ++j) {
            run += start[j];
            tmp[set.where[j]] = run;
        }
        for (int64_t k = 0; k < n_rows; ++k) start[k] = tmp[k];
        free(tmp);
    }

    for (int64_t k = 0; k < n_rows; ++k)
        for (int64_t f = 0; f < F; ++f) {
            if (out_max) out_max[k * F + f] = 0.0f;
            if (argout) argout[k * F + f] = -1;
            if (scale) scale[k * F + f] = 0.0;
        }
    for (int64_t e = 0; e < E; ++e) {
        int64_t k = row_set_find(&set, dst[e]);
        if (k < 0) continue;
        int64_t p = start[k] + seen[k];
        seen[k] += 1;
        for (int64_t f = 0; f < F; ++f) {
            float xv = feature(x, x_is_bf16, F, src[e], f);
            float m = w_coo ? (float)((double)w_coo[e] * (double)xv) : xv;
            acc[k * F + f] += (double)m;
            if (scale) scale[k * F + f] += fabs((double)m);
            if (out_max && argout && (argout[k * F + f] < 0 || m > out_max[k * F + f])) {
                out_max[k * F + f] = m;
                argout[k * F + f] = p;
            }
        }
    }
    for (int64_t k = 0; k < n_rows; ++k)
        for (int64_t f = 0; f < F; ++f) {
            if (out_sum) out_sum[k * F + f] = acc[k * F + f];
            if (out_mean) out_mean[k * F + f] = seen[k] > 0 ? acc[k * F + f] / (double)seen[k] : 0.0;
        }
    free(start); free(seen); free(acc); row_set_free(&set);
    return 0;
}

/* ---- heterogeneous sum -------------------------------------------------- */

/* Nested Eq. (1) with sum at both levels: for every destination type T,
 *   out_T[i, f] = sum over relations r with rel_dst_type[r] == T (ascending r)
 *                 of sum over r's edges e with rel_dst[r][e] == i (COO order)
 *                 of x_{rel_src_type[r]}[rel_src[r][e], f].
 * out_per_type[T] and scale_per_type[T] are [N_T, F] fp64 buffers (scale may
 * be NULL).  Returns 0, or -1 on a bad type or index. */
int oracle_hetero_sum(int n_types, const int64_t* n_per_type, const void* const* x_per_type,
                      int x_is_bf16, int64_t F, int n_rel, const int32_t* rel_src_type,
                      const int32_t* rel_dst_type, const int64_t* rel_E,
                      const int32_t* const* rel_src, const int32_t* const* rel_dst,
                      double* const* out_per_type, double* const* scale_per_type) {
    for (int t = 0; t < n_types; ++t)
        for (int64_t k = 0; k < n_per_type[t] * F; ++k) {
            out_per_type[t][k] = 0.0;
            if (scale_per_type) scale_per_type[t][k] = 0.0;
        }
    for (int r = 0; r < n_rel; ++r) {
        int st = rel_src_type[r], dt = rel_dst_type[r];
        if (st < 0 || st >= n_types || dt < 0 || dt >= n_types) return -1;
        for (int64_t e = 0; e < rel_E[r]; ++e) {
            int64_t s = rel_src[r][e], d = rel_dst[r][e];
            if (s < 0 || s >= n_per_type[st] || d < 0 || d >= n_per_type[dt]) return -1;
            for (int64_t f = 0; f < F; ++f) {
                double m = (double)feature(x_per_type[st], x_is_bf16, F, s, f);
                out_per_type[dt][d * F + f] += m;
                if (scale_per_type) scale_per_type[dt][d * F + f] += fabs(m);
            }
        }
    }
    return 0;
}

/* ---- CSR column segments of listed rows straight from COO --------------- */

/* For the listed distinct rows, the sources of their edges in COO order (which
 * is their order in the stable destination-major CSR), concatenated in list
 * order: row k's segment is cols[seg[k] .. seg[k+1]).  Pass 1 (cols == NULL)
 * fills seg[0..n_rows] only.  Returns 0, -1 on a bad index, -2 on allocation
 * failure. */
int oracle_csr_rows(int64_t E, int64_t N_dst, const int32_t* src, const int32_t* dst,
                    int64_t n_rows, const int64_t* rows, int64_t* seg, int32_t* cols) {
    row_set set;
    int rc = row_set_make(&set, N_dst, n_rows, rows);
    if (rc != 0) return rc;
    int64_t* fill = (int64_t*)calloc((size_t)(n_rows > 0 ? n_rows : 1), sizeof(int64_t));
    if (!fill) {
        row_set_free(&set);
        return -2;
    }
    if (!cols) {
        for (int64_t k = 0; k <= n_rows; ++k) seg[k] = 0;
        for (int64_t e = 0; e < E; ++e) {
            if (dst[e] < 0 || dst[e] >= N_dst) {
                free(fill); row_set_free(&set);
                return -1;
            }
            int64_t k = row_set_find(&set, dst[e]);
            if (k >= 0) seg[k + 1] += 1;
        }
        for (int64_t k = 0; k < n_rows; ++k) seg[k + 1] += seg[k];
    } else {
        for (int64_t e = 0; e < E; ++e) {
            int64_t k = row_set_find(&set, dst[e]);
            if (k >= 0) cols[seg[k] + fill[k]++] = src[e];
        }
    }
    free(fill);
    row_set_free(&set);
    return 0;
}

/* ---- transposed CSR (source-major) ------------------------------------- */

/* The same edges grouped by source: rowptrT[N_src+1]; for the t-th edge in
 * source order, colT[t] = its destination (the forward CSR row of the edge)
 * and posT[t] = its forward CSR position.  Within a source, edges keep their
 * forward CSR order (stable counting sort by col over the positions).
 * Returns 0, -1 on an out-of-range column, -2 on allocation failure. */
int oracle_csr_transpose(int64_t N_dst, int64_t N_src, const int64_t* rowptr,
                         const int32_t* col, int64_t* rowptrT, int32_t* colT, int64_t* posT) {
    int64_t E = rowptr[N_dst];
    for (int64_t p = 0; p < E; ++p)
        if (col[p] < 0 || col[p] >= N_src) return -1;
    for (int64_t u = 0; u <= N_src; ++u) rowptrT[u] = 0;
    for (int64_t p = 0; p < E; ++p) rowptrT[col[p] + 1] += 1;
    for (int64_t u = 0; u < N_src; ++u) rowptrT[u + 1] += rowptrT[u];
    int64_t* cursor = (int64_t*)malloc(sizeof(int64_t) * (size_t)(N_src > 0 ? N_src : 1));
    if (!cursor) return -2;
    for (int64_t u = 0; u < N_src; ++u) cursor[u] = rowptrT[u];
    for (int64_t v = 0; v < N_dst; ++v)
        for (int64_t p = rowptr[v]; p < rowptr[v + 1]; ++p) {
            int64_t t = cursor[col[p]]++;
            colT[t] = (int32_t)v;
            posT[t] = p;
        }
    free(cursor);
    return 0;
}

/* ---- gradients of the aggregation ---------------------------------------- */

/* reduce codes of the backward functions */
enum { ORACLE_SUM = 1, ORACLE_MEAN = 2, ORACLE_MAX = 4 };

/* Coefficient with which g[v, f] reaches edge p (in row v) for feature f:
 * sum 1, mean 1/deg(v), max 1 if argout[v, f] == p else 0. */
static inline double route(int reduce, int64_t deg, const int64_t* argout, int64_t F,
                           int64_t v, int64_t f, int64_t p) {
    if (reduce == ORACLE_SUM) return 1.0;
    if (reduce == ORACLE_MEAN) return 1.0 / (double)deg;
    return argout[v * F + f] == p ? 1.0 : 0.0;
}

/* Gradient with respect to x, for the listed source rows (rows == NULL: all
 * N_src rows, in order):
 *   gx[k, f] = sum over forward CSR edges p with col[p] == u_k, in CSR order,
 *              of route(v, f, p) * w_p * g[v, f]      (v = row of p; w_p = 1
 *              when w is NULL)
 *   scale[k, f] = the same sum of absolute values (error scale).
 * g is [N_dst, F] fp32 or bf16 bits.  argout [N_dst, F] is needed for max.
 * Returns 0, -1 on a bad index or reduce, -2 on allocation failure. */
int oracle_spmm_backward_x(int64_t n_rows, const int64_t* rows, int64_t N_dst, int64_t N_src,
                           const int64_t* rowptr, const int32_t* col, const float* w,
                           const void* g, int g_is_bf16, int64_t F, int reduce,
                           const int64_t* argout, double* gx, double* scale) {
    if (reduce != ORACLE_SUM && reduce != ORACLE_MEAN && reduce != ORACLE_MAX) return -1;
    if (reduce == ORACLE_MAX && !argout) return -1;
    int64_t n = rows ? n_rows : N_src;
    row_set set;
    if (rows) {
        int rc = row_set_make(&set, N_src, n_rows, rows);
        if (rc != 0) return rc;
    }
    for (int64_t k = 0; k < n * F; ++k) {
        gx[k] = 0.0;
        if (scale) scale[k] = 0.0;
    }
    int bad = 0;
    for (int64_t v = 0; v < N_dst && !bad; ++v) {
        int64_t deg = rowptr[v + 1] - rowptr[v];
        for (int64_t p = rowptr[v]; p < rowptr[v + 1]; ++p) {
            int64_t u = col[p];
            if (u < 0 || u >= N_src) { bad = 1; break; }
            int64_t k = rows ? row_set_find(&set, u) : u;
            if (k < 0) continue;
            double wp = w ? (double)w[p] : 1.0;
            for (int64_t f = 0; f < F; ++f) {
                double t = route(reduce, deg, argout, F, v, f, p) * wp *
                           (double)feature(g, g_is_bf16, F, v, f);
                gx[k * F + f] += t;
                if (scale) scale[k * F + f] += fabs(t);
            }
        }
    }
    if (rows) row_set_free(&set);
    return bad ? -1 : 0;
}

/* Gradient with respect to the edge weights, for every CSR edge p of the
 * listed destination rows (rows == NULL: all rows):
 *   gw[p] = sum over f of route(v, f, p) * g[v, f] * x[col[p], f]
 *   scale[p] = the same sum of absolute values.
 * Entries of unlisted rows are left untouched.  x is [N_src, F], g is
 * [N_dst, F], each fp32 or bf16 bits.  Rows are independent; nthreads > 0
 * splits them over OpenMP threads.  Returns 0, or -1 on a bad index/reduce. */
int oracle_spmm_backward_w(int64_t n_rows, const int64_t* rows, int64_t N_dst, int64_t N_src,
                           const int64_t* rowptr, const int32_t* col, const void* x,
                           int x_is_bf16, const void* g, int g_is_bf16, int64_t F, int reduce,
                           const int64_t* argout, double* gw, double* scale, int nthreads) {
    if (reduce != ORACLE_SUM && reduce != ORACLE_MEAN && reduce != ORACLE_MAX) return -1;
    if (reduce == ORACLE_MAX && !argout) return -1;
    int64_t n = rows ? n_rows : N_dst;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 64) num_threads(nthreads > 0 ? nthreads : 1) reduction(| : bad)
    for (int64_t k = 0; k < n; ++k) {
        int64_t v = rows ? rows[k] : k;
        if (v < 0 || v >= N_dst) { bad = 1; continue; }
        int64_t deg = rowptr[v + 1] - rowptr[v];
        for (int64_t p = rowptr[v]; p < rowptr[v + 1]; ++p) {
            int64_t u = col[p];
            if (u < 0 || u >= N_src) { bad = 1; break; }
            double s = 0.0, a = 0.0;
            for (int64_t f = 0; f < F; ++f) {
                double t = route(reduce, deg, argout, F, v, f, p) *
                           (double)feature(g, g_is_bf16, F, v, f) *
                           (double)feature(x, x_is_bf16, F, u, f);
                s += t;
                a += fabs(t);
            }
            gw[p] = s;
            if (scale) scale[p] = a;
        }
    }
    return bad ? -1 : 0;
}

/* ---- more aggregators ---------------------------------------------------- */

/* For each listed row (rows == NULL: rows 0..n_rows-1), each feature f, over
 * the row's messages m_p (as in oracle_spmm):
 *   out_min[k,f], argmin[k,f]: the first p with the smallest m_p ('<' scan;
 *                 0.0 and -1 for an empty row)
 *   out_var[k,f]: sum_p (m_p - mean)^2 / deg, mean = sum_p m_p / deg, both
 *                 in fp64 (two passes; 0 for an empty row)
 *   out_std[k,f]: sqrt(out_var[k,f])
 * Any output may be NULL.  Returns 0, or -1 for a bad row or column. */
int oracle_spmm_multi(int64_t n_rows, const int64_t* rows, int64_t N_dst, int64_t N_src,
                      const int64_t* rowptr, const int32_t* col, const float* w, const void* x,
                      int x_is_bf16, int64_t F, float* out_min, int64_t* argmin,
                      double* out_var, double* out_std, int nthreads) {
    int bad = 0;
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : 1) reduction(| : bad)
    for (int64_t k = 0; k < n_rows; ++k) {
        int64_t i = rows ? rows[k] : k;
        if (i < 0 || i >= N_dst) {
            bad = 1;
            continue;
        }
        int64_t p0 = rowptr[i], p1 = rowptr[i + 1];
        for (int64_t p = p0; p < p1; ++p)
            if (col[p] < 0 || col[p] >= N_src) bad = 1;
        if (bad) continue;
        int64_t deg = p1 - p0;
        for (int64_t f = 0; f < F; ++f) {
            float least = 0.0f;
            int64_t arg = -1;
            double s = 0.0;
            for (int64_t p = p0; p < p1; ++p) {
                float m = message(x, x_is_bf16, F, col[p], f, w, p);
                if (arg < 0 || m < least) {
                    least = m;
                    arg = p;
                }
                s += (double)m;
            }
            double var = 0.0;
            if (deg > 0) {
                double mean = s / (double)deg;
                for (int64_t p = p0; p < p1; ++p) {
                    double d = (double)message(x, x_is_bf16, F, col[p], f, w, p) - mean;
                    var += d * d;
                }
                var /= (double)deg;
            }
            if (out_min) out_min[k * F + f] = arg < 0 ? 0.0f : least;
            if (argmin) argmin[k * F + f] = arg;
            if (out_var) out_var[k * F + f] = var;
            if (out_std) out_std[k * F + f] = sqrt(var);
        }
    }
    return bad ? -1 : 0;
}

/* ---- segment matmul -------------------------------------------------------- */

/* value of a bf16 matrix element (bits) as fp64 */
static inline double bf(const uint16_t* a, int64_t i) { return (double)widen_bf16(a[i]); }

/* out[r, o] = sum_f X[r, f] * W[t, f, o] for every row r of segment t
 * (seg[t] <= r < seg[t+1]); scale[r, o] = sum_f |X[r, f] * W[t, f, o]|.
 * X [N, F], W [T, F, Fo] bf16 bits; out, scale [N, Fo] fp64 (scale may be
 * NULL).  Returns 0, or -1 for bad segment bounds. */
int oracle_segment_matmul(int T, const int64_t* seg, const uint16_t* X, const uint16_t* W,
                          int64_t F, int64_t Fo, double* out, double* scale) {
    if (seg[0] != 0) return -1;
    for (int t = 0; t < T; ++t)
        if (seg[t + 1] < seg[t]) return -1;
    for (int t = 0; t < T; ++t) {
        const uint16_t* Wt = W + (int64_t)t * F * Fo;
#pragma omp parallel for schedule(static)
        for (int64_t r = seg[t]; r < seg[t + 1]; ++r)
            for (int64_t o = 0; o < Fo; ++o) {
                double s = 0.0, a = 0.0;
                for (int64_t f = 0; f < F; ++f) {
                    double p = bf(X, r * F + f) * bf(Wt, f * Fo + o);
                    s += p;
                    a += fabs(p);
                }
                out[r * Fo + o] = s;
                if (scale) scale[r * Fo + o] = a;
            }
    }
    return 0;
}

/* Gradients of the segment matmul given dOut = dL/d out [N, Fo] (bf16 bits):
 *   dX[r, f]    = sum_o dOut[r, o] * W[t, f, o]           (r in segment t)
 *   dW[t, f, o] = sum_{r in segment t} X[r, f] * dOut[r, o]
 * with the matching sums of absolute values in dx_scale, dw_scale.  Any
 * output may be NULL.  Returns 0, or -1 for bad segment bounds. */
int oracle_segment_matmul_backward(int T, const int64_t* seg, const uint16_t* X,
                                   const uint16_t* W, const uint16_t* dOut, int64_t F,
                                   int64_t Fo, double* dX, double* dx_scale, double* dW,
                                   double* dw_scale) {
    if (seg[0] != 0) return -1;
    for (int t = 0; t < T; ++t)
        if (seg[t + 1] < seg[t]) return -1;
    for (int t = 0; t < T; ++t) {
        const uint16_t* Wt = W + (int64_t)t * F * Fo;
        if (dX) {
#pragma omp parallel for schedule(static)
            for (int64_t r = seg[t]; r < seg[t + 1]; ++r)
                for (int64_t f = 0; f < F; ++f) {
                    double s = 0.0, a = 0.0;
                    for (int64_t o = 0; o < Fo; ++o) {
                        double p = bf(dOut, r * Fo + o) * bf(Wt, f * Fo + o);
                        s += p;
                        a += fabs(p);
                    }
                    dX[r * F + f] = s;
                    if (dx_scale) dx_scale[r * F + f] = a;
                }
        }
        if (dW) {
#pragma omp parallel for schedule(static)
            for (int64_t i = 0; i < F * Fo; ++i) {
                int64_t f = i / Fo, o = i - f * Fo;
                double s = 0.0, a = 0.0;
                for (int64_t r = seg[t]; r < seg[t + 1]; ++r) {
                    double p = bf(X, r * F + f) * bf(dOut, r * Fo + o);
                    s += p;
                    a += fabs(p);
                }
                dW[(int64_t)t * F * Fo + i] = s;
                if (dw_scale) dw_scale[(int64_t)t * F * Fo + i] = a;
            }
        }
    }
    return 0;
}

/* ---- edge-materialized messages (explanation mode) ---------------------- */
/*
 * Sec. 2.2 recalls that the first PyG materialized every message in edge
 * space and then aggregated it into node space; in explanation mode (Sec. 2.4)
 * message passing returns to that materialization so that a callback c, a
 * map from the E x F messages to E x F messages, can edit every message
 * before the aggregation:  h_v' = f(h_v, AGG{ c(g(h_w, e_wv, h_v)) }).
 * Messages are kept in destination-major CSR order: row p holds the message
 * of CSR edge p, so aggregating materialized messages is the aggregation of
 * oracle_spmm over the rows of the message table with column p at position p.
 */

/* msg[p, f] = x[idx[p], f], or fl32(w[p] * x[idx[p], f]) when w is given
 * (the same message as oracle_spmm).  idx is any int32 index array of length
 * E into the N_src rows of x (the CSR columns give the sources' features).
 * Returns 0, or -1 for an index out of range. */
int oracle_message_gather(int64_t E, int64_t N_src, const int32_t* idx, const float* w,
                          const void* x, int x_is_bf16, int64_t F, float* msg) {
    for (int64_t p = 0; p < E; ++p)
        if (idx[p] < 0 || idx[p] >= N_src) return -1;
    for (int64_t p = 0; p < E; ++p)
        for (int64_t f = 0; f < F; ++f)
            msg[p * F + f] = message(x, x_is_bf16, F, idx[p], f, w, p);
    return 0;
}

/* The edge-mask callback (a per-edge weight on every incoming message):
 * out[p, f] = fl32(msg[p, f] * mask[j]) with j = idx[p] (idx NULL: j = p),
 * one correctly rounded fp32 product.  out may equal msg.  Returns 0, or -1
 * for an index out of range. */
int oracle_message_scale(int64_t E, int64_t F, const float* msg, const float* mask,
                         const int32_t* idx, int64_t n_mask, float* out) {
    for (int64_t p = 0; p < E; ++p) {
        int64_t j = idx ? idx[p] : p;
        if (j < 0 || j >= n_mask) return -1;
    }
    for (int64_t p = 0; p < E; ++p) {
        double s = (double)mask[idx ? idx[p] : p];
        for (int64_t f = 0; f < F; ++f) out[p * F + f] = (float)((double)msg[p * F + f] * s);
    }
    return 0;
}

/* Gradient of the aggregation of materialized messages with respect to each
 * message, given g = dL/d out [N_dst, F] (fp32 or bf16 bits), for the CSR
 * edge p of row v:
 *   sum   dmsg[p, f] = g[v, f]
 *   mean  dmsg[p, f] = fl32(g[v, f] / deg(v))   (one correctly rounded division)
 *   max   dmsg[p, f] = g[v, f] if argout[v, f] == p, else 0
 * Returns 0, or -1 for a bad reduce. */
int oracle_message_backward(int64_t N_dst, const int64_t* rowptr, const void* g, int g_is_bf16,
                            int64_t F, int reduce, const int64_t* argout, float* dmsg) {
    if (reduce != ORACLE_SUM && reduce != ORACLE_MEAN && reduce != ORACLE_MAX) return -1;
    if (reduce == ORACLE_MAX && !argout) return -1;
    for (int64_t v = 0; v < N_dst; ++v) {
        int64_t deg = rowptr[v + 1] - rowptr[v];
        for (int64_t p = rowptr[v]; p < rowptr[v + 1]; ++p)
            for (int64_t f = 0; f < F; ++f) {
                float gv = feature(g, g_is_bf16, F, v, f);
                float d;
                if (reduce == ORACLE_SUM)
                    d = gv;
                else if (reduce == ORACLE_MEAN)
                    d = (float)((double)gv / (double)deg);
                else
                    d = argout[v * F + f] == p ? gv : 0.0f;
                dmsg[p * F + f] = d;
            }
    }
    return 0;
}

/* Per-edge dot products: for p in [0, E),
 *   out[o] = sum_f a[p, f] * b[j, f],  scale[o] = sum_f |a[p, f] * b[j, f]|
 * with j = bidx[p] (bidx NULL: j = p) and o = oidx[p] (oidx NULL: o = p), in
 * fp64.  a is [E, F], b is [N_b, F], each fp32 or bf16 bits.  This is the
 * gradient of the materialized messages with respect to a per-edge factor:
 * the edge weights (a = dL/dmsg, b = x, bidx = col) or an edge mask applied
 * by the callback (a = dL/d(masked msg), b = the unmasked messages).
 * Returns 0, or -1 for an index out of range. */
int oracle_edge_dot(int64_t E, int64_t F, const void* a, int a_is_bf16, const void* b,
                    int b_is_bf16, const int32_t* bidx, int64_t N_b, const int32_t* oidx,
                    double* out, double* scale) {
    for (int64_t p = 0; p < E; ++p) {
        int64_t j = bidx ? bidx[p] : p;
        int64_t o = oidx ? oidx[p] : p;
        if (j < 0 || j >= N_b || o < 0 || o >= E) return -1;
    }
    for (int64_t p = 0; p < E; ++p) {
        int64_t j = bidx ? bidx[p] : p;
        int64_t o = oidx ? oidx[p] : p;
        double s = 0.0, sa = 0.0;
        for (int64_t f = 0; f < F; ++f) {
            double t = (double)feature(a, a_is_bf16, F, p, f) * (double)feature(b, b_is_bf16, F, j, f);
            s += t;
            sa += fabs(t);
        }
        out[o] = s;
        if (scale) scale[o] = sa;
    }
    return 0;
}

/* Gradient of the materialized messages w[p] * x[col[p], :] with respect to
 * x, given dmsg = dL/dmsg [E, F] fp32:
 *   gx[u, f] = sum over CSR edges p with col[p] == u, in CSR order, of
 *              w_p * dmsg[p, f]     (w_p = 1 when w is NULL)
 *   scale[u, f] = the same sum of absolute values.
 * Returns 0, or -1 for a column out of range. */
int oracle_message_backward_x(int64_t E, int64_t N_src, const int32_t* col, const float* w,
                              const float* dmsg, int64_t F, double* gx, double* scale) {
    for (int64_t k = 0; k < N_src * F; ++k) {
        gx[k] = 0.0;
        if (scale) scale[k] = 0.0;
    }
    for (int64_t p = 0; p < E; ++p) {
        int64_t u = col[p];
        if (u < 0 || u >= N_src) return -1;
        double wp = w ? (double)w[p] : 1.0;
        for (int64_t f = 0; f < F; ++f) {
            double t = wp * (double)dmsg[p * F + f];
            gx[u * F + f] += t;
            if (scale) scale[u * F + f] += fabs(t);
        }
    }
    return 0;
}
