/*
 * mp.h -- C ABI of the message-passing aggregation library (libmp.so).
 *
 * The library implements the AGGREGATION step of message passing as written
 * in PyG 2.0 (arXiv 2507.16991), Eq. (1):
 *
 *     h_v' = f( h_v, AGG{ g(h_w, e_wv, h_v) : w in N(v) } )
 *
 * with message g = e_wv * h_w (e_wv an optional scalar edge weight) and the
 * permutation-invariant aggregators sum, mean and max named next to Eq. (1).
 * The update f is left to the caller.  Following Sec. 2.2 ("Accelerated
 * Message Passing"), the COO edge_index is first converted into a
 * destination-sorted compressed format, after which aggregation is a
 * segmented reduction per destination row.  The heterogeneous variant
 * (Sec. 2.2, "Heterogeneous Message Passing", the nested Eq. (1)) sums the
 * per-relation aggregations into each destination node type.
 *
 * Conventions shared by every call:
 *  - Orientation.  "CSR" here is destination-major: row v lists the edges
 *    (w, v) that end at v, and col holds their sources w.  This is the CSR of
 *    A^T (equivalently the CSC of A).
 *  - Pointers.  Array arguments are DEVICE pointers, allocated and owned by
 *    the caller.  The library allocates no device memory and keeps no array
 *    pointer after a call returns.  Scratch space is passed in as a
 *    caller-allocated workspace whose size comes from the matching *_workspace
 *    or *_size query.  Host pointers are marked "host".
 *  - Streams.  `stream` is a hipStream_t passed as void* (NULL = the default
 *    stream).  Every call only enqueues work and returns without waiting for
 *    the device, except mp_spmm_plan_build (one device-to-host copy, stated
 *    there).
 *  - Errors.  Calls return MP_OK (0) or a negative mp_status.  Argument
 *    errors are detected on the host before anything is enqueued, and leave
 *    every output untouched.  MP_ERR_HIP reports a failed launch or copy.
 *    Calls that sort on the device (mp_coo_to_csr, mp_csr_transpose,
 *    mp_hetero_build) report device-side failure asynchronously through an
 *    optional device status word (see mp_coo_to_csr); mp_spmm_plan_build,
 *    which synchronizes anyway, returns it.
 *  - Index validity.  Edge indices must satisfy 0 <= src < N_src and
 *    0 <= dst < N_dst, and a rowptr must be non-decreasing with rowptr[0] = 0
 *    and rowptr[N_dst] = E.  Violations are not detected by the compute calls
 *    (their behaviour is then undefined); mp_validate_coo and mp_validate_csr
 *    count them.
 *  - Determinism.  Every output is a deterministic function of the inputs:
 *    the floating-point summation order is fixed by the plan geometry, and no
 *    floating-point atomics are used.
 */
#ifndef MP_H_
#define MP_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MP_VERSION 5

/* Status codes. */
typedef enum mp_status {
    MP_OK = 0,
    MP_ERR_NULL = -1,      /* a required pointer is NULL */
    MP_ERR_SIZE = -2,      /* negative or unsupported size (see each call) */
    MP_ERR_DTYPE = -3,     /* unknown or unsupported dtype / index type */
    MP_ERR_REDUCE = -4,    /* unknown or unsupported reduction */
    MP_ERR_WORKSPACE = -5, /* workspace or plan buffer too small */
    MP_ERR_PLAN = -6,      /* plan does not match the arguments */
    MP_ERR_HIP = -7,       /* a HIP launch, copy or query failed */
    MP_ERR_ALIGN = -8,     /* a pointer is not aligned to its element size */
    MP_ERR_CALLBACK = -9,  /* a message callback returned nonzero */
    MP_ERR_SORT = -10      /* a device sort gave up waiting for an earlier tile;
                              the CSR it was building is invalid */
} mp_status;

/* Feature / output element types. */
typedef enum mp_dtype { MP_F32 = 0, MP_BF16 = 1 } mp_dtype;

/* rowptr element types. */
typedef enum mp_itype { MP_I32 = 0, MP_I64 = 1 } mp_itype;

/* Reductions, a bit mask.  mp_spmm allows MP_SUM, MP_MEAN, MP_MAX,
 * MP_SUM|MP_MAX and MP_MEAN|MP_MAX (the fused pass: one gather feeds both);
 * MP_MIN, MP_VAR and MP_STD are for mp_spmm_multi / mp_readout_multi. */
typedef enum mp_reduce {
    MP_SUM = 1,
    MP_MEAN = 2,
    MP_MAX = 4,
    MP_MIN = 8,
    MP_VAR = 16,
    MP_STD = 32
} mp_reduce;

/* Library version (MP_VERSION). */
int mp_version(void);

/* Static description of a status code; never NULL. */
const char* mp_status_str(int status);

/* ---------------------------------------------------------------------------
 * COO -> CSR conversion (Sec. 2.2: the sorted edge_index and its CSR cache).
 * ------------------------------------------------------------------------- */

/* Workspace bytes for mp_coo_to_csr with E edges and N destination rows.
 * with_payload: 1 if the call will request perm or val_out, else 0.
 * Sizes: 0 <= E <= INT32_MAX, 1 <= N <= INT32_MAX (else MP_ERR_SIZE).
 * *bytes (host) receives the size. */
int mp_coo_to_csr_workspace(int64_t E, int64_t N, int rowptr_itype, int with_payload,
                            size_t* bytes);

/* Stable sort of the COO edges by destination, producing the
 * destination-major CSR.
 *   src, dst    [E] int32 COO edge endpoints (device, read only).
 *   rowptr      [N+1] of rowptr_itype (MP_I32 or MP_I64): rowptr[0] = 0,
 *               rowptr[v+1] - rowptr[v] = in-degree of v, rowptr[N] = E.
 *   col         [E] int32: col[p] = source of the p-th edge in CSR order.
 *   perm        [E] int32 or NULL: perm[p] = COO id of the p-th CSR edge.
 *   val_in      [E] fp32 or NULL: per-edge values in COO order.
 *   val_out     [E] fp32 or NULL (given iff val_in is): val_in[perm[p]].
 * Within a row, edges keep ascending COO id (stable), so the result is
 * unique and bit-exact.  Duplicates and self-loops are ordinary edges.
 * E = 0 is valid (rowptr all zero).  ws/ws_bytes: workspace from
 * mp_coo_to_csr_workspace.
 *   status      [1] int32 (device) or NULL: written on `stream` after the
 *               sort, MP_OK if it completed, MP_ERR_SORT if a tile of the
 *               sort gave up its bounded wait for an earlier tile's counts
 *               (then col, perm and val_out are invalid and rowptr is not
 *               written).  The wait
 *               only spans tiles that are already running, so this is a
 *               guard against a hung device, not an expected outcome; read
 *               the word once the stream's work is done.
 * Asynchronous on `stream`. */
int mp_coo_to_csr(const int32_t* src, const int32_t* dst, int64_t E, int64_t N,
                  void* rowptr, int rowptr_itype, int32_t* col, int32_t* perm,
                  const float* val_in, float* val_out, void* ws, size_t ws_bytes,
                  int32_t* status, void* stream);

/* COO edges already sorted by destination (the sort-order metadata the
 * paper's EdgeIndex carries, Sec. 2.2): the CSR is the COO itself, so rowptr
 * is derived from dst directly, col = src, perm = 0..E-1 and val_out =
 * val_in (each optional output as in mp_coo_to_csr).  The caller asserts the
 * order; mp_validate_sorted counts violations.  No workspace.  If dst is not
 * non-decreasing the outputs are unspecified (but stay in bounds, and the
 * work stays bounded: rowptr is found by one binary search per row). */
int mp_sorted_coo_to_csr(const int32_t* src, const int32_t* dst, int64_t E, int64_t N,
                         void* rowptr, int rowptr_itype, int32_t* col, int32_t* perm,
                         const float* val_in, float* val_out, void* stream);

/* ---------------------------------------------------------------------------
 * Aggregation plan: rows binned by in-degree (Sec. 2.2: a destination-sorted
 * layout lets the aggregation run in parallel over rows; the plan is built
 * once per CSR and reused, like the CSR cache).
 * ------------------------------------------------------------------------- */

typedef struct mp_plan mp_plan;

/* Device bytes of the plan buffer for a CSR with N_dst rows and E edges. */
int mp_spmm_plan_size(int64_t N_dst, int64_t E, size_t* bytes);

/* Build a plan for one CSR and one feature row width F.  Its degree classes
 * are tuned for x_dtype, but the plan also serves the other feature dtype
 * (the classification never changes results, only which kernel does a row).
 *   rowptr      [N_dst+1] of rowptr_itype (device).
 *   plan_buf    device buffer of mp_spmm_plan_size bytes, owned by the caller,
 *               which must keep it alive and unchanged while the plan is used.
 *   *out        (host) receives a host-side handle; free with
 *               mp_spmm_plan_free.
 * This call SYNCHRONIZES `stream` once: it copies the per-bin row counts to
 * the host to size later launches (and returns MP_ERR_SORT, with *out
 * untouched, if the device sort of the rows by class gave up its bounded
 * wait).  The plan stays valid while rowptr and plan_buf are unchanged. */
int mp_spmm_plan_build(const void* rowptr, int rowptr_itype, int64_t N_dst, int64_t E,
                       int64_t F, int x_dtype, void* plan_buf, size_t plan_bytes,
                       void* stream, mp_plan** out);

/* Explicit degree-class thresholds for mp_spmm_plan_build_opts (0 = the
 * default of that field).  They decide which kernel and which schedule
 * aggregate a row, and so the fp32 summation order of its sums (results stay
 * within rounding of each other; integer outputs, max and argmax do not
 * change).
 *   small_max   rows of at most this many edges get one slot of a wavefront
 *               each (at most 16383);
 *   hub_min     rows of more than this many edges (raised to small_max if
 *               lower) are cut into edge chunks aggregated by separate
 *               wavefronts and combined in chunk order;
 *   chunk_min   the fewest edges of such a chunk (at most 2048 chunks per
 *               row). */
typedef struct mp_plan_opts {
    int64_t small_max;
    int64_t hub_min;
    int64_t chunk_min;
} mp_plan_opts;

/* mp_spmm_plan_build with explicit thresholds (opts NULL: the defaults, i.e.
 * exactly mp_spmm_plan_build).  Negative fields or chunk_min > INT32_MAX give
 * MP_ERR_SIZE. */
int mp_spmm_plan_build_opts(const void* rowptr, int rowptr_itype, int64_t N_dst, int64_t E,
                            int64_t F, int x_dtype, void* plan_buf, size_t plan_bytes,
                            const mp_plan_opts* opts, void* stream, mp_plan** out);

/* Release a host handle (NULL is ignored).  Does not touch plan_buf. */
void mp_spmm_plan_free(mp_plan* plan);

/* Workspace bytes mp_spmm needs with this plan and reduction (partial
 * results of hub rows split into edge chunks).  plan may be NULL (then 0). */
int mp_spmm_workspace(const mp_plan* plan, int reduce, size_t* bytes);

/* Segmented aggregation over the destination-major CSR (Eq. (1), the
 * AGGREGATION step; messages m_p = x[col[p], :] or w[p] * x[col[p], :]).
 *   plan        from mp_spmm_plan_build for this rowptr, N_dst and F (any
 *               x_dtype), or NULL (then one wavefront per row, no hub split,
 *               no workspace); a mismatch returns MP_ERR_PLAN.
 *   rowptr      [N_dst+1] of rowptr_itype; col [rowptr[N_dst]] int32.
 *   w           [E] fp32 in CSR order, or NULL (unweighted).
 *   x           [N_src, F] of x_dtype (MP_F32 or MP_BF16), row r starting
 *               at element r * ldx (ldx >= F; ldx = F for a contiguous
 *               table).  A row stride whose row bytes are a multiple of 128
 *               starts every row on a cache line (see mp_copy_rows).
 *   reduce      MP_SUM, MP_MEAN, MP_MAX, MP_SUM|MP_MAX or MP_MEAN|MP_MAX.
 *   out         [N_dst, F] of out_dtype: the sum or mean (required iff
 *               reduce has SUM or MEAN).  Accumulation is fp32; a bf16 output
 *               is rounded to nearest even once at the end.
 *   out_max     [N_dst, F] of max_dtype: the max message (required iff
 *               reduce has MAX).  max_dtype MP_BF16 is allowed only for bf16
 *               x without weights, where it is exact.
 *   argout      [N_dst, F] int32 (required iff reduce has MAX): the CSR
 *               position p of the first edge attaining the maximum.
 * Output rows are written in full (nothing is accumulated into them).  An
 * empty row gives 0 for sum, mean and max, and -1 in argout.  Messages are
 * compared with '>' so that -0.0 and +0.0 tie and the earlier edge wins;
 * infinities are ordinary values (a row whose messages are all -inf has max
 * -inf at its first edge).  Messages must not be NaN: outputs are then
 * unspecified (but every write stays in bounds).
 * A weighted message for MAX is the fp32 product fl32(w * x); sums may fuse
 * the multiply into the add.  Size limits: 0 <= N_src, N_dst <= INT32_MAX,
 * 1 <= F <= 65536, ldx >= F, E <= INT32_MAX (argout and col are int32).
 * Asynchronous on `stream` (no host synchronization when plan != NULL). */
int mp_spmm(const mp_plan* plan, const void* rowptr, int rowptr_itype, const int32_t* col,
            const float* w, const void* x, int x_dtype, int64_t N_src, int64_t N_dst,
            int64_t F, int64_t ldx, int reduce, void* out, int out_dtype, void* out_max,
            int max_dtype, int32_t* argout, void* ws, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): mp_spmm
 * without a workspace argument.  The hub-chunk partials that mp_spmm keeps in
 * its caller's workspace live instead in a static device array of
 * MP_NOALLOC_SCRATCH_BYTES per GPU, which the library's code object reserves
 * on every GPU it is loaded on and holds until the process ends.  Arguments,
 * outputs (bit-identical to mp_spmm's with the same plan) and status codes
 * as mp_spmm, plus MP_ERR_WORKSPACE when mp_spmm_workspace(plan, reduce)
 * exceeds MP_NOALLOC_SCRATCH_BYTES.  The call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); its first call on a device looks
 * up that device's copy of the array (hipGetSymbolAddress, with the device
 * current) and keeps the address.  Every call on one GPU shares that GPU's
 * array: calls enqueued on one stream are ordered and safe, but calls that
 * overlap on one GPU (different streams, or several host threads) race on it
 * and give wrong results.  Nothing in the array needs to start at zero (every
 * partial is written before it is read).  Asynchronous on `stream`. */
#define MP_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int mp_spmm_noalloc(const mp_plan* plan, const void* rowptr, int rowptr_itype,
                    const int32_t* col, const float* w, const void* x, int x_dtype,
                    int64_t N_src, int64_t N_dst, int64_t F, int64_t ldx, int reduce, void* out,
                    int out_dtype, void* out_max, int max_dtype, int32_t* argout, void* stream);

/* Feature-table layout: out[r, 0:F] = in[r, 0:F] for 0 <= r < N, rows of in
 * ld_in and rows of out ld_out elements apart (ld_in, ld_out >= F; padding
 * elements of out are not written; in and out must not overlap).  Used to
 * give a table whose rows are not a multiple of the 128-byte cache line a
 * stride that is (e.g. bf16 rows of F = 100 stored 128 elements apart), so
 * that each row gathered by the aggregation touches the fewest lines.
 * dtype: MP_F32 or MP_BF16.  Asynchronous on `stream`. */
int mp_copy_rows(const void* in, int64_t ld_in, void* out, int64_t ld_out, int64_t N, int64_t F,
                 int dtype, void* stream);

/* ---------------------------------------------------------------------------
 * Stacked aggregations (Sec. 2.2, "Aggregations as a First-Class Principle":
 * simple aggregators (sum, mean, max), advanced ones (variance, standard
 * deviation) and stacks of several, for message passing and for global
 * readouts).  One gather of each edge's message feeds every requested output.
 * Definitions over the messages m_p of a row (deg = row length):
 *   MP_SUM  sum m_p;  MP_MEAN  sum / deg;
 *   MP_MAX / MP_MIN  the largest / smallest m_p and, in arg, the CSR position
 *           of the first edge attaining it ('>' / '<' comparisons, so -0.0
 *           and +0.0 tie and the earlier edge wins);
 *   MP_VAR  population variance, sum (m_p - mean)^2 / deg, evaluated in one
 *           pass about a shift K (the mean of up to 8 messages of the row):
 *           sum (m_p - K)^2 / deg - (sum (m_p - K) / deg)^2 in fp32, clamped
 *           at 0, so that it keeps its digits when the mean is large against
 *           the spread (rows of equal messages give exactly 0);
 *   MP_STD  its square root.
 * An empty row gives 0 everywhere and -1 in arg.  All sums accumulate in
 * fp32 in an order fixed by the plan; outputs are fp32.
 * ------------------------------------------------------------------------- */

/* One output of a stacked aggregation. */
typedef struct mp_aggr_out {
    int aggr;     /* exactly one of MP_SUM .. MP_STD; each at most once per call */
    float* out;   /* [N_dst, F] fp32, device */
    int32_t* arg; /* [N_dst, F] int32, device: required for MP_MAX and MP_MIN,
                     ignored otherwise */
} mp_aggr_out;

/* Workspace bytes for mp_spmm_multi / mp_readout_multi with this plan (hub
 * partials of every statistic); 0 for a NULL plan. */
int mp_spmm_multi_workspace(const mp_plan* plan, size_t* bytes);

/* Stacked aggregation over the destination-major CSR: arguments as in
 * mp_spmm (x fp32 or bf16 with row stride ldx >= F, optional CSR-order
 * weights w, plan optional), plus n_out (1..6) outputs described by the host
 * array outs.  Duplicate or unknown aggregators give MP_ERR_REDUCE.
 * Asynchronous on `stream`. */
int mp_spmm_multi(const mp_plan* plan, const void* rowptr, int rowptr_itype, const int32_t* col,
                  const float* w, const void* x, int x_dtype, int64_t N_src, int64_t N_dst,
                  int64_t F, int64_t ldx, int n_out, const mp_aggr_out* outs, void* ws,
                  size_t ws_bytes, void* stream);

/* Global readout: the same stacked aggregation over segments of consecutive
 * node rows, given by ptr [N_seg+1] (the CSR of a sorted batch vector, e.g.
 * from mp_sorted_coo_to_csr of (node id, batch)); ptr[N_seg] must equal
 * N_nodes.  x is [N_nodes, F] with row stride ldx >= F; arg holds node
 * indices.  plan (optional) is built on ptr with N_seg rows and E = N_nodes. */
int mp_readout_multi(const mp_plan* plan, const void* ptr, int ptr_itype, const void* x,
                     int x_dtype, int64_t N_nodes, int64_t N_seg, int64_t F, int64_t ldx,
                     int n_out, const mp_aggr_out* outs, void* ws, size_t ws_bytes,
                     void* stream);

/* ---------------------------------------------------------------------------
 * Backward pass (Sec. 2.2: the backward pass of an aggregation over A runs
 * over the transposed adjacency, so the source-major CSR is built once and
 * kept next to the destination-major one, like the cached CSC).  Given the
 * gradient G = dL/d out of mp_spmm's output, with v = the destination row of
 * CSR edge p and route(v, f, p) = 1 (MP_SUM), 1/deg(v) (MP_MEAN) or
 * [argout[v, f] == p] (MP_MAX):
 *     dL/dx[u, f] = sum over edges p with col[p] == u of route * w[p] * G[v, f]
 *     dL/dw[p]    = sum over f of route * G[v, f] * x[col[p], f]
 * The fp32 rounding of a weighted message is not differentiated.  For an
 * undirected graph with symmetric weights the forward CSR is its own
 * transpose for MP_SUM and MP_MEAN (pass it as rowptrT/colT/wT, posT NULL).
 * ------------------------------------------------------------------------- */

/* Workspace bytes for mp_csr_transpose (with_payload: posT or val_out is
 * requested). */
int mp_csr_transpose_workspace(int64_t E, int64_t N_src, int rowptrT_itype, int with_payload,
                               size_t* bytes);

/* Source-major CSR of the edges of a destination-major CSR.
 *   rowptr      [N_dst+1] of rowptr_itype, col [E] int32: the forward CSR.
 *   rowptrT     [N_src+1] of rowptrT_itype: out, edges per source.
 *   colT        [E] int32: out, the destination (forward row) of each edge.
 *   posT        [E] int32 or NULL: out, the forward CSR position of each edge.
 *   val_in      [E] fp32 in forward CSR order, or NULL; val_out [E] receives
 *               val_in[posT[t]] (both or neither).
 *   status      [1] int32 (device) or NULL: MP_OK or MP_ERR_SORT, as in
 *               mp_coo_to_csr.
 * Within a source, edges keep their forward CSR order (a stable sort by col),
 * so the result is unique and bit-exact.  Sizes: 1 <= N_dst, N_src <=
 * INT32_MAX, 0 <= E <= INT32_MAX.  Asynchronous on `stream`. */
int mp_csr_transpose(const void* rowptr, int rowptr_itype, const int32_t* col, int64_t N_dst,
                     int64_t N_src, int64_t E, void* rowptrT, int rowptrT_itype, int32_t* colT,
                     int32_t* posT, const float* val_in, float* val_out, void* ws,
                     size_t ws_bytes, int32_t* status, void* stream);

/* Workspace bytes for mp_spmm_backward_x: hub partials of planT; for MP_MEAN
 * also an fp32 copy of G divided by the in-degrees (N_dst * F * 4 bytes); for
 * MP_MAX also the win masks, ceil(F / 32) 32-bit words per edge (bit f of the
 * words of forward position p: argout[row(p), f] == p). */
int mp_spmm_backward_x_workspace(const mp_plan* planT, int64_t N_dst, int64_t E, int64_t F,
                                 int reduce, size_t* bytes);

/* dL/dx of mp_spmm for one reduction (MP_SUM, MP_MEAN or MP_MAX; for a fused
 * forward call add the gradients of its parts).
 *   planT       plan built on rowptrT (N_src rows, same F), or NULL.
 *   rowptrT, colT, posT, wT   from mp_csr_transpose (wT = the forward weights
 *               in transposed order, NULL if unweighted; posT needed for MAX).
 *   rowptr      the forward rowptr (needed for MP_MEAN: in-degrees, and for
 *               MP_MAX: the rows of the forward positions).
 *   argout      [N_dst, F] int32 from the forward call (needed for MP_MAX).
 *   grad_out    [N_dst, F] of g_dtype: G.
 *   E           number of edges (rowptr[N_dst]); must equal planT's.
 *   grad_x      [N_src, F] of out_dtype, written in full (fp32 accumulation;
 *               a bf16 output is rounded to nearest even once).
 * MP_MAX first writes the win masks into the workspace (one pass over argout),
 * then gathers, per edge, only the feature chunks the edge wins.
 * Deterministic: one gather-reduce per source row, no atomics.  Asynchronous
 * on `stream`. */
int mp_spmm_backward_x(const mp_plan* planT, const void* rowptrT, int rowptrT_itype,
                       const int32_t* colT, const int32_t* posT, const float* wT,
                       const void* rowptr, int rowptr_itype, const int32_t* argout,
                       const void* grad_out, int g_dtype, int64_t N_dst, int64_t N_src, int64_t E,
                       int64_t F, int reduce, void* grad_x, int out_dtype, void* ws,
                       size_t ws_bytes, void* stream);

/* Workspace bytes for mp_spmm_backward_w (the row of every CSR edge, 4E). */
int mp_spmm_backward_w_workspace(int64_t E, size_t* bytes);

/* dL/dw of a weighted mp_spmm for one reduction: one dot product of G[v, :]
 * and x[col[p], :] per forward CSR edge p (fp32, a fixed reduction order).
 *   x           [N_src, F] of x_dtype; grad_out [N_dst, F] of g_dtype.
 *   argout      [N_dst, F] int32 from the forward call (needed for MP_MAX).
 *   grad_w      [E] fp32 out, forward CSR order (map to COO order with perm).
 * Sizes: 1 <= N_dst, 0 <= N_src, E <= INT32_MAX, 1 <= F <= 65536.
 * Asynchronous on `stream`. */
int mp_spmm_backward_w(const void* rowptr, int rowptr_itype, const int32_t* col, const void* x,
                       int x_dtype, const void* grad_out, int g_dtype, const int32_t* argout,
                       int64_t N_src, int64_t N_dst, int64_t E, int64_t F, int reduce,
                       float* grad_w, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Segment matmul (Sec. 2.2, heterogeneous GNNs: the projections {H_T W_T}
 * over node types with a weight tensor of shape [|T|, F, F'], forward and the
 * gradients with respect to H_T and W).  Rows of x are grouped by type in
 * contiguous segments seg[t] <= r < seg[t+1]; segment t uses W[t].  Inputs
 * are bf16 (row-major), products accumulate in fp32 on the matrix cores
 * (MFMA), in an order fixed by the tiling: outputs are deterministic.
 * Shared rules: seg is a HOST array of T+1 row offsets (seg[0] = 0,
 * non-decreasing, seg[T] = N <= INT32_MAX), 1 <= T <= MP_MAX_TYPES; F and Fo
 * are multiples of 8 in [8, 65536]; bf16 arrays and workspaces are 16-byte
 * aligned.
 * ------------------------------------------------------------------------- */

/* Workspace bytes for mp_segment_matmul (W transposed, T*F*Fo*2 bytes). */
int mp_segment_matmul_workspace(int T, int64_t F, int64_t Fo, size_t* bytes);

/* out[r, :] = x[r, :] @ W[t] for every row r of segment t.
 *   x    [N, F] bf16;  W [T, F, Fo] bf16;  out [N, Fo] of out_dtype (fp32, or
 *        bf16 rounded to nearest even from the fp32 result).
 * Asynchronous on `stream`. */
int mp_segment_matmul(const int64_t* seg, int T, const void* x, const void* W, int64_t F,
                      int64_t Fo, void* out, int out_dtype, void* ws, size_t ws_bytes,
                      void* stream);

/* Workspace bytes for mp_segment_matmul_backward (fp32 partial products of
 * the weight gradient: one F x Fo tile per 2048 rows of a segment). */
int mp_segment_matmul_backward_workspace(const int64_t* seg, int T, int64_t F, int64_t Fo,
                                         size_t* bytes);

/* Gradients of mp_segment_matmul given dout = dL/d out [N, Fo] bf16:
 *   dx[r, :]  = dout[r, :] @ W[t]^T        ([N, F] of dx_dtype; needs W)
 *   dW[t]     = x[seg_t]^T @ dout[seg_t]    ([T, F, Fo] fp32; needs x and ws;
 *               each segment's rows are reduced in fixed chunks whose
 *               partials are added in order, so no atomics are used)
 * Either output may be NULL (not both).  An empty segment gives dW[t] = 0.
 * Asynchronous on `stream`. */
int mp_segment_matmul_backward(const int64_t* seg, int T, const void* x, const void* W,
                               const void* dout, int64_t F, int64_t Fo, void* dx, int dx_dtype,
                               float* dW, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Edge-materialized message passing with a message callback.  In the
 * explanation mode of Sec. 2.4, message passing falls back to the edge-level
 * materialization of the first PyG (recalled in Sec. 2.2), so that a callback
 * c mapping the E x F messages to E x F messages can edit every message
 * before the aggregation:  h_v' = f(h_v, AGG{ c(g(h_w, e_wv, h_v)) })
 * (perturbing messages, weighting them with an edge mask, or capturing them).
 * Messages live in a caller-owned [E, F] table in destination-major CSR
 * order: row p is the message of CSR edge p, i.e. of COO edge perm[p].  The
 * aggregation of the table is the segmented reduction of mp_spmm over
 * consecutive rows (no atomics: the order of every sum is fixed, so results
 * are deterministic).  Arbitrary messages g can be built by the caller from
 * gathered tables (mp_message_gather of x by col gives the source rows, by
 * the rows of mp_csr_rows the destination rows) and aggregated with
 * mp_message_aggregate.
 * The gradient with respect to x of messages w[p] * x[col[p], :] given
 * dL/dmsg is mp_spmm over the transposed CSR (mp_csr_transpose) with the
 * forward positions posT as column indices, dL/dmsg as the feature table and
 * the transposed weights: gx[u] = sum over edges p from u of w[p] dL/dmsg[p].
 * ------------------------------------------------------------------------- */

/* row[p] = the destination row v of CSR position p (rowptr[v] <= p <
 * rowptr[v+1]), int32 [E]; the destination index of every edge in CSR
 * order.  Sizes: 1 <= N_dst <= INT32_MAX, 0 <= E <= INT32_MAX.
 * Asynchronous on `stream`. */
int mp_csr_rows(const void* rowptr, int rowptr_itype, int64_t N_dst, int64_t E, int32_t* row,
                void* stream);

/* MESSAGE, materialized: msg[p, :] = w[p] * x[idx[p], :] (one correctly
 * rounded fp32 product per element, as in mp_spmm) or x[idx[p], :] when w is
 * NULL, for p in [0, E).
 *   idx  [E] int32 rows of x, 0 <= idx[p] < N_src (the CSR col for the
 *        sources' features).
 *   w    [E] fp32 or NULL.
 *   x    [N_src, F] of x_dtype.
 *   msg  [E, F] of msg_dtype: MP_F32, or MP_BF16 only for unweighted bf16 x
 *        (then an exact copy of the rows); MP_ERR_DTYPE otherwise.
 * Sizes: 0 <= E <= INT32_MAX, 0 <= N_src <= INT32_MAX, 1 <= F <= 65536.
 * Asynchronous on `stream`. */
int mp_message_gather(const int32_t* idx, const float* w, const void* x, int x_dtype,
                      int64_t N_src, int64_t E, int64_t F, void* msg, int msg_dtype,
                      void* stream);

/* The edge-mask callback of explanation mode, and its gradient with respect
 * to its input: out[p, :] = in[p, :] * mask[j] with j = idx[p] (idx NULL:
 * j = p), one correctly rounded fp32 product per element.
 *   in, out  [E, F] fp32 (out may equal in: in place).
 *   mask     [n_mask] fp32 (per COO edge with idx = perm, or per CSR edge).
 *   idx      [E] int32 in [0, n_mask), or NULL (then n_mask >= E).
 * Asynchronous on `stream`. */
int mp_message_scale(const float* in, float* out, int64_t E, int64_t F, const float* mask,
                     const int32_t* idx, int64_t n_mask, void* stream);

/* AGGREGATION of materialized messages: out[v] = AGG over rows p in
 * [rowptr[v], rowptr[v+1]) of msg[p, :], exactly as mp_spmm with column p at
 * position p and no weights (same reductions, output dtypes, empty-row values
 * and argmax convention: argout holds the message row, i.e. the CSR position).
 *   msg  [E, F] of msg_dtype (MP_F32, or MP_BF16).
 * plan (optional): built from the same rowptr with this F.  ws: as
 * mp_spmm_workspace.  Asynchronous on `stream`. */
int mp_message_aggregate(const mp_plan* plan, const void* rowptr, int rowptr_itype,
                         const void* msg, int msg_dtype, int64_t E, int64_t N_dst, int64_t F,
                         int reduce, void* out, int out_dtype, void* out_max, int max_dtype,
                         int32_t* argout, void* ws, size_t ws_bytes, void* stream);

/* A message callback c.  Called on the calling host thread, once per
 * mp_spmm_materialized call, after the message table has been enqueued on
 * `stream` and before the aggregation is: it must enqueue its own work on
 * `stream` (or finish it before returning), reading and writing the [E, F]
 * table msg of msg_dtype in place.  user is passed through unchanged.  A
 * nonzero return aborts the call with MP_ERR_CALLBACK. */
typedef int (*mp_message_fn)(void* msg, int msg_dtype, int64_t E, int64_t F, void* user,
                             void* stream);

/* Explanation-mode aggregation: msg = gather (as mp_message_gather with
 * idx = col), then c(msg, ...) if c is not NULL, then the aggregation of
 * msg (as mp_message_aggregate).  With c NULL the max and argout equal
 * mp_spmm's exactly, and so do unweighted fp32 sums; a weighted mp_spmm may
 * fuse each product into its sum (one rounding fewer), so weighted sums agree
 * within rounding.
 *   msg  caller's [E, F] table of msg_dtype (left holding the messages
 *        after the callback).
 * Every argument of the three steps is checked before anything is enqueued.
 * On MP_ERR_CALLBACK the gather (and whatever c enqueued) has run and the
 * outputs are untouched.  Asynchronous on `stream` apart from the callback. */
int mp_spmm_materialized(const mp_plan* plan, const void* rowptr, int rowptr_itype,
                         const int32_t* col, const float* w, const void* x, int x_dtype,
                         int64_t N_src, int64_t N_dst, int64_t E, int64_t F, void* msg,
                         int msg_dtype, mp_message_fn c, void* user, int reduce, void* out,
                         int out_dtype, void* out_max, int max_dtype, int32_t* argout, void* ws,
                         size_t ws_bytes, void* stream);

/* Workspace bytes for mp_message_backward: 0 (the call takes no workspace;
 * ws may be NULL and ws_bytes 0). */
int mp_message_backward_workspace(int64_t E, size_t* bytes);

/* Gradient of the aggregation of materialized messages with respect to each
 * message, given grad_out = dL/dout [N_dst, F] (fp32 or bf16), for the CSR
 * edge p of row v (reduce is exactly one of MP_SUM, MP_MEAN, MP_MAX):
 *   sum   dmsg[p, :] = grad_out[v, :]
 *   mean  dmsg[p, :] = grad_out[v, :] / deg(v)   (correctly rounded)
 *   max   dmsg[p, f] = grad_out[v, f] if argout[v, f] == p, else 0
 *   dmsg   [E, F] fp32 out;  argout [N_dst, F] int32 from the forward (max).
 * Sizes: 1 <= N_dst <= INT32_MAX, 0 <= E <= INT32_MAX, 1 <= F <= 65536.
 * Asynchronous on `stream`. */
int mp_message_backward(const void* rowptr, int rowptr_itype, const int32_t* argout,
                        const void* grad_out, int g_dtype, int64_t N_dst, int64_t E, int64_t F,
                        int reduce, float* dmsg, void* ws, size_t ws_bytes, void* stream);

/* Per-edge dot products: out[o] = sum_f a[p, f] * b[j, f] with j = bidx[p]
 * (bidx NULL: j = p) and o = oidx[p] (oidx NULL: o = p), for p in [0, E),
 * accumulated in fp32 in a fixed order.  The gradient of materialized
 * messages with respect to a per-edge factor: the edge weights (a = dL/dmsg,
 * b = x, bidx = col) or an edge mask applied by the callback (a = dL/d(masked
 * messages), b = the unmasked messages, oidx = perm for COO order).
 *   a  [E, F] of a_dtype;  b [N_b, F] of b_dtype;  out [E] fp32.
 *   oidx must be a permutation of [0, E) when given.
 * Sizes: 0 <= E <= INT32_MAX, 0 <= N_b <= INT32_MAX, 1 <= F <= 65536.
 * Asynchronous on `stream`. */
int mp_edge_dot(const void* a, int a_dtype, const void* b, int b_dtype, const int32_t* bidx,
                int64_t N_b, const int32_t* oidx, int64_t E, int64_t F, float* out,
                void* stream);

/* ---------------------------------------------------------------------------
 * Heterogeneous message passing (Sec. 2.2, nested Eq. (1)): per destination
 * node type T, out_T = sum over relations r ending at T (ascending r) of the
 * sum aggregation over r's edges.  Built as one combined destination-major
 * CSR per destination type, whose edges within a row are ordered by
 * (relation id, COO id), and whose col holds GLOBAL source ids: local id plus
 * the offset of the source type (offsets = prefix sums of N_per_type).
 * ------------------------------------------------------------------------- */

#define MP_MAX_TYPES 16
/* dst_type value selecting every destination type at once: one CSR whose
 * rows are all nodes as global ids (type t's rows are offs[t] .. offs[t+1]-1,
 * offs the prefix sums of N_per_type), built and aggregated in one pass each;
 * the rows of each type are exactly those of that type's own CSR. */
#define MP_ALL_TYPES (-1)

/* One relation: edges src_type -> dst_type with local int32 endpoints. */
typedef struct mp_relation {
    int32_t src_type;
    int32_t dst_type;
    const int32_t* src; /* [E] device, local ids in src_type */
    const int32_t* dst; /* [E] device, local ids in dst_type */
    int64_t E;
} mp_relation;

/* Workspace bytes for mp_hetero_build of destination type dst_type (or
 * MP_ALL_TYPES).  N_per_type and rels are host arrays. */
int mp_hetero_build_workspace(int n_types, const int64_t* N_per_type, int n_rel,
                              const mp_relation* rels, int dst_type, int rowptr_itype,
                              size_t* bytes);

/* Build the combined CSR of destination type dst_type:
 *   rowptr [N_per_type[dst_type]+1] of rowptr_itype, col [E_T] int32 global
 *   source ids, where E_T = sum of E over relations ending at dst_type.
 * With dst_type = MP_ALL_TYPES: rowptr [N_total+1] over all nodes (global
 * ids), col [sum of all E].
 * status: [1] int32 (device) or NULL: MP_OK or MP_ERR_SORT, as in
 * mp_coo_to_csr.
 * n_types <= MP_MAX_TYPES; the total node count must fit int32. */
int mp_hetero_build(int n_types, const int64_t* N_per_type, int n_rel,
                    const mp_relation* rels, int dst_type, void* rowptr, int rowptr_itype,
                    int32_t* col, void* ws, size_t ws_bytes, int32_t* status, void* stream);

/* Sum aggregation over a combined CSR from mp_hetero_build, gathering each
 * source row from its own type's feature table.
 *   x_per_type  host array of n_types device pointers, each [N_t, F] x_dtype.
 *   plan        from mp_spmm_plan_build on this rowptr (or NULL).
 *   reduce      MP_SUM only (the cross-relation aggregator is a sum).
 *   out         [N_per_type[dst_type], F] of out_dtype; with MP_ALL_TYPES
 *               [N_total, F] (every type's rows, in type order). */
int mp_hetero_spmm(int n_types, const int64_t* N_per_type, const void* const* x_per_type,
                   int x_dtype, int64_t F, int dst_type, const mp_plan* plan,
                   const void* rowptr, int rowptr_itype, const int32_t* col, int reduce,
                   void* out, int out_dtype, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Debug checks.  Each writes the number of violations into *d_count, a
 * device int64, on `stream`.
 * ------------------------------------------------------------------------- */

/* Counts edges with src outside [0, N_src) or dst outside [0, N_dst). */
int mp_validate_coo(const int32_t* src, const int32_t* dst, int64_t E, int64_t N_src,
                    int64_t N_dst, int64_t* d_count, void* stream);

/* Counts positions p with dst[p] < dst[p-1] (0 when dst is sorted). */
int mp_validate_sorted(const int32_t* dst, int64_t E, int64_t* d_count, void* stream);

/* Counts rowptr steps that decrease, rowptr[0] != 0, rowptr[N_dst] != E, and
 * col entries outside [0, N_src). */
int mp_validate_csr(const void* rowptr, int rowptr_itype, const int32_t* col, int64_t N_dst,
                    int64_t N_src, int64_t E, int64_t* d_count, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MP_H_ */
