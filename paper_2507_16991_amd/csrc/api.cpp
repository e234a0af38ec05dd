// C ABI of libmp (declared in include/mp.h): argument validation, workspace
// layout and launch sequencing.  Every compute step runs in the HIP kernels
// of sort.hip, scan.hip and spmm.hip; this file only checks arguments, carves
// caller-provided buffers and enqueues launches.
#include <hip/hip_runtime.h>

#include <climits>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>

#include "mp_internal.hpp"

using namespace mp;

namespace {

inline hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

inline int hip_status(hipError_t e) { return e == hipSuccess ? MP_OK : MP_ERR_HIP; }

// Sequential carve of a caller buffer into 256-byte aligned pieces.
struct Carver {
    char* base;
    size_t off = 0;
    explicit Carver(void* b) : base(static_cast<char*>(b)) {}
    template <typename T>
    T* take(size_t count) {
        T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
        off = align_up(off + count * sizeof(T), 256);
        return p;
    }
};

bool valid_itype(int t) { return t == MP_I32 || t == MP_I64; }
bool valid_dtype(int t) { return t == MP_F32 || t == MP_BF16; }
bool valid_reduce(int r) {
    return r == MP_SUM || r == MP_MEAN || r == MP_MAX || r == (MP_SUM | MP_MAX) ||
           r == (MP_MEAN | MP_MAX);
}

// ---- COO -> CSR workspace layout ---------------------------------------------

// With more than one pass, the passes before the last write (key, src)
// packed in 8-byte words, ping-ponging between kv[0] and kv[1]; the last pass
// writes the keys into the buffer it does not read and src into col.  The
// COO-id payload, when asked for, ping-pongs as a 4-byte array that ends in
// perm.  (With one pass, keys and payloads go straight to their outputs.)
#ifndef MP_SORT_PACK
#define MP_SORT_PACK 1
#endif

struct CsrLayout {
    DigitPlan dp;
    int passes;
    bool packed;
    uint32_t *kA, *kB;
    int32_t *src_tmp, *eid_tmp, *eid_final;
    uint64_t* kv[2];
    RadixScratch sc;
    size_t bytes;
};

CsrLayout csr_layout(void* ws, int64_t E, int64_t N, int with_payload) {
    CsrLayout L{};
    L.dp = digit_plan(key_bits(N));
    L.passes = L.dp.passes;
    Carver c(ws);
    const size_t e = (size_t)(E > 0 ? E : 1);
    L.packed = MP_SORT_PACK && L.passes > 1;
    if (L.packed) {
        L.kv[0] = c.take<uint64_t>(e);
        L.kv[1] = c.take<uint64_t>(e);
        // pass passes-1 reads kv[(passes-2) % 2]
        L.kA = reinterpret_cast<uint32_t*>(L.kv[(L.passes - 1) % 2]);
    } else {
        L.kA = c.take<uint32_t>(e);
        L.kB = L.passes > 1 ? c.take<uint32_t>(e) : nullptr;
        L.src_tmp = L.passes > 1 ? c.take<int32_t>(e) : nullptr;
    }
    L.eid_tmp = (with_payload && L.passes > 1) ? c.take<int32_t>(e) : nullptr;
    L.eid_final = with_payload ? c.take<int32_t>(e) : nullptr;
    char* scratch = c.take<char>(radix_scratch_bytes(E));
    if (ws) L.sc = radix_scratch(scratch, E);
    L.bytes = c.off;
    return L;
}

int check_csr_sizes(int64_t E, int64_t N) {
    if (E < 0 || E > INT32_MAX || N < 1 || N > INT32_MAX) return MP_ERR_SIZE;
    return MP_OK;
}

int coo_to_csr_impl(const int32_t* src, const int32_t* dst, int64_t E, int64_t N, void* rowptr,
                    int itype, int32_t* col, int32_t* perm, const float* val_in, float* val_out,
                    void* ws, size_t ws_bytes, int32_t* status, hipStream_t s) {
    const int rp64 = itype == MP_I64;
    if (E == 0) {
        hipError_t e = launch_fill_rowptr_zero(N, rowptr, rp64, s);
        if (e == hipSuccess) e = launch_sort_status(nullptr, status, s);
        return hip_status(e);
    }
    const int payload = (perm != nullptr || val_out != nullptr) ? 1 : 0;
    CsrLayout L = csr_layout(ws, E, N, payload);
    if (ws_bytes < L.bytes) return MP_ERR_WORKSPACE;
    int32_t* eid_final = perm ? perm : L.eid_final;

    const uint32_t* keys_in = reinterpret_cast<const uint32_t*>(dst);
    if (radix_sort_begin(keys_in, E, L.dp, L.sc, s) != hipSuccess) return MP_ERR_HIP;
    const int32_t* a_in = src;
    const int32_t* b_in = nullptr;  // COO id = element index in the first pass
    for (int p = 0; p < L.passes && L.packed; ++p) {
        const bool last_parity = ((L.passes - 1 - p) % 2) == 0;  // lands where the final pass writes
        RadixPass rp{};
        if (p == 0) {
            rp.keys_in = keys_in;
            rp.a_in = a_in;
        } else {
            rp.kv_in = L.kv[(p - 1) % 2];
        }
        if (p < L.passes - 1) {
            rp.kv_out = L.kv[p % 2];
        } else {
            rp.keys_out = L.kA;
            rp.a_out = col;
        }
        rp.b_in = b_in;
        rp.b_out = payload ? (last_parity ? eid_final : L.eid_tmp) : nullptr;
        b_in = rp.b_out;
        rp.n = E;
        rp.pass = p;
        rp.shift = L.dp.shift[p];
        rp.bits = L.dp.width[p];
        rp.sc = L.sc;
        if (radix_sort_pass(rp, s) != hipSuccess) return MP_ERR_HIP;
    }
    for (int p = 0; p < L.passes && !L.packed; ++p) {
        const bool last_parity = ((L.passes - 1 - p) % 2) == 0;  // lands where the final pass writes
        RadixPass rp{};
        rp.keys_in = keys_in;
        rp.a_in = a_in;
        rp.b_in = b_in;
        rp.keys_out = last_parity ? L.kA : L.kB;
        rp.a_out = last_parity ? col : L.src_tmp;
        rp.b_out = payload ? (last_parity ? eid_final : L.eid_tmp) : nullptr;
        rp.n = E;
        rp.pass = p;
        rp.shift = L.dp.shift[p];
        rp.bits = L.dp.width[p];
        rp.sc = L.sc;
        if (radix_sort_pass(rp, s) != hipSuccess) return MP_ERR_HIP;
        keys_in = rp.keys_out;
        a_in = rp.a_out;
        b_in = rp.b_out;
    }
    hipError_t e = launch_rowptr_from_sorted(L.kA, E, N, rowptr, rp64, L.sc.err, s);
    if (e != hipSuccess) return MP_ERR_HIP;
    if (val_in && val_out) {
        e = launch_gather_f32(val_in, eid_final, E, val_out, s);
        if (e != hipSuccess) return MP_ERR_HIP;
    }
    return hip_status(launch_sort_status(&L.sc, status, s));
}

// ---- plan --------------------------------------------------------------------

struct PlanLayout {
    uint32_t* keys;
    int32_t* rowlist;
    int32_t* rowbeg;
    int32_t* rowend;
    uint32_t* chunk_off;
    RadixScratch sc;
    void* scan_ws;
    uint32_t* header;
    size_t bytes;
};

PlanLayout plan_layout(void* buf, int64_t N) {
    PlanLayout L{};
    Carver c(buf);
    const size_t n = (size_t)(N > 0 ? N : 1);
    L.keys = c.take<uint32_t>(n);
    L.rowlist = c.take<int32_t>(n);
    L.rowbeg = c.take<int32_t>(n);
    L.rowend = c.take<int32_t>(n);
    L.chunk_off = c.take<uint32_t>(n + 1);
    char* scratch = c.take<char>(radix_scratch_bytes(N));
    if (buf) L.sc = radix_scratch(scratch, N);
    L.scan_ws = c.take<char>(scan_workspace_bytes(N + 1));
    L.header = c.take<uint32_t>(64);
    L.bytes = c.off;
    return L;
}

}  // namespace

struct mp_plan {
    const void* rowptr;
    int itype;
    int64_t N_dst, E, F;
    int x_dtype;
    int64_t small_max, hub_min;
    int chunk_min;
    int64_t n_tiny, n_small, n_mid, n_hub, n_chunks;
    int64_t mid_base, hub_base;
    int32_t* rowlist;
    int32_t* rowbeg;
    int32_t* rowend;
    uint32_t* chunk_off;
};

namespace {

// A single feature table of `rows` rows, `ld` elements apart, is addressed
// with 32-bit byte offsets from its base: it spans under 4 GiB, and row
// indices and the row stride in bytes fit 24 bits, so that the kernels form
// an offset with one 24-bit multiply-add.
inline int fits_off32(int64_t rows, int64_t ld, int elem_bytes) {
    return rows * ld * elem_bytes <= (int64_t)UINT32_MAX && rows <= ((int64_t)1 << 24) &&
                   ld * elem_bytes < ((int64_t)1 << 24)
               ? 1
               : 0;
}

// Fill the work description of SpmmParams from a plan (or the plan-free
// generic layout) and launch the main kernel plus the hub fix-up.
int run_spmm(const mp_plan* plan, SpmmParams& P, const Geometry& g, int x_dtype, int64_t N_dst,
             void* ws, size_t ws_bytes, hipStream_t s) {
    if (P.ldx == 0) P.ldx = P.F;  // contiguous feature rows
    P.L = g.L;
    P.S = g.S;
    P.FT = g.FT;
    P.ltot = g.ltot;
    const bool hx = P.stats != 0;
    const bool hs = hx || (P.reduce & (MP_SUM | MP_MEAN)) != 0;
    const bool hm = hx || (P.reduce & MP_MAX) != 0;
    const bool tiny = plan && plan->n_tiny > 0 && g.L > kTinyDeg;
    if (plan) {
        P.rowlist = plan->rowlist;
        P.rowbeg = plan->rowbeg;
        P.rowend = plan->rowend;
        P.chunk_off = plan->chunk_off;
        P.chunk_min = plan->chunk_min;
        // tiny rows go to their own kernel when slots are wide enough
        P.n_tiny = tiny ? plan->n_tiny : 0;
        P.small_base = P.n_tiny;
        P.n_small = plan->n_small - P.n_tiny;
        P.n_hub = plan->n_hub;
        P.mid_base = plan->mid_base;
        P.hub_base = plan->hub_base;
        P.n_hub_waves = plan->n_chunks * g.FT;
        P.n_mid_waves = plan->n_mid * g.FT;
        P.n_small_waves = ceil_div(P.n_small, g.S) * g.FT;
        if (plan->n_chunks > 0) {
            Carver c(ws);
            const size_t cells = (size_t)plan->n_chunks * (size_t)P.F;
            P.part_sum = hs ? c.take<float>(cells) : nullptr;
            P.part_max = hm ? c.take<float>(cells) : nullptr;
            P.part_arg = hm ? c.take<int32_t>(cells) : nullptr;
            P.part_dsum = hx ? c.take<float>(cells) : nullptr;
            P.part_sq = hx ? c.take<float>(cells) : nullptr;
            P.part_min = hx ? c.take<float>(cells) : nullptr;
            P.part_amin = hx ? c.take<int32_t>(cells) : nullptr;
            if (ws_bytes < c.off || !ws) return MP_ERR_WORKSPACE;
        }
    } else {
        P.rowlist = nullptr;
        P.n_mid_waves = N_dst * g.FT;
    }
    const int64_t waves = P.n_hub_waves + P.n_mid_waves + P.n_small_waves;
    if (ceil_div(waves, 4) > (int64_t)UINT32_MAX) return MP_ERR_SIZE;
    hipError_t e = launch_spmm_tiny(P, x_dtype, g.epl, s);
    if (e != hipSuccess) return MP_ERR_HIP;
    e = launch_spmm(P, x_dtype, g.epl, s);
    if (e != hipSuccess) return MP_ERR_HIP;
    if (plan && plan->n_hub > 0) {
        e = launch_spmm_fixup(P, s);
        if (e != hipSuccess) return MP_ERR_HIP;
    }
    return MP_OK;
}

// The row classes only steer work to kernels (any classification gives the
// same result), so a plan built for one feature dtype serves the other too;
// F must match because hub partials are sized by it.
int check_plan(const mp_plan* plan, const void* rowptr, int itype, int64_t N_dst, int64_t F) {
    if (!plan) return MP_OK;
    if (plan->rowptr != rowptr || plan->itype != itype || plan->N_dst != N_dst || plan->F != F)
        return MP_ERR_PLAN;
    return MP_OK;
}

// ---- stacked aggregations ---------------------------------------------------------

constexpr int kAllAggr = MP_SUM | MP_MEAN | MP_MAX | MP_MIN | MP_VAR | MP_STD;

// Check the output list and fill the stats-mode outputs of P.
int fill_multi_outputs(int n_out, const mp_aggr_out* outs, int64_t rows, SpmmParams& P) {
    if (n_out < 1 || n_out > 6) return MP_ERR_SIZE;
    if (!outs) return MP_ERR_NULL;
    int seen = 0;
    uintptr_t all = 0;
    for (int k = 0; k < n_out; ++k) {
        const mp_aggr_out& o = outs[k];
        const int a = o.aggr;
        if ((a & kAllAggr) != a || a == 0 || (a & (a - 1)) != 0 || (seen & a)) return MP_ERR_REDUCE;
        seen |= a;
        const bool has_arg = a == MP_MAX || a == MP_MIN;
        if (rows > 0 && (!o.out || (has_arg && !o.arg))) return MP_ERR_NULL;
        if ((uintptr_t)o.out % 4 || (uintptr_t)o.arg % 4) return MP_ERR_ALIGN;
        all |= (uintptr_t)o.out | (has_arg ? (uintptr_t)o.arg : 0);
        switch (a) {
            case MP_SUM: P.o_sum = o.out; break;
            case MP_MEAN: P.o_mean = o.out; break;
            case MP_MAX: P.o_max = o.out; P.o_amax = o.arg; break;
            case MP_MIN: P.o_min = o.out; P.o_amin = o.arg; break;
            case MP_VAR: P.o_var = o.out; break;
            default: P.o_std = o.out; break;
        }
    }
    P.stats = 1;
    P.reduce = MP_SUM | MP_MAX;
    P.vec_store = (all % 16) == 0;
    return MP_OK;
}

int multi_impl(const mp_plan* plan, const void* rowptr, int rowptr_itype, const int32_t* col,
               const float* w, const void* x, int x_dtype, int64_t N_src, int64_t N_dst, int64_t F,
               int64_t ldx, int n_out, const mp_aggr_out* outs, void* ws, size_t ws_bytes,
               hipStream_t s) {
    if (!valid_itype(rowptr_itype) || !valid_dtype(x_dtype)) return MP_ERR_DTYPE;
    if (N_src < 0 || N_src > INT32_MAX || N_dst < 0 || N_dst > INT32_MAX || F < 1 || F > 65536 ||
        ldx < F)
        return MP_ERR_SIZE;
    if (!rowptr) return MP_ERR_NULL;
    if (N_dst > 0 && !x) return MP_ERR_NULL;
    SpmmParams P{};
    int st = fill_multi_outputs(n_out, outs, N_dst, P);
    if (st != MP_OK) return st;
    st = check_plan(plan, rowptr, rowptr_itype, N_dst, F);
    if (st != MP_OK) return st;
    const int eb = x_dtype == MP_BF16 ? 2 : 4;
    if ((uintptr_t)x % eb || (uintptr_t)rowptr % (rowptr_itype == MP_I64 ? 8 : 4) ||
        (uintptr_t)col % 4 || (uintptr_t)w % 4)
        return MP_ERR_ALIGN;
    if (N_dst == 0) return MP_OK;
    Geometry g = make_geometry(F, x_dtype, (uintptr_t)x | (uintptr_t)(ldx * eb));
    P.rowptr = rowptr;
    P.rp64 = rowptr_itype == MP_I64;
    P.col = col;
    P.w = w;
    P.n_tables = 1;
    P.table_ptr[0] = static_cast<const char*>(x);
    P.F = F;
    P.ldx = ldx;
    P.off32 = fits_off32(N_src, ldx, eb);
    return run_spmm(plan, P, g, x_dtype, N_dst, ws, ws_bytes, s);
}

// ---- aggregation call (mp_spmm, mp_message_aggregate) ---------------------------

// The arguments of one aggregation; col == nullptr reads position p as
// column p (a table of materialized messages).
struct SpmmCall {
    const mp_plan* plan;
    const void* rowptr;
    int rowptr_itype;
    const int32_t* col;
    const float* w;
    const void* x;
    int x_dtype;
    int64_t N_src, N_dst, F;
    int64_t ldx;  // row stride of x in elements (>= F)
    int reduce;
    void* out;
    int out_dtype;
    void* out_max;
    int max_dtype;
    int32_t* argout;
    void* ws;
    size_t ws_bytes;
};

// Every argument check of an aggregation, before anything is enqueued.
int spmm_check(const SpmmCall& c) {
    if (!valid_reduce(c.reduce)) return MP_ERR_REDUCE;
    if (!valid_itype(c.rowptr_itype) || !valid_dtype(c.x_dtype)) return MP_ERR_DTYPE;
    const bool hs = (c.reduce & (MP_SUM | MP_MEAN)) != 0;
    const bool hm = (c.reduce & MP_MAX) != 0;
    if (hs && !valid_dtype(c.out_dtype)) return MP_ERR_DTYPE;
    if (hm && !valid_dtype(c.max_dtype)) return MP_ERR_DTYPE;
    if (hm && c.max_dtype == MP_BF16 && (c.x_dtype != MP_BF16 || c.w != nullptr))
        return MP_ERR_DTYPE;
    if (c.N_src < 0 || c.N_src > INT32_MAX || c.N_dst < 0 || c.N_dst > INT32_MAX || c.F < 1 ||
        c.F > 65536 || c.ldx < c.F)
        return MP_ERR_SIZE;
    if (!c.rowptr) return MP_ERR_NULL;
    if (c.N_dst > 0) {
        if (!c.x) return MP_ERR_NULL;
        if (hs && !c.out) return MP_ERR_NULL;
        if (hm && (!c.out_max || !c.argout)) return MP_ERR_NULL;
    }
    int st = check_plan(c.plan, c.rowptr, c.rowptr_itype, c.N_dst, c.F);
    if (st != MP_OK) return st;
    const int eb = c.x_dtype == MP_BF16 ? 2 : 4;
    if ((uintptr_t)c.x % eb || (uintptr_t)c.rowptr % (c.rowptr_itype == MP_I64 ? 8 : 4) ||
        (uintptr_t)c.col % 4 || (uintptr_t)c.w % 4 || (uintptr_t)c.argout % 4 ||
        (hs && (uintptr_t)c.out % (c.out_dtype == MP_BF16 ? 2 : 4)) ||
        (hm && (uintptr_t)c.out_max % (c.max_dtype == MP_BF16 ? 2 : 4)))
        return MP_ERR_ALIGN;
    size_t need = 0;
    mp_spmm_workspace(c.plan, c.reduce, &need);
    if (c.N_dst > 0 && need > 0 && (c.ws_bytes < need || !c.ws)) return MP_ERR_WORKSPACE;
    return MP_OK;
}

// Enqueue a checked aggregation.
int spmm_launch(const SpmmCall& c, hipStream_t s) {
    if (c.N_dst == 0) return MP_OK;
    const int eb = c.x_dtype == MP_BF16 ? 2 : 4;
    Geometry g = make_geometry(c.F, c.x_dtype, (uintptr_t)c.x | (uintptr_t)(c.ldx * eb));
    SpmmParams P{};
    P.rowptr = c.rowptr;
    P.rp64 = c.rowptr_itype == MP_I64;
    P.col = c.col;
    P.w = c.w;
    P.n_tables = 1;
    P.table_ptr[0] = static_cast<const char*>(c.x);
    P.table_off[0] = 0;
    P.F = c.F;
    P.ldx = c.ldx;
    P.off32 = fits_off32(c.N_src, c.ldx, eb);
    P.reduce = c.reduce;
    P.out = c.out;
    P.out_bf16 = c.out_dtype == MP_BF16;
    P.out_max = c.out_max;
    P.max_bf16 = c.max_dtype == MP_BF16;
    P.argout = c.argout;
    P.vec_store = (((uintptr_t)c.out | (uintptr_t)c.out_max | (uintptr_t)c.argout) % 16) == 0;
    return run_spmm(c.plan, P, g, c.x_dtype, c.N_dst, c.ws, c.ws_bytes, s);
}

// ---- edge-materialized messages ---------------------------------------------------

// Check a message gather and describe it.
int gather_check(const int32_t* idx, const float* w, const void* x, int x_dtype, int64_t N_src,
                 int64_t E, int64_t F, void* msg, int msg_dtype, MessageGather* a) {
    if (!valid_dtype(x_dtype) || !valid_dtype(msg_dtype)) return MP_ERR_DTYPE;
    if (msg_dtype == MP_BF16 && (x_dtype != MP_BF16 || w != nullptr)) return MP_ERR_DTYPE;
    if (E < 0 || E > INT32_MAX || N_src < 0 || N_src > INT32_MAX || F < 1 || F > 65536)
        return MP_ERR_SIZE;
    if (E > 0 && (!idx || !x || !msg)) return MP_ERR_NULL;
    const int bx = x_dtype == MP_BF16 ? 2 : 4, bm = msg_dtype == MP_BF16 ? 2 : 4;
    if ((uintptr_t)idx % 4 || (uintptr_t)w % 4 || (uintptr_t)x % bx || (uintptr_t)msg % bm)
        return MP_ERR_ALIGN;
    const uintptr_t ptrs[2] = {(uintptr_t)x, (uintptr_t)msg};
    const int sizes[2] = {bx, bm};
    *a = MessageGather{idx, w, x, x_dtype == MP_BF16, msg, msg_dtype == MP_BF16, E, F,
                       message_epl(F, ptrs, sizes, 2, 8)};
    return MP_OK;
}

// ---- segment matmul ------------------------------------------------------------

constexpr int64_t kGmmRowsPerChunk = 2048;  // rows per partial of the weight gradient

// Validate the host segment offsets; fill P.seg and return the row count.
int gmm_segments(const int64_t* seg, int T, GmmParams& P, int64_t* N_rows) {
    if (!seg) return MP_ERR_NULL;
    if (T < 1 || T > MP_MAX_TYPES) return MP_ERR_SIZE;
    if (seg[0] != 0) return MP_ERR_SIZE;
    for (int t = 0; t < T; ++t)
        if (seg[t + 1] < seg[t]) return MP_ERR_SIZE;
    if (seg[T] > INT32_MAX) return MP_ERR_SIZE;
    P.T = T;
    for (int t = 0; t <= T; ++t) P.seg[t] = seg[t];
    *N_rows = seg[T];
    return MP_OK;
}

int gmm_dims(int64_t F, int64_t Fo) {
    // 16-byte row chunks of bf16
    if (F < 8 || Fo < 8 || F > 65536 || Fo > 65536 || F % 8 || Fo % 8) return MP_ERR_SIZE;
    return MP_OK;
}

int64_t gmm_chunks(const int64_t* seg, int T, int64_t* off) {
    int64_t c = 0;
    for (int t = 0; t < T; ++t) {
        off[t] = c;
        c += ceil_div(seg[t + 1] - seg[t], kGmmRowsPerChunk);
    }
    off[T] = c;
    return c;
}

}  // namespace

extern "C" {

int mp_version(void) { return MP_VERSION; }

const char* mp_status_str(int status) {
    switch (status) {
        case MP_OK: return "ok";
        case MP_ERR_NULL: return "a required pointer is NULL";
        case MP_ERR_SIZE: return "size out of range";
        case MP_ERR_DTYPE: return "unsupported dtype or index type";
        case MP_ERR_REDUCE: return "unsupported reduction";
        case MP_ERR_WORKSPACE: return "workspace or plan buffer too small";
        case MP_ERR_PLAN: return "plan does not match the arguments";
        case MP_ERR_HIP: return "HIP launch or copy failed";
        case MP_ERR_ALIGN: return "pointer not aligned to its element size";
        case MP_ERR_CALLBACK: return "the message callback failed";
        case MP_ERR_SORT: return "a device sort gave up waiting; its output is invalid";
        default: return "unknown status";
    }
}

int mp_coo_to_csr_workspace(int64_t E, int64_t N, int rowptr_itype, int with_payload,
                            size_t* bytes) {
    if (!bytes) return MP_ERR_NULL;
    if (!valid_itype(rowptr_itype)) return MP_ERR_DTYPE;
    int st = check_csr_sizes(E, N);
    if (st != MP_OK) return st;
    *bytes = E == 0 ? 0 : csr_layout(nullptr, E, N, with_payload ? 1 : 0).bytes;
    return MP_OK;
}

int mp_coo_to_csr(const int32_t* src, const int32_t* dst, int64_t E, int64_t N, void* rowptr,
                  int rowptr_itype, int32_t* col, int32_t* perm, const float* val_in,
                  float* val_out, void* ws, size_t ws_bytes, int32_t* status, void* stream) {
    if (!valid_itype(rowptr_itype)) return MP_ERR_DTYPE;
    int st = check_csr_sizes(E, N);
    if (st != MP_OK) return st;
    if (!rowptr) return MP_ERR_NULL;
    if (E > 0 && (!src || !dst || !col || !ws)) return MP_ERR_NULL;
    if (E > 0 && (val_in == nullptr) != (val_out == nullptr)) return MP_ERR_NULL;
    if ((uintptr_t)rowptr % (rowptr_itype == MP_I64 ? 8 : 4) || (uintptr_t)status % 4)
        return MP_ERR_ALIGN;
    return coo_to_csr_impl(src, dst, E, N, rowptr, rowptr_itype, col, perm, val_in, val_out, ws,
                           ws_bytes, status, as_stream(stream));
}

int mp_sorted_coo_to_csr(const int32_t* src, const int32_t* dst, int64_t E, int64_t N,
                         void* rowptr, int rowptr_itype, int32_t* col, int32_t* perm,
                         const float* val_in, float* val_out, void* stream) {
    if (!valid_itype(rowptr_itype)) return MP_ERR_DTYPE;
    int st = check_csr_sizes(E, N);
    if (st != MP_OK) return st;
    if (!rowptr) return MP_ERR_NULL;
    if (E > 0 && (!src || !dst || !col)) return MP_ERR_NULL;
    if (E > 0 && (val_in == nullptr) != (val_out == nullptr)) return MP_ERR_NULL;
    if ((uintptr_t)rowptr % (rowptr_itype == MP_I64 ? 8 : 4)) return MP_ERR_ALIGN;
    hipStream_t s = as_stream(stream);
    const int rp64 = rowptr_itype == MP_I64;
    if (E == 0) return hip_status(launch_fill_rowptr_zero(N, rowptr, rp64, s));
    // the sorted keys are dst itself (non-negative int32 read as uint32);
    // a binary search per row keeps the work bounded if dst is not sorted
    hipError_t e = launch_rowptr_by_search(reinterpret_cast<const uint32_t*>(dst), E, N,
                                           rowptr, rp64, s);
    if (e == hipSuccess) e = launch_offset_copy(src, E, 0, col, s);
    if (e == hipSuccess && perm) e = launch_iota(E, perm, s);
    if (e == hipSuccess && val_in) e = launch_copy_f32(val_in, E, val_out, s);
    return hip_status(e);
}

int mp_spmm_plan_size(int64_t N_dst, int64_t E, size_t* bytes) {
    if (!bytes) return MP_ERR_NULL;
    if (N_dst < 0 || N_dst > INT32_MAX || E < 0 || E > INT32_MAX) return MP_ERR_SIZE;
    *bytes = plan_layout(nullptr, N_dst).bytes;
    return MP_OK;
}

int mp_spmm_plan_build(const void* rowptr, int rowptr_itype, int64_t N_dst, int64_t E, int64_t F,
                       int x_dtype, void* plan_buf, size_t plan_bytes, void* stream,
                       mp_plan** out) {
    return mp_spmm_plan_build_opts(rowptr, rowptr_itype, N_dst, E, F, x_dtype, plan_buf,
                                   plan_bytes, nullptr, stream, out);
}

int mp_spmm_plan_build_opts(const void* rowptr, int rowptr_itype, int64_t N_dst, int64_t E,
                            int64_t F, int x_dtype, void* plan_buf, size_t plan_bytes,
                            const mp_plan_opts* opts, void* stream, mp_plan** out) {
    if (!out || !rowptr || !plan_buf) return MP_ERR_NULL;
    if (!valid_itype(rowptr_itype) || !valid_dtype(x_dtype)) return MP_ERR_DTYPE;
    if (N_dst < 0 || N_dst > INT32_MAX || E < 0 || E > INT32_MAX || F < 1 || F > 65536)
        return MP_ERR_SIZE;
    const mp_plan_opts o = opts ? *opts : mp_plan_opts{0, 0, 0};
    if (o.small_max < 0 || o.hub_min < 0 || o.chunk_min < 0 || o.chunk_min > INT32_MAX)
        return MP_ERR_SIZE;
    PlanLayout L = plan_layout(plan_buf, N_dst);
    if (plan_bytes < L.bytes) return MP_ERR_WORKSPACE;
    hipStream_t s = as_stream(stream);
    const int rp64 = rowptr_itype == MP_I64;

    mp_plan* p = new (std::nothrow) mp_plan{};
    if (!p) return MP_ERR_SIZE;
    p->rowptr = rowptr;
    p->itype = rowptr_itype;
    p->N_dst = N_dst;
    p->E = E;
    p->F = F;
    p->x_dtype = x_dtype;
    // rows of up to 16 edges per slot get one slot; longer rows a wavefront
    const Geometry geo = make_geometry(F, x_dtype, 16);
    p->small_max = o.small_max > 0 ? o.small_max : 16 * (int64_t)geo.S;
    if (p->small_max > 16383) p->small_max = 16383;
    // a wavefront takes S * U edges per step; rows longer than 32 steps are
    // split into chunks of at least 32 steps, so that no wavefront runs a
    // long chain of dependent steps on its own
    const int64_t step_edges = (int64_t)geo.S * (geo.S * 8 > 64 ? 64 / geo.S : 8);
    p->hub_min = o.hub_min > 0 ? o.hub_min : 32 * step_edges;
    if (p->hub_min < p->small_max) p->hub_min = p->small_max;
    p->chunk_min = (int)(o.chunk_min > 0 ? o.chunk_min : 32 * step_edges);
    p->rowlist = L.rowlist;
    p->rowbeg = L.rowbeg;
    p->rowend = L.rowend;
    p->chunk_off = L.chunk_off;
    if (N_dst == 0) {
        *out = p;
        return MP_OK;
    }
    hipError_t e = launch_plan_classes(rowptr, rp64, N_dst, p->small_max, p->hub_min, L.keys, s);
    if (e == hipSuccess) {
        DigitPlan dp{};
        dp.passes = 1;
        dp.width[0] = dp.max_width = kPlanClassBits;
        e = radix_sort_begin(L.keys, N_dst, dp, L.sc, s);
    }
    if (e == hipSuccess) {
        RadixPass rp{};
        rp.keys_in = L.keys;
        rp.a_out = L.rowlist;  // payload = row id
        rp.n = N_dst;
        rp.pass = 0;
        rp.shift = 0;
        rp.bits = kPlanClassBits;
        rp.sc = L.sc;
        e = radix_sort_pass(rp, s);
    }
    if (e == hipSuccess)
        e = launch_plan_rows(rowptr, rp64, L.rowlist, N_dst, p->hub_min, p->chunk_min, L.rowbeg,
                             L.rowend, L.chunk_off, s);
    // only hub rows have chunks, and they end the class-sorted list: the
    // entries before the hub class's start are zero
    if (e == hipSuccess)
        e = exclusive_scan_u32(L.chunk_off, N_dst + 1, L.scan_ws, s, L.sc.gbase + kClassHub);
    const int nclass = kClassHub + 1;
    if (e == hipSuccess)
        e = launch_plan_header(L.sc.gbase, nclass, L.chunk_off, N_dst, L.sc.err, L.header, s);
    uint32_t h[64] = {0};
    if (e == hipSuccess)
        e = hipMemcpyAsync(h, L.header, sizeof(uint32_t) * (nclass + 3), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess || h[nclass + 2] != 0) {
        delete p;
        return e != hipSuccess ? MP_ERR_HIP : MP_ERR_SORT;
    }
    p->mid_base = h[kClassMid];
    p->hub_base = h[kClassHub];
    p->n_small = p->mid_base;
    // rows of classes below kTinyClassEnd have at most kTinyDeg edges
    p->n_tiny = h[kTinyClassEnd] < (uint32_t)p->mid_base ? h[kTinyClassEnd] : p->mid_base;
    p->n_mid = p->hub_base - p->mid_base;
    p->n_hub = N_dst - p->hub_base;
    p->n_chunks = h[nclass + 1];
    *out = p;
    return MP_OK;
}

void mp_spmm_plan_free(mp_plan* plan) { delete plan; }

int mp_spmm_workspace(const mp_plan* plan, int reduce, size_t* bytes) {
    if (!bytes) return MP_ERR_NULL;
    if (!valid_reduce(reduce)) return MP_ERR_REDUCE;
    if (!plan || plan->n_chunks == 0) {
        *bytes = 0;
        return MP_OK;
    }
    const size_t cells = (size_t)plan->n_chunks * (size_t)plan->F;
    size_t b = 0;
    if (reduce & (MP_SUM | MP_MEAN)) b += align_up(cells * 4, 256);
    if (reduce & MP_MAX) b += 2 * align_up(cells * 4, 256);
    *bytes = b;
    return MP_OK;
}

int mp_spmm_multi_workspace(const mp_plan* plan, size_t* bytes) {
    if (!bytes) return MP_ERR_NULL;
    if (!plan || plan->n_chunks == 0) {
        *bytes = 0;
        return MP_OK;
    }
    // hub partials: sum, shifted sum and sum of squares, max and min values,
    // their positions
    *bytes = 7 * align_up((size_t)plan->n_chunks * (size_t)plan->F * 4, 256);
    return MP_OK;
}

int mp_spmm_multi(const mp_plan* plan, const void* rowptr, int rowptr_itype, const int32_t* col,
                  const float* w, const void* x, int x_dtype, int64_t N_src, int64_t N_dst,
                  int64_t F, int64_t ldx, int n_out, const mp_aggr_out* outs, void* ws,
                  size_t ws_bytes, void* stream) {
    if (N_dst > 0 && !col) return MP_ERR_NULL;
    return multi_impl(plan, rowptr, rowptr_itype, col, w, x, x_dtype, N_src, N_dst, F, ldx, n_out,
                      outs, ws, ws_bytes, as_stream(stream));
}

int mp_readout_multi(const mp_plan* plan, const void* ptr, int ptr_itype, const void* x,
                     int x_dtype, int64_t N_nodes, int64_t N_seg, int64_t F, int64_t ldx,
                     int n_out, const mp_aggr_out* outs, void* ws, size_t ws_bytes,
                     void* stream) {
    // segments of consecutive node rows: the CSR of the sorted batch vector,
    // whose column of position p is p itself
    return multi_impl(plan, ptr, ptr_itype, nullptr, nullptr, x, x_dtype, N_nodes, N_seg, F, ldx,
                      n_out, outs, ws, ws_bytes, as_stream(stream));
}

}  // extern "C"

// ---- mp_spmm_noalloc: hub partials in a static device array --------------------

// The workspace of mp_spmm_noalloc.  In host code its name is only the host
// stand-in of the device symbol: host code uses the address that
// hipGetSymbolAddress returns for the current device (each GPU holds its own
// copy), never the name.
static __device__ __align__(256) unsigned char scratch[MP_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up once per device.
int noalloc_scratch(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return MP_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return MP_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
            return MP_ERR_HIP;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return MP_OK;
}

}  // namespace

extern "C" {

int mp_spmm_noalloc(const mp_plan* plan, const void* rowptr, int rowptr_itype,
                    const int32_t* col, const float* w, const void* x, int x_dtype,
                    int64_t N_src, int64_t N_dst, int64_t F, int64_t ldx, int reduce, void* out,
                    int out_dtype, void* out_max, int max_dtype, int32_t* argout, void* stream) {
    if (N_dst > 0 && !col) return MP_ERR_NULL;
    size_t need = 0;
    int st = mp_spmm_workspace(plan, reduce, &need);
    if (st != MP_OK) return st;
    if (need > MP_NOALLOC_SCRATCH_BYTES) return MP_ERR_WORKSPACE;
    SpmmCall c{plan, rowptr, rowptr_itype, col, w, x, x_dtype, N_src, N_dst, F, ldx, reduce,
               out, out_dtype, out_max, max_dtype, argout, nullptr, 0};
    if (need > 0) {
        // every other argument is checked before the array is looked up; the
        // check only needs to know that a large enough workspace will come
        c.ws = &g_scratch_ptr;
        c.ws_bytes = MP_NOALLOC_SCRATCH_BYTES;
    }
    st = spmm_check(c);
    if (st != MP_OK) return st;
    if (need > 0 && N_dst > 0) {
        st = noalloc_scratch(&c.ws);
        if (st != MP_OK) return st;
    }
    return spmm_launch(c, as_stream(stream));
}

int mp_spmm(const mp_plan* plan, const void* rowptr, int rowptr_itype, const int32_t* col,
            const float* w, const void* x, int x_dtype, int64_t N_src, int64_t N_dst, int64_t F,
            int64_t ldx, int reduce, void* out, int out_dtype, void* out_max, int max_dtype,
            int32_t* argout, void* ws, size_t ws_bytes, void* stream) {
    if (N_dst > 0 && !col) return MP_ERR_NULL;
    SpmmCall c{plan, rowptr, rowptr_itype, col, w, x, x_dtype, N_src, N_dst, F, ldx, reduce,
               out, out_dtype, out_max, max_dtype, argout, ws, ws_bytes};
    const int st = spmm_check(c);
    return st != MP_OK ? st : spmm_launch(c, as_stream(stream));
}

// ---- backward ------------------------------------------------------------------

int mp_csr_transpose_workspace(int64_t E, int64_t N_src, int rowptrT_itype, int with_payload,
                               size_t* bytes) {
    if (!bytes) return MP_ERR_NULL;
    if (!valid_itype(rowptrT_itype)) return MP_ERR_DTYPE;
    int st = check_csr_sizes(E, N_src);
    if (st != MP_OK) return st;
    if (E == 0) {
        *bytes = 0;
        return MP_OK;
    }
    *bytes = align_up((size_t)E * 4, 256) + csr_layout(nullptr, E, N_src, with_payload ? 1 : 0).bytes;
    return MP_OK;
}

int mp_csr_transpose(const void* rowptr, int rowptr_itype, const int32_t* col, int64_t N_dst,
                     int64_t N_src, int64_t E, void* rowptrT, int rowptrT_itype, int32_t* colT,
                     int32_t* posT, const float* val_in, float* val_out, void* ws,
                     size_t ws_bytes, int32_t* status, void* stream) {
    if (!valid_itype(rowptr_itype) || !valid_itype(rowptrT_itype)) return MP_ERR_DTYPE;
    int st = check_csr_sizes(E, N_src);
    if (st != MP_OK) return st;
    if (N_dst < 1 || N_dst > INT32_MAX) return MP_ERR_SIZE;
    if (!rowptr || !rowptrT) return MP_ERR_NULL;
    if (E > 0 && (!col || !colT || !ws)) return MP_ERR_NULL;
    if (E > 0 && (val_in == nullptr) != (val_out == nullptr)) return MP_ERR_NULL;
    if ((uintptr_t)rowptr % (rowptr_itype == MP_I64 ? 8 : 4) ||
        (uintptr_t)rowptrT % (rowptrT_itype == MP_I64 ? 8 : 4) || (uintptr_t)status % 4)
        return MP_ERR_ALIGN;
    hipStream_t s = as_stream(stream);
    if (E == 0) {
        hipError_t e = launch_fill_rowptr_zero(N_src, rowptrT, rowptrT_itype == MP_I64, s);
        if (e == hipSuccess) e = launch_sort_status(nullptr, status, s);
        return hip_status(e);
    }
    size_t need = 0;
    mp_csr_transpose_workspace(E, N_src, rowptrT_itype, posT || val_out, &need);
    if (ws_bytes < need) return MP_ERR_WORKSPACE;
    // the forward CSR listed as COO (row of every position, col) is already in
    // position order, so a stable sort by col keeps forward order per source
    Carver c(ws);
    int32_t* row = c.take<int32_t>((size_t)E);
    if (launch_rows_of_edges(rowptr, rowptr_itype == MP_I64, N_dst, E, row, s) != hipSuccess)
        return MP_ERR_HIP;
    return coo_to_csr_impl(row, col, E, N_src, rowptrT, rowptrT_itype, colT, posT, val_in,
                           val_out, static_cast<char*>(ws) + c.off, ws_bytes - c.off, status, s);
}

// Extra workspace of mp_spmm_backward_x beyond the aggregation's own: the
// fp32 grad_out / in-degree table (mean) or the win masks (max).
size_t backward_x_extra(int64_t N_dst, int64_t E, int64_t F, int reduce) {
    if (reduce == MP_MEAN) return align_up((size_t)N_dst * (size_t)F * 4, 256);
    // (at least one position's words: the gather may load word 0 unread)
    if (reduce == MP_MAX)
        return align_up((size_t)(E > 0 ? E : 1) * (size_t)win_mask_words(F) * 4, 256);
    return 0;
}

int mp_spmm_backward_x_workspace(const mp_plan* planT, int64_t N_dst, int64_t E, int64_t F,
                                 int reduce, size_t* bytes) {
    if (!bytes) return MP_ERR_NULL;
    if (reduce != MP_SUM && reduce != MP_MEAN && reduce != MP_MAX) return MP_ERR_REDUCE;
    if (N_dst < 0 || N_dst > INT32_MAX || E < 0 || E > INT32_MAX || F < 1 || F > 65536)
        return MP_ERR_SIZE;
    size_t b = 0;
    int st = mp_spmm_workspace(planT, MP_SUM, &b);
    if (st != MP_OK) return st;
    const size_t extra = backward_x_extra(N_dst, E, F, reduce);
    if (extra) b = align_up(b, 256) + extra;
    *bytes = b;
    return MP_OK;
}

int mp_spmm_backward_x(const mp_plan* planT, const void* rowptrT, int rowptrT_itype,
                       const int32_t* colT, const int32_t* posT, const float* wT,
                       const void* rowptr, int rowptr_itype, const int32_t* argout,
                       const void* grad_out, int g_dtype, int64_t N_dst, int64_t N_src, int64_t E,
                       int64_t F, int reduce, void* grad_x, int out_dtype, void* ws,
                       size_t ws_bytes, void* stream) {
    if (reduce != MP_SUM && reduce != MP_MEAN && reduce != MP_MAX) return MP_ERR_REDUCE;
    const bool need_rp = reduce != MP_SUM;
    if (!valid_itype(rowptrT_itype) || !valid_dtype(g_dtype) || !valid_dtype(out_dtype))
        return MP_ERR_DTYPE;
    if (need_rp && !valid_itype(rowptr_itype)) return MP_ERR_DTYPE;
    if (N_src < 0 || N_src > INT32_MAX || N_dst < 0 || N_dst > INT32_MAX || E < 0 ||
        E > INT32_MAX || F < 1 || F > 65536)
        return MP_ERR_SIZE;
    if (!rowptrT) return MP_ERR_NULL;
    if (N_src > 0) {
        if (!colT || !grad_out || !grad_x) return MP_ERR_NULL;
        if (need_rp && !rowptr) return MP_ERR_NULL;
        if (reduce == MP_MAX && (!argout || !posT)) return MP_ERR_NULL;
    }
    int st = check_plan(planT, rowptrT, rowptrT_itype, N_src, F);
    if (st != MP_OK) return st;
    if (planT && planT->E != E) return MP_ERR_PLAN;
    const int eb = g_dtype == MP_BF16 ? 2 : 4;
    if ((uintptr_t)grad_out % eb || (uintptr_t)rowptrT % (rowptrT_itype == MP_I64 ? 8 : 4) ||
        (uintptr_t)colT % 4 || (uintptr_t)posT % 4 || (uintptr_t)wT % 4 ||
        (uintptr_t)argout % 4 || (uintptr_t)grad_x % (out_dtype == MP_BF16 ? 2 : 4) ||
        (need_rp && (uintptr_t)rowptr % (rowptr_itype == MP_I64 ? 8 : 4)))
        return MP_ERR_ALIGN;
    // workspace: the aggregation's hub partials, then the reduction's extra
    size_t part = 0;
    mp_spmm_workspace(planT, MP_SUM, &part);
    const size_t extra = backward_x_extra(N_dst, E, F, reduce);
    if (extra) {
        part = align_up(part, 256);
        if (ws_bytes < part + extra || !ws) return MP_ERR_WORKSPACE;
    }
    if (N_src == 0) return MP_OK;
    hipStream_t s = as_stream(stream);
    const void* table = grad_out;
    int t_dtype = g_dtype;
    void* spmm_ws = ws;
    size_t spmm_ws_bytes = extra ? part : ws_bytes;
    char* extra_buf = extra ? static_cast<char*>(ws) + part : nullptr;
    if (reduce == MP_MEAN) {
        // mean: a sum over the transposed CSR of grad_out / in-degree
        float* scaled = reinterpret_cast<float*>(extra_buf);
        if (launch_scale_inv_deg(grad_out, g_dtype == MP_BF16, rowptr, rowptr_itype == MP_I64,
                                 N_dst, F, scaled, s) != hipSuccess)
            return MP_ERR_HIP;
        table = scaled;
        t_dtype = MP_F32;
    }
    uint32_t* mbits = nullptr;
    if (reduce == MP_MAX) {
        // max: the win masks of every forward position, then a sum over the
        // transposed CSR that keeps the features each edge wins
        mbits = reinterpret_cast<uint32_t*>(extra_buf);
        if (E > 0 && launch_win_masks(rowptr, rowptr_itype == MP_I64, argout, N_dst, F, mbits,
                                      s) != hipSuccess)
            return MP_ERR_HIP;
    }
    Geometry g = make_geometry(F, t_dtype, (uintptr_t)table);
    SpmmParams P{};
    P.rowptr = rowptrT;
    P.rp64 = rowptrT_itype == MP_I64;
    P.col = colT;
    P.w = wT;
    P.n_tables = 1;
    P.table_ptr[0] = static_cast<const char*>(table);
    P.F = F;
    P.off32 = fits_off32(N_dst, F, t_dtype == MP_BF16 ? 2 : 4);
    P.reduce = MP_SUM;
    P.out = grad_x;
    P.out_bf16 = out_dtype == MP_BF16;
    P.vec_store = ((uintptr_t)grad_x % 16) == 0;
    if (reduce == MP_MAX) {
        P.ekey = posT;
        P.mbits = mbits;
        P.mw = win_mask_words(F);
    }
    return run_spmm(planT, P, g, t_dtype, N_src, spmm_ws, spmm_ws_bytes, s);
}

int mp_spmm_backward_w_workspace(int64_t E, size_t* bytes) {
    if (!bytes) return MP_ERR_NULL;
    if (E < 0 || E > INT32_MAX) return MP_ERR_SIZE;
    *bytes = E == 0 ? 0 : align_up((size_t)E * 4, 256);
    return MP_OK;
}

int mp_spmm_backward_w(const void* rowptr, int rowptr_itype, const int32_t* col, const void* x,
                       int x_dtype, const void* grad_out, int g_dtype, const int32_t* argout,
                       int64_t N_src, int64_t N_dst, int64_t E, int64_t F, int reduce,
                       float* grad_w, void* ws, size_t ws_bytes, void* stream) {
    if (reduce != MP_SUM && reduce != MP_MEAN && reduce != MP_MAX) return MP_ERR_REDUCE;
    if (!valid_itype(rowptr_itype) || !valid_dtype(x_dtype) || !valid_dtype(g_dtype))
        return MP_ERR_DTYPE;
    if (N_src < 0 || N_src > INT32_MAX || N_dst < 1 || N_dst > INT32_MAX || E < 0 ||
        E > INT32_MAX || F < 1 || F > 65536)
        return MP_ERR_SIZE;
    if (!rowptr) return MP_ERR_NULL;
    if (E == 0) return MP_OK;
    if (!col || !x || !grad_out || !grad_w || !ws) return MP_ERR_NULL;
    if (reduce == MP_MAX && !argout) return MP_ERR_NULL;
    if (ws_bytes < align_up((size_t)E * 4, 256)) return MP_ERR_WORKSPACE;
    const int ex = x_dtype == MP_BF16 ? 2 : 4, eg = g_dtype == MP_BF16 ? 2 : 4;
    if ((uintptr_t)rowptr % (rowptr_itype == MP_I64 ? 8 : 4) || (uintptr_t)col % 4 ||
        (uintptr_t)x % ex || (uintptr_t)grad_out % eg || (uintptr_t)argout % 4 ||
        (uintptr_t)grad_w % 4)
        return MP_ERR_ALIGN;
    hipStream_t s = as_stream(stream);
    int32_t* row = static_cast<int32_t*>(ws);
    if (launch_rows_of_edges(rowptr, rowptr_itype == MP_I64, N_dst, E, row, s) != hipSuccess)
        return MP_ERR_HIP;
    // one lane-chunk of EPL elements per table: x's vector width must keep
    // every table's chunk aligned (g and argout scaled to x's element size)
    uintptr_t al = (uintptr_t)x;
    al |= eg == ex ? (uintptr_t)grad_out : (eg > ex ? (uintptr_t)grad_out >> 1 : (uintptr_t)grad_out << 1);
    if (reduce == MP_MAX) al |= ex == 4 ? (uintptr_t)argout : (uintptr_t)argout >> 1;
    Geometry g = make_geometry(F, x_dtype, al);
    GradWParams P{};
    P.rowptr = rowptr;
    P.rp64 = rowptr_itype == MP_I64;
    P.col = col;
    P.row = row;
    P.x = x;
    P.g = grad_out;
    P.argout = argout;
    P.F = F;
    P.E = E;
    P.L = g.L;
    P.S = g.S;
    P.FT = g.FT;
    P.ltot = g.ltot;
    P.reduce = reduce;
    P.grad_w = grad_w;
    return hip_status(launch_spmm_grad_w(P, x_dtype, g_dtype, g.epl, s));
}

// ---- feature-table layout --------------------------------------------------------

int mp_copy_rows(const void* in, int64_t ld_in, void* out, int64_t ld_out, int64_t N, int64_t F,
                 int dtype, void* stream) {
    if (!valid_dtype(dtype)) return MP_ERR_DTYPE;
    if (N < 0 || F < 1 || ld_in < F || ld_out < F) return MP_ERR_SIZE;
    if (N == 0) return MP_OK;
    if (!in || !out) return MP_ERR_NULL;
    const int eb = dtype == MP_BF16 ? 2 : 4;
    if ((uintptr_t)in % eb || (uintptr_t)out % eb) return MP_ERR_ALIGN;
    return hip_status(launch_copy_rows(in, ld_in, out, ld_out, N, F, eb, as_stream(stream)));
}

// ---- edge-materialized messages ------------------------------------------------

int mp_csr_rows(const void* rowptr, int rowptr_itype, int64_t N_dst, int64_t E, int32_t* row,
                void* stream) {
    if (!valid_itype(rowptr_itype)) return MP_ERR_DTYPE;
    if (N_dst < 1 || N_dst > INT32_MAX || E < 0 || E > INT32_MAX) return MP_ERR_SIZE;
    if (!rowptr || (E > 0 && !row)) return MP_ERR_NULL;
    if ((uintptr_t)rowptr % (rowptr_itype == MP_I64 ? 8 : 4) || (uintptr_t)row % 4)
        return MP_ERR_ALIGN;
    return hip_status(launch_rows_of_edges(rowptr, rowptr_itype == MP_I64, N_dst, E, row,
                                           as_stream(stream)));
}

int mp_message_gather(const int32_t* idx, const float* w, const void* x, int x_dtype,
                      int64_t N_src, int64_t E, int64_t F, void* msg, int msg_dtype,
                      void* stream) {
    MessageGather a{};
    const int st = gather_check(idx, w, x, x_dtype, N_src, E, F, msg, msg_dtype, &a);
    return st != MP_OK ? st : hip_status(launch_message_gather(a, as_stream(stream)));
}

int mp_message_scale(const float* in, float* out, int64_t E, int64_t F, const float* mask,
                     const int32_t* idx, int64_t n_mask, void* stream) {
    if (E < 0 || E > INT32_MAX || F < 1 || F > 65536 || n_mask < 0) return MP_ERR_SIZE;
    if (E == 0) return MP_OK;
    if (!in || !out || !mask) return MP_ERR_NULL;
    if (!idx && n_mask < E) return MP_ERR_SIZE;
    if ((uintptr_t)in % 4 || (uintptr_t)out % 4 || (uintptr_t)mask % 4 || (uintptr_t)idx % 4)
        return MP_ERR_ALIGN;
    const uintptr_t ptrs[2] = {(uintptr_t)in, (uintptr_t)out};
    const int sizes[2] = {4, 4};
    const int epl = message_epl(F, ptrs, sizes, 2, 4);
    return hip_status(launch_message_scale(in, out, mask, idx, E, F, epl, as_stream(stream)));
}

int mp_message_aggregate(const mp_plan* plan, const void* rowptr, int rowptr_itype,
                         const void* msg, int msg_dtype, int64_t E, int64_t N_dst, int64_t F,
                         int reduce, void* out, int out_dtype, void* out_max, int max_dtype,
                         int32_t* argout, void* ws, size_t ws_bytes, void* stream) {
    if (E < 0 || E > INT32_MAX) return MP_ERR_SIZE;
    SpmmCall c{plan, rowptr, rowptr_itype, nullptr, nullptr, msg, msg_dtype, E, N_dst, F, F,
               reduce, out, out_dtype, out_max, max_dtype, argout, ws, ws_bytes};
    const int st = spmm_check(c);
    return st != MP_OK ? st : spmm_launch(c, as_stream(stream));
}

int mp_spmm_materialized(const mp_plan* plan, const void* rowptr, int rowptr_itype,
                         const int32_t* col, const float* w, const void* x, int x_dtype,
                         int64_t N_src, int64_t N_dst, int64_t E, int64_t F, void* msg,
                         int msg_dtype, mp_message_fn c, void* user, int reduce, void* out,
                         int out_dtype, void* out_max, int max_dtype, int32_t* argout, void* ws,
                         size_t ws_bytes, void* stream) {
    if (E < 0 || E > INT32_MAX) return MP_ERR_SIZE;
    if (plan && plan->E != E) return MP_ERR_PLAN;
    MessageGather a{};
    int st = gather_check(col, w, x, x_dtype, N_src, E, F, msg, msg_dtype, &a);
    if (st != MP_OK) return st;
    SpmmCall agg{plan, rowptr, rowptr_itype, nullptr, nullptr, msg, msg_dtype, E, N_dst, F, F,
                 reduce, out, out_dtype, out_max, max_dtype, argout, ws, ws_bytes};
    st = spmm_check(agg);
    if (st != MP_OK) return st;
    hipStream_t s = as_stream(stream);
    if (launch_message_gather(a, s) != hipSuccess) return MP_ERR_HIP;
    if (c && c(msg, msg_dtype, E, F, user, stream) != 0) return MP_ERR_CALLBACK;
    return spmm_launch(agg, s);
}

int mp_message_backward_workspace(int64_t E, size_t* bytes) {
    if (!bytes) return MP_ERR_NULL;
    if (E < 0 || E > INT32_MAX) return MP_ERR_SIZE;
    *bytes = 0;  // the kernels need none
    return MP_OK;
}

int mp_message_backward(const void* rowptr, int rowptr_itype, const int32_t* argout,
                        const void* grad_out, int g_dtype, int64_t N_dst, int64_t E, int64_t F,
                        int reduce, float* dmsg, void* ws, size_t ws_bytes, void* stream) {
    if (reduce != MP_SUM && reduce != MP_MEAN && reduce != MP_MAX) return MP_ERR_REDUCE;
    if (!valid_itype(rowptr_itype) || !valid_dtype(g_dtype)) return MP_ERR_DTYPE;
    if (N_dst < 1 || N_dst > INT32_MAX || E < 0 || E > INT32_MAX || F < 1 || F > 65536)
        return MP_ERR_SIZE;
    if (!rowptr) return MP_ERR_NULL;
    (void)ws;
    (void)ws_bytes;
    if (E == 0) return MP_OK;
    if (!grad_out || !dmsg) return MP_ERR_NULL;
    if (reduce == MP_MAX && !argout) return MP_ERR_NULL;
    const int eg = g_dtype == MP_BF16 ? 2 : 4;
    if ((uintptr_t)rowptr % (rowptr_itype == MP_I64 ? 8 : 4) || (uintptr_t)argout % 4 ||
        (uintptr_t)grad_out % eg || (uintptr_t)dmsg % 4)
        return MP_ERR_ALIGN;
    hipStream_t s = as_stream(stream);
    const uintptr_t ptrs[3] = {(uintptr_t)grad_out, (uintptr_t)dmsg,
                               reduce == MP_MAX ? (uintptr_t)argout : 0};
    const int sizes[3] = {eg, 4, 4};
    MessageBackward b{rowptr, rowptr_itype == MP_I64, argout, grad_out, g_dtype == MP_BF16,
                      N_dst, E, F, reduce, message_epl(F, ptrs, sizes, 3, 4), dmsg};
    return hip_status(launch_message_backward(b, s));
}

int mp_edge_dot(const void* a, int a_dtype, const void* b, int b_dtype, const int32_t* bidx,
                int64_t N_b, const int32_t* oidx, int64_t E, int64_t F, float* out,
                void* stream) {
    if (!valid_dtype(a_dtype) || !valid_dtype(b_dtype)) return MP_ERR_DTYPE;
    if (E < 0 || E > INT32_MAX || N_b < 0 || N_b > INT32_MAX || F < 1 || F > 65536)
        return MP_ERR_SIZE;
    if (!bidx && N_b < E) return MP_ERR_SIZE;
    if (E == 0) return MP_OK;
    if (!a || !b || !out) return MP_ERR_NULL;
    const int ea = a_dtype == MP_BF16 ? 2 : 4, eb = b_dtype == MP_BF16 ? 2 : 4;
    if ((uintptr_t)a % ea || (uintptr_t)b % eb || (uintptr_t)bidx % 4 || (uintptr_t)oidx % 4 ||
        (uintptr_t)out % 4)
        return MP_ERR_ALIGN;
    // one lane-chunk of EPL elements per table: b's vector width must keep a's
    // chunk aligned too (a's address scaled to b's element size)
    uintptr_t al = (uintptr_t)b;
    al |= ea == eb ? (uintptr_t)a : (ea > eb ? (uintptr_t)a >> 1 : (uintptr_t)a << 1);
    Geometry g = make_geometry(F, b_dtype, al);
    GradWParams P{};
    P.col = bidx;
    P.row = nullptr;
    P.x = b;
    P.g = a;
    P.F = F;
    P.E = E;
    P.L = g.L;
    P.S = g.S;
    P.FT = g.FT;
    P.ltot = g.ltot;
    P.reduce = MP_SUM;
    P.grad_w = out;
    P.oidx = oidx;
    return hip_status(launch_spmm_grad_w(P, b_dtype, a_dtype, g.epl, as_stream(stream)));
}

int mp_segment_matmul_workspace(int T, int64_t F, int64_t Fo, size_t* bytes) {
    if (!bytes) return MP_ERR_NULL;
    if (T < 1 || T > MP_MAX_TYPES) return MP_ERR_SIZE;
    int st = gmm_dims(F, Fo);
    if (st != MP_OK) return st;
    *bytes = align_up((size_t)T * (size_t)F * (size_t)Fo * 2, 256);  // W transposed
    return MP_OK;
}

int mp_segment_matmul(const int64_t* seg, int T, const void* x, const void* W, int64_t F,
                      int64_t Fo, void* out, int out_dtype, void* ws, size_t ws_bytes,
                      void* stream) {
    if (!valid_dtype(out_dtype)) return MP_ERR_DTYPE;
    GmmParams P{};
    int64_t N = 0;
    int st = gmm_segments(seg, T, P, &N);
    if (st != MP_OK) return st;
    st = gmm_dims(F, Fo);
    if (st != MP_OK) return st;
    if (!W || !ws || (N > 0 && (!x || !out))) return MP_ERR_NULL;
    if ((uintptr_t)x % 16 || (uintptr_t)W % 16 || (uintptr_t)ws % 16 ||
        (uintptr_t)out % (out_dtype == MP_BF16 ? 2 : 4))
        return MP_ERR_ALIGN;
    size_t need = 0;
    mp_segment_matmul_workspace(T, F, Fo, &need);
    if (ws_bytes < need) return MP_ERR_WORKSPACE;
    hipStream_t s = as_stream(stream);
    uint16_t* Wt = static_cast<uint16_t*>(ws);
    if (launch_transpose_w(static_cast<const uint16_t*>(W), T, F, Fo, Wt, s) != hipSuccess)
        return MP_ERR_HIP;
    const int64_t ntn = ceil_div(Fo, gmm_tile_cols());
    int64_t tiles = 0;
    for (int t = 0; t < T; ++t) {
        P.tile_off[t] = tiles;
        tiles += ceil_div(seg[t + 1] - seg[t], gmm_tile_rows()) * ntn;
    }
    P.tile_off[T] = tiles;
    P.A = static_cast<const uint16_t*>(x);
    P.lda = F;
    P.K = F;
    P.B = Wt;
    P.ldb = F;
    P.b_stride = Fo * F;
    P.N = Fo;
    P.C = out;
    P.ldc = Fo;
    P.c_bf16 = out_dtype == MP_BF16;
    return hip_status(launch_gmm_nt(P, tiles, s));
}

int mp_segment_matmul_backward_workspace(const int64_t* seg, int T, int64_t F, int64_t Fo,
                                         size_t* bytes) {
    if (!bytes) return MP_ERR_NULL;
    GmmParams P{};
    int64_t N = 0;
    int st = gmm_segments(seg, T, P, &N);
    if (st != MP_OK) return st;
    st = gmm_dims(F, Fo);
    if (st != MP_OK) return st;
    int64_t off[MP_MAX_TYPES + 1];
    const int64_t chunks = gmm_chunks(seg, T, off);
    *bytes = align_up((size_t)(chunks > 0 ? chunks : 1) * (size_t)F * (size_t)Fo * 4, 256);
    return MP_OK;
}

int mp_segment_matmul_backward(const int64_t* seg, int T, const void* x, const void* W,
                               const void* dout, int64_t F, int64_t Fo, void* dx, int dx_dtype,
                               float* dW, void* ws, size_t ws_bytes, void* stream) {
    if (!valid_dtype(dx_dtype)) return MP_ERR_DTYPE;
    GmmParams P{};
    int64_t N = 0;
    int st = gmm_segments(seg, T, P, &N);
    if (st != MP_OK) return st;
    st = gmm_dims(F, Fo);
    if (st != MP_OK) return st;
    if (!dx && !dW) return MP_ERR_NULL;
    if (N > 0 && !dout) return MP_ERR_NULL;
    if (dx && !W) return MP_ERR_NULL;
    if (dW && (!ws || (N > 0 && !x))) return MP_ERR_NULL;
    if ((uintptr_t)x % 16 || (uintptr_t)W % 16 || (uintptr_t)dout % 16 || (uintptr_t)ws % 16 ||
        (uintptr_t)dx % (dx_dtype == MP_BF16 ? 2 : 4) || (uintptr_t)dW % 4)
        return MP_ERR_ALIGN;
    hipStream_t s = as_stream(stream);
    if (dx && N > 0) {
        // dX = dOut W^T: W[t] stored [F][Fo] is already the transposed operand
        GmmParams Q = P;
        const int64_t ntn = ceil_div(F, gmm_tile_cols());
        int64_t tiles = 0;
        for (int t = 0; t < T; ++t) {
            Q.tile_off[t] = tiles;
            tiles += ceil_div(seg[t + 1] - seg[t], gmm_tile_rows()) * ntn;
        }
        Q.tile_off[T] = tiles;
        Q.A = static_cast<const uint16_t*>(dout);
        Q.lda = Fo;
        Q.K = Fo;
        Q.B = static_cast<const uint16_t*>(W);
        Q.ldb = Fo;
        Q.b_stride = F * Fo;
        Q.N = F;
        Q.C = dx;
        Q.ldc = F;
        Q.c_bf16 = dx_dtype == MP_BF16;
        if (launch_gmm_nt(Q, tiles, s) != hipSuccess) return MP_ERR_HIP;
    }
    if (dW) {
        size_t need = 0;
        mp_segment_matmul_backward_workspace(seg, T, F, Fo, &need);
        if (ws_bytes < need) return MP_ERR_WORKSPACE;
        const int64_t chunks = gmm_chunks(seg, T, P.tile_off);
        P.A = static_cast<const uint16_t*>(x);
        P.lda = F;
        P.B = static_cast<const uint16_t*>(dout);
        P.ldb = Fo;
        P.M = F;
        P.N = Fo;
        P.part = static_cast<float*>(ws);
        P.rows_per_chunk = kGmmRowsPerChunk;
        if (launch_gmm_weight_grad(P, chunks, dW, s) != hipSuccess) return MP_ERR_HIP;
    }
    return MP_OK;
}

// ---- heterogeneous ----------------------------------------------------------

static int hetero_check(int n_types, const int64_t* N_per_type, int n_rel, const mp_relation* rels,
                        int dst_type, int64_t* E_T, int64_t* offs, int64_t* N_rows) {
    if (!N_per_type || (n_rel > 0 && !rels)) return MP_ERR_NULL;
    const bool all = dst_type == MP_ALL_TYPES;
    if (n_types < 1 || n_types > MP_MAX_TYPES || n_rel < 0 ||
        (!all && (dst_type < 0 || dst_type >= n_types)))
        return MP_ERR_SIZE;
    int64_t tot = 0;
    for (int t = 0; t < n_types; ++t) {
        if (N_per_type[t] < 0) return MP_ERR_SIZE;
        offs[t] = tot;
        tot += N_per_type[t];
    }
    offs[n_types] = tot;
    if (tot > INT32_MAX) return MP_ERR_SIZE;
    int64_t e = 0;
    for (int r = 0; r < n_rel; ++r) {
        const mp_relation& R = rels[r];
        if (R.src_type < 0 || R.src_type >= n_types || R.dst_type < 0 || R.dst_type >= n_types ||
            R.E < 0)
            return MP_ERR_SIZE;
        if (all || R.dst_type == dst_type) {
            if (R.E > 0 && (!R.src || !R.dst)) return MP_ERR_NULL;
            e += R.E;
        }
    }
    if (e > INT32_MAX) return MP_ERR_SIZE;
    const int64_t rows = all ? tot : N_per_type[dst_type];
    if (rows < 1) return MP_ERR_SIZE;
    *E_T = e;
    *N_rows = rows;
    return MP_OK;
}

int mp_hetero_build_workspace(int n_types, const int64_t* N_per_type, int n_rel,
                              const mp_relation* rels, int dst_type, int rowptr_itype,
                              size_t* bytes) {
    if (!bytes) return MP_ERR_NULL;
    if (!valid_itype(rowptr_itype)) return MP_ERR_DTYPE;
    int64_t E_T = 0, N_rows = 0, offs[MP_MAX_TYPES + 1];
    int st = hetero_check(n_types, N_per_type, n_rel, rels, dst_type, &E_T, offs, &N_rows);
    if (st != MP_OK) return st;
    size_t cw = 0;
    st = mp_coo_to_csr_workspace(E_T, N_rows, rowptr_itype, 0, &cw);
    if (st != MP_OK) return st;
    *bytes = 2 * align_up((size_t)(E_T > 0 ? E_T : 1) * 4, 256) + cw;
    return MP_OK;
}

int mp_hetero_build(int n_types, const int64_t* N_per_type, int n_rel, const mp_relation* rels,
                    int dst_type, void* rowptr, int rowptr_itype, int32_t* col, void* ws,
                    size_t ws_bytes, int32_t* status, void* stream) {
    if (!valid_itype(rowptr_itype)) return MP_ERR_DTYPE;
    int64_t E_T = 0, N_rows = 0, offs[MP_MAX_TYPES + 1];
    int st = hetero_check(n_types, N_per_type, n_rel, rels, dst_type, &E_T, offs, &N_rows);
    if (st != MP_OK) return st;
    if (!rowptr || (E_T > 0 && (!col || !ws))) return MP_ERR_NULL;
    if ((uintptr_t)status % 4) return MP_ERR_ALIGN;
    size_t need = 0;
    st = mp_hetero_build_workspace(n_types, N_per_type, n_rel, rels, dst_type, rowptr_itype, &need);
    if (st != MP_OK) return st;
    if (ws_bytes < need) return MP_ERR_WORKSPACE;
    hipStream_t s = as_stream(stream);
    Carver c(ws);
    const size_t e = (size_t)(E_T > 0 ? E_T : 1);
    int32_t* src_g = c.take<int32_t>(e);
    int32_t* dst_c = c.take<int32_t>(e);
    int64_t off = 0;
    const bool all = dst_type == MP_ALL_TYPES;
    for (int r = 0; r < n_rel; ++r) {
        const mp_relation& R = rels[r];
        if ((!all && R.dst_type != dst_type) || R.E == 0) continue;
        // sources (and, over all types, destinations) as global node ids
        hipError_t he = launch_offset_copy(R.src, R.E, (int32_t)offs[R.src_type], src_g + off, s);
        if (he == hipSuccess)
            he = launch_offset_copy(R.dst, R.E, all ? (int32_t)offs[R.dst_type] : 0, dst_c + off, s);
        if (he != hipSuccess) return MP_ERR_HIP;
        off += R.E;
    }
    return coo_to_csr_impl(src_g, dst_c, E_T, N_rows, rowptr, rowptr_itype, col, nullptr,
                           nullptr, nullptr, c.base + c.off, ws_bytes - c.off, status, s);
}

int mp_hetero_spmm(int n_types, const int64_t* N_per_type, const void* const* x_per_type,
                   int x_dtype, int64_t F, int dst_type, const mp_plan* plan, const void* rowptr,
                   int rowptr_itype, const int32_t* col, int reduce, void* out, int out_dtype,
                   void* ws, size_t ws_bytes, void* stream) {
    if (reduce != MP_SUM) return MP_ERR_REDUCE;
    if (!valid_itype(rowptr_itype) || !valid_dtype(x_dtype) || !valid_dtype(out_dtype))
        return MP_ERR_DTYPE;
    int64_t E_T = 0, N_dst = 0, offs[MP_MAX_TYPES + 1];
    int st = hetero_check(n_types, N_per_type, 0, nullptr, dst_type, &E_T, offs, &N_dst);
    if (st != MP_OK) return st;
    if (F < 1 || F > 65536) return MP_ERR_SIZE;
    if (!x_per_type || !rowptr || !out || !col) return MP_ERR_NULL;
    st = check_plan(plan, rowptr, rowptr_itype, N_dst, F);
    if (st != MP_OK) return st;
    const int eb = x_dtype == MP_BF16 ? 2 : 4;
    uintptr_t xa = 0;
    for (int t = 0; t < n_types; ++t) {
        if (N_per_type[t] > 0 && !x_per_type[t]) return MP_ERR_NULL;
        if ((uintptr_t)x_per_type[t] % eb) return MP_ERR_ALIGN;
        xa |= (uintptr_t)x_per_type[t];
    }
    if ((uintptr_t)out % (out_dtype == MP_BF16 ? 2 : 4) || (uintptr_t)col % 4 ||
        (uintptr_t)rowptr % (rowptr_itype == MP_I64 ? 8 : 4))
        return MP_ERR_ALIGN;
    Geometry g = make_geometry(F, x_dtype, xa);
    SpmmParams P{};
    P.rowptr = rowptr;
    P.rp64 = rowptr_itype == MP_I64;
    P.col = col;
    P.w = nullptr;
    // tables laid out back to back in one allocation (one typed feature
    // tensor) are a single table indexed by global id
    bool contiguous = true;
    for (int t = 1; t < n_types; ++t)
        if ((uintptr_t)x_per_type[t] != (uintptr_t)x_per_type[0] + (uintptr_t)(offs[t] * F * eb))
            contiguous = false;
    P.n_tables = contiguous ? 1 : n_types;
    for (int t = 0; t < n_types; ++t) {
        P.table_ptr[t] = static_cast<const char*>(x_per_type[t]);
        P.table_off[t] = offs[t];
        P.voff[t] = ((int64_t)(uintptr_t)x_per_type[t] - (int64_t)(uintptr_t)x_per_type[0]) -
                    offs[t] * F * eb;
    }
    P.table_off[n_types] = offs[n_types];
    P.F = F;
    P.reduce = reduce;
    P.out = out;
    P.out_bf16 = out_dtype == MP_BF16;
    P.vec_store = ((uintptr_t)out % 16) == 0;
    return run_spmm(plan, P, g, x_dtype, N_dst, ws, ws_bytes, as_stream(stream));
}

int mp_probe_read(const void* p, int64_t bytes, uint32_t* sink, void* stream) {
    if (!p || !sink) return MP_ERR_NULL;
    if (bytes < 16 || bytes % 16) return MP_ERR_SIZE;
    if ((uintptr_t)p % 16 || (uintptr_t)sink % 4) return MP_ERR_ALIGN;
    return hip_status(launch_probe_read(p, bytes / 16, sink, as_stream(stream)));
}

int mp_probe_copy(const void* in, void* out, int64_t bytes, void* stream) {
    if (!in || !out) return MP_ERR_NULL;
    if (bytes < 16 || bytes % 16) return MP_ERR_SIZE;
    if ((uintptr_t)in % 16 || (uintptr_t)out % 16) return MP_ERR_ALIGN;
    return hip_status(launch_probe_copy(in, out, bytes / 16, as_stream(stream)));
}

int mp_probe_gather(const int32_t* idx, int64_t n, const void* table, int64_t stride_bytes,
                    int64_t row_bytes, uint32_t* sink, void* stream) {
    if (!sink || (n > 0 && (!idx || !table))) return MP_ERR_NULL;
    if (n < 0 || n > INT32_MAX || row_bytes < 16 || row_bytes > 1024 || row_bytes % 16 ||
        stride_bytes < row_bytes)
        return MP_ERR_SIZE;
    if ((uintptr_t)table % 16 || stride_bytes % 16 || (uintptr_t)idx % 4 || (uintptr_t)sink % 4)
        return MP_ERR_ALIGN;
    if (n == 0) return MP_OK;
    return hip_status(launch_probe_gather(idx, n, table, stride_bytes, (int)(row_bytes / 16), sink,
                                          as_stream(stream)));
}

int mp_probe_scatter(const void* in, const int32_t* dest, int64_t n, int64_t elem_bytes, void* out,
                     void* stream) {
    if (n > 0 && (!in || !dest || !out)) return MP_ERR_NULL;
    if (n < 0 || n > INT32_MAX || (elem_bytes != 4 && elem_bytes != 8)) return MP_ERR_SIZE;
    if ((uintptr_t)in % elem_bytes || (uintptr_t)out % elem_bytes || (uintptr_t)dest % 4)
        return MP_ERR_ALIGN;
    if (n == 0) return MP_OK;
    return hip_status(launch_probe_scatter(in, dest, n, (int)elem_bytes, out, as_stream(stream)));
}

int mp_validate_coo(const int32_t* src, const int32_t* dst, int64_t E, int64_t N_src,
                    int64_t N_dst, int64_t* d_count, void* stream) {
    if (!d_count || (E > 0 && (!src || !dst))) return MP_ERR_NULL;
    if (E < 0 || N_src < 0 || N_dst < 0) return MP_ERR_SIZE;
    return hip_status(launch_validate_coo(src, dst, E, N_src, N_dst, d_count, as_stream(stream)));
}

int mp_validate_sorted(const int32_t* dst, int64_t E, int64_t* d_count, void* stream) {
    if (!d_count || (E > 0 && !dst)) return MP_ERR_NULL;
    if (E < 0) return MP_ERR_SIZE;
    return hip_status(launch_validate_sorted(dst, E, d_count, as_stream(stream)));
}

int mp_validate_csr(const void* rowptr, int rowptr_itype, const int32_t* col, int64_t N_dst,
                    int64_t N_src, int64_t E, int64_t* d_count, void* stream) {
    if (!d_count || !rowptr || (E > 0 && !col)) return MP_ERR_NULL;
    if (!valid_itype(rowptr_itype)) return MP_ERR_DTYPE;
    if (E < 0 || N_src < 0 || N_dst < 0) return MP_ERR_SIZE;
    return hip_status(launch_validate_csr(rowptr, rowptr_itype == MP_I64, col, N_dst, N_src, E,
                                          d_count, as_stream(stream)));
}

}  // extern "C"
