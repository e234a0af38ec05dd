// Internal declarations shared by the HIP translation units of libmp.
// Nothing here is part of the public ABI (include/mp.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "mp.h"
#include "mp_probe.h"

namespace mp {

constexpr int kWave = 64;

// ---- radix sort geometry (COO -> CSR) ---------------------------------------
#ifndef MP_SORT_BLOCK
#define MP_SORT_BLOCK 1024
#endif
#ifndef MP_SORT_ITEMS
#define MP_SORT_ITEMS 16
#endif
constexpr int kSortBlock = MP_SORT_BLOCK;          // threads per workgroup
constexpr int kSortItems = MP_SORT_ITEMS;          // keys per thread
constexpr int kSortTile = kSortBlock * kSortItems; // keys per workgroup
constexpr int kSortMaxBits = 9;                    // digit width cap (512 buckets)

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Number of key bits for keys in [0, n): at least 1.
inline int key_bits(int64_t n) {
    int b = 1;
    while (b < 62 && (int64_t(1) << b) < n) ++b;
    return b;
}

// The digits of an LSD sort of `bits`-bit keys: as few passes of at most
// kSortMaxBits as cover the key, the bits split as evenly as possible, with
// the one-bit-wider digits on the last passes.  (The low digits of
// destination ids take all their values evenly, so a narrower digit there
// lengthens every digit run of a tile; the top bits of ids below N often
// take fewer values than their width allows.)
struct DigitPlan {
    int passes;
    int shift[4], width[4];
    int max_width;
};
inline DigitPlan digit_plan(int bits) {
    DigitPlan d{};
    d.passes = (bits + kSortMaxBits - 1) / kSortMaxBits;
    const int base = bits / d.passes, extra = bits % d.passes;
    for (int p = 0, s = 0; p < d.passes; ++p) {
        d.width[p] = base + (p >= d.passes - extra ? 1 : 0);
        d.shift[p] = s;
        s += d.width[p];
        if (d.width[p] > d.max_width) d.max_width = d.width[p];
    }
    return d;
}

// ---- exclusive scan of uint32 (scan.hip) -----------------------------------
constexpr int kScanBlock = 256;
constexpr int kScanItems = 16;
constexpr int kScanTile = kScanBlock * kScanItems;
size_t scan_workspace_bytes(int64_t n);
// In-place exclusive scan of data[0..n); returns the hipError of the launches.
// zero_below (device word, or nullptr): the caller guarantees data[i] = 0 for
// i < *zero_below, and the tiles wholly below it are skipped.
hipError_t exclusive_scan_u32(uint32_t* data, int64_t n, void* ws, hipStream_t s,
                              const uint32_t* zero_below = nullptr);

// ---- stable LSD radix sort, one sweep per digit (sort.hip) ----------------
//
// radix_sort_begin() computes the global digit histogram of every pass in one
// read of the keys (and clears the look-back descriptors); then each
// radix_sort_pass() ranks, offsets and scatters in a single kernel, getting
// the offsets of earlier tiles by decoupled look-back.
constexpr int kMaxPasses = 4;  // keys of at most 31 bits, digits of at most 9 bits

struct RadixScratch {
    uint64_t* desc;     // [tiles * R] look-back descriptors (R = 2^bits <= 512)
    uint32_t* gbase;    // [kMaxPasses * 512] global digit histogram -> exclusive starts
    uint32_t* counter;  // [kMaxPasses] dynamic tile ids
    uint32_t* err;      // nonzero: a look-back wait gave up (the result is invalid)
};
size_t radix_scratch_bytes(int64_t n);
RadixScratch radix_scratch(void* base, int64_t n);

struct RadixPass {
    const uint32_t* keys_in;  // [n]
    const int32_t* a_in;      // [n] or nullptr: payload a = element index
    const int32_t* b_in;      // [n] or nullptr: payload b = element index
    uint32_t* keys_out;       // [n] or nullptr
    int32_t* a_out;           // [n] or nullptr
    int32_t* b_out;           // [n] or nullptr
    // packed (key << 32 | payload a) words in place of keys_in and a_in
    // (kv_in) or keys_out and a_out (kv_out)
    const uint64_t* kv_in;    // [n] or nullptr
    uint64_t* kv_out;         // [n] or nullptr
    int64_t n;
    int pass, shift, bits;
    RadixScratch sc;
};
hipError_t radix_sort_begin(const uint32_t* keys, int64_t n, const DigitPlan& dp,
                            const RadixScratch& sc, hipStream_t s);
hipError_t radix_sort_pass(const RadixPass& p, hipStream_t s);

// Write the caller's status word (nullptr: nothing) from the error word of
// the sort that used sc (sc nullptr: no sort ran, MP_OK).
hipError_t launch_sort_status(const RadixScratch* sc, int32_t* status, hipStream_t s);
// rowptr of keys sorted by a radix sort whose error word is sort_err (the
// kernel does nothing when the sort failed); nullptr: no such word
hipError_t launch_rowptr_from_sorted(const uint32_t* keys, int64_t E, int64_t N, void* rowptr,
                                     int rp64, const uint32_t* sort_err, hipStream_t s);
// rowptr of keys sorted by the caller, by binary search (bounded work for
// any order of keys)
hipError_t launch_rowptr_by_search(const uint32_t* keys, int64_t E, int64_t N, void* rowptr,
                                   int rp64, hipStream_t s);
hipError_t launch_fill_rowptr_zero(int64_t N, void* rowptr, int rp64, hipStream_t s);
hipError_t launch_gather_f32(const float* in, const int32_t* idx, int64_t n, float* out,
                             hipStream_t s);
hipError_t launch_validate_coo(const int32_t* src, const int32_t* dst, int64_t E, int64_t N_src,
                               int64_t N_dst, int64_t* d_count, hipStream_t s);
hipError_t launch_validate_csr(const void* rowptr, int rp64, const int32_t* col, int64_t N_dst,
                               int64_t N_src, int64_t E, int64_t* d_count, hipStream_t s);
hipError_t launch_offset_copy(const int32_t* in, int64_t n, int32_t add, int32_t* out,
                              hipStream_t s);
hipError_t launch_iota(int64_t n, int32_t* out, hipStream_t s);
hipError_t launch_copy_f32(const float* in, int64_t n, float* out, hipStream_t s);
hipError_t launch_validate_sorted(const int32_t* dst, int64_t E, int64_t* d_count, hipStream_t s);

// ---- aggregation (spmm.hip) --------------------------------------------------
enum : int { kSum = MP_SUM, kMean = MP_MEAN, kMax = MP_MAX };

// Feature-row geometry of one launch: a row of F elements is cut into Ltot
// lane-chunks of EPL elements (one vector load each).  A wavefront holds S
// slots of L lanes; when Ltot > 64 the row is split into FT feature tiles of
// 64 lanes, each handled by its own wavefront.
struct Geometry {
    int elem_bytes;  // 4 (fp32) or 2 (bf16)
    int epl;         // elements per lane-chunk: vector bytes / elem_bytes
    int64_t ltot;    // lane-chunks per feature row
    int L, S, FT;    // lanes per slot, slots per wave, feature tiles
};
// x_align: the feature pointer value(s) and row strides in bytes, OR-ed
// (only the low bits matter).
Geometry make_geometry(int64_t F, int x_dtype, uintptr_t x_align);

// Degree classes of the plan (keys of the row sort).
constexpr int kSmallClasses = 16;       // class c < 16: small row, deg < 2^c ... see plan
constexpr int kClassMid = kSmallClasses;
constexpr int kClassHub = kSmallClasses + 1;
constexpr int kPlanClassBits = 5;       // 32 buckets (18 used)
constexpr int kMaxChunksPerHub = 2048;  // hub rows are split into <= this many chunks
constexpr int kTinyDeg = 7;             // rows of at most this many edges: tiny-row kernel
constexpr int kTinyClassEnd = 4;        // classes 0..3 (bit length <= 3) are tiny

struct SpmmParams {
    const void* rowptr;
    int rp64;
    const int32_t* col;  // nullptr: col[p] = p (a readout over contiguous segments)
    const float* w;
    int n_tables;
    const char* table_ptr[MP_MAX_TYPES];
    int64_t table_off[MP_MAX_TYPES + 1];
    // byte offset from table_ptr[0] such that global row c of table t starts
    // at table_ptr[0] + voff[t] + c * ldx * elem_bytes
    int64_t voff[MP_MAX_TYPES];
    int64_t F;
    int64_t ldx;  // row stride of the feature tables in elements (>= F)
    int off32;    // one table, all of it within 4 GiB of table_ptr[0]
    int L, S, FT;
    int64_t ltot;
    // work list (waves, in launch order): hub chunks, mid rows, small groups
    const int32_t* rowlist;  // nullptr: rows 0..N-1 all handled as "mid"
    const int32_t* rowbeg;   // [N] rowptr[rowlist[k]] (plan only)
    const int32_t* rowend;   // [N] rowptr[rowlist[k] + 1] (plan only)
    int64_t n_hub_waves, n_mid_waves, n_small_waves;
    int64_t hub_base, mid_base, small_base, n_small, n_hub;
    int64_t n_tiny;          // rowlist[0, n_tiny): rows for the tiny-row kernel
    const uint32_t* chunk_off;  // indexed by rowlist position
    int chunk_min;
    int reduce;
    void* out;
    int out_bf16;
    void* out_max;
    int max_bf16;
    int32_t* argout;
    int vec_store;  // 1: out, out_max and argout are 16-byte aligned
    // masked sum (gradient of max): edge t contributes feature f only where
    // bit f of the win mask of forward position ekey[t] is set (word
    // mbits[ekey[t] * mw + f / 32], bit f % 32); both nullptr otherwise.
    // mbits holds at least mw words even without edges: the kernels load
    // word 0 for invalid edges and discard it.
    const int32_t* ekey;
    const uint32_t* mbits;
    int64_t mw;
    // stats mode (stacked statistics from one gather): each non-null output
    // [N_dst, F] fp32 (arguments int32) is written
    int stats;
    float* o_sum;
    float* o_mean;
    float* o_max;
    int32_t* o_amax;
    float* o_min;
    int32_t* o_amin;
    float* o_var;
    float* o_std;
    float* part_sum;
    float* part_max;
    int32_t* part_arg;
    float* part_dsum;  // stats: hub partial sums of (m - K)
    float* part_sq;    // stats: hub partial sums of (m - K)^2
    float* part_min;
    int32_t* part_amin;
};

// ---- backward (backward.hip) -----------------------------------------------
struct GradWParams {
    const void* rowptr;
    int rp64;
    const int32_t* col;     // row of x read by position p; nullptr: p itself
    const int32_t* row;     // destination row of every CSR position; nullptr: p
    const void* x;          // [N_src, F]
    const void* g;          // [N_dst, F] gradient of the aggregation output
    const int32_t* argout;  // [N_dst, F] (max only)
    int64_t F, E;
    int L, S, FT;
    int64_t ltot;
    int reduce;             // exactly one of kSum, kMean, kMax
    float* grad_w;          // [E]
    const int32_t* oidx;    // nullptr, or grad_w[oidx[p]] receives position p's dot
};
hipError_t launch_rows_of_edges(const void* rowptr, int rp64, int64_t N, int64_t E, int32_t* row,
                                hipStream_t s);
hipError_t launch_scale_inv_deg(const void* g, int g_bf16, const void* rowptr, int rp64, int64_t N,
                                int64_t F, float* out, hipStream_t s);
hipError_t launch_spmm_grad_w(const GradWParams& p, int x_dtype, int g_dtype, int epl,
                              hipStream_t s);
// Win masks of the max aggregation: for every forward CSR position p, mw =
// ceil(F / 32) words whose bit f says argout[row(p), f] == p.
inline int64_t win_mask_words(int64_t F) { return (F + 31) / 32; }
hipError_t launch_win_masks(const void* rowptr, int rp64, const int32_t* argout, int64_t N,
                            int64_t F, uint32_t* bits, hipStream_t s);

// ---- segment matmul (gmm.hip) --------------------------------------------------
struct GmmParams {
    const uint16_t* A;  // bf16 rows of the left operand
    const uint16_t* B;  // bf16: per segment Bt[t] = B + t * b_stride (gmm_nt), or G (weight grad)
    void* C;            // output (gmm_nt)
    float* part;        // fp32 partial tiles (weight grad)
    int64_t lda, ldb, ldc, b_stride;
    int64_t M, N, K;    // gmm_nt: N columns, K inner; weight grad: M x N = F x Fo
    int T;
    int64_t seg[MP_MAX_TYPES + 1];       // row offsets of the segments
    int64_t tile_off[MP_MAX_TYPES + 1];  // first tile (gmm_nt) or chunk (weight grad) of each
    int64_t rows_per_chunk;
    int c_bf16;
};
hipError_t launch_gmm_nt(const GmmParams& p, int64_t tiles, hipStream_t s);
hipError_t launch_gmm_weight_grad(const GmmParams& p, int64_t chunks, float* dW, hipStream_t s);
hipError_t launch_transpose_w(const uint16_t* W, int64_t T, int64_t F, int64_t Fo, uint16_t* Wt,
                              hipStream_t s);
int64_t gmm_tile_rows();
int64_t gmm_tile_cols();

hipError_t launch_spmm(const SpmmParams& p, int x_dtype, int epl, hipStream_t s);
hipError_t launch_spmm_tiny(const SpmmParams& p, int x_dtype, int epl, hipStream_t s);
hipError_t launch_spmm_fixup(const SpmmParams& p, hipStream_t s);
hipError_t launch_plan_classes(const void* rowptr, int rp64, int64_t N, int64_t small_max,
                               int64_t hub_min, uint32_t* keys, hipStream_t s);
// per rowlist entry: row range and hub chunk count (nch[N] = 0)
hipError_t launch_plan_rows(const void* rowptr, int rp64, const int32_t* rowlist, int64_t N,
                            int64_t hub_min, int chunk_min, int32_t* rowbeg, int32_t* rowend,
                            uint32_t* nch, hipStream_t s);
// header[c] = first rowlist position of class c (c < nclass, from the class
// sort's exclusive digit starts), header[nclass] = N, header[nclass+1] = chunks
hipError_t launch_plan_header(const uint32_t* class_start, int nclass, const uint32_t* chunk_off,
                              int64_t N, const uint32_t* sort_err, uint32_t* header, hipStream_t s);

// ---- edge-materialized messages (messages.hip) ----------------------------------
struct MessageGather {
    const int32_t* idx;  // [E] row of x of every message
    const float* w;      // [E] or nullptr
    const void* x;       // [N_src, F]
    int x_bf16;
    void* msg;           // [E, F]: fp32, or bf16 (unweighted bf16 x, an exact copy)
    int msg_bf16;
    int64_t E, F;
    int epl;             // elements per lane-chunk (message_epl)
};
struct MessageBackward {
    const void* rowptr;
    int rp64;
    const int32_t* argout;  // [N_dst, F] (max only)
    const void* g;          // [N_dst, F] dL/dout
    int g_bf16;
    int64_t N, E, F;
    int reduce;             // exactly one of kSum, kMean, kMax
    int epl;
    float* dmsg;            // [E, F]
};
// Largest lane-chunk width in {max_epl, ..., 2, 1} that divides F, keeps each
// listed element size within 16 bytes per access and divides every pointer.
int message_epl(int64_t F, const uintptr_t* ptrs, const int* elem_bytes, int n, int max_epl);
hipError_t launch_message_gather(const MessageGather& a, hipStream_t s);
hipError_t launch_message_scale(const float* in, float* out, const float* mask,
                                const int32_t* idx, int64_t E, int64_t F, int epl, hipStream_t s);
hipError_t launch_message_backward(const MessageBackward& a, hipStream_t s);

// ---- feature-table layout (layout.hip) -------------------------------------------
// out[r, 0:F] = in[r, 0:F] for r < N, rows ld_in / ld_out elements apart.
hipError_t launch_copy_rows(const void* in, int64_t ld_in, void* out, int64_t ld_out, int64_t N,
                            int64_t F, int elem_bytes, hipStream_t s);

// ---- bandwidth probes (probe.hip) ---------------------------------------------
hipError_t launch_probe_read(const void* p, int64_t n16, uint32_t* sink, hipStream_t s);
hipError_t launch_probe_copy(const void* in, void* out, int64_t n16, hipStream_t s);
hipError_t launch_probe_scatter(const void* in, const int32_t* dest, int64_t n, int elem_bytes,
                                void* out, hipStream_t s);
hipError_t launch_probe_gather(const int32_t* idx, int64_t n, const void* table,
                               int64_t stride_bytes, int L, uint32_t* sink, hipStream_t s);

}  // namespace mp
