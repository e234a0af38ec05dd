// Segmented aggregation over the destination-major CSR (the AGGREGATION step
// of Eq. (1) in PyG 2.0, with message w * x[src]), and its degree-binned plan.
//
// Work is split three ways by in-degree (Sec. 2.2: a destination-sorted layout
// lets the aggregation run in parallel over rows), all inside ONE launch whose wavefronts take, in
// order: hub-row edge chunks (longest first), mid rows (one wavefront per
// row, its slots interleaving the row's edges), and groups of small rows (one
// slot of L lanes per row).  A slot is a group of L lanes that together hold
// one feature row: lane j loads elements [j*EPL, (j+1)*EPL) with one vector
// load, so a feature-row gather is one coalesced access per slot.  The column
// indices (and weights) of an iteration are loaded once, coalesced, by the
// first lanes and broadcast with cross-lane permutes.
//
// Determinism: every output element is reduced in an order fixed by the
// geometry (slot, unroll index, accumulator, then a fixed tree over
// accumulators and slots; hub chunks are combined in chunk order by a second
// kernel).  No floating-point atomics anywhere.
//
// Max: (value, CSR position) pairs; a later edge replaces the running pair
// only when strictly greater (a partial left empty, position -1, after
// receiving messages saw only -inf and takes its first edge), and pairs are combined preferring a non-empty pair, then the
// larger value, then the smaller position -- the first edge attaining the
// maximum, also for rows of -inf messages.  (NaN messages are outside the contract: the
// strided partials would not reproduce a sequential scan's answer.)
#include <type_traits>

#include "mp_internal.hpp"

namespace mp {
namespace {

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;
#ifndef MP_UNROLL
#define MP_UNROLL 8         // edges gathered per slot per iteration
#endif
#ifndef MP_MAX_PARTIALS
#define MP_MAX_PARTIALS 1   // independent (value, position) partials of a max-only call
#endif
constexpr int kUnroll = MP_UNROLL;
#ifndef MP_STATS_UNROLL
#define MP_STATS_UNROLL 8   // the same for the stacked statistics
#endif
#ifndef MP_STATS_WAVES
#define MP_STATS_WAVES 4    // stats mode: wavefronts per SIMD the registers must allow
#endif
#ifndef MP_SUM_WAVES
#define MP_SUM_WAVES 6      // unweighted bf16 sums with 32-bit row offsets: the same
#endif
// The masked sum (gradient of max) is bound by the latency of its dependent
// loads: 6 rows per slot step and 2 partials (96 registers, 5 wavefronts per
// SIMD) measured 8.89 -> 8.51 ms against 8 and 4 on the 124M-edge graph
#ifndef MP_MASKED_UNROLL
#define MP_MASKED_UNROLL 6  // rows per slot step of the masked sum
#endif
#ifndef MP_MASKED_PARTIALS
#define MP_MASKED_PARTIALS 2  // partial sums per element of the masked sum
#endif

// Kernel modes: the plain aggregation (sum/mean and/or max); the masked sum
// (the gradient of max); and the stacked statistics (sum, sum of squares, max
// and min with their positions, from one gather: sum, mean, max, min,
// variance and standard deviation).
constexpr int kModePlain = 0;
constexpr int kModeMasked = 1;
constexpr int kModeStats = 2;

// Edges per slot per iteration of a mode (array sizes of the gather loops).
// A max-only call keeps fewer rows in flight per slot (6 instead of 8, one
// (value, position) partial): the registers this frees buy a wavefront more
// per SIMD (bf16 features: 92 -> 76 registers, 5 -> 6 wavefronts; measured
// 5.40 -> 5.05 ms on the 124M-edge graph, fp32 9.27 -> 9.00 ms).
#ifndef MP_MAX_UNROLL
#define MP_MAX_UNROLL 6
#endif
template <int MODE, bool HS = true, bool HM = false>
constexpr int unroll_of() {
    return MODE == kModeStats    ? MP_STATS_UNROLL
           : MODE == kModeMasked ? MP_MASKED_UNROLL
           : (HM && !HS)         ? MP_MAX_UNROLL
                                 : kUnroll;
}

// ---- feature loads ----------------------------------------------------------

template <typename TX, int EPL>
struct RawVec;
template <> struct RawVec<float, 4> { using T = float4; };
template <> struct RawVec<float, 2> { using T = float2; };
template <> struct RawVec<float, 1> { using T = float; };
template <> struct RawVec<uint16_t, 8> { using T = uint4; };
template <> struct RawVec<uint16_t, 4> { using T = uint2; };
template <> struct RawVec<uint16_t, 2> { using T = uint32_t; };
template <> struct RawVec<uint16_t, 1> { using T = uint16_t; };

// Byte offset of element fe of row c from the table's base when the table is
// addressed with 32-bit offsets (O32): the table spans under 4 GiB, has at
// most 2^24 rows and a row stride under 2^24 bytes, so one full-rate 24-bit
// multiply-add forms the offset (a 32-bit multiply is a quarter-rate
// instruction, and the gathers issue one per row).
template <typename TX>
__device__ inline uint32_t off32(const SpmmParams& P, int32_t c, int64_t fe) {
    return __umul24((uint32_t)c, (uint32_t)P.ldx * (uint32_t)sizeof(TX)) +
           (uint32_t)fe * (uint32_t)sizeof(TX);
}

__device__ inline float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ inline float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

template <typename TX, int EPL>
__device__ inline void widen(const typename RawVec<TX, EPL>::T& r, float (&v)[EPL]) {
    if constexpr (std::is_same<TX, float>::value) {
        if constexpr (EPL == 4) { v[0] = r.x; v[1] = r.y; v[2] = r.z; v[3] = r.w; }
        else if constexpr (EPL == 2) { v[0] = r.x; v[1] = r.y; }
        else { v[0] = r; }
    } else {
        if constexpr (EPL == 8) {
            v[0] = bf16_lo(r.x); v[1] = bf16_hi(r.x); v[2] = bf16_lo(r.y); v[3] = bf16_hi(r.y);
            v[4] = bf16_lo(r.z); v[5] = bf16_hi(r.z); v[6] = bf16_lo(r.w); v[7] = bf16_hi(r.w);
        } else if constexpr (EPL == 4) {
            v[0] = bf16_lo(r.x); v[1] = bf16_hi(r.x); v[2] = bf16_lo(r.y); v[3] = bf16_hi(r.y);
        } else if constexpr (EPL == 2) {
            v[0] = bf16_lo(r); v[1] = bf16_hi(r);
        } else {
            v[0] = bf16_lo((uint32_t)r);
        }
    }
}

// The EPL bits of a win-mask word that belong to features [fe, fe + EPL) of
// a lane-chunk (EPL divides 32 and fe is a multiple of EPL, so they never
// straddle two words).
template <int EPL>
__device__ inline uint32_t lane_bits(uint32_t word, int64_t fe) {
    return (word >> (fe & 31)) & ((1u << EPL) - 1u);
}

// Keep only the features whose win bit is set (bit k of bits: element k).
template <int EPL>
__device__ inline void apply_mask(float (&v)[EPL], uint32_t bits) {
#pragma unroll
    for (int k = 0; k < EPL; ++k) v[k] = (bits >> k) & 1u ? v[k] : 0.f;
}

// fp32 -> bf16 bits, round to nearest even (finite values).
__device__ inline uint16_t to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ inline int64_t load_rp(const void* rp, int rp64, int64_t i) {
    return rp64 ? static_cast<const int64_t*>(rp)[i] : (int64_t) static_cast<const int32_t*>(rp)[i];
}

// Address of feature element `fe` of source row c (rows ldx elements apart).
// With NT > 1 tables (typed nodes; NT is a compile-time bound on n_tables), c
// is a global id and its table is the last one whose offset is <= c: one
// compare and one 64-bit select per table.  Addresses stay offsets from the
// first table's pointer, so loads remain global-memory loads.
template <typename TX, int NT>
__device__ inline const char* feat_addr(const SpmmParams& P, int32_t c, int64_t fe) {
    if constexpr (NT == 1) {
        return P.table_ptr[0] + ((int64_t)c * P.ldx + fe) * (int64_t)sizeof(TX);
    } else {
        int64_t vo = 0;
#pragma unroll
        for (int k = 1; k < NT; ++k)
            vo = (k < P.n_tables && c >= (int32_t)P.table_off[k]) ? P.voff[k] : vo;
        return P.table_ptr[0] + vo + ((int64_t)c * P.ldx + fe) * (int64_t)sizeof(TX);
    }
}

// One lane-chunk (EPL elements from fe) of source row c.  O32: the address is
// the table's base plus a 32-bit byte offset (one register per gathered row
// instead of two), which frees registers for more rows in flight.
template <typename TX, int EPL, int NT, bool O32>
__device__ inline typename RawVec<TX, EPL>::T load_chunk(const SpmmParams& P, int32_t c,
                                                          int64_t fe) {
    using R = typename RawVec<TX, EPL>::T;
    if constexpr (O32) {
        static_assert(NT == 1, "32-bit offsets address one table");
        return *reinterpret_cast<const R*>(P.table_ptr[0] + off32<TX>(P, c, fe));
    } else {
        return *reinterpret_cast<const R*>(feat_addr<TX, NT>(P, c, fe));
    }
}

// A wave-uniform 64-bit value held in scalar registers.
__device__ inline int64_t uniform64(int64_t x) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// a - b, never fused with the product that formed a: a weighted message is
// the rounded product fl(w * x), and a deviation fused into fma(w, x, -K)
// would belong to the unrounded one (a one-edge row would get a variance of
// the product's rounding error squared instead of 0)
__device__ inline float sub_rounded(float a, float b) {
#pragma clang fp contract(off)
    return a - b;
}

// Keep the pair with the larger value; on equal values the smaller position.
__device__ inline void max_merge(float& va, int32_t& ia, float vb, int32_t ib) {
    const bool take = (ib >= 0) && (ia < 0 || vb > va || (vb == va && ib < ia));
    va = take ? vb : va;
    ia = take ? ib : ia;
}

// Keep the pair with the smaller value; on equal values the smaller position.
__device__ inline void min_merge(float& va, int32_t& ia, float vb, int32_t ib) {
    const bool take = (ib >= 0) && (ia < 0 || vb < va || (vb == va && ib < ia));
    va = take ? vb : va;
    ia = take ? ib : ia;
}

// ---- accumulator state -------------------------------------------------------

// HX (stats mode, which also sets HS and HM): the (min, position) pair and,
// for the variance, the sum and the sum of squares of the messages minus a
// shift K, are kept as well.  K is the mean of a few messages of the row (the
// same K for every partial, slot and hub chunk of the row), so the shifted
// messages are small whenever the row's spread is small next to its mean,
// and  var = sum (m-K)^2 / deg - (sum (m-K) / deg)^2  subtracts terms of the
// size of the variance itself instead of E[m^2] and E[m]^2 (whose difference
// loses every digit when the mean is large against the spread).
template <int EPL, bool HS, bool HM, bool HX = false, int NA = (HM ? 2 : 4)>
struct Acc {
    static constexpr int A = NA;  // independent partial accumulators
    static constexpr int AX = HX ? NA : 1;
    float s[A][EPL];
    float m[A][EPL];
    int32_t i[A][EPL];
    float d[AX][EPL];  // sum of (m - K)
    float q[AX][EPL];  // sum of (m - K)^2
    float n[AX][EPL];
    int32_t j[AX][EPL];
    float K[HX ? EPL : 1];  // the row's shift

    __device__ inline void init() {
#pragma unroll
        for (int a = 0; a < A; ++a)
#pragma unroll
            for (int k = 0; k < EPL; ++k) {
                if constexpr (HS) s[a][k] = 0.f;
                // empty: position -1 (the first message always replaces it)
                if constexpr (HM) { m[a][k] = -__builtin_huge_valf(); i[a][k] = -1; }
                if constexpr (HX) {
                    d[a][k] = 0.f;
                    q[a][k] = 0.f;
                    n[a][k] = __builtin_huge_valf();
                    j[a][k] = -1;
                }
            }
#pragma unroll
        for (int k = 0; k < (HX ? EPL : 1); ++k) K[k] = 0.f;
    }
    // the shift: the mean of cnt >= 1 messages whose fp32 sum is t
    __device__ inline void set_shift(const float (&t)[EPL], int cnt) {
        if constexpr (HX) {
            const float c = (float)(cnt > 0 ? cnt : 1);
#pragma unroll
            for (int k = 0; k < EPL; ++k) K[k] = t[k] / c;
        }
    }
    // message values v (already weighted) of CSR position pos
    __device__ inline void add(int a, const float (&v)[EPL], int32_t pos) {
#pragma unroll
        for (int k = 0; k < EPL; ++k) {
            if constexpr (HS) s[a][k] += v[k];
            if constexpr (HM) {
                const bool take = v[k] > m[a][k];
                m[a][k] = take ? v[k] : m[a][k];
                i[a][k] = take ? pos : i[a][k];
            }
            if constexpr (HX) {
                const float dv = sub_rounded(v[k], K[k]);
                d[a][k] += dv;
                q[a][k] = __builtin_fmaf(dv, dv, q[a][k]);
                const bool take = v[k] < n[a][k];
                n[a][k] = take ? v[k] : n[a][k];
                j[a][k] = take ? pos : j[a][k];
            }
        }
    }
    // add() when ok, else no change, by selects instead of a branch: the sum
    // keeps its value, the shifted terms add an exact zero, and max / min take
    // nothing
    __device__ inline void add_masked(int a, const float (&v)[EPL], int32_t pos, bool ok) {
#pragma unroll
        for (int k = 0; k < EPL; ++k) {
            if constexpr (HS) s[a][k] = ok ? s[a][k] + v[k] : s[a][k];
            if constexpr (HM) {
                const bool take = ok && v[k] > m[a][k];
                m[a][k] = take ? v[k] : m[a][k];
                i[a][k] = take ? pos : i[a][k];
            }
            if constexpr (HX) {
                const float dv = ok ? sub_rounded(v[k], K[k]) : 0.f;
                d[a][k] += dv;
                q[a][k] = __builtin_fmaf(dv, dv, q[a][k]);
                const bool take = ok && v[k] < n[a][k];
                n[a][k] = take ? v[k] : n[a][k];
                j[a][k] = take ? pos : j[a][k];
            }
        }
    }
    // After the gather: a partial that received messages but is still empty
    // (position -1) saw only -inf messages (+inf for min), since any other
    // message replaces the initial -inf; its answer is its first message,
    // at position `first`.  (Testing for the empty pair on every message
    // instead costs a compare per element per edge: 6% on the max kernels.)
    __device__ inline void settle(int a, int32_t first, bool had) {
#pragma unroll
        for (int k = 0; k < EPL; ++k) {
            if constexpr (HM) i[a][k] = had && i[a][k] < 0 ? first : i[a][k];
            if constexpr (HX) j[a][k] = had && j[a][k] < 0 ? first : j[a][k];
        }
    }
    // fold the A partials into slot 0 (fixed tree)
    __device__ inline void fold() {
#pragma unroll
        for (int step = 1; step < A; step <<= 1)
#pragma unroll
            for (int a = 0; a + step < A; a += 2 * step)
#pragma unroll
                for (int k = 0; k < EPL; ++k) {
                    if constexpr (HS) s[a][k] += s[a + step][k];
                    if constexpr (HM) max_merge(m[a][k], i[a][k], m[a + step][k], i[a + step][k]);
                    if constexpr (HX) {
                        d[a][k] += d[a + step][k];
                        q[a][k] += q[a + step][k];
                        min_merge(n[a][k], j[a][k], n[a + step][k], j[a + step][k]);
                    }
                }
    }
    // fixed tree across the S slots of the wavefront (slot s at lanes s*L..);
    // the result lands in slot 0
    __device__ inline void reduce_slots(int S, int L, int slot, int lane) {
        for (int off = 1; off < S; off <<= 1) {
            const int src = lane + off * L;
            const bool use = (slot % (2 * off) == 0) && (slot + off < S);
#pragma unroll
            for (int k = 0; k < EPL; ++k) {
                if constexpr (HS) {
                    const float o = __shfl(s[0][k], src);
                    if (use) s[0][k] += o;
                }
                if constexpr (HM) {
                    const float om = __shfl(m[0][k], src);
                    const int32_t oi = __shfl(i[0][k], src);
                    if (use) max_merge(m[0][k], i[0][k], om, oi);
                }
                if constexpr (HX) {
                    const float od = __shfl(d[0][k], src);
                    const float oq = __shfl(q[0][k], src);
                    const float on = __shfl(n[0][k], src);
                    const int32_t oj = __shfl(j[0][k], src);
                    if (use) {
                        d[0][k] += od;
                        q[0][k] += oq;
                        min_merge(n[0][k], j[0][k], on, oj);
                    }
                }
            }
        }
    }
};

// Accumulator of a kernel instance.  Stats mode keeps seven running values
// per element in one partial for either feature dtype: the kernel is bound by
// its vector instructions, and a second partial costs registers and
// instructions (bf16 statistics: 8.79 -> 8.57 ms with one partial on the
// 124M-edge graph) without shortening anything that limits it.
template <typename TX, int EPL, bool HS, bool HM, int MODE>
using AccFor = Acc<EPL, HS, HM, MODE == kModeStats,
                   MODE == kModeStats    ? 1
                   : MODE == kModeMasked ? MP_MASKED_PARTIALS
                                         : (HM ? (HS ? 2 : MP_MAX_PARTIALS) : 4)>;

// Steps with missing edges accumulate by selects (no branches) for sums and
// fp32 max, whose kernels are bound by memory: the branches cost more than
// the work of the missing edges.  bf16 max, fused sum and max, and the
// statistics skip missing edges instead: the first and the last are bound by
// their vector instructions, which a select step spends on every edge slot
// (fp32 statistics measured 10.32 -> 10.72 ms with selects), and for fused
// sum and max the selects cost more registers than the branches.  Typed
// tables (short relation rows, mostly tail steps) skip them too.
template <typename TX, bool HS, bool HM>
constexpr bool kSelectTail = HS ? !HM : sizeof(TX) == 4;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Store EPL consecutive 4-byte values; 16-byte stores when allowed.
template <int EPL, typename T>
__device__ inline void store4(T* out, const T (&v)[EPL], bool vec) {
    static_assert(sizeof(T) == 4, "4-byte elements");
    if constexpr (EPL == 4 || EPL == 8) {
        if (vec) {
#pragma unroll
            for (int q = 0; q < EPL / 4; ++q) {
                u32x4 u;
                u.x = __builtin_bit_cast(uint32_t, v[4 * q + 0]);
                u.y = __builtin_bit_cast(uint32_t, v[4 * q + 1]);
                u.z = __builtin_bit_cast(uint32_t, v[4 * q + 2]);
                u.w = __builtin_bit_cast(uint32_t, v[4 * q + 3]);
                __builtin_nontemporal_store(u, reinterpret_cast<u32x4*>(out) + q);
            }
            return;
        }
    }
#pragma unroll
    for (int k = 0; k < EPL; ++k) out[k] = v[k];
}

// Store EPL consecutive bf16 values (as bits); 8/16-byte stores when allowed.
template <int EPL>
__device__ inline void store2(uint16_t* out, const uint16_t (&b)[EPL], bool vec) {
    if constexpr (EPL == 4 || EPL == 8) {
        if (vec) {
#pragma unroll
            for (int q = 0; q < EPL / 4; ++q) {
                u32x2 u;
                u.x = (uint32_t)b[4 * q + 0] | ((uint32_t)b[4 * q + 1] << 16);
                u.y = (uint32_t)b[4 * q + 2] | ((uint32_t)b[4 * q + 3] << 16);
                __builtin_nontemporal_store(u, reinterpret_cast<u32x2*>(out) + q);
            }
            return;
        }
    }
#pragma unroll
    for (int k = 0; k < EPL; ++k) out[k] = b[k];
}

template <int EPL>
__device__ inline void store_row(const SpmmParams& P, int64_t row, int64_t fe, int64_t deg,
                                 const float (&s)[EPL], const float (&m)[EPL],
                                 const int32_t (&idx)[EPL], bool hs, bool hm) {
    const int64_t o = row * P.F + fe;
    const bool vec = P.vec_store != 0;
    if (hs) {
        float v[EPL];
        const bool mean = (P.reduce & kMean) != 0;
        // one division per lane, then products (within 2 ulp of the quotient)
        const float inv = deg > 0 ? 1.f / (float)deg : 0.f;
#pragma unroll
        for (int k = 0; k < EPL; ++k) v[k] = mean ? s[k] * inv : s[k];
        if (P.out_bf16) {
            uint16_t b[EPL];
#pragma unroll
            for (int k = 0; k < EPL; ++k) b[k] = to_bf16(v[k]);
            store2<EPL>(static_cast<uint16_t*>(P.out) + o, b, vec);
        } else {
            store4<EPL>(static_cast<float*>(P.out) + o, v, vec);
        }
    }
    if (hm) {
        float mv[EPL];
#pragma unroll
        for (int k = 0; k < EPL; ++k) mv[k] = idx[k] < 0 ? 0.f : m[k];
        if (P.max_bf16) {
            // exact: the max is one of the bf16 inputs (unweighted only)
            uint16_t b[EPL];
#pragma unroll
            for (int k = 0; k < EPL; ++k) b[k] = (uint16_t)(__float_as_uint(mv[k]) >> 16);
            store2<EPL>(static_cast<uint16_t*>(P.out_max) + o, b, vec);
        } else {
            store4<EPL>(static_cast<float*>(P.out_max) + o, mv, vec);
        }
        store4<EPL>(P.argout + o, idx, vec);
    }
}

// Stats mode: write every requested statistic of a finished row (fp32).
// s is the plain sum; d and q the sums of (m - K) and (m - K)^2 for the
// row's shift K.  Variance is the population variance
// q / deg - (d / deg)^2 (shift-invariant), clamped at 0, with exact
// quotients (they cancel exactly on a row of equal messages, whose variance
// is then exactly 0); the mean is a product with one reciprocal of the
// degree per lane (within 2 ulp of the quotient).
template <int EPL>
__device__ inline void store_stats(const SpmmParams& P, int64_t row, int64_t fe, int64_t deg,
                                   const float (&s)[EPL], const float (&d)[EPL],
                                   const float (&q)[EPL], const float (&m)[EPL],
                                   const int32_t (&im)[EPL], const float (&n)[EPL],
                                   const int32_t (&in)[EPL], bool vec) {
    const int64_t o = row * P.F + fe;
    const float dv = (float)deg;
    const float inv = deg > 0 ? 1.f / dv : 0.f;
    float mean[EPL], var[EPL], sd[EPL], mx[EPL], mn[EPL];
#pragma unroll
    for (int k = 0; k < EPL; ++k) {
        mean[k] = s[k] * inv;
        const float c = d[k] / dv;
        const float v = deg > 0 ? q[k] / dv - c * c : 0.f;
        var[k] = v > 0.f ? v : 0.f;
        sd[k] = __builtin_sqrtf(var[k]);
        mx[k] = im[k] < 0 ? 0.f : m[k];
        mn[k] = in[k] < 0 ? 0.f : n[k];
    }
    if (P.o_sum) store4<EPL>(P.o_sum + o, s, vec);
    if (P.o_mean) store4<EPL>(P.o_mean + o, mean, vec);
    if (P.o_max) { store4<EPL>(P.o_max + o, mx, vec); store4<EPL>(P.o_amax + o, im, vec); }
    if (P.o_min) { store4<EPL>(P.o_min + o, mn, vec); store4<EPL>(P.o_amin + o, in, vec); }
    if (P.o_var) store4<EPL>(P.o_var + o, var, vec);
    if (P.o_std) store4<EPL>(P.o_std + o, sd, vec);
}

// Column of CSR position p: col[p], or p itself when col is absent (a
// readout over contiguous segments of nodes).
__device__ inline int32_t col_at(const SpmmParams& P, int64_t p) {
    return P.col ? __builtin_nontemporal_load(P.col + p) : (int32_t)p;
}

// Gather-and-accumulate over edges [e0, e1) with all S slots of the wavefront
// interleaved.  The column indices (and weights) of up to 64 edges are loaded
// once, coalesced, one per lane; each inner step then covers SU = S*U edges:
// slot s takes edges base + u*S + s (u < U), gets their columns by cross-lane
// permute, issues all U feature-row loads, and only then accumulates.  A step
// whose SU edges all exist (every step of a range but its last, and the
// first one of a row that sets the variance shift) runs without per-edge
// conditions: lanes that hold no feature chunk load the row's first chunk
// instead (a line the slot's first lane fetches anyway) and accumulate values
// that are never stored, so the step needs no exec-mask branches.  (The
// masked sum has its own pipelined variant below.)
template <typename TX, int EPL, bool HS, bool HM, int NT, bool W, int MODE, bool O32>
__device__ inline void wave_range(const SpmmParams& P,
                                  AccFor<TX, EPL, HS, HM, MODE>& acc, int64_t e0,
                                  int64_t e1, int lane, int slot, bool feat_ok, int64_t fe, int U,
                                  bool shift_first) {
    using R = typename RawVec<TX, EPL>::T;
    constexpr int A = AccFor<TX, EPL, HS, HM, MODE>::A;
    constexpr int UN = unroll_of<MODE, HS, HM>();
    const int S = P.S;
    const int j = lane - slot * P.L;  // lane within the slot
    const int SU = S * U;
    const int steps = kWave / SU;
    const int tile = steps * SU;
    e0 = uniform64(e0);
    e1 = uniform64(e1);
    const int64_t fe_ld = feat_ok ? fe : 0;
    const bool full_u = U == UN;
    constexpr bool SEL = kSelectTail<TX, HS, HM> && NT == 1;
    // column indices (and weights) of the tile at q, one per lane
    auto load_tile = [&](int64_t q, int32_t& c, float& w) {
        c = 0;
        w = 1.f;
        if (lane < tile && lane < e1 - q) {
            c = col_at(P, q + lane);
            if constexpr (W) w = __builtin_nontemporal_load(P.w + q + lane);
        }
    };
    // a step whose edges may run past the range (t >= rem) or with U < UN;
    // set_shift: the row's first step, whose slot-0 messages (edges u * S of
    // the row) give the row's shift, passed from slot 0's lane j to lane j of
    // every slot.  With one reduction (sum or max), loads are unconditional
    // (a lane's column is a valid row even for a missing edge: a column of the
    // tile, or 0 past its end) and missing edges accumulate nothing, by
    // selects; with both (fused sum and max, statistics) the selects cost more
    // registers than the branches, and missing edges are skipped.
    auto general_step = [&](int64_t p0, int32_t myc, float myw, int base, bool set_shift) {
        const int64_t rem = e1 - p0;
        bool ok[UN];
        R raw[UN];
#pragma unroll
        for (int u = 0; u < UN; ++u) {
            const int t = base + u * S + slot;
            ok[u] = feat_ok && (u < U) && (t < rem);
            // every lane takes part in the permute (an inactive source lane
            // would not supply its column)
            const int32_t c = __shfl(myc, t);
            if constexpr (SEL)
                raw[u] = load_chunk<TX, EPL, NT, O32>(P, c, fe_ld);
            else if (ok[u])
                raw[u] = load_chunk<TX, EPL, NT, O32>(P, c, fe);
        }
        if constexpr (MODE == kModeStats) {
            if (set_shift) {
                float t[EPL] = {};
                int cnt = 0;
#pragma unroll
                for (int u = 0; u < UN; ++u) {
                    float wt = 1.f;
                    if constexpr (W) wt = __shfl(myw, (u * S + slot) & (kWave - 1));
                    if (u < U && u * S < rem) ++cnt;
                    if (slot == 0 && ok[u]) {
                        float v[EPL];
                        widen<TX, EPL>(raw[u], v);
#pragma unroll
                        for (int k = 0; k < EPL; ++k) t[k] += W ? __fmul_rn(wt, v[k]) : v[k];
                    }
                }
#pragma unroll
                for (int k = 0; k < EPL; ++k) t[k] = __shfl(t[k], j);
                acc.set_shift(t, cnt);
            }
        }
#pragma unroll
        for (int u = 0; u < UN; ++u) {
            const int t = base + u * S + slot;
            float wt = 1.f;
            if constexpr (W) wt = __shfl(myw, t);
            if (SEL || ok[u]) {
                float v[EPL];
                widen<TX, EPL>(raw[u], v);
                if constexpr (W) {
#pragma unroll
                    for (int k = 0; k < EPL; ++k) v[k] = __fmul_rn(wt, v[k]);
                }
                if constexpr (SEL)
                    acc.add_masked(u % A, v, (int32_t)(p0 + t), ok[u]);
                else
                    acc.add(u % A, v, (int32_t)(p0 + t));
            }
        }
    };
    // a full step: every edge exists, no per-edge conditions; set_shift:
    // the row's first step, as in general_step
    auto full_step = [&](int64_t p0, int32_t myc, float myw, int base, bool set_shift) {
        R raw[UN];
#pragma unroll
        for (int u = 0; u < UN; ++u)
            raw[u] = load_chunk<TX, EPL, NT, O32>(P, __shfl(myc, base + u * S + slot), fe_ld);
        const int32_t pos = (int32_t)(p0 + base) + slot;
        // message u of this lane's slot (weighted)
        auto message = [&](int u, float (&v)[EPL]) {
            widen<TX, EPL>(raw[u], v);
            if constexpr (W) {
                const float wt = __shfl(myw, base + u * S + slot);
#pragma unroll
                for (int k = 0; k < EPL; ++k) v[k] = __fmul_rn(wt, v[k]);
            }
        };
        if constexpr (MODE == kModeStats) {
            if (set_shift) {
                float t[EPL] = {};
#pragma unroll
                for (int u = 0; u < UN; ++u) {
                    float v[EPL];
                    message(u, v);
#pragma unroll
                    for (int k = 0; k < EPL; ++k) t[k] += v[k];
                }
#pragma unroll
                for (int k = 0; k < EPL; ++k) t[k] = __shfl(t[k], j);
                acc.set_shift(t, UN);
            }
        }
#pragma unroll
        for (int u = 0; u < UN; ++u) {
            float v[EPL];
            message(u, v);
            acc.add(u % A, v, pos + u * S);
        }
    };
    int32_t myc;
    float myw;
    load_tile(e0, myc, myw);
    int st0 = 0;
    if constexpr (MODE == kModeStats) {
        if (shift_first && e0 < e1) {
            if (full_u && SU <= e1 - e0)
                full_step(e0, myc, myw, 0, true);
            else
                general_step(e0, myc, myw, 0, true);
            st0 = 1;
        }
    }
    for (int64_t p0 = e0; p0 < e1; p0 += tile) {
        const int64_t rem = e1 - p0;
        const int64_t nf = full_u ? rem / SU : 0;
        const int nfull = nf < steps ? (int)nf : steps;
        int st = st0;
        for (; st < nfull; ++st) full_step(p0, myc, myw, st * SU, false);
        for (; st < steps; ++st) {
            const int base = st * SU;
            if (base >= rem) break;
            general_step(p0, myc, myw, base, false);
        }
        st0 = 0;
        load_tile(p0 + tile, myc, myw);
    }
    if constexpr (HM) {
        // partial a's first message: edge u = a of the range's first step
#pragma unroll
        for (int a = 0; a < A; ++a)
            acc.settle(a, (int32_t)(e0 + a * S + slot), feat_ok && a < U && a * S + slot < e1 - e0);
    }
}

// The masked sum (gradient of max) over edges [e0, e1): the same edge
// schedule as wave_range, but a feature chunk is gathered only when its
// edge wins one of its features, which needs that edge's win-mask word
// first.  The mask words of a step are loaded cooperatively, one per lane
// (lane l takes word l % mww of the step's edge l / mww, where mww words
// starting at w_lo cover this wavefront's feature tile), and each lane picks
// the words it needs by cross-lane permute; U is capped so that a step's
// words fit the wavefront.  To keep one memory round trip per step, the
// loads run one step ahead: while step st gathers its chunks, the mask words
// of step st + 1 are in flight, and while a tile is gathered, the column
// indices and forward positions of the next tile are too.
template <typename TX, int EPL, bool HS, bool HM, int NT, bool W, bool O32>
__device__ inline void wave_range_masked(const SpmmParams& P,
                                         AccFor<TX, EPL, HS, HM, kModeMasked>& acc, int64_t e0,
                                         int64_t e1, int lane, int slot, bool feat_ok, int64_t fe,
                                         int64_t w_lo, int mww) {
    using R = typename RawVec<TX, EPL>::T;
    constexpr int A = AccFor<TX, EPL, HS, HM, kModeMasked>::A;
    constexpr int UN = unroll_of<kModeMasked>();
    if (e0 >= e1) return;
    const int S = P.S;
    int U = UN;
    if (S * U > kWave) U = kWave / S;
    if (S * U * mww > kWave) U = kWave / (S * mww);  // S * mww <= 64, so U >= 1
    const int SU = S * U;
    const int steps = kWave / SU;
    const int tile = steps * SU;
    const int me = lane / mww;          // edge of a step whose word this lane loads
    const int mq = lane - me * mww;     // and which of its words
    const int wi = (int)((fe >> 5) - w_lo);  // the word of an edge this lane needs
    // indices of the tile starting at q (lanes past its end keep 0 / -1)
    auto indices = [&](int64_t q, int32_t& c, int32_t& k, float& w) {
        c = 0;
        k = -1;
        w = 1.f;
        if (lane < tile && lane < e1 - q) {
            c = col_at(P, q + lane);
            if constexpr (W) w = __builtin_nontemporal_load(P.w + q + lane);
            k = __builtin_nontemporal_load(P.ekey + q + lane);
        }
    };
    // this lane's share of the mask words of the step at `base` of a tile
    // with `rem` edges left and forward positions in k: an unconditional load
    // (word 0 for a lane or edge past the end, never read)
    auto mword = [&](int32_t k, int base, int64_t rem) -> uint32_t {
        const int32_t key = __shfl(k, (base + me) & (kWave - 1));
        const bool v = me < SU && base + me < rem;
        return P.mbits[v ? (int64_t)key * P.mw + w_lo + mq : 0];
    };
    int32_t myc, myk;
    float myw;
    indices(e0, myc, myk, myw);
    uint32_t mcur = mword(myk, 0, e1 - e0);
    for (int64_t p0 = e0; p0 < e1; p0 += tile) {
        const int64_t rem = e1 - p0;
        const int64_t nxt = p0 + tile;
        int32_t nc, nk;
        float nw;
        indices(nxt, nc, nk, nw);
        for (int st = 0; st < steps; ++st) {
            const int base = st * SU;
            if (base >= rem) break;
            // row-chunk addresses: 32-bit byte offsets from the table base
            // when the table spans under 4 GiB (one register each)
            const char* addr[O32 ? 1 : UN];
            uint32_t off[O32 ? UN : 1];
            bool ok[UN];
            uint64_t bits = 0;  // EPL bits per edge of this lane's slot
#pragma unroll
            for (int u = 0; u < UN; ++u) {
                const int t = base + u * S + slot;
                const uint32_t w = __shfl(mcur, ((u * S + slot) * mww + wi) & (kWave - 1));
                const uint32_t b = feat_ok && u < U && t < rem ? lane_bits<EPL>(w, fe) : 0u;
                ok[u] = b != 0u;
                bits |= (uint64_t)b << (u * EPL);
                const int32_t c = __shfl(myc, t & (kWave - 1));
                if constexpr (O32)
                    off[u] = off32<TX>(P, c, fe);
                else
                    addr[u] = feat_addr<TX, NT>(P, c, fe);
            }
            // the next step's words: of this tile, or the first step of the
            // next one
            const uint32_t mnext = st + 1 < steps && base + SU < rem ? mword(myk, base + SU, rem)
                                                                     : mword(nk, 0, e1 - nxt);
            R raw[UN];
#pragma unroll
            for (int u = 0; u < UN; ++u) {
                if (ok[u]) {
                    if constexpr (O32)
                        raw[u] = *reinterpret_cast<const R*>(P.table_ptr[0] + off[u]);
                    else
                        raw[u] = *reinterpret_cast<const R*>(addr[u]);
                }
            }
#pragma unroll
            for (int u = 0; u < UN; ++u) {
                const int t = base + u * S + slot;
                float wt = 1.f;
                if constexpr (W) wt = __shfl(myw, t & (kWave - 1));
                if (ok[u]) {
                    float v[EPL];
                    widen<TX, EPL>(raw[u], v);
                    if constexpr (W) {
#pragma unroll
                        for (int k = 0; k < EPL; ++k) v[k] = __fmul_rn(wt, v[k]);
                    }
                    apply_mask<EPL>(v, (uint32_t)(bits >> (u * EPL)));
                    acc.add(u % A, v, (int32_t)(p0 + t));
                }
            }
            mcur = mnext;
        }
        myc = nc;
        myk = nk;
        myw = nw;
    }
}

// The masked sum over small rows (one slot per row, as in slot_row): an
// iteration covers U edges of every slot's row, U capped so that the
// iteration's win-mask words fit the wavefront one per lane (lane l takes
// word l % mww of edge u of slot s, l / mww = u * S + s), shared by
// cross-lane permute as in wave_range_masked.  Loads run ahead: the indices
// two iterations ahead and the mask words one iteration ahead are in flight
// while an iteration gathers its chunks.
template <typename TX, int EPL, bool HS, bool HM, int NT, bool W, bool O32>
__device__ inline void slot_row_masked(const SpmmParams& P,
                                       AccFor<TX, EPL, HS, HM, kModeMasked>& acc, int64_t e0,
                                       int32_t my_n, int32_t max_n, int lane, int slot, int j,
                                       bool feat_ok, int64_t fe, int64_t w_lo, int mww) {
    using R = typename RawVec<TX, EPL>::T;
    constexpr int A = AccFor<TX, EPL, HS, HM, kModeMasked>::A;
    constexpr int UN = unroll_of<kModeMasked>();
    if (max_n <= 0) return;
    const int L = P.L, S = P.S;
    int U = UN;
    if (U > L) U = L;  // the first U lanes of a slot load its indices
    if (S * U * mww > kWave) U = kWave / (S * mww);  // S * mww <= 64, so U >= 1
    const int me = lane / mww;  // edge of an iteration whose word this lane loads
    const int mq = lane - me * mww;
    const int mu = me / S, ms = me - mu * S;
    const bool mload = me < S * U;
    const int32_t n_ms = __shfl(my_n, (ms * L) & (kWave - 1));  // row length of slot ms
    const int wi = (int)((fe >> 5) - w_lo);
    // lanes j < U of each slot: column, weight and forward position of edge
    // it + j of the slot's row
    auto indices = [&](int32_t it, int32_t& c, int32_t& k, float& w) {
        c = 0;
        k = -1;
        w = 1.f;
        if (slot < S && j < U && it + j < my_n) {
            c = col_at(P, e0 + it + j);
            if constexpr (W) w = __builtin_nontemporal_load(P.w + e0 + it + j);
            k = __builtin_nontemporal_load(P.ekey + e0 + it + j);
        }
    };
    // this lane's share of the mask words of iteration it (unconditional
    // load: word 0 for a lane or edge past the end, never read)
    auto mword = [&](int32_t it, int32_t k) -> uint32_t {
        const int32_t key = __shfl(k, (ms * L + mu) & (kWave - 1));
        const bool v = mload && it + mu < n_ms;
        return P.mbits[v ? (int64_t)key * P.mw + w_lo + mq : 0];
    };
    int32_t c0, k0, c1, k1;
    float w0, w1;
    indices(0, c0, k0, w0);
    indices(U, c1, k1, w1);
    uint32_t mcur = mword(0, k0);
    for (int32_t it = 0; it < max_n; it += U) {
        const char* addr[O32 ? 1 : UN];
        uint32_t off[O32 ? UN : 1];
        bool ok[UN];
        uint64_t bits = 0;  // EPL bits per edge of this lane's slot
#pragma unroll
        for (int u = 0; u < UN; ++u) {
            const uint32_t w = __shfl(mcur, ((u * S + slot) * mww + wi) & (kWave - 1));
            const uint32_t b = feat_ok && u < U && it + u < my_n ? lane_bits<EPL>(w, fe) : 0u;
            ok[u] = b != 0u;
            bits |= (uint64_t)b << (u * EPL);
            const int32_t c = __shfl(c0, (slot * L + u) & (kWave - 1));
            if constexpr (O32)
                off[u] = off32<TX>(P, c, fe);
            else
                addr[u] = feat_addr<TX, NT>(P, c, fe);
        }
        // the next iteration's words (its indices arrived during this one),
        // then the indices of the iteration after it
        const uint32_t mnext = mword(it + U, k1);
        int32_t c2, k2;
        float w2;
        indices(it + 2 * U, c2, k2, w2);
        R raw[UN];
#pragma unroll
        for (int u = 0; u < UN; ++u) {
            if (ok[u]) {
                if constexpr (O32)
                    raw[u] = *reinterpret_cast<const R*>(P.table_ptr[0] + off[u]);
                else
                    raw[u] = *reinterpret_cast<const R*>(addr[u]);
            }
        }
#pragma unroll
        for (int u = 0; u < UN; ++u) {
            float wt = 1.f;
            if constexpr (W) wt = __shfl(w0, (slot * L + u) & (kWave - 1));
            if (ok[u]) {
                float v[EPL];
                widen<TX, EPL>(raw[u], v);
                if constexpr (W) {
#pragma unroll
                    for (int k = 0; k < EPL; ++k) v[k] = __fmul_rn(wt, v[k]);
                }
                apply_mask<EPL>(v, (uint32_t)(bits >> (u * EPL)));
                acc.add(u % A, v, (int32_t)(e0 + it + u));
            }
        }
        mcur = mnext;
        c0 = c1;
        k0 = k1;
        w0 = w1;
        c1 = c2;
        k1 = k2;
        w1 = w2;
    }
}

// One slot per row: every slot walks its own row's edges, U at a time.
// COOP: the slot has at least U lanes, which load its next U columns
// together; otherwise each lane loads the columns itself.  With COOP, the
// iterations in which every slot's row still has U edges (min_n: the
// shortest row of the wavefront) run without per-edge conditions, as the full
// steps of wave_range do.  (The masked sum has its own pipelined variant
// above.)
template <typename TX, int EPL, bool HS, bool HM, int NT, bool W, int MODE, bool COOP, bool O32>
__device__ inline void slot_row(const SpmmParams& P, AccFor<TX, EPL, HS, HM, MODE>& acc,
                                int64_t e0, int32_t my_n, int32_t max_n, int32_t min_n,
                                int slot, int j, bool feat_ok, int64_t fe) {
    using R = typename RawVec<TX, EPL>::T;
    constexpr int A = AccFor<TX, EPL, HS, HM, MODE>::A;
    constexpr int UN = unroll_of<MODE, HS, HM>();
    const int L = P.L;
    const int64_t fe_ld = feat_ok ? fe : 0;
    constexpr bool SEL = kSelectTail<TX, HS, HM> && NT == 1;
    // an iteration in which a slot's row may end (it + u >= my_n); set_shift:
    // the first one, whose messages give the row's shift.  With one
    // reduction, loads are unconditional (a missing edge's column is 0, a
    // valid row) and missing edges accumulate nothing, by selects; with both,
    // missing edges are skipped (as in wave_range).
    auto general_iter = [&](int32_t it, bool set_shift) {
        int32_t cc[UN];
        bool ok[UN];
        float wt[UN];
        if constexpr (COOP) {
            int32_t myc = 0;
            float myw = 1.f;
            if (j < UN && it + j < my_n) {
                myc = col_at(P, e0 + it + j);
                if constexpr (W) myw = __builtin_nontemporal_load(P.w + e0 + it + j);
            }
#pragma unroll
            for (int u = 0; u < UN; ++u) {
                const int srcl = slot * L + u;
                cc[u] = __shfl(myc, srcl);
                wt[u] = 1.f;
                if constexpr (W) wt[u] = __shfl(myw, srcl);
                ok[u] = feat_ok && (it + u < my_n);
            }
        } else {
#pragma unroll
            for (int u = 0; u < UN; ++u) {
                ok[u] = feat_ok && (it + u < my_n);
                cc[u] = ok[u] ? (P.col ? P.col[e0 + it + u] : (int32_t)(e0 + it + u)) : 0;
                wt[u] = 1.f;
                if constexpr (W) wt[u] = ok[u] ? P.w[e0 + it + u] : 1.f;
            }
        }
        R raw[UN];
#pragma unroll
        for (int u = 0; u < UN; ++u) {
            if constexpr (SEL)
                raw[u] = load_chunk<TX, EPL, NT, O32>(P, cc[u], fe_ld);
            else if (ok[u])
                raw[u] = load_chunk<TX, EPL, NT, O32>(P, cc[u], fe);
        }
        if constexpr (MODE == kModeStats) {
            if (set_shift) {  // the mean of the row's first UN messages
                float t[EPL] = {};
#pragma unroll
                for (int u = 0; u < UN; ++u) {
                    if (ok[u]) {
                        float v[EPL];
                        widen<TX, EPL>(raw[u], v);
#pragma unroll
                        for (int k = 0; k < EPL; ++k) t[k] += W ? __fmul_rn(wt[u], v[k]) : v[k];
                    }
                }
                acc.set_shift(t, my_n < UN ? my_n : UN);
            }
        }
#pragma unroll
        for (int u = 0; u < UN; ++u) {
            if (SEL || ok[u]) {
                float v[EPL];
                widen<TX, EPL>(raw[u], v);
                if constexpr (W) {
#pragma unroll
                    for (int k = 0; k < EPL; ++k) v[k] = __fmul_rn(wt[u], v[k]);
                }
                if constexpr (SEL)
                    acc.add_masked(u % A, v, (int32_t)(e0 + it + u), ok[u]);
                else
                    acc.add(u % A, v, (int32_t)(e0 + it + u));
            }
        }
    };
    // every slot's row has UN more edges: no per-edge conditions (COOP);
    // set_shift: the first iteration, as in general_iter
    auto full_iter = [&](int32_t it, bool set_shift) {
        int32_t myc = 0;
        float myw = 1.f;
        if (j < UN && it + j < my_n) {
            myc = col_at(P, e0 + it + j);
            if constexpr (W) myw = __builtin_nontemporal_load(P.w + e0 + it + j);
        }
        R raw[UN];
#pragma unroll
        for (int u = 0; u < UN; ++u)
            raw[u] = load_chunk<TX, EPL, NT, O32>(P, __shfl(myc, slot * L + u), fe_ld);
        const int32_t pos = (int32_t)(e0 + it);
        // message u of this lane's row (weighted)
        auto message = [&](int u, float (&v)[EPL]) {
            widen<TX, EPL>(raw[u], v);
            if constexpr (W) {
                const float wt = __shfl(myw, slot * L + u);
#pragma unroll
                for (int k = 0; k < EPL; ++k) v[k] = __fmul_rn(wt, v[k]);
            }
        };
        if constexpr (MODE == kModeStats) {
            if (set_shift) {
                float t[EPL] = {};
#pragma unroll
                for (int u = 0; u < UN; ++u) {
                    float v[EPL];
                    message(u, v);
#pragma unroll
                    for (int k = 0; k < EPL; ++k) t[k] += v[k];
                }
                acc.set_shift(t, UN);
            }
        }
#pragma unroll
        for (int u = 0; u < UN; ++u) {
            float v[EPL];
            message(u, v);
            acc.add(u % A, v, pos + u);
        }
    };
    int32_t it = 0;
    if constexpr (MODE == kModeStats) {
        if (COOP && UN <= min_n)
            full_iter(0, true);
        else
            general_iter(0, true);
        it = UN;
    }
    if constexpr (COOP) {
        for (; it + UN <= min_n; it += UN) full_iter(it, false);
    }
    for (; it < max_n; it += UN) general_iter(it, false);
    if constexpr (HM) {
#pragma unroll
        for (int a = 0; a < A; ++a) acc.settle(a, (int32_t)(e0 + a), feat_ok && a < my_n);
    }
}

// The shift of a hub row for the variance: the mean of the row's first
// min(deg, 8) messages, summed in edge order.  Every wavefront of every chunk
// of the row loads the same messages and so computes the identical shift
// (one extra pair of dependent loads per hub chunk, which spans 32 or more
// steps).
template <typename TX, int EPL, int NT, bool W, bool O32>
__device__ inline void hub_shift(const SpmmParams& P, int64_t r0, int64_t deg, bool feat_ok,
                                 int64_t fe, float (&t)[EPL], int& cnt) {
    using R = typename RawVec<TX, EPL>::T;
    constexpr int KS = 8;
    cnt = deg < KS ? (int)deg : KS;
    int32_t c[KS];
    float w[KS];
#pragma unroll
    for (int u = 0; u < KS; ++u) {
        c[u] = u < cnt ? col_at(P, r0 + u) : 0;
        w[u] = 1.f;
        if constexpr (W) w[u] = u < cnt ? P.w[r0 + u] : 1.f;
    }
    R raw[KS];
#pragma unroll
    for (int u = 0; u < KS; ++u)
        if (feat_ok && u < cnt)
            raw[u] = load_chunk<TX, EPL, NT, O32>(P, c[u], fe);
#pragma unroll
    for (int k = 0; k < EPL; ++k) t[k] = 0.f;
#pragma unroll
    for (int u = 0; u < KS; ++u) {
        if (feat_ok && u < cnt) {
            float v[EPL];
            widen<TX, EPL>(raw[u], v);
#pragma unroll
            for (int k = 0; k < EPL; ++k) t[k] += W ? __fmul_rn(w[u], v[k]) : v[k];
        }
    }
}

// Stats mode keeps seven running values per element.  Where they fit
// (unweighted, 32-bit row offsets, at most 4 elements per lane in one
// partial), the register budget is capped so that MP_STATS_WAVES wavefronts
// fit a SIMD without spilling: the gathers need wavefronts in flight more
// than the scheduler needs the registers.  (Eight bf16 elements per lane
// would spill under that cap.)  Unweighted bf16 sums of up to 4 elements per
// lane with 32-bit row offsets are capped likewise (MP_SUM_WAVES).
template <typename TX, int EPL, bool HS, bool HM, bool W, int MODE, bool O32>
constexpr int waves_hint() {
    if (MODE == kModeStats && !W && O32 && AccFor<TX, EPL, HS, HM, MODE>::A * EPL <= 4)
        return MP_STATS_WAVES;
    if (MODE == kModePlain && HS && !HM && !W && O32 && sizeof(TX) == 2 && EPL <= 4)
        return MP_SUM_WAVES;
    return 1;
}

template <typename TX, int EPL, bool HS, bool HM, int NT, bool W, int MODE, bool O32 = false>
__global__ __launch_bounds__(kBlock)
__attribute__((amdgpu_waves_per_eu(waves_hint<TX, EPL, HS, HM, W, MODE, O32>())))
void spmm_main(SpmmParams P) {
    constexpr bool HX = MODE == kModeStats;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave)) +
                       (int64_t)blockIdx.x * kWavesPerBlock;
    const int L = P.L, S = P.S;
    const int slot = lane / L;
    const int j = lane - slot * L;
    const bool slot_ok = slot < S;

    AccFor<TX, EPL, HS, HM, MODE> acc;
    acc.init();

    if (wv < P.n_hub_waves + P.n_mid_waves) {
        // ---- one wavefront per mid row, or per hub-row edge chunk ----
        const bool hub = wv < P.n_hub_waves;
        const int64_t local = hub ? wv : wv - P.n_hub_waves;
        const int64_t item = local / P.FT;
        const int ft = (int)(local - item * P.FT);
        const int64_t chunk_j = ft * (int64_t)kWave + j;  // lane-chunk index in the row
        const bool feat_ok = slot_ok && chunk_j < P.ltot;
        const int64_t fe = chunk_j * EPL;
        int U = unroll_of<MODE, HS, HM>();
        if (S * U > kWave) U = kWave / S;

        int64_t row, e0, e1, cidx = 0;
        if (hub) {
            // item = global chunk id; find its hub by binary search over the
            // chunk offsets of the hub rows (rowlist positions hub_base..)
            int64_t lo = 0, hi = P.n_hub - 1;
            while (lo < hi) {
                const int64_t mid = (lo + hi + 1) >> 1;
                if ((int64_t)P.chunk_off[P.hub_base + mid] <= item) lo = mid; else hi = mid - 1;
            }
            row = P.rowlist[P.hub_base + lo];
            const int64_t r0 = load_rp(P.rowptr, P.rp64, row);
            const int64_t r1 = load_rp(P.rowptr, P.rp64, row + 1);
            const int64_t deg = r1 - r0;
            int64_t csz = (deg + kMaxChunksPerHub - 1) / kMaxChunksPerHub;
            if (csz < P.chunk_min) csz = P.chunk_min;
            const int64_t k = item - (int64_t)P.chunk_off[P.hub_base + lo];
            e0 = r0 + k * csz;
            e1 = e0 + csz < r1 ? e0 + csz : r1;
            cidx = item;
            if constexpr (HX) {
                float t[EPL];
                int cnt;
                hub_shift<TX, EPL, NT, W, O32>(P, r0, deg, feat_ok, fe, t, cnt);
                acc.set_shift(t, cnt);
            }
        } else {
            if (P.rowbeg) {
                row = P.rowlist[P.mid_base + item];
                e0 = P.rowbeg[P.mid_base + item];
                e1 = P.rowend[P.mid_base + item];
            } else {
                row = P.rowlist ? (int64_t)P.rowlist[P.mid_base + item] : item;
                e0 = load_rp(P.rowptr, P.rp64, row);
                e1 = load_rp(P.rowptr, P.rp64, row + 1);
            }
        }
        if constexpr (MODE == kModeMasked) {
            // win-mask words covering this feature tile
            const int64_t w_lo = (int64_t)ft * 2 * EPL;
            const int64_t wmax = P.mw - w_lo;
            const int mww = (int)(wmax < 2 * EPL ? wmax : 2 * EPL);
            wave_range_masked<TX, EPL, HS, HM, NT, W, O32>(P, acc, e0, e1, lane, slot, feat_ok, fe,
                                                           w_lo, mww);
        }
        else
            wave_range<TX, EPL, HS, HM, NT, W, MODE, O32>(P, acc, e0, e1, lane, slot, feat_ok, fe, U,
                                                          !hub);
        acc.fold();
        acc.reduce_slots(S, L, slot, lane);
        if (slot == 0 && feat_ok) {
            if (hub) {
                const int64_t o = cidx * P.F + fe;
#pragma unroll
                for (int k = 0; k < EPL; ++k) {
                    if constexpr (HS) P.part_sum[o + k] = acc.s[0][k];
                    if constexpr (HM) { P.part_max[o + k] = acc.m[0][k]; P.part_arg[o + k] = acc.i[0][k]; }
                    if constexpr (HX) {
                        P.part_dsum[o + k] = acc.d[0][k];
                        P.part_sq[o + k] = acc.q[0][k];
                        P.part_min[o + k] = acc.n[0][k];
                        P.part_amin[o + k] = acc.j[0][k];
                    }
                }
            } else if constexpr (HX) {
                store_stats<EPL>(P, row, fe, e1 - e0, acc.s[0], acc.d[0], acc.q[0], acc.m[0],
                                 acc.i[0], acc.n[0], acc.j[0], P.vec_store != 0);
            } else {
                store_row<EPL>(P, row, fe, e1 - e0, acc.s[0], acc.m[0], acc.i[0], HS, HM);
            }
        }
        return;
    }

    // ---- small rows: one slot per row ----
    const int64_t local = wv - P.n_hub_waves - P.n_mid_waves;
    if (local >= P.n_small_waves) return;
    const int64_t group = local / P.FT;
    const int ft = (int)(local - group * P.FT);
    const int64_t chunk_j = ft * (int64_t)kWave + j;
    const int64_t k_row = group * S + slot;
    const bool row_ok = slot_ok && k_row < P.n_small;
    const bool feat_ok = row_ok && chunk_j < P.ltot;
    const int64_t fe = chunk_j * EPL;
    int64_t row = 0, e0 = 0, e1 = 0;
    if (row_ok) {
        row = P.rowlist[P.small_base + k_row];
        e0 = P.rowbeg[P.small_base + k_row];
        e1 = P.rowend[P.small_base + k_row];
    }
    const int32_t my_n = (int32_t)(e1 - e0);
    int32_t max_n = my_n;
    int32_t min_n = row_ok ? my_n : INT32_MAX;  // the shortest row of the wavefront
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int32_t o = __shfl_xor(max_n, off);
        max_n = o > max_n ? o : max_n;
        const int32_t on = __shfl_xor(min_n, off);
        min_n = on < min_n ? on : min_n;
    }
    max_n = __builtin_amdgcn_readfirstlane(max_n);
    min_n = __builtin_amdgcn_readfirstlane(min_n);
    if constexpr (MODE == kModeMasked) {
        const int64_t w_lo = (int64_t)ft * 2 * EPL;
        const int64_t wmax = P.mw - w_lo;
        const int mww = (int)(wmax < 2 * EPL ? wmax : 2 * EPL);
        slot_row_masked<TX, EPL, HS, HM, NT, W, O32>(P, acc, e0, my_n, max_n, lane, slot, j,
                                                     feat_ok, fe, w_lo, mww);
    } else if (L >= unroll_of<MODE, HS, HM>()) {
        slot_row<TX, EPL, HS, HM, NT, W, MODE, true, O32>(P, acc, e0, my_n, max_n, min_n, slot, j,
                                                         feat_ok, fe);
    } else {
        slot_row<TX, EPL, HS, HM, NT, W, MODE, false, O32>(P, acc, e0, my_n, max_n, min_n, slot, j,
                                                          feat_ok, fe);
    }
    acc.fold();
    if (feat_ok) {
        if constexpr (HX)
            store_stats<EPL>(P, row, fe, e1 - e0, acc.s[0], acc.d[0], acc.q[0], acc.m[0],
                             acc.i[0], acc.n[0], acc.j[0], P.vec_store != 0);
        else
            store_row<EPL>(P, row, fe, e1 - e0, acc.s[0], acc.m[0], acc.i[0], HS, HM);
    }
}

// Rows of at most kTinyDeg edges (most rows of low-degree graphs): one slot
// per row as in the small-row path, but wavefronts are persistent and
// software-pipelined: while the rows of group g are gathered, the column
// indices of the next group and the row ranges of the one after are already
// in flight, so a group costs about one memory round trip.  Requires slots of
// at least kTinyDeg + 1 lanes (the columns of a row are loaded one per lane).
// One accumulator per element: a row has at most 7 edges.
template <typename TX, int EPL, bool HS, bool HM, bool W, int NT, int MODE>
__global__ __launch_bounds__(kBlock) void spmm_tiny(SpmmParams P) {
    constexpr bool MK = MODE == kModeMasked;
    constexpr bool HX = MODE == kModeStats;
    using R = typename RawVec<TX, EPL>::T;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t tw = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave)) +
                       (int64_t)blockIdx.x * kWavesPerBlock;
    const int64_t nw = (int64_t)gridDim.x * kWavesPerBlock;
    const int L = P.L, S = P.S;
    const int slot = lane / L;
    const int j = lane - slot * L;
    const bool slot_ok = slot < S;
    const int64_t items = ((P.n_tiny + S - 1) / S) * P.FT;

    // row record (row, first edge, degree) of work item `it` for this slot
    auto rec = [&](int64_t it, int32_t& row, int32_t& beg, int32_t& deg) {
        row = -1;
        beg = 0;
        deg = 0;
        if (it < items) {
            const int64_t k = (it / P.FT) * S + slot;
            if (slot_ok && k < P.n_tiny) {
                row = P.rowlist[k];
                beg = P.rowbeg[k];
                deg = P.rowend[k] - beg;
            }
        }
    };
    auto cols = [&](int32_t beg, int32_t deg, int32_t& c, float& w, int32_t& key) {
        c = 0;
        w = 1.f;
        key = -1;
        if (j < deg) {
            c = col_at(P, (int64_t)beg + j);
            if constexpr (W) w = __builtin_nontemporal_load(P.w + beg + j);
            if constexpr (MK) key = __builtin_nontemporal_load(P.ekey + beg + j);
        }
    };

    int64_t it = tw;
    int32_t row, beg, deg, nrow, nbeg, ndeg;
    int32_t cv, kv;
    float wv;
    rec(it, row, beg, deg);
    cols(beg, deg, cv, wv, kv);
    rec(it + nw, nrow, nbeg, ndeg);
    for (; it < items; it += nw) {
        const int ft = (int)(it % P.FT);
        const int64_t chunk_j = ft * (int64_t)kWave + j;
        const bool feat_ok = row >= 0 && chunk_j < P.ltot;
        const int64_t fe = chunk_j * EPL;
        R raw[kTinyDeg];
        uint32_t mb[MK ? kTinyDeg : 1];
        bool ok[kTinyDeg];
        int32_t cc[kTinyDeg];
#pragma unroll
        for (int u = 0; u < kTinyDeg; ++u) {
            cc[u] = __shfl(cv, slot * L + u);
            ok[u] = feat_ok && (u < deg);
            if constexpr (MK) {
                // unconditional load (word 0 for an invalid edge)
                const int32_t key = __shfl(kv, slot * L + u);
                mb[u] = P.mbits[ok[u] ? (int64_t)key * P.mw + (fe >> 5) : 0];
            }
        }
        if constexpr (MK) {
            // gather a chunk only if one of its features is won by this edge
#pragma unroll
            for (int u = 0; u < kTinyDeg; ++u) {
                mb[u] = ok[u] ? lane_bits<EPL>(mb[u], fe) : 0u;
                ok[u] = ok[u] && mb[u] != 0u;
            }
        }
#pragma unroll
        for (int u = 0; u < kTinyDeg; ++u)
            if (ok[u]) raw[u] = *reinterpret_cast<const R*>(feat_addr<TX, NT>(P, cc[u], fe));
        float wt[kTinyDeg];
#pragma unroll
        for (int u = 0; u < kTinyDeg; ++u) {
            wt[u] = 1.f;
            if constexpr (W) wt[u] = __shfl(wv, slot * L + u);
        }
        // next group's columns, and the row ranges of the group after it
        int32_t ncv, nkv;
        float nwv;
        cols(nbeg, ndeg, ncv, nwv, nkv);
        int32_t row2, beg2, deg2;
        rec(it + 2 * nw, row2, beg2, deg2);

        Acc<EPL, HS, HM, HX, 1> acc;
        acc.init();
        if constexpr (HX) {  // the shift: the mean of all (at most kTinyDeg) messages
            float t[EPL] = {};
#pragma unroll
            for (int u = 0; u < kTinyDeg; ++u) {
                if (ok[u]) {
                    float v[EPL];
                    widen<TX, EPL>(raw[u], v);
#pragma unroll
                    for (int k = 0; k < EPL; ++k) t[k] += W ? __fmul_rn(wt[u], v[k]) : v[k];
                }
            }
            acc.set_shift(t, deg);
        }
#pragma unroll
        for (int u = 0; u < kTinyDeg; ++u) {
            if (ok[u]) {
                float v[EPL];
                widen<TX, EPL>(raw[u], v);
                if constexpr (W) {
#pragma unroll
                    for (int k = 0; k < EPL; ++k) v[k] = __fmul_rn(wt[u], v[k]);
                }
                if constexpr (MK) apply_mask<EPL>(v, mb[u]);
                acc.add(0, v, beg + u);
            }
        }
        if constexpr (HM) acc.settle(0, beg, feat_ok && deg > 0);
        if (feat_ok) {
            if constexpr (HX)
                store_stats<EPL>(P, row, fe, deg, acc.s[0], acc.d[0], acc.q[0], acc.m[0],
                                 acc.i[0], acc.n[0], acc.j[0], P.vec_store != 0);
            else
                store_row<EPL>(P, row, fe, deg, acc.s[0], acc.m[0], acc.i[0], HS, HM);
        }
        row = nrow;
        beg = nbeg;
        deg = ndeg;
        cv = ncv;
        wv = nwv;
        kv = nkv;
        nrow = row2;
        nbeg = beg2;
        ndeg = deg2;
    }
}

// Combine the chunk partials of every hub row, in chunk order, and write the
// row.  One wavefront per (hub row, 64-feature tile); lane = one feature.
// HX: the stats partials too (the shifted sums and sums of squares, all
// chunks of a row using the same shift, and min with its position).
template <bool HS, bool HM, bool HX>
__global__ __launch_bounds__(kBlock) void spmm_fixup(SpmmParams P) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave)) +
                       (int64_t)blockIdx.x * kWavesPerBlock;
    const int64_t ftiles = (P.F + kWave - 1) / kWave;
    const int64_t h = wv / ftiles;
    if (h >= P.n_hub) return;
    const int64_t f = (wv - h * ftiles) * kWave + lane;
    if (f >= P.F) return;
    const int64_t row = P.rowlist[P.hub_base + h];
    const int64_t c0 = P.chunk_off[P.hub_base + h], c1 = P.chunk_off[P.hub_base + h + 1];
    constexpr int A = 4;
    float s[A] = {0.f, 0.f, 0.f, 0.f};
    float ds[A] = {0.f, 0.f, 0.f, 0.f};
    float qs[A] = {0.f, 0.f, 0.f, 0.f};
    float m = 0.f, mn = 0.f;
    int32_t mi = -1, ni = -1;
    for (int64_t c = c0; c < c1; c += A) {
        float ps[A], pm[A], pd[A], pq[A], pn[A];
        int32_t pi[A], pj[A];
#pragma unroll
        for (int a = 0; a < A; ++a) {
            const bool ok = c + a < c1;
            const int64_t o = (c + a) * P.F + f;
            if constexpr (HS) ps[a] = ok ? P.part_sum[o] : 0.f;
            if constexpr (HM) { pm[a] = ok ? P.part_max[o] : 0.f; pi[a] = ok ? P.part_arg[o] : -1; }
            if constexpr (HX) {
                pd[a] = ok ? P.part_dsum[o] : 0.f;
                pq[a] = ok ? P.part_sq[o] : 0.f;
                pn[a] = ok ? P.part_min[o] : 0.f;
                pj[a] = ok ? P.part_amin[o] : -1;
            }
        }
#pragma unroll
        for (int a = 0; a < A; ++a) {
            if constexpr (HS) s[a] += ps[a];
            if constexpr (HM) max_merge(m, mi, pm[a], pi[a]);
            if constexpr (HX) {
                ds[a] += pd[a];
                qs[a] += pq[a];
                min_merge(mn, ni, pn[a], pj[a]);
            }
        }
    }
    const int64_t deg = load_rp(P.rowptr, P.rp64, row + 1) - load_rp(P.rowptr, P.rp64, row);
    const int64_t o = row * P.F + f;
    if constexpr (HX) {
        const float sum[1] = {(s[0] + s[1]) + (s[2] + s[3])};
        const float dsum[1] = {(ds[0] + ds[1]) + (ds[2] + ds[3])};
        const float sq[1] = {(qs[0] + qs[1]) + (qs[2] + qs[3])};
        const float mx[1] = {m}, nn[1] = {mn};
        const int32_t im[1] = {mi}, in[1] = {ni};
        store_stats<1>(P, row, f, deg, sum, dsum, sq, mx, im, nn, in, false);
        return;
    }
    if constexpr (HS) {
        float v = (s[0] + s[1]) + (s[2] + s[3]);
        if (P.reduce & kMean) v = deg > 0 ? v / (float)deg : 0.f;
        if (P.out_bf16) static_cast<uint16_t*>(P.out)[o] = to_bf16(v);
        else static_cast<float*>(P.out)[o] = v;
    }
    if constexpr (HM) {
        const float mv = mi < 0 ? 0.f : m;
        if (P.max_bf16) static_cast<uint16_t*>(P.out_max)[o] = (uint16_t)(__float_as_uint(mv) >> 16);
        else static_cast<float*>(P.out_max)[o] = mv;
        P.argout[o] = mi;
    }
}

// ---- plan kernels -------------------------------------------------------------

// class of row i: small rows by bit length of the degree (0 for an empty
// row), then mid, then hub.
__global__ __launch_bounds__(256) void plan_classes(const void* rowptr, int rp64, int64_t N,
                                                    int64_t small_max, int64_t hub_min,
                                                    uint32_t* __restrict__ keys) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= N) return;
    const int64_t d = load_rp(rowptr, rp64, i + 1) - load_rp(rowptr, rp64, i);
    uint32_t c;
    if (d > hub_min) c = kClassHub;
    else if (d > small_max) c = kClassMid;
    else c = d == 0 ? 0u : (uint32_t)(64 - __clzll((unsigned long long)d));
    keys[i] = c;
}

// Per rowlist entry k: the row's range (rowbeg, rowend) and its chunk count
// (0 unless the row is a hub); entry N gets 0 chunks, so that the scan of
// the counts ends in the total.  One read of the row's two rowptr entries.
__global__ __launch_bounds__(256) void plan_rows(const void* rowptr, int rp64,
                                                 const int32_t* __restrict__ rowlist, int64_t N,
                                                 int64_t hub_min, int chunk_min,
                                                 int32_t* __restrict__ rowbeg,
                                                 int32_t* __restrict__ rowend,
                                                 uint32_t* __restrict__ nch) {
    const int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (k > N) return;
    if (k == N) { nch[k] = 0; return; }
    const int64_t row = rowlist[k];
    const int64_t b = load_rp(rowptr, rp64, row);
    const int64_t e = load_rp(rowptr, rp64, row + 1);
    rowbeg[k] = (int32_t)b;
    rowend[k] = (int32_t)e;
    const int64_t d = e - b;
    uint32_t c = 0;
    if (d > hub_min) {
        int64_t csz = (d + kMaxChunksPerHub - 1) / kMaxChunksPerHub;
        if (csz < chunk_min) csz = chunk_min;
        c = (uint32_t)((d + csz - 1) / csz);
    }
    nch[k] = c;
}

// header[c] = start of class c in rowlist (c < nclass), header[nclass] = N,
// header[nclass + 1] = total hub chunks
// header: class starts, N, the chunk count and the sort's error word
__global__ void plan_header(const uint32_t* __restrict__ class_start, int nclass,
                            const uint32_t* __restrict__ chunk_off, int64_t N,
                            const uint32_t* __restrict__ sort_err, uint32_t* __restrict__ header) {
    const int c = threadIdx.x;
    if (c < nclass) header[c] = class_start[c];
    if (c == 0) {
        header[nclass] = (uint32_t)N;
        header[nclass + 1] = chunk_off[N];
        header[nclass + 2] = *sort_err;
    }
}

// masked sum: the gradient of max
template <typename TX, int EPL, bool O32>
hipError_t launch_masked(const SpmmParams& p, unsigned grid, hipStream_t s) {
    if (p.w)
        hipLaunchKernelGGL((spmm_main<TX, EPL, true, false, 1, true, kModeMasked, O32>), dim3(grid), dim3(kBlock), 0, s, p);
    else
        hipLaunchKernelGGL((spmm_main<TX, EPL, true, false, 1, false, kModeMasked, O32>), dim3(grid), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

template <typename TX, int EPL, bool W, bool O32>
hipError_t launch_w(const SpmmParams& p, unsigned grid, hipStream_t s) {
    const bool hs = (p.reduce & (kSum | kMean)) != 0;
    const bool hm = (p.reduce & kMax) != 0;
    if (p.stats)
        hipLaunchKernelGGL((spmm_main<TX, EPL, true, true, 1, W, kModeStats, O32>), dim3(grid), dim3(kBlock), 0, s, p);
    else if (hs && hm)
        hipLaunchKernelGGL((spmm_main<TX, EPL, true, true, 1, W, kModePlain, O32>), dim3(grid), dim3(kBlock), 0, s, p);
    else if (hm)
        hipLaunchKernelGGL((spmm_main<TX, EPL, false, true, 1, W, kModePlain, O32>), dim3(grid), dim3(kBlock), 0, s, p);
    else
        hipLaunchKernelGGL((spmm_main<TX, EPL, true, false, 1, W, kModePlain, O32>), dim3(grid), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

template <typename TX, int EPL>
hipError_t launch_typed(const SpmmParams& p, unsigned grid, hipStream_t s) {
    if (p.n_tables > 1) {
        // typed-node tables: unweighted sum only
        if (p.n_tables <= 2)
            hipLaunchKernelGGL((spmm_main<TX, EPL, true, false, 2, false, kModePlain>), dim3(grid), dim3(kBlock), 0, s, p);
        else if (p.n_tables <= 4)
            hipLaunchKernelGGL((spmm_main<TX, EPL, true, false, 4, false, kModePlain>), dim3(grid), dim3(kBlock), 0, s, p);
        else
            hipLaunchKernelGGL((spmm_main<TX, EPL, true, false, MP_MAX_TYPES, false, kModePlain>), dim3(grid), dim3(kBlock), 0, s, p);
        return hipGetLastError();
    }
    // the masked sum is bound by memory latency rather than bandwidth: the
    // registers that 32-bit row offsets free buy more wavefronts in flight
    if (p.mbits)
        return p.off32 ? launch_masked<TX, EPL, true>(p, grid, s) : launch_masked<TX, EPL, false>(p, grid, s);
    // 32-bit row offsets pay off for bf16 rows (measured: 7% on the
    // 124M-edge graph; fp32 rows are unaffected), so only those are built
    if constexpr (std::is_same<TX, uint16_t>::value) {
        if (p.off32)
            return p.w ? launch_w<TX, EPL, true, true>(p, grid, s)
                       : launch_w<TX, EPL, false, true>(p, grid, s);
    }
    // ... and for fp32 rows in stats mode, where the registers they free
    // keep the kernel at four wavefronts per SIMD
    if constexpr (std::is_same<TX, float>::value) {
        if (p.off32 && p.stats)
            return p.w ? launch_w<TX, EPL, true, true>(p, grid, s)
                       : launch_w<TX, EPL, false, true>(p, grid, s);
    }
    return p.w ? launch_w<TX, EPL, true, false>(p, grid, s) : launch_w<TX, EPL, false, false>(p, grid, s);
}

}  // namespace

Geometry make_geometry(int64_t F, int x_dtype, uintptr_t x_align) {
    Geometry g;
    g.elem_bytes = x_dtype == MP_BF16 ? 2 : 4;
    const int64_t row_bytes = F * g.elem_bytes;
    int vec = 16;
    while (vec > g.elem_bytes && (row_bytes % vec != 0 || x_align % vec != 0)) vec >>= 1;
    g.epl = vec / g.elem_bytes;
    g.ltot = row_bytes / vec;
    if (g.ltot <= kWave) {
        g.L = (int)g.ltot;
        g.S = kWave / g.L;
        g.FT = 1;
    } else {
        g.L = kWave;
        g.S = 1;
        g.FT = (int)ceil_div(g.ltot, kWave);
    }
    return g;
}

hipError_t launch_spmm(const SpmmParams& p, int x_dtype, int epl, hipStream_t s) {
    const int64_t waves = p.n_hub_waves + p.n_mid_waves + p.n_small_waves;
    if (waves <= 0) return hipSuccess;
    const unsigned grid = (unsigned)ceil_div(waves, kWavesPerBlock);
    if (x_dtype == MP_F32) {
        switch (epl) {
            case 4: return launch_typed<float, 4>(p, grid, s);
            case 2: return launch_typed<float, 2>(p, grid, s);
            default: return launch_typed<float, 1>(p, grid, s);
        }
    }
    switch (epl) {
        case 8: return launch_typed<uint16_t, 8>(p, grid, s);
        case 4: return launch_typed<uint16_t, 4>(p, grid, s);
        case 2: return launch_typed<uint16_t, 2>(p, grid, s);
        default: return launch_typed<uint16_t, 1>(p, grid, s);
    }
}

template <typename TX, int EPL>
hipError_t launch_tiny_typed(const SpmmParams& p, unsigned grid, hipStream_t s) {
    const bool hs = (p.reduce & (kSum | kMean)) != 0;
    const bool hm = (p.reduce & kMax) != 0;
    const bool w = p.w != nullptr;
#define MP_TINY(HS, HM, WW) \
    hipLaunchKernelGGL((spmm_tiny<TX, EPL, HS, HM, WW, 1, kModePlain>), dim3(grid), dim3(kBlock), 0, s, p)
    if (p.n_tables > 1) {
        // typed-node tables: unweighted sum only
        if (p.n_tables <= 2)
            hipLaunchKernelGGL((spmm_tiny<TX, EPL, true, false, false, 2, kModePlain>), dim3(grid), dim3(kBlock), 0, s, p);
        else if (p.n_tables <= 4)
            hipLaunchKernelGGL((spmm_tiny<TX, EPL, true, false, false, 4, kModePlain>), dim3(grid), dim3(kBlock), 0, s, p);
        else
            hipLaunchKernelGGL((spmm_tiny<TX, EPL, true, false, false, MP_MAX_TYPES, kModePlain>), dim3(grid), dim3(kBlock), 0, s, p);
    } else if (p.mbits) {
        // masked sum: the gradient of max
        if (w) hipLaunchKernelGGL((spmm_tiny<TX, EPL, true, false, true, 1, kModeMasked>), dim3(grid), dim3(kBlock), 0, s, p);
        else hipLaunchKernelGGL((spmm_tiny<TX, EPL, true, false, false, 1, kModeMasked>), dim3(grid), dim3(kBlock), 0, s, p);
    } else if (p.stats) {
        if (w) hipLaunchKernelGGL((spmm_tiny<TX, EPL, true, true, true, 1, kModeStats>), dim3(grid), dim3(kBlock), 0, s, p);
        else hipLaunchKernelGGL((spmm_tiny<TX, EPL, true, true, false, 1, kModeStats>), dim3(grid), dim3(kBlock), 0, s, p);
    } else if (hs && hm) { if (w) MP_TINY(true, true, true); else MP_TINY(true, true, false); }
    else if (hm) { if (w) MP_TINY(false, true, true); else MP_TINY(false, true, false); }
    else { if (w) MP_TINY(true, false, true); else MP_TINY(true, false, false); }
#undef MP_TINY
    return hipGetLastError();
}

hipError_t launch_spmm_tiny(const SpmmParams& p, int x_dtype, int epl, hipStream_t s) {
    if (p.n_tiny <= 0) return hipSuccess;
    const int64_t items = ceil_div(p.n_tiny, p.S) * p.FT;
    const int64_t waves = items < 4096 ? items : 4096;
    const unsigned grid = (unsigned)ceil_div(waves, kWavesPerBlock);
    if (x_dtype == MP_F32) {
        switch (epl) {
            case 4: return launch_tiny_typed<float, 4>(p, grid, s);
            case 2: return launch_tiny_typed<float, 2>(p, grid, s);
            default: return launch_tiny_typed<float, 1>(p, grid, s);
        }
    }
    switch (epl) {
        case 8: return launch_tiny_typed<uint16_t, 8>(p, grid, s);
        case 4: return launch_tiny_typed<uint16_t, 4>(p, grid, s);
        case 2: return launch_tiny_typed<uint16_t, 2>(p, grid, s);
        default: return launch_tiny_typed<uint16_t, 1>(p, grid, s);
    }
}

hipError_t launch_spmm_fixup(const SpmmParams& p, hipStream_t s) {
    if (p.n_hub <= 0) return hipSuccess;
    const int64_t waves = p.n_hub * ceil_div(p.F, kWave);
    const unsigned grid = (unsigned)ceil_div(waves, kWavesPerBlock);
    const bool hs = (p.reduce & (kSum | kMean)) != 0;
    const bool hm = (p.reduce & kMax) != 0;
    if (p.stats) hipLaunchKernelGGL((spmm_fixup<true, true, true>), dim3(grid), dim3(kBlock), 0, s, p);
    else if (hs && hm) hipLaunchKernelGGL((spmm_fixup<true, true, false>), dim3(grid), dim3(kBlock), 0, s, p);
    else if (hm) hipLaunchKernelGGL((spmm_fixup<false, true, false>), dim3(grid), dim3(kBlock), 0, s, p);
    else hipLaunchKernelGGL((spmm_fixup<true, false, false>), dim3(grid), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_plan_classes(const void* rowptr, int rp64, int64_t N, int64_t small_max,
                               int64_t hub_min, uint32_t* keys, hipStream_t s) {
    if (N <= 0) return hipSuccess;
    hipLaunchKernelGGL(plan_classes, dim3((unsigned)ceil_div(N, 256)), dim3(256), 0, s, rowptr,
                       rp64, N, small_max, hub_min, keys);
    return hipGetLastError();
}

hipError_t launch_plan_rows(const void* rowptr, int rp64, const int32_t* rowlist, int64_t N,
                            int64_t hub_min, int chunk_min, int32_t* rowbeg, int32_t* rowend,
                            uint32_t* nch, hipStream_t s) {
    hipLaunchKernelGGL(plan_rows, dim3((unsigned)ceil_div(N + 1, 256)), dim3(256), 0, s, rowptr,
                       rp64, rowlist, N, hub_min, chunk_min, rowbeg, rowend, nch);
    return hipGetLastError();
}

hipError_t launch_plan_header(const uint32_t* class_start, int nclass, const uint32_t* chunk_off,
                              int64_t N, const uint32_t* sort_err, uint32_t* header, hipStream_t s) {
    hipLaunchKernelGGL(plan_header, dim3(1), dim3(64), 0, s, class_start, nclass, chunk_off, N,
                       sort_err, header);
    return hipGetLastError();
}

}  // namespace mp
