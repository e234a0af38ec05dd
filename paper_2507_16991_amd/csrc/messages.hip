// Edge-materialized message passing (the explanation mode of PyG 2.0,
// Sec. 2.4, which falls back to the edge-level materialization of PyG 1
// recalled in Sec. 2.2 so that a callback can edit every message before it is
// aggregated).
//
// Messages live in an [E, F] table in destination-major CSR order (row p is
// the message of CSR edge p), so the aggregation that follows is the
// segmented reduction of spmm.hip over consecutive message rows: no atomics,
// deterministic.  The kernels here are the edge-space steps around it:
//
//   * message_gather:   msg[p, :] = w[p] * x[idx[p], :] (or x[idx[p], :])
//   * message_scale:    out[p, :] = in[p, :] * mask[idx[p]] (the edge-mask
//                       callback, and its backward with respect to the input)
//   * message_backward: dL/dmsg[p, :] from dL/dout[row(p), :] (sum: a copy;
//                       mean: divided by the in-degree; max: routed to the
//                       argmax edge only)
//
// The gather and the scale are streaming kernels over the flat [E, F] table
// cut into lane-chunks of EPL elements (one vector access each): consecutive
// threads take consecutive chunks, so the table side is read and written
// fully coalesced, and a gathered feature row is read by consecutive lanes.
// Each thread handles a few chunks spaced one block apart, issuing all index
// loads, then all row loads, before any store.  The gradient goes row by
// row: a destination row's gradient is loaded once and written to the
// consecutive message rows of its edges.
#include <type_traits>

#include "mp_internal.hpp"

namespace mp {
namespace {

constexpr int kBlock = 256;
// lane-chunks per thread of the gather and the scale
constexpr int kItems = 4;

__device__ inline float bf16_bits(uint32_t b) { return __uint_as_float(b << 16); }

// EPL consecutive elements of a fp32 or bf16 row, widened to fp32; p is
// aligned to EPL * sizeof(T) bytes (at most 16).
template <typename T, int EPL>
__device__ inline void load_chunk(const T* p, float (&v)[EPL]) {
    if constexpr (std::is_same<T, float>::value) {
        if constexpr (EPL == 4) {
            const float4 a = *reinterpret_cast<const float4*>(p);
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        } else if constexpr (EPL == 2) {
            const float2 a = *reinterpret_cast<const float2*>(p);
            v[0] = a.x; v[1] = a.y;
        } else {
            v[0] = *p;
        }
    } else {
        if constexpr (EPL == 8) {
            const uint4 a = *reinterpret_cast<const uint4*>(p);
            const uint32_t u[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                v[2 * k] = bf16_bits(u[k] & 0xFFFFu);
                v[2 * k + 1] = __uint_as_float(u[k] & 0xFFFF0000u);
            }
        } else if constexpr (EPL == 4) {
            const uint2 a = *reinterpret_cast<const uint2*>(p);
            v[0] = bf16_bits(a.x & 0xFFFFu); v[1] = __uint_as_float(a.x & 0xFFFF0000u);
            v[2] = bf16_bits(a.y & 0xFFFFu); v[3] = __uint_as_float(a.y & 0xFFFF0000u);
        } else if constexpr (EPL == 2) {
            const uint32_t a = *reinterpret_cast<const uint32_t*>(p);
            v[0] = bf16_bits(a & 0xFFFFu); v[1] = __uint_as_float(a & 0xFFFF0000u);
        } else {
            v[0] = bf16_bits(*reinterpret_cast<const uint16_t*>(p));
        }
    }
}

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Store EPL fp32 values (16/8/4-byte stores; p aligned to EPL * 4 bytes).
template <int EPL>
__device__ inline void store_f32(float* p, const float (&v)[EPL]) {
    if constexpr (EPL == 4) {
        const f32x4 u = {v[0], v[1], v[2], v[3]};
        __builtin_nontemporal_store(u, reinterpret_cast<f32x4*>(p));
    } else if constexpr (EPL == 2) {
        const f32x2 u = {v[0], v[1]};
        __builtin_nontemporal_store(u, reinterpret_cast<f32x2*>(p));
    } else {
        __builtin_nontemporal_store(v[0], p);
    }
}

// Copy EPL bf16 values unchanged (the exact message of an unweighted bf16
// row); p and q aligned to EPL * 2 bytes.
template <int EPL>
__device__ inline void copy_bf16(const uint16_t* p, uint16_t* q) {
    if constexpr (EPL == 8) {
        __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(p), reinterpret_cast<u32x4*>(q));
    } else if constexpr (EPL == 4) {
        __builtin_nontemporal_store(*reinterpret_cast<const u32x2*>(p), reinterpret_cast<u32x2*>(q));
    } else if constexpr (EPL == 2) {
        __builtin_nontemporal_store(*reinterpret_cast<const uint32_t*>(p), reinterpret_cast<uint32_t*>(q));
    } else {
        *q = *p;
    }
}

template <int EPL>
__device__ inline void load_ints(const int32_t* p, int32_t (&v)[EPL]) {
    if constexpr (EPL >= 4) {
#pragma unroll
        for (int q = 0; q < EPL / 4; ++q) {
            const int4 a = reinterpret_cast<const int4*>(p)[q];
            v[4 * q + 0] = a.x; v[4 * q + 1] = a.y; v[4 * q + 2] = a.z; v[4 * q + 3] = a.w;
        }
    } else if constexpr (EPL == 2) {
        const int2 a = *reinterpret_cast<const int2*>(p);
        v[0] = a.x; v[1] = a.y;
    } else {
        v[0] = *p;
    }
}

// The chunks of this thread in virtual block vb: chunk g = vb * kBlock *
// ITEMS + i * kBlock + tid lies in table row p = g / cpr at lane-chunk
// k = g % cpr.  One 64-bit division per virtual block (uniform), 32-bit
// divisions per chunk.  Virtual blocks are walked with a grid stride, so the
// grid stays within the launch limits for any table size.
template <int ITEMS>
struct ChunkPos {
    int64_t g[ITEMS];
    int64_t p[ITEMS];
    int32_t k[ITEMS];
    bool ok[ITEMS];
};

template <int ITEMS>
__device__ inline ChunkPos<ITEMS> chunk_positions(int64_t vb, int64_t total, int64_t cpr) {
    ChunkPos<ITEMS> c;
    const int64_t g0 = vb * (int64_t)(kBlock * ITEMS);
    const int64_t p0 = g0 / cpr;
    const uint32_t r0 = (uint32_t)(g0 - p0 * cpr);
    const uint32_t ucpr = (uint32_t)cpr;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
        const uint32_t local = r0 + (uint32_t)(i * kBlock) + threadIdx.x;
        const uint32_t dp = local / ucpr;
        c.g[i] = g0 + i * kBlock + threadIdx.x;
        c.p[i] = p0 + dp;
        c.k[i] = (int32_t)(local - dp * ucpr);
        c.ok[i] = c.g[i] < total;
    }
    return c;
}

// Virtual blocks of the table: the grid walks them with a stride.
template <int ITEMS>
__device__ inline int64_t vblocks(int64_t total) {
    return (total + kBlock * ITEMS - 1) / (kBlock * ITEMS);
}

// msg[p, k-th chunk] = (w[p] *) x[idx[p], k-th chunk].  TM = float: the
// fp32 message (one correctly rounded product when weighted); TM = uint16_t:
// an unweighted bf16 row copied unchanged.
template <typename TX, typename TM, int EPL, bool W>
__device__ inline void gather_vblock(const ChunkPos<kItems>& c, const int32_t* __restrict__ idx,
                                     const float* __restrict__ w, const TX* __restrict__ x,
                                     int64_t F, TM* __restrict__ msg) {
    int32_t src[kItems];
    float wt[kItems];
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        src[i] = c.ok[i] ? idx[c.p[i]] : 0;
        wt[i] = 1.f;
        if constexpr (W) wt[i] = c.ok[i] ? w[c.p[i]] : 1.f;
    }
    if constexpr (std::is_same<TM, float>::value) {
        float v[kItems][EPL];
#pragma unroll
        for (int i = 0; i < kItems; ++i)
            if (c.ok[i]) load_chunk<TX, EPL>(x + (int64_t)src[i] * F + (int64_t)c.k[i] * EPL, v[i]);
#pragma unroll
        for (int i = 0; i < kItems; ++i) {
            if (!c.ok[i]) continue;
            if constexpr (W) {
#pragma unroll
                for (int e = 0; e < EPL; ++e) v[i][e] = __fmul_rn(wt[i], v[i][e]);
            }
            store_f32<EPL>(msg + c.g[i] * EPL, v[i]);
        }
    } else {
#pragma unroll
        for (int i = 0; i < kItems; ++i)
            if (c.ok[i])
                copy_bf16<EPL>(reinterpret_cast<const uint16_t*>(x) + (int64_t)src[i] * F +
                                   (int64_t)c.k[i] * EPL,
                               msg + c.g[i] * EPL);
    }
}

template <typename TX, typename TM, int EPL, bool W>
__global__ __launch_bounds__(kBlock) void message_gather(const int32_t* __restrict__ idx,
                                                         const float* __restrict__ w,
                                                         const TX* __restrict__ x, int64_t F,
                                                         int64_t cpr, int64_t total,
                                                         TM* __restrict__ msg) {
    const int64_t nvb = vblocks<kItems>(total);
    for (int64_t vb = blockIdx.x; vb < nvb; vb += gridDim.x)
        gather_vblock<TX, TM, EPL, W>(chunk_positions<kItems>(vb, total, cpr), idx, w, x, F, msg);
}

// out[p, :] = in[p, :] * mask[idx ? idx[p] : p], fp32, one rounding.
template <int EPL>
__global__ __launch_bounds__(kBlock) void message_scale(const float* __restrict__ in,
                                                        float* __restrict__ out,
                                                        const float* __restrict__ mask,
                                                        const int32_t* __restrict__ idx,
                                                        int64_t cpr, int64_t total) {
    const int64_t nvb = vblocks<kItems>(total);
    for (int64_t vb = blockIdx.x; vb < nvb; vb += gridDim.x) {
        const ChunkPos<kItems> c = chunk_positions<kItems>(vb, total, cpr);
        float s[kItems], v[kItems][EPL];
#pragma unroll
        for (int i = 0; i < kItems; ++i) {
            s[i] = 1.f;
            if (c.ok[i]) {
                const int64_t j = idx ? (int64_t)idx[c.p[i]] : c.p[i];
                s[i] = mask[j];
                load_chunk<float, EPL>(in + c.g[i] * EPL, v[i]);
            }
        }
#pragma unroll
        for (int i = 0; i < kItems; ++i) {
            if (!c.ok[i]) continue;
#pragma unroll
            for (int e = 0; e < EPL; ++e) v[i][e] = __fmul_rn(v[i][e], s[i]);
            store_f32<EPL>(out + c.g[i] * EPL, v[i]);
        }
    }
}

__device__ inline int64_t rp_load(const void* rp, int rp64, int64_t i) {
    return rp64 ? static_cast<const int64_t*>(rp)[i] : (int64_t) static_cast<const int32_t*>(rp)[i];
}

// dmsg[p, :] for the CSR edges p of destination row v, from g = dL/dout
// [N, F]: sum g[v, :]; mean g[v, :] / deg(v) (correctly rounded; in fp64 for
// degrees beyond 2^24, which fp32 cannot hold); max g[v, f] where
// argout[v, f] == p.  One wavefront per row: its lanes load the row's
// gradient chunks once (and, for max, its argmax chunks), then stream them
// to the message rows of all of v's edges, which are consecutive: slot s of
// the S slots of L lanes writes edges s, s + S, ..., so one store
// instruction covers S whole consecutive rows.  Rows wider than 64
// lane-chunks take one more pass per 64 chunks.  No loads in the store loop.
template <typename TG, int EPL, int MODE>
__global__ __launch_bounds__(kBlock) void message_backward(const void* __restrict__ rowptr,
                                                           int rp64,
                                                           const int32_t* __restrict__ argout,
                                                           const TG* __restrict__ g, int64_t N,
                                                           int64_t F, int64_t cpr, int L, int S,
                                                           float* __restrict__ dmsg) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t v = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave)) +
                      (int64_t)blockIdx.x * (kBlock / kWave);
    if (v >= N) return;
    const int64_t beg = rp_load(rowptr, rp64, v);
    const int64_t deg = rp_load(rowptr, rp64, v + 1) - beg;
    const int slot = lane / L;
    const int j = lane - slot * L;
    if (deg <= 0 || slot >= S) return;
    for (int64_t k = j; k < cpr; k += L) {
        const int64_t o = v * F + k * EPL;
        float gv[EPL];
        load_chunk<TG, EPL>(g + o, gv);
        int32_t am[MODE == kMax ? EPL : 1];
        if constexpr (MODE == kMax) load_ints<EPL>(argout + o, am);
        if constexpr (MODE == kMean) {
#pragma unroll
            for (int e = 0; e < EPL; ++e)
                gv[e] = deg <= (int64_t(1) << 24) ? gv[e] / (float)deg
                                                 : (float)((double)gv[e] / (double)deg);
        }
        float* out = dmsg + (beg + slot) * F + k * EPL;
        const int64_t step = (int64_t)S * F;
        for (int64_t e = slot; e < deg; e += S, out += step) {
            float d[EPL];
#pragma unroll
            for (int x = 0; x < EPL; ++x) {
                if constexpr (MODE == kMax)
                    d[x] = am[x] == (int32_t)(beg + e) ? gv[x] : 0.f;
                else
                    d[x] = gv[x];
            }
            // plain stores: measured faster here than non-temporal ones
            // (which the read-and-write kernels above prefer)
            if constexpr (EPL == 4)
                *reinterpret_cast<float4*>(out) = make_float4(d[0], d[1], d[2], d[3]);
            else if constexpr (EPL == 2)
                *reinterpret_cast<float2*>(out) = make_float2(d[0], d[1]);
            else
                *out = d[0];
        }
    }
}

// Launch at most this many blocks; larger tables are walked by the grid stride.
constexpr int64_t kMaxGrid = int64_t(1) << 20;

unsigned grid_for(int64_t total, int items = kItems) {
    const int64_t b = ceil_div(total, (int64_t)kBlock * items);
    return (unsigned)(b < kMaxGrid ? b : kMaxGrid);
}

template <typename TX, int EPL>
hipError_t gather_w(const MessageGather& a, hipStream_t s) {
    const int64_t cpr = a.F / EPL, total = a.E * cpr;
    const TX* x = static_cast<const TX*>(a.x);
    if (a.msg_bf16) {
        // a bf16 table is only the exact copy of unweighted bf16 rows
        if constexpr (std::is_same<TX, uint16_t>::value) {
            hipLaunchKernelGGL((message_gather<TX, uint16_t, EPL, false>), dim3(grid_for(total)),
                               dim3(kBlock), 0, s, a.idx, a.w, x, a.F, cpr, total,
                               static_cast<uint16_t*>(a.msg));
            return hipGetLastError();
        } else {
            return hipErrorInvalidValue;
        }
    }
    if (a.w)
        hipLaunchKernelGGL((message_gather<TX, float, EPL, true>), dim3(grid_for(total)),
                           dim3(kBlock), 0, s, a.idx, a.w, x, a.F, cpr, total,
                           static_cast<float*>(a.msg));
    else
        hipLaunchKernelGGL((message_gather<TX, float, EPL, false>), dim3(grid_for(total)),
                           dim3(kBlock), 0, s, a.idx, a.w, x, a.F, cpr, total,
                           static_cast<float*>(a.msg));
    return hipGetLastError();
}

template <typename TX>
hipError_t gather_epl(const MessageGather& a, hipStream_t s) {
    switch (a.epl) {
        case 8: if constexpr (std::is_same<TX, uint16_t>::value) return gather_w<TX, 8>(a, s);
                return hipErrorInvalidValue;
        case 4: return gather_w<TX, 4>(a, s);
        case 2: return gather_w<TX, 2>(a, s);
        default: return gather_w<TX, 1>(a, s);
    }
}

template <typename TG, int EPL>
hipError_t backward_mode(const MessageBackward& a, hipStream_t s) {
    const int64_t cpr = a.F / EPL;
    const int L = cpr < kWave ? (int)cpr : kWave;
    const int S = kWave / L;
    const TG* g = static_cast<const TG*>(a.g);
    const dim3 grid((unsigned)ceil_div(a.N, kBlock / kWave)), block(kBlock);
    if (a.reduce == kMax)
        hipLaunchKernelGGL((message_backward<TG, EPL, kMax>), grid, block, 0, s, a.rowptr, a.rp64,
                           a.argout, g, a.N, a.F, cpr, L, S, a.dmsg);
    else if (a.reduce == kMean)
        hipLaunchKernelGGL((message_backward<TG, EPL, kMean>), grid, block, 0, s, a.rowptr, a.rp64,
                           a.argout, g, a.N, a.F, cpr, L, S, a.dmsg);
    else
        hipLaunchKernelGGL((message_backward<TG, EPL, kSum>), grid, block, 0, s, a.rowptr, a.rp64,
                           a.argout, g, a.N, a.F, cpr, L, S, a.dmsg);
    return hipGetLastError();
}

template <typename TG>
hipError_t backward_epl(const MessageBackward& a, hipStream_t s) {
    switch (a.epl) {
        case 4: return backward_mode<TG, 4>(a, s);
        case 2: return backward_mode<TG, 2>(a, s);
        default: return backward_mode<TG, 1>(a, s);
    }
}

}  // namespace

// Largest chunk width EPL in {8, 4, 2, 1} that divides F, whose byte size
// stays within 16 for every element size listed, and to which every listed
// pointer is aligned.
int message_epl(int64_t F, const uintptr_t* ptrs, const int* elem_bytes, int n, int max_epl) {
    for (int e = max_epl; e > 1; e >>= 1) {
        bool ok = F % e == 0;
        for (int i = 0; i < n && ok; ++i)
            ok = e * elem_bytes[i] <= 16 && ptrs[i] % (uintptr_t)(e * elem_bytes[i]) == 0;
        if (ok) return e;
    }
    return 1;
}

hipError_t launch_message_gather(const MessageGather& a, hipStream_t s) {
    if (a.E <= 0) return hipSuccess;
    return a.x_bf16 ? gather_epl<uint16_t>(a, s) : gather_epl<float>(a, s);
}

hipError_t launch_message_scale(const float* in, float* out, const float* mask,
                                const int32_t* idx, int64_t E, int64_t F, int epl, hipStream_t s) {
    if (E <= 0) return hipSuccess;
    const int64_t cpr = F / epl, total = E * cpr;
    const dim3 grid(grid_for(total)), block(kBlock);
    if (epl == 4)
        hipLaunchKernelGGL(message_scale<4>, grid, block, 0, s, in, out, mask, idx, cpr, total);
    else if (epl == 2)
        hipLaunchKernelGGL(message_scale<2>, grid, block, 0, s, in, out, mask, idx, cpr, total);
    else
        hipLaunchKernelGGL(message_scale<1>, grid, block, 0, s, in, out, mask, idx, cpr, total);
    return hipGetLastError();
}

hipError_t launch_message_backward(const MessageBackward& a, hipStream_t s) {
    if (a.E <= 0 || a.N <= 0) return hipSuccess;
    return a.g_bf16 ? backward_epl<uint16_t>(a, s) : backward_epl<float>(a, s);
}

}  // namespace mp
