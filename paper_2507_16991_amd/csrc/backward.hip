// Backward pass of the aggregation (Sec. 2.2 of PyG 2.0: the gradient of an
// aggregation over A runs over the transposed adjacency, which the library
// builds once as a source-major CSR, the analogue of the cached CSC).
//
//   * rows_of_edges: the destination row of every forward CSR position (the
//     keys the transposed CSR is sorted by carry it as payload), one
//     wavefront per 64 rows.
//   * scale_inv_deg: grad_out / in-degree per destination row, the input of
//     the gradient of mean.
//   * spmm_grad_w: the gradient with respect to the edge weights, one dot
//     product of grad_out[v] and x[col[p]] per CSR edge p of row v (a
//     sampled dense-dense product).  Edge-parallel: every wavefront takes 64
//     consecutive CSR positions, so hub rows need no special handling; the
//     per-edge dots are reduced over the lanes of a slot by recursive
//     halving, a fixed pattern.  With
//     the row or column array absent (position p reads row p) the same kernel
//     gives the per-edge dot products of the edge-materialized path.
//   * win_masks: for the gradient of max, the features each forward edge
//     wins (one bit per feature), so that the masked sum over the transposed
//     CSR reads one mask word per edge and lane instead of the argmax chunk
//     of the edge's destination row.
//
// The gradient with respect to x reuses the aggregation kernels of spmm.hip
// over the transposed CSR (sum, mean after scale_inv_deg, and a masked sum
// for max).
#include <type_traits>

#include "mp_internal.hpp"

namespace mp {
namespace {

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;
#ifndef MP_GW_UNROLL
#define MP_GW_UNROLL 4  // edges per slot per step of the weight gradient (sum, mean)
#endif

__device__ inline int64_t rp_at(const void* rp, int rp64, int64_t i) {
    return rp64 ? static_cast<const int64_t*>(rp)[i] : (int64_t) static_cast<const int32_t*>(rp)[i];
}

// row[p] = the v with rowptr[v] <= p < rowptr[v+1].  Each wavefront takes 64
// consecutive rows: it stages their 65 bounds in LDS, then writes the
// positions from its first row's start to its last row's end 64 at a time
// (one store instruction each, however long or short the rows), each lane
// finding the row of its position by a binary search over the staged
// bounds.  Bounds are read as 0 for row 0 and E for row N and clamped to
// [0, E], so every position is written, with a row id below N, whatever the
// input (an inconsistent rowptr only makes ids wrong).
template <typename IT>
__global__ __launch_bounds__(kBlock) void rows_of_edges(const IT* __restrict__ rowptr, int64_t N,
                                                        int64_t E, int32_t* __restrict__ row) {
    __shared__ int64_t s_b[kWavesPerBlock][kWave + 1];
    const int lane = threadIdx.x & (kWave - 1);
    const int wl = threadIdx.x / kWave;
    const int64_t v0 = ((int64_t)blockIdx.x * kWavesPerBlock + wl) * kWave;
    if (v0 >= N) return;  // uniform per wavefront
    auto bound = [&](int64_t v) -> int64_t {
        if (v <= 0) return 0;
        if (v >= N) return E;
        const int64_t b = (int64_t)rowptr[v];
        return b < 0 ? 0 : (b > E ? E : b);
    };
    s_b[wl][lane] = bound(v0 + lane);
    if (lane == 0) s_b[wl][kWave] = bound(v0 + kWave);
    // the wavefront reads what its own lanes wrote: LDS operations of one
    // wavefront complete in order
    __builtin_amdgcn_wave_barrier();
    const int nr = (int)(N - v0 < kWave ? N - v0 : kWave);  // rows of this wavefront
    const int64_t p1 = s_b[wl][nr];
    for (int64_t p = s_b[wl][0] + lane; p < p1; p += kWave) {
        int lo = 0, hi = nr - 1;  // the last row whose start is <= p
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_b[wl][mid] <= p) lo = mid; else hi = mid - 1;
        }
        row[p] = (int32_t)(v0 + lo);
    }
}

__device__ inline float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// out[v, f] = g[v, f] / deg(v) in fp32 (0 for an empty row).  Each thread
// takes V consecutive elements of one row (V divides F); the row index uses
// 32-bit division when the table has under 2^32 elements.
template <bool GB, int V>
__global__ __launch_bounds__(kBlock) void scale_inv_deg(const void* __restrict__ g,
                                                        const void* __restrict__ rowptr, int rp64,
                                                        int64_t N, int64_t F,
                                                        float* __restrict__ out) {
    const int64_t n = N * F;
    const int64_t i = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * V;
    if (i >= n) return;
    const int64_t v = n <= (int64_t)UINT32_MAX ? (int64_t)((uint32_t)i / (uint32_t)F) : i / F;
    const int64_t deg = rp_at(rowptr, rp64, v + 1) - rp_at(rowptr, rp64, v);
    float gv[V];
    if constexpr (GB) {
        const uint16_t* gb = static_cast<const uint16_t*>(g) + i;
        if constexpr (V == 4) {
            const uint2 u = *reinterpret_cast<const uint2*>(gb);
            gv[0] = bf16_bits_to_f32(u.x & 0xFFFFu); gv[1] = __uint_as_float(u.x & 0xFFFF0000u);
            gv[2] = bf16_bits_to_f32(u.y & 0xFFFFu); gv[3] = __uint_as_float(u.y & 0xFFFF0000u);
        } else {
            gv[0] = bf16_bits_to_f32(gb[0]);
        }
    } else {
        const float* gf = static_cast<const float*>(g) + i;
        if constexpr (V == 4) {
            const float4 a = *reinterpret_cast<const float4*>(gf);
            gv[0] = a.x; gv[1] = a.y; gv[2] = a.z; gv[3] = a.w;
        } else {
            gv[0] = gf[0];
        }
    }
#pragma unroll
    for (int k = 0; k < V; ++k) gv[k] = deg > 0 ? gv[k] / (float)deg : 0.f;
    if constexpr (V == 4)
        *reinterpret_cast<float4*>(out + i) = make_float4(gv[0], gv[1], gv[2], gv[3]);
    else
        out[i] = gv[0];
}

// bits[p * MW + w], bit b: feature f = 32 w + b of row v = row(p) has its
// maximum at CSR position p (argout[v, f] == p).  A wavefront takes
// kMaskRows consecutive rows, whose row ranges and first argout loads are
// issued together (a row's own work is short next to a memory round trip).
// The features go in pairs of 64-feature tiles (two argout values per lane,
// up to four words per position); a row's positions in chunks of 64.  For
// each chunk the wavefront clears 4 LDS words per position, every feature
// whose winner lies in the chunk ORs its bit into its winner's word (an
// integer OR, so the order does not matter), and lane i stores the words of
// position i.  Every word of every position is written exactly once.  The
// LDS region is the wavefront's own; LDS operations of one wavefront execute
// in program order, so no barrier is needed.
constexpr int kMaskRows = 4;

template <typename IT>
__global__ __launch_bounds__(kBlock) void win_masks(const IT* __restrict__ rowptr,
                                                    const int32_t* __restrict__ argout, int64_t N,
                                                    int64_t F, int64_t MW,
                                                    uint32_t* __restrict__ bits) {
    __shared__ __align__(16) uint32_t lds[kWavesPerBlock][kWave * 4];
    const int lane = threadIdx.x & (kWave - 1);
    const int wid = threadIdx.x / kWave;
    const int64_t v0 =
        (__builtin_amdgcn_readfirstlane(wid) + (int64_t)blockIdx.x * kWavesPerBlock) * kMaskRows;
    if (v0 >= N) return;
    uint32_t* my = lds[wid];
    int64_t rb[kMaskRows + 1];
#pragma unroll
    for (int i = 0; i <= kMaskRows; ++i) rb[i] = (int64_t)rowptr[v0 + i < N ? v0 + i : N];
    // features f0 + lane and f0 + 64 + lane (clamped to the row, masked below)
    const int64_t la = lane < F ? lane : F - 1;
    const int64_t lb = kWave + lane < F ? kWave + lane : F - 1;
    int32_t a0[kMaskRows], b0[kMaskRows];
#pragma unroll
    for (int i = 0; i < kMaskRows; ++i) {
        const int64_t v = v0 + i < N ? v0 + i : N - 1;
        a0[i] = argout[v * F + la];
        b0[i] = argout[v * F + lb];
    }
    const uint32_t bit = 1u << (lane & 31);
    const int half = lane >> 5;
#pragma unroll
    for (int i = 0; i < kMaskRows; ++i) {
        const int64_t v = v0 + i;
        const int64_t beg = rb[i];
        const int64_t deg = rb[i + 1] - beg;
        if (v >= N || deg <= 0) continue;
        for (int64_t f0 = 0; f0 < F; f0 += 2 * kWave) {
            // winners of features f0 + lane and f0 + 64 + lane, relative to
            // the row start (-1: no such feature)
            const int64_t fa = f0 + lane, fb = f0 + kWave + lane;
            int32_t aa = a0[i], ab = b0[i];
            if (f0 > 0) {
                aa = argout[v * F + (fa < F ? fa : F - 1)];
                ab = argout[v * F + (fb < F ? fb : F - 1)];
            }
            const int64_t ra = fa < F ? (int64_t)aa - beg : -1;
            const int64_t rbv = fb < F ? (int64_t)ab - beg : -1;
            const int64_t w0 = f0 >> 5;  // a multiple of 4
            const int nw = (int)(MW - w0 < 4 ? MW - w0 : 4);
            for (int64_t c0 = 0; c0 < deg; c0 += kWave) {
                const int n = (int)(deg - c0 < kWave ? deg - c0 : kWave);
                const int64_t qa = ra - c0, qb = rbv - c0;
                *reinterpret_cast<uint4*>(my + 4 * lane) = make_uint4(0u, 0u, 0u, 0u);
                __builtin_amdgcn_wave_barrier();
                if (qa >= 0 && qa < n) atomicOr(my + 4 * qa + half, bit);
                if (qb >= 0 && qb < n) atomicOr(my + 4 * qb + 2 + half, bit);
                __builtin_amdgcn_wave_barrier();
                if (lane < n) {
                    const uint4 r = *reinterpret_cast<const uint4*>(my + 4 * lane);
                    uint32_t* o = bits + (beg + c0 + lane) * MW + w0;
                    if (nw == 4 && (MW & 3) == 0) {
                        *reinterpret_cast<uint4*>(o) = r;  // 16-byte aligned
                    } else {
                        o[0] = r.x;
                        if (nw > 1) o[1] = r.y;
                        if (nw > 2) o[2] = r.z;
                        if (nw > 3) o[3] = r.w;
                    }
                }
                __builtin_amdgcn_wave_barrier();
            }
        }
    }
}

// EPL consecutive values of a fp32 or bf16 row, widened to fp32; p is aligned
// to min(16, EPL * sizeof(T)) bytes.
template <typename T, int EPL>
__device__ inline void load_vals(const T* p, float (&v)[EPL]) {
    if constexpr (std::is_same<T, float>::value) {
        if constexpr (EPL >= 4) {
#pragma unroll
            for (int q = 0; q < EPL / 4; ++q) {
                const float4 a = reinterpret_cast<const float4*>(p)[q];
                v[4 * q + 0] = a.x; v[4 * q + 1] = a.y; v[4 * q + 2] = a.z; v[4 * q + 3] = a.w;
            }
        } else if constexpr (EPL == 2) {
            const float2 a = *reinterpret_cast<const float2*>(p);
            v[0] = a.x; v[1] = a.y;
        } else {
            v[0] = *p;
        }
    } else {
        uint32_t u[(EPL + 1) / 2];
        if constexpr (EPL == 8) {
            const uint4 a = *reinterpret_cast<const uint4*>(p);
            u[0] = a.x; u[1] = a.y; u[2] = a.z; u[3] = a.w;
        } else if constexpr (EPL == 4) {
            const uint2 a = *reinterpret_cast<const uint2*>(p);
            u[0] = a.x; u[1] = a.y;
        } else if constexpr (EPL == 2) {
            u[0] = *reinterpret_cast<const uint32_t*>(p);
        } else {
            u[0] = *reinterpret_cast<const uint16_t*>(p);
        }
#pragma unroll
        for (int k = 0; k < EPL; ++k)
            v[k] = (k & 1) ? __uint_as_float(u[k / 2] & 0xFFFF0000u) : bf16_bits_to_f32(u[k / 2] & 0xFFFFu);
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

// grad_w[p] = sum_f route(v, f, p) * g[v, f] * x[col[p], f] for the CSR edge
// p of row v = row[p]; route is 1 (sum), 1/deg(v) (mean, applied to the
// finished dot) or [argout[v, f] == p] (max).  A wavefront takes 64
// consecutive positions; slot s of its S slots takes positions base + u*S + s
// (u < U) of each step, its L lanes (a power of two, slots aligned) covering
// the feature row in FT tiles.
template <typename TX, typename TG, int EPL, int MODE>
__global__ __launch_bounds__(kBlock) void spmm_grad_w(GradWParams P) {
    constexpr int U = MODE == kMax ? 4 : MP_GW_UNROLL;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave)) +
                       (int64_t)blockIdx.x * kWavesPerBlock;
    const int64_t p0 = wv * kWave;
    if (p0 >= P.E) return;
    const int L = P.L, S = P.S;
    const int slot = lane / L;
    const int j = lane - slot * L;
    const bool slot_ok = slot < S;
    const int64_t rem = P.E - p0;

    // absent index arrays are the identity (per-edge dot products of two
    // edge-space tables, or of one edge-space table and gathered rows)
    int32_t myc = 0, myv = 0;
    if (lane < rem) {
        myc = P.col ? __builtin_nontemporal_load(P.col + p0 + lane) : (int32_t)(p0 + lane);
        myv = P.row ? __builtin_nontemporal_load(P.row + p0 + lane) : (int32_t)(p0 + lane);
    }
    // values per lane left by the slot reduction (L < U), and the lane
    // stride between the holders of consecutive edges (L >= U)
    const int nv = U > L ? U / L : 1;
    const int hstride = U > L ? 1 : L / U;

    float result = 0.f;  // lane t ends with the dot of position p0 + t
    const int SU = S * U;
    for (int base = 0; base < kWave && base < rem; base += SU) {
        float dot[U];
#pragma unroll
        for (int u = 0; u < U; ++u) dot[u] = 0.f;
        for (int ft = 0; ft < P.FT; ++ft) {
            const int64_t chunk = (int64_t)ft * kWave + j;
            const bool feat_ok = slot_ok && chunk < P.ltot;
            const int64_t fe = chunk * EPL;
            float xv[U][EPL], gv[U][EPL];
            int32_t mv[MODE == kMax ? U : 1][EPL];
            bool ok[U], fresh[U];
            int32_t vprev = -1;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int t = base + u * S + slot;
                const int32_t c = __shfl(myc, t & (kWave - 1));
                const int32_t v = __shfl(myv, t & (kWave - 1));
                ok[u] = feat_ok && t < kWave && t < rem;
                // consecutive edges of a slot mostly share their row: its
                // gradient chunk (and argmax chunk) is loaded once and reused
                fresh[u] = u == 0 || v != vprev;
                vprev = v;
                if (ok[u]) {
                    load_vals<TX, EPL>(reinterpret_cast<const TX*>(P.x) + (int64_t)c * P.F + fe, xv[u]);
                    if (fresh[u]) {
                        load_vals<TG, EPL>(reinterpret_cast<const TG*>(P.g) + (int64_t)v * P.F + fe, gv[u]);
                        if constexpr (MODE == kMax) load_ints<EPL>(P.argout + (int64_t)v * P.F + fe, mv[u]);
                    }
                }
            }
#pragma unroll
            for (int u = 1; u < U; ++u) {
                if (fresh[u]) continue;  // a valid edge's predecessor in the slot is valid
#pragma unroll
                for (int k = 0; k < EPL; ++k) {
                    gv[u][k] = gv[u - 1][k];
                    if constexpr (MODE == kMax) mv[u][k] = mv[u - 1][k];
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (!ok[u]) continue;
                const int32_t pos = (int32_t)(p0 + base + u * S + slot);
#pragma unroll
                for (int k = 0; k < EPL; ++k) {
                    float t = gv[u][k] * xv[u][k];
                    if constexpr (MODE == kMax) t = mv[u][k] == pos ? t : 0.f;
                    dot[u] += t;
                }
            }
        }
        // reduce the U dots over the slot's L lanes (L a power of two, slots
        // aligned) by recursive halving: at stride m the lanes with bit m set
        // keep the upper half of their values, the others the lower half, and
        // each adds its partner's copy of the half it keeps; once one value
        // is left, plain butterflies finish the sum.  A fixed pattern, so the
        // result is deterministic.  Afterwards lane j holds in dot[i] (i < nv)
        // the total of edge u = (j / hstride) * nv + i.
        int m = L >> 1;
#pragma unroll
        for (int h = U / 2; h >= 1; h >>= 1) {
            if (m >= 1) {
                const bool up = (lane & m) != 0;
#pragma unroll
                for (int i = 0; i < h; ++i) {
                    const float send = up ? dot[i] : dot[i + h];
                    const float keep = up ? dot[i + h] : dot[i];
                    dot[i] = keep + __shfl_xor(send, m);
                }
                m >>= 1;
            }
        }
        for (; m >= 1; m >>= 1) dot[0] += __shfl_xor(dot[0], m);
        // lane t picks the total of position base + u*S + s from its holder
        const int rel = lane - base;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int s = rel - u * S;
            const bool mine = s >= 0 && s < S;
            const int src = ((mine ? s : 0) * L + (u / nv) * hstride) & (kWave - 1);
            float o = __shfl(dot[0], src);
            if (nv > 1) {
#pragma unroll
                for (int i = 1; i < U; ++i) {
                    if (i < nv) {
                        const float q = __shfl(dot[i], src);
                        if (i == u % nv) o = q;
                    }
                }
            }
            if (mine) result = o;
        }
    }
    if (lane < rem) {
        if constexpr (MODE == kMean) {
            const int64_t deg = rp_at(P.rowptr, P.rp64, (int64_t)myv + 1) - rp_at(P.rowptr, P.rp64, myv);
            result = result / (float)deg;
        }
        P.grad_w[P.oidx ? (int64_t)P.oidx[p0 + lane] : p0 + lane] = result;
    }
}

template <typename TX, typename TG, int EPL>
hipError_t launch_gw_mode(const GradWParams& p, unsigned grid, hipStream_t s) {
    if (p.reduce == kMax)
        hipLaunchKernelGGL((spmm_grad_w<TX, TG, EPL, kMax>), dim3(grid), dim3(kBlock), 0, s, p);
    else if (p.reduce == kMean)
        hipLaunchKernelGGL((spmm_grad_w<TX, TG, EPL, kMean>), dim3(grid), dim3(kBlock), 0, s, p);
    else
        hipLaunchKernelGGL((spmm_grad_w<TX, TG, EPL, kSum>), dim3(grid), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

template <typename TX, typename TG>
hipError_t launch_gw_epl(const GradWParams& p, int epl, unsigned grid, hipStream_t s) {
    switch (epl) {
        case 8: return launch_gw_mode<TX, TG, 8>(p, grid, s);
        case 4: return launch_gw_mode<TX, TG, 4>(p, grid, s);
        case 2: return launch_gw_mode<TX, TG, 2>(p, grid, s);
        default: return launch_gw_mode<TX, TG, 1>(p, grid, s);
    }
}

}  // namespace

hipError_t launch_rows_of_edges(const void* rowptr, int rp64, int64_t N, int64_t E, int32_t* row,
                                hipStream_t s) {
    if (E <= 0 || N <= 0) return hipSuccess;
    const unsigned grid = (unsigned)ceil_div(ceil_div(N, kWave), kWavesPerBlock);
    if (rp64)
        hipLaunchKernelGGL(rows_of_edges<int64_t>, dim3(grid), dim3(kBlock), 0, s,
                           static_cast<const int64_t*>(rowptr), N, E, row);
    else
        hipLaunchKernelGGL(rows_of_edges<int32_t>, dim3(grid), dim3(kBlock), 0, s,
                           static_cast<const int32_t*>(rowptr), N, E, row);
    return hipGetLastError();
}

hipError_t launch_win_masks(const void* rowptr, int rp64, const int32_t* argout, int64_t N,
                            int64_t F, uint32_t* bits, hipStream_t s) {
    if (N <= 0) return hipSuccess;
    const unsigned grid = (unsigned)ceil_div(ceil_div(N, kMaskRows), kWavesPerBlock);
    if (rp64)
        hipLaunchKernelGGL(win_masks<int64_t>, dim3(grid), dim3(kBlock), 0, s,
                           static_cast<const int64_t*>(rowptr), argout, N, F, win_mask_words(F),
                           bits);
    else
        hipLaunchKernelGGL(win_masks<int32_t>, dim3(grid), dim3(kBlock), 0, s,
                           static_cast<const int32_t*>(rowptr), argout, N, F, win_mask_words(F),
                           bits);
    return hipGetLastError();
}

hipError_t launch_scale_inv_deg(const void* g, int g_bf16, const void* rowptr, int rp64, int64_t N,
                                int64_t F, float* out, hipStream_t s) {
    const int64_t n = N * F;
    if (n <= 0) return hipSuccess;
    // four elements per thread when rows hold whole groups of four and the
    // gradient is aligned for it (out is a 256-byte aligned workspace)
    const bool v4 = F % 4 == 0 && (uintptr_t)g % (g_bf16 ? 8 : 16) == 0;
    const unsigned grid = (unsigned)ceil_div(v4 ? n / 4 : n, kBlock);
    if (g_bf16 && v4)
        hipLaunchKernelGGL((scale_inv_deg<true, 4>), dim3(grid), dim3(kBlock), 0, s, g, rowptr, rp64, N, F, out);
    else if (g_bf16)
        hipLaunchKernelGGL((scale_inv_deg<true, 1>), dim3(grid), dim3(kBlock), 0, s, g, rowptr, rp64, N, F, out);
    else if (v4)
        hipLaunchKernelGGL((scale_inv_deg<false, 4>), dim3(grid), dim3(kBlock), 0, s, g, rowptr, rp64, N, F, out);
    else
        hipLaunchKernelGGL((scale_inv_deg<false, 1>), dim3(grid), dim3(kBlock), 0, s, g, rowptr, rp64, N, F, out);
    return hipGetLastError();
}

hipError_t launch_spmm_grad_w(const GradWParams& p0, int x_dtype, int g_dtype, int epl,
                              hipStream_t s) {
    if (p0.E <= 0) return hipSuccess;
    // slots of a power-of-two width at aligned lanes, as the dot reduction
    // needs (lanes past the feature row hold zeros)
    GradWParams p = p0;
    if (p.L < kWave) {
        int lp = 1;
        while (lp < p.L) lp *= 2;
        p.L = lp;
        p.S = kWave / lp;
    }
    const int64_t waves = ceil_div(p.E, kWave);
    const unsigned grid = (unsigned)ceil_div(waves, kWavesPerBlock);
    if (x_dtype == MP_F32)
        return g_dtype == MP_F32 ? launch_gw_epl<float, float>(p, epl, grid, s)
                                 : launch_gw_epl<float, uint16_t>(p, epl, grid, s);
    return g_dtype == MP_F32 ? launch_gw_epl<uint16_t, float>(p, epl, grid, s)
                             : launch_gw_epl<uint16_t, uint16_t>(p, epl, grid, s);
}

}  // namespace mp
