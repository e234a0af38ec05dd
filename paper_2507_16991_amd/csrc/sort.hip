// Stable LSD radix sort of COO edges by destination, and the small kernels
// around it (rowptr from the sorted keys, payload gather, validation).
//
// One pass over a digit: (1) every 4096-key tile counts its digits in LDS;
// (2) the digit-major table counts[d * tiles + t] is exclusive-scanned, giving
// each (digit, tile) its global output start; (3) every tile ranks its keys
// stably (wave-level multisplit with ballots, per-wave LDS counters), stages
// them in LDS in digit order and writes each digit's run contiguously.  Ranks
// follow (wave, round, lane) order, which is element order, so each pass is
// stable and the whole LSD sort keeps ascending COO id within a destination
// (the order the CSR of Sec. 2.2 must have to be unique).  Only integer
// arithmetic: the result is bit-exact.
#include "mp_internal.hpp"

#ifndef MP_SORT_NT_STORE
#define MP_SORT_NT_STORE 0
#endif

namespace mp {
namespace {

constexpr int kSortWaves = kSortBlock / kWave;
constexpr int kWaveKeys = kWave * kSortItems;  // keys per wavefront per tile
constexpr int kMaxBuckets = 1 << kSortMaxBits;

__global__ __launch_bounds__(kSortBlock) void radix_hist(const uint32_t* __restrict__ keys,
                                                         int64_t n, int shift, int bits,
                                                         uint32_t* __restrict__ counts,
                                                         int64_t tiles) {
    __shared__ uint32_t h[kMaxBuckets];
    const int R = 1 << bits;
    for (int i = threadIdx.x; i < R; i += kSortBlock) h[i] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
#pragma unroll 4
    for (int k = 0; k < kSortItems; ++k) {
        int64_t i = base + (int64_t)k * kSortBlock + threadIdx.x;
        if (i < n) atomicAdd(&h[(keys[i] >> shift) & (R - 1)], 1u);
    }
    __syncthreads();
    for (int d = threadIdx.x; d < R; d += kSortBlock) counts[(int64_t)d * tiles + blockIdx.x] = h[d];
}

// HAS_B: the second payload is carried (it costs 16 KB of LDS per tile, so
// the payload-free variant fits one more workgroup per CU).
template <bool HAS_B>
__global__ __launch_bounds__(kSortBlock) void radix_scatter(RadixPass p, int64_t tiles) {
    __shared__ uint32_t s_key[kSortTile];
    __shared__ int32_t s_a[kSortTile];
    __shared__ int32_t s_b[HAS_B ? kSortTile : 1];
    __shared__ uint32_t s_cnt[kSortWaves][kMaxBuckets];
    __shared__ uint32_t s_start[kMaxBuckets];
    __shared__ uint32_t s_gbase[kMaxBuckets];

    const int R = 1 << p.bits;
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x / kWave;
    for (int i = threadIdx.x; i < kSortWaves * kMaxBuckets; i += kSortBlock)
        (&s_cnt[0][0])[i] = 0;
    for (int d = threadIdx.x; d < R; d += kSortBlock)
        s_gbase[d] = p.counts[(int64_t)d * tiles + blockIdx.x];
    __syncthreads();

    const int64_t tbase = (int64_t)blockIdx.x * kSortTile;
    const int64_t wbase = tbase + (int64_t)wv * kWaveKeys;
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));

    uint32_t key[kSortItems];
    int32_t va[kSortItems], vb[kSortItems];
    uint32_t rank[kSortItems];
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = wbase + (int64_t)k * kWave + lane;
        const bool ok = i < p.n;
        key[k] = ok ? __builtin_nontemporal_load(p.keys_in + i) : 0u;
        va[k] = p.a_in ? (ok ? __builtin_nontemporal_load(p.a_in + i) : 0) : (int32_t)i;
        if constexpr (HAS_B) vb[k] = p.b_in ? (ok ? __builtin_nontemporal_load(p.b_in + i) : 0) : (int32_t)i;
    }
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = wbase + (int64_t)k * kWave + lane;
        const bool ok = i < p.n;
        const uint32_t d = (key[k] >> p.shift) & (uint32_t)(R - 1);
        // lanes holding a valid key with the same digit
        uint64_t peers = __ballot(ok);
        for (int b = 0; b < p.bits; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t bal = __ballot(bit);
            peers &= bit ? bal : ~bal;
        }
        const uint32_t below = (uint32_t)__popcll(peers & lt_mask);
        const uint32_t base = s_cnt[wv][d];
        rank[k] = base + below;
        // the lowest peer advances the counter for all of them; every lane has
        // read the old value above (LDS ops of one wavefront run in order)
        if (ok && below == 0) s_cnt[wv][d] = base + (uint32_t)__popcll(peers);
    }
    __syncthreads();

    // per digit: start of each wave's run inside the digit, tile total
    for (int d = threadIdx.x; d < R; d += kSortBlock) {
        uint32_t run = 0;
#pragma unroll
        for (int w = 0; w < kSortWaves; ++w) {
            uint32_t c = s_cnt[w][d];
            s_cnt[w][d] = run;
            run += c;
        }
        s_start[d] = run;
    }
    __syncthreads();
    // exclusive scan of the digit totals (R <= 256) by wavefront 0
    if (wv == 0) {
        uint32_t t[kMaxBuckets / kWave];
        uint32_t s = 0;
#pragma unroll
        for (int k = 0; k < kMaxBuckets / kWave; ++k) {
            int d = lane * (kMaxBuckets / kWave) + k;
            t[k] = d < R ? s_start[d] : 0u;
            s += t[k];
        }
        uint32_t inc = s;
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
            uint32_t o = __shfl_up(inc, off, kWave);
            if (lane >= off) inc += o;
        }
        uint32_t run = inc - s;
#pragma unroll
        for (int k = 0; k < kMaxBuckets / kWave; ++k) {
            int d = lane * (kMaxBuckets / kWave) + k;
            if (d < R) s_start[d] = run;
            run += t[k];
        }
    }
    __syncthreads();

#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = wbase + (int64_t)k * kWave + lane;
        if (i < p.n) {
            const uint32_t d = (key[k] >> p.shift) & (uint32_t)(R - 1);
            const uint32_t lp = s_start[d] + s_cnt[wv][d] + rank[k];
            s_key[lp] = key[k];
            s_a[lp] = va[k];
            if constexpr (HAS_B) s_b[lp] = vb[k];
        }
    }
    __syncthreads();

    const int64_t nvalid = (p.n - tbase) < kSortTile ? (p.n - tbase) : kSortTile;
    for (int i = threadIdx.x; i < nvalid; i += kSortBlock) {
        const uint32_t kk = s_key[i];
        const uint32_t d = (kk >> p.shift) & (uint32_t)(R - 1);
        const int64_t pos = (int64_t)s_gbase[d] + (i - (int64_t)s_start[d]);
        if (pos >= p.n) continue;  // cannot happen for consistent counts; never write past n
#if MP_SORT_NT_STORE
        if (p.keys_out) __builtin_nontemporal_store(kk, p.keys_out + pos);
        if (p.a_out) __builtin_nontemporal_store(s_a[i], p.a_out + pos);
        if constexpr (HAS_B) {
            if (p.b_out) __builtin_nontemporal_store(s_b[i], p.b_out + pos);
        }
#else
        if (p.keys_out) p.keys_out[pos] = kk;
        if (p.a_out) p.a_out[pos] = s_a[i];
        if constexpr (HAS_B) {
            if (p.b_out) p.b_out[pos] = s_b[i];
        }
#endif
    }
}

// rowptr[v] = first CSR position whose key is >= v, from the sorted keys:
// position p writes every v in (keys[p-1], keys[p]] (keys[-1] = -1,
// keys[E] = N), so each of the N+1 entries is written exactly once.  Each
// thread covers kRowptrItems consecutive positions.
constexpr int kRowptrItems = 8;

template <typename RP>
__global__ __launch_bounds__(256) void rowptr_from_sorted(const uint32_t* __restrict__ keys,
                                                          int64_t E, int64_t N, RP* __restrict__ rowptr) {
    const int64_t p0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * kRowptrItems;
    if (p0 > E) return;
    int64_t prev = p0 == 0 ? -1 : (int64_t)keys[p0 - 1];
#pragma unroll
    for (int k = 0; k < kRowptrItems; ++k) {
        const int64_t p = p0 + k;
        if (p > E) break;
        int64_t cur = p == E ? N : (int64_t)keys[p];
        if (cur > N) cur = N;  // keys are < N for valid input; stay inside rowptr regardless
        for (int64_t v = prev + 1; v <= cur; ++v) rowptr[v] = (RP)p;
        if (cur > prev) prev = cur;
    }
}

template <typename RP>
__global__ __launch_bounds__(256) void fill_zero(int64_t n, RP* __restrict__ out) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
        out[i] = 0;
}

__global__ __launch_bounds__(256) void gather_f32(const float* __restrict__ in,
                                                  const int32_t* __restrict__ idx, int64_t n,
                                                  float* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) out[i] = in[idx[i]];
}

__global__ __launch_bounds__(256) void offset_copy(const int32_t* __restrict__ in, int64_t n,
                                                   int32_t add, int32_t* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) out[i] = in[i] + add;
}

__global__ void zero_i64(int64_t* p) { *p = 0; }

__global__ __launch_bounds__(256) void validate_coo(const int32_t* __restrict__ src,
                                                    const int32_t* __restrict__ dst, int64_t E,
                                                    int64_t N_src, int64_t N_dst,
                                                    unsigned long long* count) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    unsigned bad = 0;
    if (i < E) {
        bad += (src[i] < 0 || src[i] >= N_src) ? 1u : 0u;
        bad += (dst[i] < 0 || dst[i] >= N_dst) ? 1u : 0u;
    }
    if (bad) atomicAdd(count, (unsigned long long)bad);
}

template <typename RP>
__global__ __launch_bounds__(256) void validate_csr(const RP* __restrict__ rowptr,
                                                    const int32_t* __restrict__ col,
                                                    int64_t N_dst, int64_t N_src, int64_t E,
                                                    unsigned long long* count) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    unsigned bad = 0;
    if (i < N_dst) bad += (rowptr[i + 1] < rowptr[i]) ? 1u : 0u;
    if (i == 0) {
        bad += (rowptr[0] != 0) ? 1u : 0u;
        bad += ((int64_t)rowptr[N_dst] != E) ? 1u : 0u;
    }
    if (i < E) bad += (col[i] < 0 || col[i] >= N_src) ? 1u : 0u;
    if (bad) atomicAdd(count, (unsigned long long)bad);
}

inline unsigned grid_for(int64_t n, int per_block) {
    return (unsigned)ceil_div(n > 0 ? n : 1, per_block);
}

}  // namespace

size_t radix_pass_counts_bytes(int64_t n, int bits) {
    const int64_t tiles = ceil_div(n > 0 ? n : 1, kSortTile);
    return align_up((size_t)tiles * ((size_t)1 << bits) * sizeof(uint32_t), 256);
}

hipError_t radix_pass(const RadixPass& p, hipStream_t s) {
    if (p.n <= 0) return hipSuccess;
    const int64_t tiles = ceil_div(p.n, kSortTile);
    hipLaunchKernelGGL(radix_hist, dim3((unsigned)tiles), dim3(kSortBlock), 0, s, p.keys_in, p.n,
                       p.shift, p.bits, p.counts, tiles);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = exclusive_scan_u32(p.counts, tiles << p.bits, p.scan_ws, s);
    if (e != hipSuccess) return e;
    if (p.b_out)
        hipLaunchKernelGGL(radix_scatter<true>, dim3((unsigned)tiles), dim3(kSortBlock), 0, s, p, tiles);
    else
        hipLaunchKernelGGL(radix_scatter<false>, dim3((unsigned)tiles), dim3(kSortBlock), 0, s, p, tiles);
    return hipGetLastError();
}

hipError_t launch_rowptr_from_sorted(const uint32_t* keys, int64_t E, int64_t N, void* rowptr,
                                     int rp64, hipStream_t s) {
    const unsigned g = grid_for(ceil_div(E + 1, kRowptrItems), 256);
    if (rp64)
        hipLaunchKernelGGL(rowptr_from_sorted<int64_t>, dim3(g), dim3(256), 0, s, keys, E, N,
                           static_cast<int64_t*>(rowptr));
    else
        hipLaunchKernelGGL(rowptr_from_sorted<int32_t>, dim3(g), dim3(256), 0, s, keys, E, N,
                           static_cast<int32_t*>(rowptr));
    return hipGetLastError();
}

hipError_t launch_fill_rowptr_zero(int64_t N, void* rowptr, int rp64, hipStream_t s) {
    const int64_t n = N + 1;
    unsigned g = grid_for(n, 256);
    if (g > 65536) g = 65536;
    if (rp64)
        hipLaunchKernelGGL(fill_zero<int64_t>, dim3(g), dim3(256), 0, s, n,
                           static_cast<int64_t*>(rowptr));
    else
        hipLaunchKernelGGL(fill_zero<int32_t>, dim3(g), dim3(256), 0, s, n,
                           static_cast<int32_t*>(rowptr));
    return hipGetLastError();
}

hipError_t launch_gather_f32(const float* in, const int32_t* idx, int64_t n, float* out,
                             hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(gather_f32, dim3(grid_for(n, 256)), dim3(256), 0, s, in, idx, n, out);
    return hipGetLastError();
}

hipError_t launch_offset_copy(const int32_t* in, int64_t n, int32_t add, int32_t* out,
                              hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(offset_copy, dim3(grid_for(n, 256)), dim3(256), 0, s, in, n, add, out);
    return hipGetLastError();
}

hipError_t launch_validate_coo(const int32_t* src, const int32_t* dst, int64_t E, int64_t N_src,
                               int64_t N_dst, int64_t* d_count, hipStream_t s) {
    hipLaunchKernelGGL(zero_i64, dim3(1), dim3(1), 0, s, d_count);
    if (E > 0)
        hipLaunchKernelGGL(validate_coo, dim3(grid_for(E, 256)), dim3(256), 0, s, src, dst, E,
                           N_src, N_dst, reinterpret_cast<unsigned long long*>(d_count));
    return hipGetLastError();
}

hipError_t launch_validate_csr(const void* rowptr, int rp64, const int32_t* col, int64_t N_dst,
                               int64_t N_src, int64_t E, int64_t* d_count, hipStream_t s) {
    hipLaunchKernelGGL(zero_i64, dim3(1), dim3(1), 0, s, d_count);
    const int64_t n = (N_dst > E ? N_dst : E) + 1;
    auto* c = reinterpret_cast<unsigned long long*>(d_count);
    if (rp64)
        hipLaunchKernelGGL(validate_csr<int64_t>, dim3(grid_for(n, 256)), dim3(256), 0, s,
                           static_cast<const int64_t*>(rowptr), col, N_dst, N_src, E, c);
    else
        hipLaunchKernelGGL(validate_csr<int32_t>, dim3(grid_for(n, 256)), dim3(256), 0, s,
                           static_cast<const int32_t*>(rowptr), col, N_dst, N_src, E, c);
    return hipGetLastError();
}

}  // namespace mp
