// Bandwidth probes: the simplest kernels with the aggregation's memory
// traffic, used to measure what the hardware delivers for it (the achievable
// ceiling the aggregation kernels are compared with, next to the published
// HBM peak).  A streaming read and a streaming copy of a buffer, and a row
// gather that reads, for every index of a given stream, one row of a table in
// that order -- the aggregation's own gather (its CSR column stream) with no
// reduction, no output rows and no degree structure.  Every loaded word is
// folded into an XOR that each wavefront stores once, so no load is dead.
// And a scatter that writes every element of a buffer to the position a
// destination stream gives it -- a radix pass's data movement (its digit
// runs) with no ranking, no staging and no look-back.
#include "mp_internal.hpp"

namespace mp {
namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / kWave;
constexpr int kReadUnroll = 4;       // 16-byte loads in flight per thread per iteration
constexpr int kGatherUnroll = 8;     // rows per slot per step, as in the aggregation
constexpr int64_t kGatherPerWave = 1024;  // indices per wavefront

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline uint32_t fold(const u32x4& v) { return v.x ^ v.y ^ v.z ^ v.w; }

// XOR over the wavefront; lane 0 stores it.
__device__ inline void sink_wave(uint32_t x, uint32_t* __restrict__ sink, int64_t slot) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x ^= (uint32_t)__shfl_xor((int)x, off);
    if ((threadIdx.x & (kWave - 1)) == 0) sink[slot] = x;
}

__global__ __launch_bounds__(kBlock) void probe_read(const u32x4* __restrict__ p, int64_t n,
                                                     uint32_t* __restrict__ sink) {
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    uint32_t x = 0;
    int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    for (; i + (kReadUnroll - 1) * stride < n; i += kReadUnroll * stride) {
        u32x4 v[kReadUnroll];
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) x ^= fold(v[u]);
    }
    for (; i < n; i += stride) x ^= fold(p[i]);
    sink_wave(x, sink, (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave);
}

__global__ __launch_bounds__(kBlock) void probe_copy(const u32x4* __restrict__ in,
                                                     u32x4* __restrict__ out, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    for (; i + (kReadUnroll - 1) * stride < n; i += kReadUnroll * stride) {
        u32x4 v[kReadUnroll];
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) v[u] = in[i + u * stride];
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) out[i + u * stride] = v[u];
    }
    for (; i < n; i += stride) out[i] = in[i];
}

// Each wavefront walks chunks of kGatherPerWave consecutive indices (chunk
// wv, wv + waves, ...): slots of L lanes (L = 16-byte chunks of a row, S =
// 64 / L slots), U rows per slot per step, the indices loaded once per 64,
// coalesced, and passed by cross-lane permute -- the geometry of the
// aggregation's gather.
__global__ __launch_bounds__(kBlock) void probe_gather(const int32_t* __restrict__ idx, int64_t n,
                                                       const char* __restrict__ table,
                                                       int64_t stride_bytes, int L,
                                                       uint32_t* __restrict__ sink) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wv = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave;
    const int64_t nw = (int64_t)gridDim.x * kWaves;
    const int S = kWave / L;
    const int slot = lane / L;
    const int j = lane - slot * L;
    const bool lane_ok = slot < S;
    int U = kGatherUnroll;
    if (S * U > kWave) U = kWave / S;
    const int SU = S * U;
    const int steps = kWave / SU;
    const int tile = steps * SU;
    uint32_t x = 0;
    for (int64_t e0 = wv * kGatherPerWave; e0 < n; e0 += nw * kGatherPerWave) {
        const int64_t e1 = e0 + kGatherPerWave < n ? e0 + kGatherPerWave : n;
        for (int64_t p0 = e0; p0 < e1; p0 += tile) {
            const int64_t rem = e1 - p0;
            const int32_t myc =
                (lane < tile && lane < rem) ? __builtin_nontemporal_load(idx + p0 + lane) : 0;
            for (int st = 0; st < steps; ++st) {
                const int base = st * SU;
                if (base >= rem) break;
                u32x4 v[kGatherUnroll];
                bool ok[kGatherUnroll];
#pragma unroll
                for (int u = 0; u < kGatherUnroll; ++u) {
                    const int t = base + u * S + slot;
                    const int32_t c = __shfl(myc, t & (kWave - 1));
                    ok[u] = lane_ok && u < U && t < rem;
                    if (ok[u])
                        v[u] = *reinterpret_cast<const u32x4*>(table + (int64_t)c * stride_bytes +
                                                               j * 16);
                }
#pragma unroll
                for (int u = 0; u < kGatherUnroll; ++u)
                    if (ok[u]) x ^= fold(v[u]);
            }
        }
    }
    sink_wave(x, sink, wv);
}

// out[dest[i]] = in[i] for i in [0, n): in and dest read in order, out
// written where dest says (dest is a permutation of [0, n), which the caller
// guarantees).
template <typename T>
__global__ __launch_bounds__(kBlock) void probe_scatter(const T* __restrict__ in,
                                                        const int32_t* __restrict__ dest,
                                                        int64_t n, T* __restrict__ out) {
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    for (; i + (kReadUnroll - 1) * stride < n; i += kReadUnroll * stride) {
        T v[kReadUnroll];
        int32_t d[kReadUnroll];
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) {
            v[u] = __builtin_nontemporal_load(in + i + u * stride);
            d[u] = __builtin_nontemporal_load(dest + i + u * stride);
        }
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) out[d[u]] = v[u];
    }
    for (; i < n; i += stride) out[dest[i]] = in[i];
}

constexpr int64_t kMaxGrid = MP_PROBE_SINK_WORDS / kWaves;  // one sink word per wavefront

unsigned grid_for(int64_t n16) {
    int64_t g = (n16 + kBlock * kReadUnroll - 1) / (kBlock * kReadUnroll);
    if (g > kMaxGrid) g = kMaxGrid;
    if (g < 1) g = 1;
    return (unsigned)g;
}

}  // namespace

hipError_t launch_probe_read(const void* p, int64_t n16, uint32_t* sink, hipStream_t s) {
    hipLaunchKernelGGL(probe_read, dim3(grid_for(n16)), dim3(kBlock), 0, s,
                       static_cast<const u32x4*>(p), n16, sink);
    return hipGetLastError();
}

hipError_t launch_probe_copy(const void* in, void* out, int64_t n16, hipStream_t s) {
    hipLaunchKernelGGL(probe_copy, dim3(grid_for(n16)), dim3(kBlock), 0, s,
                       static_cast<const u32x4*>(in), static_cast<u32x4*>(out), n16);
    return hipGetLastError();
}

hipError_t launch_probe_scatter(const void* in, const int32_t* dest, int64_t n, int elem_bytes,
                                void* out, hipStream_t s) {
    if (elem_bytes == 8)
        hipLaunchKernelGGL(probe_scatter<uint64_t>, dim3(grid_for(n)), dim3(kBlock), 0, s,
                           static_cast<const uint64_t*>(in), dest, n, static_cast<uint64_t*>(out));
    else
        hipLaunchKernelGGL(probe_scatter<uint32_t>, dim3(grid_for(n)), dim3(kBlock), 0, s,
                           static_cast<const uint32_t*>(in), dest, n, static_cast<uint32_t*>(out));
    return hipGetLastError();
}

hipError_t launch_probe_gather(const int32_t* idx, int64_t n, const void* table,
                               int64_t stride_bytes, int L, uint32_t* sink, hipStream_t s) {
    const int64_t chunks = (n + kGatherPerWave - 1) / kGatherPerWave;
    int64_t grid = (chunks + kWaves - 1) / kWaves;
    if (grid > kMaxGrid) grid = kMaxGrid;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(probe_gather, dim3((unsigned)grid), dim3(kBlock), 0, s, idx, n,
                       static_cast<const char*>(table), stride_bytes, L, sink);
    return hipGetLastError();
}

}  // namespace mp
