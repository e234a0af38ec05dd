// Device exclusive scan of uint32 arrays (reduce, scan the tile sums, apply).
// Used for the radix-sort digit offsets and the plan's chunk offsets.  All
// sums are integer, so the result is exact and independent of scheduling.
#include "mp_internal.hpp"

namespace mp {
namespace {

__device__ inline uint32_t wave_inclusive_scan(uint32_t v) {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        uint32_t t = __shfl_up(v, off, kWave);
        if (lane >= off) v += t;
    }
    return v;
}

// Exclusive scan of one value per thread across a block of kScanBlock threads.
// Returns the exclusive prefix; *total receives the block total.
__device__ inline uint32_t block_exclusive_scan(uint32_t v, uint32_t* total) {
    __shared__ uint32_t wsum[kScanBlock / kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x / kWave;
    uint32_t inc = wave_inclusive_scan(v);
    if (lane == kWave - 1) wsum[wv] = inc;
    __syncthreads();
    uint32_t before = 0, all = 0;
#pragma unroll
    for (int k = 0; k < kScanBlock / kWave; ++k) {
        uint32_t t = wsum[k];
        before += (k < wv) ? t : 0u;
        all += t;
    }
    __syncthreads();  // wsum may be reused by the caller's next call
    *total = all;
    return before + inc - v;
}

// zero_below (device, or nullptr): data[i] = 0 for every i below *zero_below,
// so tiles that end there have sum 0 and keep their (all-zero) prefixes.
__device__ inline bool tile_all_zero(const uint32_t* zero_below, int64_t base) {
    return zero_below && base + kScanTile <= (int64_t)*zero_below;
}

__global__ __launch_bounds__(kScanBlock) void scan_tile_sums(const uint32_t* __restrict__ in,
                                                             int64_t n, uint32_t* __restrict__ part,
                                                             const uint32_t* zero_below) {
    const int64_t base = (int64_t)blockIdx.x * kScanTile;
    if (tile_all_zero(zero_below, base)) {
        if (threadIdx.x == 0) part[blockIdx.x] = 0;
        return;
    }
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        int64_t i = base + (int64_t)k * kScanBlock + threadIdx.x;
        if (i < n) s += in[i];
    }
    uint32_t total;
    block_exclusive_scan(s, &total);
    if (threadIdx.x == 0) part[blockIdx.x] = total;
}

// Single workgroup: exclusive scan of the tile sums, in chunks of kScanBlock.
__global__ __launch_bounds__(kScanBlock) void scan_partials(uint32_t* __restrict__ part,
                                                            int64_t m) {
    uint32_t carry = 0;
    for (int64_t base = 0; base < m; base += kScanBlock) {
        int64_t i = base + threadIdx.x;
        uint32_t v = i < m ? part[i] : 0u;
        uint32_t total;
        uint32_t ex = block_exclusive_scan(v, &total);
        if (i < m) part[i] = carry + ex;
        carry += total;
    }
}

// Each thread owns kScanItems consecutive elements of the tile.
__global__ __launch_bounds__(kScanBlock) void scan_apply(uint32_t* __restrict__ data, int64_t n,
                                                         const uint32_t* __restrict__ part,
                                                         const uint32_t* zero_below) {
    if (tile_all_zero(zero_below, (int64_t)blockIdx.x * kScanTile)) return;
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    uint32_t v[kScanItems];
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        int64_t i = base + k;
        v[k] = i < n ? data[i] : 0u;
        s += v[k];
    }
    uint32_t total;
    uint32_t run = part[blockIdx.x] + block_exclusive_scan(s, &total);
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        int64_t i = base + k;
        if (i < n) data[i] = run;
        run += v[k];
    }
}

}  // namespace

size_t scan_workspace_bytes(int64_t n) {
    int64_t tiles = ceil_div(n > 0 ? n : 1, kScanTile);
    return align_up((size_t)tiles * sizeof(uint32_t), 256);
}

hipError_t exclusive_scan_u32(uint32_t* data, int64_t n, void* ws, hipStream_t s,
                              const uint32_t* zero_below) {
    if (n <= 0) return hipSuccess;
    const int64_t tiles = ceil_div(n, kScanTile);
    uint32_t* part = static_cast<uint32_t*>(ws);
    hipLaunchKernelGGL(scan_tile_sums, dim3((unsigned)tiles), dim3(kScanBlock), 0, s, data, n, part,
                       zero_below);
    hipLaunchKernelGGL(scan_partials, dim3(1), dim3(kScanBlock), 0, s, part, tiles);
    hipLaunchKernelGGL(scan_apply, dim3((unsigned)tiles), dim3(kScanBlock), 0, s, data, n, part,
                       zero_below);
    return hipGetLastError();
}

}  // namespace mp
