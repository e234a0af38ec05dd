// Feature-table layout: copy the F elements of each row between tables whose
// rows lie ld_in and ld_out elements apart.  With an output stride whose row
// bytes are a multiple of the 128-byte cache line, every gathered row starts
// on a line boundary: a 200-byte bf16 row (F = 100) then spans two lines
// instead of two and a half on average, which the aggregation's random row
// gathers pay for in full.
#include "mp_internal.hpp"

namespace mp {
namespace {

constexpr int kBlock = 256;

// One thread per VB-byte chunk of a row (VB divides the row bytes and both
// strides in bytes, and the pointers are VB-aligned); a block covers whole
// rows, walked with a grid stride.
template <typename V>
__global__ __launch_bounds__(kBlock) void copy_rows(const char* __restrict__ in, int64_t ld_in,
                                                    char* __restrict__ out, int64_t ld_out,
                                                    int64_t N, int64_t cpr,
                                                    int64_t rows_per_block) {
    const int64_t nvb = (N + rows_per_block - 1) / rows_per_block;
    const uint32_t ucpr = (uint32_t)cpr;
    for (int64_t vb = blockIdx.x; vb < nvb; vb += gridDim.x) {
        const int64_t r0 = vb * rows_per_block;
        const int64_t nr = N - r0 < rows_per_block ? N - r0 : rows_per_block;
        const uint32_t n = (uint32_t)(nr * cpr);
        for (uint32_t l = threadIdx.x; l < n; l += kBlock) {
            const uint32_t dr = l / ucpr;
            const int64_t r = r0 + dr;
            const int64_t k = l - dr * ucpr;
            const V v = reinterpret_cast<const V*>(in + r * ld_in)[k];
            reinterpret_cast<V*>(out + r * ld_out)[k] = v;
        }
    }
}

}  // namespace

hipError_t launch_copy_rows(const void* in, int64_t ld_in, void* out, int64_t ld_out, int64_t N,
                            int64_t F, int elem_bytes, hipStream_t s) {
    if (N <= 0) return hipSuccess;
    const int64_t rb = F * elem_bytes, bi = ld_in * elem_bytes, bo = ld_out * elem_bytes;
    const uintptr_t al = (uintptr_t)in | (uintptr_t)out | (uintptr_t)rb | (uintptr_t)bi |
                         (uintptr_t)bo;
    int vb = 16;
    while (vb > 1 && al % (uintptr_t)vb != 0) vb >>= 1;
    const int64_t cpr = rb / vb;
    int64_t rpb = 4096 / cpr;
    if (rpb < 1) rpb = 1;
    int64_t grid = (N + rpb - 1) / rpb;
    if (grid > (int64_t(1) << 20)) grid = int64_t(1) << 20;
    const char* ci = static_cast<const char*>(in);
    char* co = static_cast<char*>(out);
    const dim3 g((unsigned)grid), b(kBlock);
    switch (vb) {
        case 16: hipLaunchKernelGGL(copy_rows<uint4>, g, b, 0, s, ci, bi, co, bo, N, cpr, rpb); break;
        case 8: hipLaunchKernelGGL(copy_rows<uint2>, g, b, 0, s, ci, bi, co, bo, N, cpr, rpb); break;
        case 4: hipLaunchKernelGGL(copy_rows<uint32_t>, g, b, 0, s, ci, bi, co, bo, N, cpr, rpb); break;
        case 2: hipLaunchKernelGGL(copy_rows<uint16_t>, g, b, 0, s, ci, bi, co, bo, N, cpr, rpb); break;
        default: hipLaunchKernelGGL(copy_rows<uint8_t>, g, b, 0, s, ci, bi, co, bo, N, cpr, rpb); break;
    }
    return hipGetLastError();
}

}  // namespace mp
