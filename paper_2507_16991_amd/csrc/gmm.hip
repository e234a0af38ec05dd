// Segment matmul on the matrix cores (Sec. 2.2, heterogeneous GNNs: the
// projections {H_T W_T} over node types with a weight tensor [|T|, F, F'],
// and their gradients with respect to H_T and W).
//
// Rows of X are grouped by type in contiguous segments; segment t is
// multiplied by W[t].  All products use the gfx950 bf16 MFMA
// v_mfma_f32_32x32x16_bf16 with fp32 accumulation:
//   * gmm_nt: C[r, n] = sum_k A[r, k] * Bt[t][n, k] for the rows r of segment
//     t (forward with Bt = W^T; input gradient with A = dOut, Bt = W).
//     Block tile 128 x 128, K in steps of 32 through LDS, four wavefronts of
//     64 x 64 (2 x 2 MFMA tiles each).  A tile never spans two segments.
//   * gmm_tn_partial + reduce_partials: the weight gradient dW[t] =
//     X_t^T dOut_t, a reduction over the segment's rows: fixed chunks of rows
//     give fp32 partial tiles that a second kernel adds in a fixed order (no
//     atomics, deterministic).
//
// MFMA operand layout (32x32x16 bf16, wave64): lane l holds A[l % 32][8 (l/32)
// + 0..7] and B[8 (l/32) + 0..7][l % 32]; accumulator element v of lane l is
// C[8 (v/4) + 4 (l/32) + v % 4][l % 32].
#include "mp_internal.hpp"

namespace mp {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kBM = 128, kBN = 128, kBK = 32;
constexpr int kPad = 8;               // bf16 of padding per LDS row (bank spread)
constexpr int kLds = kBK + kPad;      // LDS row length in bf16
constexpr int kThreads = 256;         // four wavefronts, 2 x 2 over the tile

__device__ inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Accumulate one 128 x 128 tile from the LDS tiles As[m][k], Bs[n][k] of one
// K step (two MFMA K16 steps).  acc[i][j]: rows wm*64 + i*32, cols wn*64 + j*32.
__device__ inline void mma_step(const uint16_t (*As)[kLds], const uint16_t (*Bs)[kLds], int wm,
                                int wn, int lane, f32x16 (&acc)[2][2]) {
#pragma unroll
    for (int s = 0; s < kBK / 16; ++s) {
        const int kk = s * 16 + 8 * (lane >> 5);
        bf16x8 a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const uint4 va = *reinterpret_cast<const uint4*>(&As[wm * 64 + i * 32 + (lane & 31)][kk]);
            a[i] = __builtin_bit_cast(bf16x8, va);
            const uint4 vb = *reinterpret_cast<const uint4*>(&Bs[wn * 64 + i * 32 + (lane & 31)][kk]);
            b[i] = __builtin_bit_cast(bf16x8, vb);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
}

// Write the 128 x 128 accumulator tile to C (fp32 or bf16), rows below
// row_end and columns below ncols only.
__device__ inline void store_tile(const f32x16 (&acc)[2][2], int64_t r0, int64_t row_end,
                                  int64_t n0, int64_t ncols, int wm, int wn, int lane, void* C,
                                  int64_t ldc, int c_bf16) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t col = n0 + wn * 64 + j * 32 + (lane & 31);
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t row = r0 + wm * 64 + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                if (row < row_end && col < ncols) {
                    if (c_bf16)
                        static_cast<uint16_t*>(C)[row * ldc + col] = f32_to_bf16_rne(acc[i][j][v]);
                    else
                        static_cast<float*>(C)[row * ldc + col] = acc[i][j][v];
                }
            }
        }
}

// C[r, n] = sum_k A[r, k] Bt[t][n, k] for the rows of segment t.
__global__ __launch_bounds__(kThreads) void gmm_nt(GmmParams P) {
    __shared__ __attribute__((aligned(16))) uint16_t As[kBM][kLds];  // rows of 80 B: 16-B reads
    __shared__ __attribute__((aligned(16))) uint16_t Bs[kBN][kLds];
    const int64_t tile = blockIdx.x;
    int t = 0;
    while (t + 1 < P.T && P.tile_off[t + 1] <= tile) ++t;
    const int64_t local = tile - P.tile_off[t];
    const int64_t ntn = (P.N + kBN - 1) / kBN;
    const int64_t rt = local / ntn, ct = local - rt * ntn;
    const int64_t r0 = P.seg[t] + rt * kBM, row_end = P.seg[t + 1];
    const int64_t n0 = ct * kBN;
    const uint16_t* A = P.A;
    const uint16_t* Bt = P.B + (int64_t)t * P.b_stride;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int wm = w >> 1, wn = w & 1;

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // the next K step's tiles are loaded into registers while this one's
    // products run
    uint4 ra[2], rb[2];
    auto load = [&](int64_t k0) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int c = tid + kThreads * q;  // 512 chunks of 8 bf16 per tile
            const int row = c >> 2, kc = (c & 3) * 8;
            const int64_t gr = r0 + row, gn = n0 + row, gk = k0 + kc;
            ra[q] = make_uint4(0, 0, 0, 0);
            rb[q] = make_uint4(0, 0, 0, 0);
            if (gr < row_end && gk < P.K) ra[q] = *reinterpret_cast<const uint4*>(A + gr * P.lda + gk);
            if (gn < P.N && gk < P.K) rb[q] = *reinterpret_cast<const uint4*>(Bt + gn * P.ldb + gk);
        }
    };
    load(0);
    for (int64_t k0 = 0; k0 < P.K; k0 += kBK) {
        __syncthreads();  // the previous step's reads of As/Bs are done
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int c = tid + kThreads * q;
            const int row = c >> 2, kc = (c & 3) * 8;
            *reinterpret_cast<uint4*>(&As[row][kc]) = ra[q];
            *reinterpret_cast<uint4*>(&Bs[row][kc]) = rb[q];
        }
        __syncthreads();
        if (k0 + kBK < P.K) load(k0 + kBK);
        mma_step(As, Bs, wm, wn, lane, acc);
    }
    store_tile(acc, r0, row_end, n0, P.N, wm, wn, lane, P.C, P.ldc, P.c_bf16);
}

// Partial weight gradient of one chunk of rows of segment t:
// Part[chunk][m, n] = sum over the chunk's rows r of X[r, m] * G[r, n].
// The reduction index k is the row r, so the operand tiles are kept in LDS
// in their natural row-major layout, [k][m] and [k][n], written with 8-byte
// stores; a fragment (eight consecutive k at one m) is then gathered with
// eight 2-byte reads.  Rows of kTnLds bf16 (264 B) put rows k and k + 8 on
// different banks, so the two halves of a wavefront do not collide.
constexpr int kTnLds = kBM + 4;

__device__ inline void mma_step_tn(const uint16_t (*As)[kTnLds], const uint16_t (*Bs)[kTnLds],
                                   int wm, int wn, int lane, f32x16 (&acc)[2][2]) {
#pragma unroll
    for (int s = 0; s < kBK / 16; ++s) {
        const int kk = s * 16 + 8 * (lane >> 5);
        bf16x8 a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int m = wm * 64 + i * 32 + (lane & 31);
            const int n = wn * 64 + i * 32 + (lane & 31);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                a[i][j] = __builtin_bit_cast(__bf16, As[kk + j][m]);
                b[i][j] = __builtin_bit_cast(__bf16, Bs[kk + j][n]);
            }
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
}

__global__ __launch_bounds__(kThreads) void gmm_tn_partial(GmmParams P) {
    __shared__ __attribute__((aligned(16))) uint16_t As[kBK][kTnLds];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[kBK][kTnLds];
    const int64_t tile = blockIdx.x;
    const int64_t ntm = (P.M + kBM - 1) / kBM, ntn = (P.N + kBN - 1) / kBN;
    const int64_t chunk = tile / (ntm * ntn);
    const int64_t rest = tile - chunk * ntm * ntn;
    const int64_t mt = rest / ntn, nt = rest - mt * ntn;
    int t = 0;
    while (t + 1 < P.T && P.tile_off[t + 1] <= chunk) ++t;  // tile_off: chunk offsets here
    const int64_t r_begin = P.seg[t] + (chunk - P.tile_off[t]) * P.rows_per_chunk;
    const int64_t r_end_seg = P.seg[t + 1];
    const int64_t r_end = r_begin + P.rows_per_chunk < r_end_seg ? r_begin + P.rows_per_chunk : r_end_seg;
    const int64_t m0 = mt * kBM, n0 = nt * kBN;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int wm = w >> 1, wn = w & 1;

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    uint4 ra[2], rb[2];
    auto load = [&](int64_t k0) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int c = tid + kThreads * q;  // 32 rows x 16 chunks of 8 bf16
            const int kr = c >> 4, mc = (c & 15) * 8;
            const int64_t gr = k0 + kr;
            ra[q] = make_uint4(0, 0, 0, 0);
            rb[q] = make_uint4(0, 0, 0, 0);
            if (gr < r_end && m0 + mc < P.M) ra[q] = *reinterpret_cast<const uint4*>(P.A + gr * P.lda + m0 + mc);
            if (gr < r_end && n0 + mc < P.N) rb[q] = *reinterpret_cast<const uint4*>(P.B + gr * P.ldb + n0 + mc);
        }
    };
    load(r_begin);
    for (int64_t k0 = r_begin; k0 < r_end; k0 += kBK) {
        __syncthreads();
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int c = tid + kThreads * q;
            const int kr = c >> 4, mc = (c & 15) * 8;
            uint2* pa = reinterpret_cast<uint2*>(&As[kr][mc]);
            uint2* pb = reinterpret_cast<uint2*>(&Bs[kr][mc]);
            pa[0] = make_uint2(ra[q].x, ra[q].y);
            pa[1] = make_uint2(ra[q].z, ra[q].w);
            pb[0] = make_uint2(rb[q].x, rb[q].y);
            pb[1] = make_uint2(rb[q].z, rb[q].w);
        }
        __syncthreads();
        if (k0 + kBK < r_end) load(k0 + kBK);  // in flight during the products
        mma_step_tn(As, Bs, wm, wn, lane, acc);
    }
    float* part = P.part + chunk * P.M * P.N;
    store_tile(acc, m0, P.M, n0, P.N, wm, wn, lane, part, P.N, 0);
}

// dW[t][i] = sum over the chunks of segment t of Part[chunk][i], in a fixed
// order: eight running sums over chunks c = 8q + s, then a fixed tree.  Eight
// independent loads per iteration keep the long sums from waiting on each
// load in turn.
__global__ __launch_bounds__(256) void reduce_partials(GmmParams P, float* __restrict__ dW) {
    const int64_t mn = P.M * P.N;
    const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (g >= (int64_t)P.T * mn) return;
    const int t = (int)(g / mn);
    const int64_t i = g - (int64_t)t * mn;
    const int64_t c0 = P.tile_off[t], c1 = P.tile_off[t + 1];
    float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int64_t c = c0; c < c1; c += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = c + u < c1 ? P.part[(c + u) * mn + i] : 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u) s[u] += v[u];
    }
    dW[g] = ((s[0] + s[1]) + (s[2] + s[3])) + ((s[4] + s[5]) + (s[6] + s[7]));
}

// Wt[t][o][f] = W[t][f][o] (bf16).
__global__ __launch_bounds__(256) void transpose_w(const uint16_t* __restrict__ W, int64_t T,
                                                   int64_t F, int64_t Fo,
                                                   uint16_t* __restrict__ Wt) {
    const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (g >= T * F * Fo) return;
    const int64_t t = g / (F * Fo);
    const int64_t r = g - t * F * Fo;
    const int64_t o = r / F, f = r - o * F;
    Wt[g] = W[t * F * Fo + f * Fo + o];
}

}  // namespace

hipError_t launch_gmm_nt(const GmmParams& p, int64_t tiles, hipStream_t s) {
    if (tiles <= 0) return hipSuccess;
    hipLaunchKernelGGL(gmm_nt, dim3((unsigned)tiles), dim3(kThreads), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_gmm_weight_grad(const GmmParams& p, int64_t chunks, float* dW, hipStream_t s) {
    const int64_t tiles = chunks * ((p.M + kBM - 1) / kBM) * ((p.N + kBN - 1) / kBN);
    if (tiles > 0) hipLaunchKernelGGL(gmm_tn_partial, dim3((unsigned)tiles), dim3(kThreads), 0, s, p);
    const int64_t n = (int64_t)p.T * p.M * p.N;
    hipLaunchKernelGGL(reduce_partials, dim3((unsigned)ceil_div(n, 256)), dim3(256), 0, s, p, dW);
    return hipGetLastError();
}

hipError_t launch_transpose_w(const uint16_t* W, int64_t T, int64_t F, int64_t Fo, uint16_t* Wt,
                              hipStream_t s) {
    const int64_t n = T * F * Fo;
    hipLaunchKernelGGL(transpose_w, dim3((unsigned)ceil_div(n, 256)), dim3(256), 0, s, W, T, F, Fo,
                       Wt);
    return hipGetLastError();
}

int64_t gmm_tile_rows() { return kBM; }
int64_t gmm_tile_cols() { return kBN; }

}  // namespace mp
