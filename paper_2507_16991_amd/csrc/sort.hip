// Stable LSD radix sort of COO edges by destination, and the small kernels
// around it (rowptr from the sorted keys, payload gather, validation).
//
// The sort is one-sweep: radix_ghist counts the digits of every pass in one
// read of the keys; then each pass is ONE kernel, radix_onesweep, in which a
// tile of kSortTile keys (tile ids taken from an atomic counter in launch
// order) ranks its keys stably (wave-level multisplit: one ballot per digit
// bit, per-wavefront LDS counters), publishes its per-digit counts, obtains
// the running totals of all earlier tiles by decoupled look-back over their
// published descriptors, stages the tile in LDS in digit order and writes
// each digit's run contiguously.  Ranks follow (wave, round, lane) order,
// which is element order, so each pass is stable and the whole LSD sort keeps
// ascending COO id within a destination (the order the CSR of Sec. 2.2 must
// have to be unique).  Only integer arithmetic: the result is bit-exact.
//
// The look-back only waits on tiles that started earlier (their ids were
// taken first), so it always ends; its wait is nevertheless bounded, and a
// tile that gives up records it in an error word that the caller turns into
// MP_ERR_SORT (radix_status) instead of hanging the device.
#include "mp_internal.hpp"

namespace mp {
namespace {

constexpr int kSortWaves = kSortBlock / kWave;
constexpr int kWaveKeys = kWave * kSortItems;  // keys per wavefront per tile
constexpr int kMaxBuckets = 1 << kSortMaxBits;

constexpr int kGhistBlock = 256;
constexpr int kGhistItems = 8;
constexpr uint32_t kSpinLimit = 1u << 20;

// look-back descriptor: flag (bits 63..62: 1 tile count, 2 inclusive prefix),
// pass tag (bits 61..56, pass + 1), value (bits 55..0)
constexpr uint64_t kFlagAgg = 1ull << 62;
constexpr uint64_t kFlagPre = 2ull << 62;
__device__ inline uint64_t desc_make(uint64_t flag, uint32_t tag, uint64_t v) {
    return flag | ((uint64_t)tag << 56) | v;
}

// Lanes of the wavefront that hold a valid key with the same digit as this
// lane: one ballot per digit bit; a lane differs from this one where the
// ballot's bit differs from this lane's own bit (sign-extended to a full
// word, so that one XOR per half-mask finds those lanes).  The bits are
// unrolled up to kSortMaxBits under a wave-uniform test.
__device__ inline uint64_t digit_peers(bool ok, uint32_t d, int bits) {
    uint32_t dlo = 0, dhi = 0;  // lanes whose digit differs in some bit
#pragma unroll
    for (int b = 0; b < kSortMaxBits; ++b) {
        if (b < bits) {
            const int32_t sb = (int32_t)(d << (31 - b)) >> 31;  // 0 or -1
            const uint64_t bal = __ballot(sb != 0);
            dlo |= (uint32_t)bal ^ (uint32_t)sb;
            dhi |= (uint32_t)(bal >> 32) ^ (uint32_t)sb;
        }
    }
    return __ballot(ok) & ~(((uint64_t)dhi << 32) | dlo);
}

// Set bits of m below this lane.
__device__ inline uint32_t count_below(uint64_t m) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__global__ __launch_bounds__(256) void radix_clear(uint64_t* __restrict__ desc, int64_t ndesc,
                                                   uint32_t* __restrict__ gbase,
                                                   uint32_t* __restrict__ counter,
                                                   uint32_t* __restrict__ err) {
    const int64_t i0 = (int64_t)blockIdx.x * 256 + threadIdx.x;
    for (int64_t i = i0; i < ndesc; i += (int64_t)gridDim.x * 256) desc[i] = 0;
    if (i0 < kMaxPasses * kMaxBuckets) gbase[i0] = 0;
    if (i0 < kMaxPasses) counter[i0] = 0;
    if (i0 == 0) *err = 0;
}

// Global histogram of every pass's digit.  Counts do not depend on order, so
// each wavefront adds into its own LDS copy with integer atomics (no ranking
// needed), then one integer atomic per (pass, digit) per workgroup.
// shifts and widths: one byte per pass (pass p in bits 8p..8p+7).
__global__ __launch_bounds__(kGhistBlock) void radix_ghist(const uint32_t* __restrict__ keys,
                                                           int64_t n, int passes, uint32_t shifts,
                                                           uint32_t widths,
                                                           uint32_t* __restrict__ ghist) {
    constexpr int W = kGhistBlock / kWave;
    __shared__ uint32_t h[W][kMaxPasses][kMaxBuckets];
    for (int i = threadIdx.x; i < W * kMaxPasses * kMaxBuckets; i += kGhistBlock)
        (&h[0][0][0])[i] = 0;
    __syncthreads();
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x / kWave;
    const int64_t stride = (int64_t)gridDim.x * W * kWave * kGhistItems;
    for (int64_t base = ((int64_t)blockIdx.x * W + wv) * kWave * kGhistItems; base < n;
         base += stride) {
        uint32_t key[kGhistItems];
#pragma unroll
        for (int k = 0; k < kGhistItems; ++k) {
            const int64_t i = base + (int64_t)k * kWave + lane;
            key[k] = i < n ? __builtin_nontemporal_load(keys + i) : 0u;
        }
#pragma unroll
        for (int k = 0; k < kGhistItems; ++k) {
            if (base + (int64_t)k * kWave + lane >= n) continue;
            for (int p = 0; p < passes; ++p) {
                const uint32_t sh = (shifts >> (8 * p)) & 255u;
                const uint32_t mask = (1u << ((widths >> (8 * p)) & 255u)) - 1u;
                atomicAdd(&h[wv][p][(key[k] >> sh) & mask], 1u);
            }
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < passes * kMaxBuckets; i += kGhistBlock) {
        uint32_t t = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) t += (&h[w][0][0])[i];
        if (t) atomicAdd(&ghist[i], t);
    }
}

// In place: per pass, exclusive scan over its digit counts (the counts of
// digits beyond a pass's width are zero).
__global__ void radix_gscan(uint32_t* __restrict__ g, int passes) {
    const int p = threadIdx.x;
    if (p >= passes) return;
    uint32_t run = 0;
    for (int d = 0; d < kMaxBuckets; ++d) {
        const uint32_t c = g[p * kMaxBuckets + d];
        g[p * kMaxBuckets + d] = run;
        run += c;
    }
}

// One LSD pass: rank the tile's keys stably (wave-level multisplit, per-wave
// LDS counters), publish the tile's digit counts, stage the tile in LDS in
// digit order, then look back over earlier tiles for their running totals
// and write every digit run contiguously.  Ranks follow (wave, round, lane)
// order, which is element order, and tiles are numbered in the order they
// start, so the pass is stable.  Staging before the look-back frees the
// registers of the keys while the tile waits on its predecessors, so the
// look-back can keep kLookWindow descriptor loads in flight.  Descriptors of
// a pass over R = 2^bits digits lie R apart per tile.
//   HAS_B: the second payload is carried.
//   WIDE:  digits of up to 9 bits (512 buckets: twice the per-wave counters).
//   PIN, POUT: the keys and payload a are read (written) as one array of
//          (key << 32 | a) words instead of two arrays; between passes this
//          makes each digit run one contiguous stretch of memory of twice the
//          length rather than two, which the scattered writes of a pass
//          favour.  A pass that stages one array at a time (ONEBUF) writes a
//          word's two halves in turn, the key with the keys and a with the
//          payload, to the same lines shortly apart.
// A tile's arrays are staged in LDS all at once where they fit beside the
// counters (one payload); otherwise (ONEBUF) the keys and then each payload
// go through one staging buffer in turn: keys before the look-back, each
// payload after the previous array is written.
constexpr int kLookWindow = 4;
// tiles resident per CU, as the LDS allows: two of 512 threads or one of 1024
constexpr int kSortTilesPerCU = kSortBlock >= 1024 ? 1 : 2;
constexpr int kMaxLdsBytes = 160 * 1024;  // LDS of one workgroup on gfx950

template <bool HAS_B, bool WIDE, bool PIN, bool POUT>
__global__ __launch_bounds__(kSortBlock)
__attribute__((amdgpu_waves_per_eu(HAS_B ? 1 : kSortTilesPerCU * kSortBlock / 256)))
void radix_onesweep(RadixPass p) {
    static_assert(kSortTile <= 65536, "16-bit counters and staged slots");
    constexpr int NB = WIDE ? kMaxBuckets : kMaxBuckets / 2;  // buckets this variant handles
    // per-wave digit counts, then each wave's run start inside its digit
    using cnt_t = uint16_t;
    // all arrays staged at once where they fit in LDS, else one at a time
    constexpr int kFixedLds = kSortWaves * NB * (int)sizeof(cnt_t) + 3 * NB * 4 + 16;
    constexpr bool ONEBUF = (HAS_B ? 3 : 2) * kSortTile * 4 + kFixedLds > kMaxLdsBytes;
    constexpr int NSTAGE = ONEBUF ? 1 : (HAS_B ? 3 : 2);  // staging arrays
    __shared__ uint32_t s_stage[NSTAGE][kSortTile];
    __shared__ uint16_t s_lp[ONEBUF ? kSortTile : 1];  // ONEBUF: staged slot of every key
    __shared__ cnt_t s_cnt[kSortWaves][NB];
    __shared__ uint32_t s_tcnt[NB];   // the tile's count of each digit
    __shared__ uint32_t s_start[NB];  // ... and its exclusive scan
    __shared__ uint32_t s_gbase[NB];
    __shared__ uint32_t s_tile;

    const int R = 1 << p.bits;
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x / kWave;
    for (int i = threadIdx.x; i < kSortWaves * NB; i += kSortBlock) (&s_cnt[0][0])[i] = 0;
    if (threadIdx.x == 0) s_tile = atomicAdd(&p.sc.counter[p.pass], 1u);
    __syncthreads();
    const int64_t tile = s_tile;
    uint64_t* const desc = p.sc.desc + tile * R;

    const int64_t tbase = tile * kSortTile;
    const int64_t wbase = tbase + (int64_t)wv * kWaveKeys;

    uint32_t key[kSortItems];
    int32_t va[kSortItems], vb[kSortItems];
    uint32_t rank[kSortItems];
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = wbase + (int64_t)k * kWave + lane;
        const bool ok = i < p.n;
        if constexpr (PIN) {
            const uint64_t kv = ok ? __builtin_nontemporal_load(p.kv_in + i) : 0ull;
            key[k] = (uint32_t)(kv >> 32);
            va[k] = (int32_t)(uint32_t)kv;
        } else {
            key[k] = ok ? __builtin_nontemporal_load(p.keys_in + i) : 0u;
            va[k] = p.a_in ? (ok ? __builtin_nontemporal_load(p.a_in + i) : 0) : (int32_t)i;
        }
        if constexpr (HAS_B) vb[k] = p.b_in ? (ok ? __builtin_nontemporal_load(p.b_in + i) : 0) : (int32_t)i;
    }
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        const bool ok = wbase + (int64_t)k * kWave + lane < p.n;
        const uint32_t d = (key[k] >> p.shift) & (uint32_t)(R - 1);
        const uint64_t peers = digit_peers(ok, d, p.bits);
        const uint32_t below = count_below(peers);
        const uint32_t base = s_cnt[wv][d];
        rank[k] = base + below;
        // the lowest peer advances the counter for all of them; every lane has
        // read the old value above (LDS ops of one wavefront run in order)
        if (ok && below == 0) s_cnt[wv][d] = (cnt_t)(base + (uint32_t)__popcll(peers));
    }
    __syncthreads();

    // per digit: each wave's run start inside the digit, and the tile count,
    // which is published at once (earlier publication shortens the waits of
    // later tiles)
    const uint32_t tag = (uint32_t)p.pass + 1u;
    for (int d = threadIdx.x; d < R; d += kSortBlock) {
        uint32_t run = 0;
#pragma unroll
        for (int w = 0; w < kSortWaves; ++w) {
            uint32_t c = s_cnt[w][d];
            s_cnt[w][d] = (cnt_t)run;
            run += c;
        }
        s_tcnt[d] = run;
        __hip_atomic_store(desc + d, desc_make(tile == 0 ? kFlagPre : kFlagAgg, tag, run),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    // exclusive scan of the tile's digit counts (R <= NB) by wavefront 0
    if (wv == 0) {
        constexpr int PER = NB / kWave;
        uint32_t t[PER];
        uint32_t sum = 0;
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            int d = lane * PER + k;
            t[k] = d < R ? s_tcnt[d] : 0u;
            sum += t[k];
        }
        uint32_t inc = sum;
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
            uint32_t o = __shfl_up(inc, off, kWave);
            if (lane >= off) inc += o;
        }
        uint32_t run = inc - sum;
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            int d = lane * PER + k;
            if (d < R) s_start[d] = run;
            run += t[k];
        }
    }
    __syncthreads();

    // stage the tile in LDS in digit order (tile-local positions only): all
    // arrays, or with ONEBUF the keys alone (each key's slot is kept in LDS
    // for the payloads)
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = wbase + (int64_t)k * kWave + lane;
        const uint32_t d = (key[k] >> p.shift) & (uint32_t)(R - 1);
        const uint32_t lp = s_start[d] + s_cnt[wv][d] + rank[k];
        if (i < p.n) {
            s_stage[0][lp] = key[k];
            if constexpr (ONEBUF) {
                s_lp[k * kSortBlock + threadIdx.x] = (uint16_t)lp;
            } else {
                s_stage[1][lp] = (uint32_t)va[k];
                if constexpr (HAS_B) s_stage[2][lp] = (uint32_t)vb[k];
            }
        }
    }

    // decoupled look-back, one thread per digit: add up earlier tiles'
    // counts until one that carries an inclusive prefix, kLookWindow
    // descriptors per round (a descriptor not yet published ends the round;
    // the wait on it is bounded)
    if (threadIdx.x < R) {
        const int d = threadIdx.x;
        const uint64_t* col = p.sc.desc + d;
        uint64_t excl = 0;
        if (tile > 0) {
            int64_t look = tile - 1;
            uint32_t spins = 0;
            bool done = false;
            while (!done) {
                uint64_t v[kLookWindow];
#pragma unroll
                for (int w = 0; w < kLookWindow; ++w)
                    v[w] = look - w >= 0
                               ? __hip_atomic_load(col + (look - w) * R, __ATOMIC_RELAXED,
                                                   __HIP_MEMORY_SCOPE_AGENT)
                               : 0ull;
                int used = 0;
#pragma unroll
                for (int w = 0; w < kLookWindow; ++w) {
                    if (done || used < w) continue;  // stopped earlier in this round
                    const bool ready = (uint32_t)((v[w] >> 56) & 63u) == tag && (v[w] >> 62) != 0;
                    if (!ready) continue;
                    excl += v[w] & ((1ull << 56) - 1);
                    used = w + 1;
                    if ((v[w] >> 62) == 2 || look - w == 0) done = true;
                }
                if (done) break;
                look -= used;
                if (used == 0) {
                    if (++spins > kSpinLimit) {  // bounded: never hang; flag it instead
                        atomicOr(p.sc.err, 1u);
                        break;
                    }
                    __builtin_amdgcn_s_sleep(1);
                }
            }
            __hip_atomic_store(desc + d, desc_make(kFlagPre, tag, excl + s_tcnt[d]),
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        s_gbase[d] = p.sc.gbase[p.pass * kMaxBuckets + d] + (uint32_t)excl;
    }
    __syncthreads();

    // write the digit runs: thread t takes staged slots t, t + kSortBlock, ...
    const int64_t nvalid = (p.n - tbase) < kSortTile ? (p.n - tbase) : kSortTile;
    int32_t pos[ONEBUF ? kSortItems : 1];
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        const int i = (int)threadIdx.x + k * kSortBlock;
        if constexpr (ONEBUF) pos[k] = -1;
        if (i < nvalid) {
            const uint32_t kk = s_stage[0][i];
            const uint32_t d = (kk >> p.shift) & (uint32_t)(R - 1);
            const int64_t q = (int64_t)s_gbase[d] + (i - (int64_t)s_start[d]);
            if (q < p.n) {  // cannot fail for consistent counts; never write past n
                if constexpr (ONEBUF) pos[k] = (int32_t)q;
                if constexpr (POUT && ONEBUF) {
                    // the word's key half now, its payload half with the payload
                    reinterpret_cast<uint32_t*>(p.kv_out)[2 * q + 1] = kk;
                } else if constexpr (POUT) {
                    p.kv_out[q] = ((uint64_t)kk << 32) | s_stage[1][i];
                } else if (p.keys_out) {
                    p.keys_out[q] = kk;
                }
                if constexpr (!ONEBUF && !POUT) {
                    if (p.a_out) p.a_out[q] = (int32_t)s_stage[1][i];
                    if constexpr (HAS_B) {
                        if (p.b_out) p.b_out[q] = (int32_t)s_stage[2][i];
                    }
                }
            }
        }
    }
    if constexpr (ONEBUF) {
        // the payloads, one at a time through the same buffer
        for (int which = 0; which < (HAS_B ? 2 : 1); ++which) {
            // payload a of a packed write: the low halves of the words
            const bool half = POUT && which == 0;
            int32_t* out = half ? reinterpret_cast<int32_t*>(p.kv_out)
                                : (which == 0 ? p.a_out : p.b_out);
            __syncthreads();  // every read of the buffer's previous contents is done
#pragma unroll
            for (int k = 0; k < kSortItems; ++k) {
                const int64_t i = wbase + (int64_t)k * kWave + lane;
                if (i < p.n)
                    s_stage[0][s_lp[k * kSortBlock + threadIdx.x]] =
                        (uint32_t)(which == 0 ? va[k] : vb[k]);
            }
            __syncthreads();
            if (!out) continue;
#pragma unroll
            for (int k = 0; k < kSortItems; ++k)
                if (pos[k] >= 0)
                    out[half ? 2 * (int64_t)pos[k] : (int64_t)pos[k]] =
                        (int32_t)s_stage[0][threadIdx.x + k * kSortBlock];
        }
    }
}

// The caller's status word: MP_ERR_SORT if any look-back of the sort gave up,
// else MP_OK (err NULL: no sort ran).
__global__ void radix_status(const uint32_t* __restrict__ err, int32_t* __restrict__ status) {
    if (threadIdx.x == 0) *status = (err && *err) ? (int32_t)MP_ERR_SORT : (int32_t)MP_OK;
}

// rowptr[v] = first CSR position whose key is >= v, from the sorted keys:
// position p writes every v in (keys[p-1], keys[p]] (keys[-1] = -1,
// keys[E] = N), so each of the N+1 entries is written exactly once.  Each
// thread covers kRowptrItems consecutive positions.
constexpr int kRowptrItems = 8;

template <typename RP, bool VEC>
__global__ __launch_bounds__(256) void rowptr_from_sorted(const uint32_t* __restrict__ keys,
                                                          int64_t E, int64_t N, RP* __restrict__ rowptr,
                                                          const uint32_t* __restrict__ sort_err) {
    static_assert(kRowptrItems == 8, "two 16-byte loads per thread");
    const int64_t p0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * kRowptrItems;
    if (p0 > E) return;
    // keys left unsorted by a failed sort would make the fills below run
    // over up to N rows per thread; the caller gets MP_ERR_SORT instead
    if (sort_err && *sort_err) return;
    uint32_t k8[kRowptrItems];
    if (VEC && p0 + kRowptrItems <= E) {
        // VEC: keys is 16-byte aligned and p0 a multiple of 8, so the loads are aligned
        const uint4 a = reinterpret_cast<const uint4*>(keys + p0)[0];
        const uint4 b = reinterpret_cast<const uint4*>(keys + p0)[1];
        k8[0] = a.x; k8[1] = a.y; k8[2] = a.z; k8[3] = a.w;
        k8[4] = b.x; k8[5] = b.y; k8[6] = b.z; k8[7] = b.w;
    } else {
#pragma unroll
        for (int k = 0; k < kRowptrItems; ++k) k8[k] = p0 + k < E ? keys[p0 + k] : 0u;
    }
    int64_t prev = p0 == 0 ? -1 : (int64_t)keys[p0 - 1];
#pragma unroll
    for (int k = 0; k < kRowptrItems; ++k) {
        const int64_t p = p0 + k;
        if (p > E) break;
        int64_t cur = p == E ? N : (int64_t)k8[k];
        if (cur > N) cur = N;  // keys are < N for valid input; stay inside rowptr regardless
        for (int64_t v = prev + 1; v <= cur; ++v) rowptr[v] = (RP)p;
        if (cur > prev) prev = cur;
    }
}

// rowptr[v] = the first position p with keys[p] >= v (E if none), by binary
// search: the CSR of keys sorted by the caller, with work bounded by
// (N + 1) * log2(E) reads whatever the order of keys.
template <typename RP>
__global__ __launch_bounds__(256) void rowptr_by_search(const uint32_t* __restrict__ keys,
                                                        int64_t E, int64_t N, RP* __restrict__ rowptr) {
    for (int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x; v <= N;
         v += (int64_t)gridDim.x * 256) {
        int64_t lo = 0, hi = E;
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if ((int64_t)keys[mid] < v) lo = mid + 1; else hi = mid;
        }
        rowptr[v] = (RP)(v == N ? E : lo);
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

__global__ __launch_bounds__(256) void iota_i32(int64_t n, int32_t* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) out[i] = (int32_t)i;
}

__global__ __launch_bounds__(256) void copy_f32(const float* __restrict__ in, int64_t n,
                                                float* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) out[i] = in[i];
}

__global__ void zero_i64(int64_t* p) { *p = 0; }

__global__ __launch_bounds__(256) void validate_sorted(const int32_t* __restrict__ dst, int64_t E,
                                                       unsigned long long* count) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i > 0 && i < E && dst[i] < dst[i - 1]) atomicAdd(count, 1ull);
}

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

size_t radix_scratch_bytes(int64_t n) {
    const int64_t tiles = ceil_div(n > 0 ? n : 1, kSortTile);
    return align_up((size_t)tiles * kMaxBuckets * sizeof(uint64_t), 256) +
           align_up(kMaxPasses * kMaxBuckets * sizeof(uint32_t), 256) + 256 + 256;
}

RadixScratch radix_scratch(void* base, int64_t n) {
    const int64_t tiles = ceil_div(n > 0 ? n : 1, kSortTile);
    char* b = static_cast<char*>(base);
    RadixScratch sc;
    sc.desc = reinterpret_cast<uint64_t*>(b);
    b += align_up((size_t)tiles * kMaxBuckets * sizeof(uint64_t), 256);
    sc.gbase = reinterpret_cast<uint32_t*>(b);
    b += align_up(kMaxPasses * kMaxBuckets * sizeof(uint32_t), 256);
    sc.counter = reinterpret_cast<uint32_t*>(b);
    b += 256;
    sc.err = reinterpret_cast<uint32_t*>(b);
    return sc;
}

hipError_t radix_sort_begin(const uint32_t* keys, int64_t n, const DigitPlan& dp,
                            const RadixScratch& sc, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    if (dp.passes < 1 || dp.passes > kMaxPasses) return hipErrorInvalidValue;
    uint32_t shifts = 0, widths = 0;
    for (int p = 0; p < dp.passes; ++p) {
        if (dp.width[p] < 1 || dp.width[p] > kSortMaxBits || dp.shift[p] < 0 ||
            dp.shift[p] + dp.width[p] > 32)
            return hipErrorInvalidValue;
        shifts |= (uint32_t)dp.shift[p] << (8 * p);
        widths |= (uint32_t)dp.width[p] << (8 * p);
    }
    const int64_t tiles = ceil_div(n, kSortTile);
    // a pass over R = 2^width digits uses R descriptors per tile
    const int64_t ndesc = tiles * ((int64_t)1 << dp.max_width);
    unsigned g = grid_for(ndesc, 256);
    if (g > 8192) g = 8192;
    // every histogram word needs a thread, however few descriptors there are
    if (g < (unsigned)ceil_div(kMaxPasses * kMaxBuckets, 256)) g = (unsigned)ceil_div(kMaxPasses * kMaxBuckets, 256);
    hipLaunchKernelGGL(radix_clear, dim3(g), dim3(256), 0, s, sc.desc, ndesc, sc.gbase,
                       sc.counter, sc.err);
    const int64_t per_block = (int64_t)kGhistBlock * kGhistItems;
    unsigned gh = grid_for(n, (int)per_block);
    if (gh > 2048) gh = 2048;
    hipLaunchKernelGGL(radix_ghist, dim3(gh), dim3(kGhistBlock), 0, s, keys, n, dp.passes, shifts,
                       widths, sc.gbase);
    hipLaunchKernelGGL(radix_gscan, dim3(1), dim3(kWave), 0, s, sc.gbase, dp.passes);
    return hipGetLastError();
}

template <bool HAS_B, bool WIDE>
void launch_onesweep(const RadixPass& p, int64_t tiles, hipStream_t s) {
    const dim3 g((unsigned)tiles), b(kSortBlock);
    if (p.kv_in && p.kv_out)
        hipLaunchKernelGGL((radix_onesweep<HAS_B, WIDE, true, true>), g, b, 0, s, p);
    else if (p.kv_in)
        hipLaunchKernelGGL((radix_onesweep<HAS_B, WIDE, true, false>), g, b, 0, s, p);
    else if (p.kv_out)
        hipLaunchKernelGGL((radix_onesweep<HAS_B, WIDE, false, true>), g, b, 0, s, p);
    else
        hipLaunchKernelGGL((radix_onesweep<HAS_B, WIDE, false, false>), g, b, 0, s, p);
}

hipError_t radix_sort_pass(const RadixPass& p, hipStream_t s) {
    if (p.n <= 0) return hipSuccess;
    const int64_t tiles = ceil_div(p.n, kSortTile);
    const bool wide = p.bits > kSortMaxBits - 1;
    if (p.b_out) {
        if (wide) launch_onesweep<true, true>(p, tiles, s);
        else launch_onesweep<true, false>(p, tiles, s);
    } else {
        if (wide) launch_onesweep<false, true>(p, tiles, s);
        else launch_onesweep<false, false>(p, tiles, s);
    }
    return hipGetLastError();
}

hipError_t launch_sort_status(const RadixScratch* sc, int32_t* status, hipStream_t s) {
    if (!status) return hipSuccess;
    hipLaunchKernelGGL(radix_status, dim3(1), dim3(64), 0, s, sc ? sc->err : nullptr, status);
    return hipGetLastError();
}

hipError_t launch_rowptr_from_sorted(const uint32_t* keys, int64_t E, int64_t N, void* rowptr,
                                     int rp64, const uint32_t* sort_err, hipStream_t s) {
    const unsigned g = grid_for(ceil_div(E + 1, kRowptrItems), 256);
    const bool vec = reinterpret_cast<uintptr_t>(keys) % 16 == 0;
    if (rp64) {
        auto* rp = static_cast<int64_t*>(rowptr);
        if (vec)
            hipLaunchKernelGGL((rowptr_from_sorted<int64_t, true>), dim3(g), dim3(256), 0, s, keys, E, N, rp, sort_err);
        else
            hipLaunchKernelGGL((rowptr_from_sorted<int64_t, false>), dim3(g), dim3(256), 0, s, keys, E, N, rp, sort_err);
    } else {
        auto* rp = static_cast<int32_t*>(rowptr);
        if (vec)
            hipLaunchKernelGGL((rowptr_from_sorted<int32_t, true>), dim3(g), dim3(256), 0, s, keys, E, N, rp, sort_err);
        else
            hipLaunchKernelGGL((rowptr_from_sorted<int32_t, false>), dim3(g), dim3(256), 0, s, keys, E, N, rp, sort_err);
    }
    return hipGetLastError();
}

hipError_t launch_rowptr_by_search(const uint32_t* keys, int64_t E, int64_t N, void* rowptr,
                                   int rp64, hipStream_t s) {
    const unsigned g = grid_for(N + 1, 256);
    if (rp64)
        hipLaunchKernelGGL((rowptr_by_search<int64_t>), dim3(g), dim3(256), 0, s, keys, E, N,
                           static_cast<int64_t*>(rowptr));
    else
        hipLaunchKernelGGL((rowptr_by_search<int32_t>), dim3(g), dim3(256), 0, s, keys, E, N,
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

hipError_t launch_iota(int64_t n, int32_t* out, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(iota_i32, dim3(grid_for(n, 256)), dim3(256), 0, s, n, out);
    return hipGetLastError();
}

hipError_t launch_copy_f32(const float* in, int64_t n, float* out, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(copy_f32, dim3(grid_for(n, 256)), dim3(256), 0, s, in, n, out);
    return hipGetLastError();
}

hipError_t launch_validate_sorted(const int32_t* dst, int64_t E, int64_t* d_count,
                                  hipStream_t s) {
    hipLaunchKernelGGL(zero_i64, dim3(1), dim3(1), 0, s, d_count);
    if (E > 1)
        hipLaunchKernelGGL(validate_sorted, dim3(grid_for(E, 256)), dim3(256), 0, s, dst, E,
                           reinterpret_cast<unsigned long long*>(d_count));
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
