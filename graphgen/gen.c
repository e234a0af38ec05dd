/*
 * Seeded synthetic graph and feature generators.
 *
 * This module only draws inputs: random endpoints, random features and the
 * GCN-style edge weights that one workload asks for.  It computes none of the
 * aggregation arithmetic (no gather, no reduction, no sort), so both the CPU
 * oracle and the device path can be fed from it without sharing any of the
 * method's code.
 *
 * Random numbers.  Every value is a pure function of (seed, stream, index):
 *   key(seed, stream)  = mix(mix(seed + G) ^ (stream * G + C))
 *   draw(key, i)       = mix(key + (i + 1) * G)
 * where G = 0x9E3779B97F4A7C15 and mix() is the output function of
 * SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014).  draw(key, i) is therefore the (i+1)-th output
 * of a SplitMix64 stream started at state `key`.  Results do not depend on the
 * number of threads used.
 *
 * Power-law endpoints use rank weights w_r = r^-beta (r = 1..N), sampled with
 * Vose's alias method (Vose, IEEE TSE 1991), then mapped to node ids through a
 * seeded Fisher-Yates permutation so that hubs carry no id locality.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define GG_G 0x9E3779B97F4A7C15ULL
#define GG_C 0x632BE59BD9B4E019ULL

static inline uint64_t gg_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

uint64_t gg_key(uint64_t seed, uint64_t stream) {
    return gg_mix(gg_mix(seed + GG_G) ^ (stream * GG_G + GG_C));
}

uint64_t gg_draw(uint64_t key, uint64_t i) { return gg_mix(key + (i + 1) * GG_G); }

/* floor(r * n / 2^64): an integer in [0, n). */
static inline uint64_t gg_below(uint64_t r, uint64_t n) {
    return (uint64_t)(((__uint128_t)r * (__uint128_t)n) >> 64);
}

/* Uniform in (0, 1): ((r >> 11) + 0.5) * 2^-53, never 0 or 1. */
static inline double gg_open01(uint64_t r) {
    return ((double)(r >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

/* Uniform in [0, 1): (r >> 11) * 2^-53. */
static inline double gg_half01(uint64_t r) {
    return (double)(r >> 11) * (1.0 / 9007199254740992.0);
}

/* ---- integers ---------------------------------------------------------- */

void gg_uniform_ints(uint64_t seed, uint64_t stream, int64_t n, int64_t range,
                     int32_t* out) {
    const uint64_t key = gg_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = (int32_t)gg_below(gg_draw(key, (uint64_t)i), (uint64_t)range);
}

/* Seeded Fisher-Yates permutation of 0..n-1 (sequential by definition). */
void gg_permutation(uint64_t seed, uint64_t stream, int64_t n, int32_t* perm) {
    const uint64_t key = gg_key(seed, stream);
    for (int64_t i = 0; i < n; ++i) perm[i] = (int32_t)i;
    for (int64_t i = n - 1; i > 0; --i) {
        int64_t j = (int64_t)gg_below(gg_draw(key, (uint64_t)i), (uint64_t)(i + 1));
        int32_t t = perm[i];
        perm[i] = perm[j];
        perm[j] = t;
    }
}

/* Vose alias table for weights w_r = (r+1)^-beta, r = 0..n-1.
 * prob[k] in [0,1], alias[k] in [0,n).  Returns 0, or -1 on allocation
 * failure. */
int gg_alias_powerlaw(int64_t n, double beta, double* prob, int32_t* alias) {
    double total = 0.0;
    for (int64_t r = 0; r < n; ++r) total += pow((double)(r + 1), -beta);
    int32_t* small = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    int32_t* large = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    if (!small || !large) {
        free(small);
        free(large);
        return -1;
    }
    int64_t ns = 0, nl = 0;
    for (int64_t r = 0; r < n; ++r) {
        prob[r] = (double)n * pow((double)(r + 1), -beta) / total;
        alias[r] = (int32_t)r;
        if (prob[r] < 1.0)
            small[ns++] = (int32_t)r;
        else
            large[nl++] = (int32_t)r;
    }
    while (ns > 0 && nl > 0) {
        int32_t s = small[--ns];
        int32_t l = large[nl - 1];
        alias[s] = l;
        prob[l] = (prob[l] + prob[s]) - 1.0;
        if (prob[l] < 1.0) {
            --nl;
            small[ns++] = l;
        }
    }
    while (nl > 0) prob[large[--nl]] = 1.0;
    while (ns > 0) prob[small[--ns]] = 1.0; /* rounding leftovers */
    free(small);
    free(large);
    return 0;
}

/* E endpoints drawn i.i.d. with P(rank r) proportional to (r+1)^-beta, mapped
 * to node ids by perm (rank -> id).  Column draw from `stream`, the alias coin
 * from `stream` with bit 32 set. */
void gg_sample_alias(uint64_t seed, uint64_t stream, int64_t e, int64_t n,
                     const double* prob, const int32_t* alias, const int32_t* perm,
                     int32_t* out) {
    const uint64_t kc = gg_key(seed, stream);
    const uint64_t kb = gg_key(seed, stream | (1ULL << 32));
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < e; ++i) {
        int64_t k = (int64_t)gg_below(gg_draw(kc, (uint64_t)i), (uint64_t)n);
        double coin = gg_half01(gg_draw(kb, (uint64_t)i));
        int64_t r = coin < prob[k] ? k : (int64_t)alias[k];
        out[i] = perm[r];
    }
}

/* Sum_{r=1..n} r^-beta. */
double gg_zeta_partial(int64_t n, double beta) {
    double s = 0.0;
    for (int64_t r = n; r >= 1; --r) s += pow((double)r, -beta);
    return s;
}

/* beta in (lo, hi) with e / sum_{r<=n} r^-beta == dmax (the expected degree
 * of rank 1 under Chung-Lu weights r^-beta), by bisection. */
double gg_fit_beta(int64_t n, int64_t e, double dmax, double lo, double hi,
                   int iters) {
    for (int it = 0; it < iters; ++it) {
        double mid = 0.5 * (lo + hi);
        double d1 = (double)e / gg_zeta_partial(n, mid);
        if (d1 < dmax)
            lo = mid; /* too flat: more skew needed */
        else
            hi = mid;
    }
    return 0.5 * (lo + hi);
}

/* ---- features ---------------------------------------------------------- */

/* U(-1,1) in fp32: (2k + 1 - 2^24) * 2^-24 with k the top 24 bits; exact,
 * symmetric, never zero. */
void gg_uniform_f32(uint64_t seed, uint64_t stream, int64_t n, float* out) {
    const uint64_t key = gg_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        int64_t k = (int64_t)(gg_draw(key, (uint64_t)i) >> 40);
        out[i] = (float)((double)(2 * k + 1 - (1LL << 24)) * (1.0 / 16777216.0));
    }
}

/* N(0,1) by Box-Muller in fp64, rounded once to fp32.  u1 from `stream`,
 * u2 from `stream` with its top bit flipped. */
void gg_normal_f32(uint64_t seed, uint64_t stream, int64_t n, float* out) {
    const uint64_t k1 = gg_key(seed, stream);
    const uint64_t k2 = gg_key(seed, stream ^ 0x8000000000000000ULL);
    const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double u1 = gg_open01(gg_draw(k1, (uint64_t)i));
        double u2 = gg_half01(gg_draw(k2, (uint64_t)i));
        out[i] = (float)(sqrt(-2.0 * log(u1)) * cos(two_pi * u2));
    }
}

/* fp32 -> bfloat16 bits, round to nearest even (finite inputs). */
void gg_f32_to_bf16(int64_t n, const float* in, uint16_t* out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        uint32_t u;
        memcpy(&u, &in[i], 4);
        uint32_t lsb = (u >> 16) & 1u;
        out[i] = (uint16_t)((u + 0x7FFFu + lsb) >> 16);
    }
}

/* ---- GCN-style edge weights -------------------------------------------- */

/* w_e = fl32(1 / sqrt(outdeg(src_e) * indeg(dst_e))) in fp64, degrees counted
 * with duplicates.  Returns -1 on a bad index or allocation failure. */
int gg_gcn_weights(int64_t e, const int32_t* src, const int32_t* dst, int64_t n_src,
                   int64_t n_dst, float* w) {
    int64_t* od = (int64_t*)calloc((size_t)(n_src > 0 ? n_src : 1), sizeof(int64_t));
    int64_t* id = (int64_t*)calloc((size_t)(n_dst > 0 ? n_dst : 1), sizeof(int64_t));
    if (!od || !id) {
        free(od);
        free(id);
        return -1;
    }
    for (int64_t i = 0; i < e; ++i) {
        if (src[i] < 0 || src[i] >= n_src || dst[i] < 0 || dst[i] >= n_dst) {
            free(od);
            free(id);
            return -1;
        }
        od[src[i]]++;
        id[dst[i]]++;
    }
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < e; ++i)
        w[i] = (float)(1.0 / sqrt((double)od[src[i]] * (double)id[dst[i]]));
    free(od);
    free(id);
    return 0;
}

/* U(-1,1) drawn exactly as gg_uniform_f32, then rounded to bfloat16 (RNE),
 * without materializing the fp32 array. */
void gg_uniform_bf16(uint64_t seed, uint64_t stream, int64_t n, uint16_t* out) {
    const uint64_t key = gg_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        int64_t k = (int64_t)(gg_draw(key, (uint64_t)i) >> 40);
        float f = (float)((double)(2 * k + 1 - (1LL << 24)) * (1.0 / 16777216.0));
        uint32_t u;
        memcpy(&u, &f, 4);
        out[i] = (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
    }
}
