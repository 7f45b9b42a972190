/*
 * Seeded synthetic inputs shared by the CPU oracle, the tests and the benchmark:
 * RMAT graphs in CSR form, N(0,1) feature matrices and distinct target lists.
 *
 * This module holds none of the method's arithmetic.  Its random words come from
 * SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014), a generator unrelated to the one the sampler uses.
 *
 * Graph model: R-MAT (Chakrabarti, Zhan and Faloutsos, SDM 2004).  Every edge
 * descends `scale` levels of the adjacency matrix; at each level it picks one of
 * the four quadrants with probabilities (a, b, c, 1-a-b-c).  Edges are then
 * sorted by (src, dst), duplicates and self-loops are dropped, and the result is
 * written as CSR with source rows.  Node ids are not permuted.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#define GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* Word i of the stream named `tag` under `seed`: SplitMix64 output for state
 * base + (i + 1) * GAMMA, where base is itself a mixed function of (seed, tag). */
static inline uint64_t stream_base(uint64_t seed, uint64_t tag) {
    return mix64(mix64(seed + GAMMA) ^ (tag * 0xD1B54A32D192ED03ULL));
}
static inline uint64_t word_at(uint64_t base, uint64_t i) {
    return mix64(base + (i + 1) * GAMMA);
}

enum { TAG_GRAPH = 1, TAG_FEAT = 2, TAG_TARGET = 3 };

uint64_t synth_word(uint64_t seed, uint64_t tag, uint64_t i) {
    return word_at(stream_base(seed, tag), i);
}

/* ---------------------------------------------------------------- R-MAT */

/* Quadrant thresholds at 32-bit resolution: one 64-bit word drives two levels. */
static inline uint64_t rmat_key(uint64_t base, uint64_t e, int scale, uint32_t ta,
                                uint32_t tab, uint32_t tabc) {
    uint64_t src = 0, dst = 0;
    uint64_t w = 0;
    for (int d = 0; d < scale; d++) {
        if ((d & 1) == 0) w = word_at(base, e * (uint64_t)((scale + 1) / 2) + (uint64_t)(d >> 1));
        uint32_t r = (d & 1) ? (uint32_t)(w >> 32) : (uint32_t)w;
        int sb, db;
        if (r < ta) { sb = 0; db = 0; }
        else if (r < tab) { sb = 0; db = 1; }
        else if (r < tabc) { sb = 1; db = 0; }
        else { sb = 1; db = 1; }
        src = (src << 1) | (uint64_t)sb;
        dst = (dst << 1) | (uint64_t)db;
    }
    return (src << 32) | dst;
}

static uint32_t prob_threshold(double p) {
    double t = p * 4294967296.0;
    if (t <= 0.0) return 0;
    if (t >= 4294967295.0) return 0xFFFFFFFFu;
    return (uint32_t)t;
}

/* LSD radix sort of n keys on bit range [0, bits) with 11-bit digits. */
static void radix_sort_u64(uint64_t* a, uint64_t* tmp, int64_t n, int bits) {
    const int DB = 11, NB = 1 << DB;
    int64_t cnt[1 << 11];
    uint64_t *src = a, *dst = tmp;
    int passes = (bits + DB - 1) / DB;
    for (int p = 0; p < passes; p++) {
        int sh = p * DB;
        memset(cnt, 0, sizeof(cnt));
        for (int64_t i = 0; i < n; i++) cnt[(src[i] >> sh) & (NB - 1)]++;
        int64_t s = 0;
        for (int d = 0; d < NB; d++) { int64_t c = cnt[d]; cnt[d] = s; s += c; }
        for (int64_t i = 0; i < n; i++) dst[cnt[(src[i] >> sh) & (NB - 1)]++] = src[i];
        uint64_t* t = src; src = dst; dst = t;
    }
    if (src != a) memcpy(a, src, (size_t)n * sizeof(uint64_t));
}

/*
 * Build an R-MAT graph with 2^scale nodes from m generated edges.
 * offsets: caller-owned int64 array of 2^scale + 1 entries.
 * indices: caller-owned int32 array with room for m entries.
 * Returns the number of edges kept (after dropping duplicates and self-loops),
 * or -1 on allocation failure.
 */
int64_t synth_rmat_csr(int scale, int64_t m, double a, double b, double c, uint64_t seed,
                       int64_t* offsets, int32_t* indices) {
    const int64_t N = (int64_t)1 << scale;
    const uint64_t base = stream_base(seed, TAG_GRAPH);
    const uint32_t ta = prob_threshold(a), tab = prob_threshold(a + b),
                   tabc = prob_threshold(a + b + c);
    const int PB = scale < 10 ? scale : 10;     /* partition on the top PB bits of src */
    const int64_t P = (int64_t)1 << PB;
    const int low_bits = scale - PB;            /* src bits that vary within a partition */

    uint64_t* keys = (uint64_t*)malloc((size_t)(m > 0 ? m : 1) * sizeof(uint64_t));
    uint64_t* tmp = (uint64_t*)malloc((size_t)(m > 0 ? m : 1) * sizeof(uint64_t));
    int nt = omp_get_max_threads();
    int64_t* hist = (int64_t*)calloc((size_t)nt * (size_t)P, sizeof(int64_t));
    int64_t* part_start = (int64_t*)malloc((size_t)(P + 1) * sizeof(int64_t));
    int64_t* part_kept = (int64_t*)calloc((size_t)(P + 1), sizeof(int64_t));
    int64_t* deg = (int64_t*)calloc((size_t)N, sizeof(int64_t));
    if (!keys || !tmp || !hist || !part_start || !part_kept || !deg) {
        free(keys); free(tmp); free(hist); free(part_start); free(part_kept); free(deg);
        return -1;
    }

    /* 1. generate edges and count them per partition (per thread) */
#pragma omp parallel num_threads(nt)
    {
        int t = omp_get_thread_num();
        int64_t lo = m * t / nt, hi = m * (t + 1) / nt;
        int64_t* h = hist + (int64_t)t * P;
        for (int64_t e = lo; e < hi; e++) {
            uint64_t k = rmat_key(base, (uint64_t)e, scale, ta, tab, tabc);
            keys[e] = k;
            h[(k >> 32) >> low_bits]++;
        }
    }
    /* 2. scatter into partitions (stable per thread) */
    {
        int64_t s = 0;
        for (int64_t p = 0; p < P; p++) {
            part_start[p] = s;
            for (int t = 0; t < nt; t++) {
                int64_t c = hist[(int64_t)t * P + p];
                hist[(int64_t)t * P + p] = s;
                s += c;
            }
        }
        part_start[P] = s;
    }
#pragma omp parallel num_threads(nt)
    {
        int t = omp_get_thread_num();
        int64_t lo = m * t / nt, hi = m * (t + 1) / nt;
        int64_t* h = hist + (int64_t)t * P;
        for (int64_t e = lo; e < hi; e++) {
            uint64_t k = keys[e];
            tmp[h[(k >> 32) >> low_bits]++] = k;
        }
    }
    /* 3. sort each partition by (src, dst), drop duplicates and self-loops, count degrees */
    const uint64_t low_mask = ((uint64_t)1 << low_bits) - 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
    for (int64_t p = 0; p < P; p++) {
        int64_t s0 = part_start[p], s1 = part_start[p + 1], n = s1 - s0;
        uint64_t* x = tmp + s0;
        uint64_t* y = keys + s0;
        for (int64_t i = 0; i < n; i++) {
            uint64_t src = x[i] >> 32, dst = x[i] & 0xFFFFFFFFULL;
            x[i] = ((src & low_mask) << scale) | dst;
        }
        radix_sort_u64(x, y, n, low_bits + scale);
        int64_t kept = 0;
        uint64_t prev = ~(uint64_t)0;
        for (int64_t i = 0; i < n; i++) {
            uint64_t k = x[i];
            if (k == prev) continue;
            prev = k;
            uint64_t src = ((uint64_t)p << low_bits) | (k >> scale);
            uint64_t dst = k & (((uint64_t)1 << scale) - 1);
            if (src == dst) continue;
            x[kept++] = (src << 32) | dst;
            deg[src]++;
        }
        part_kept[p] = kept;
    }
    /* 4. offsets and indices */
    int64_t* out_start = (int64_t*)malloc((size_t)(P + 1) * sizeof(int64_t));
    int64_t E = 0;
    for (int64_t p = 0; p < P; p++) { out_start[p] = E; E += part_kept[p]; }
    out_start[P] = E;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
    for (int64_t p = 0; p < P; p++) {
        uint64_t* x = tmp + part_start[p];
        int32_t* o = indices + out_start[p];
        for (int64_t i = 0; i < part_kept[p]; i++) o[i] = (int32_t)(x[i] & 0xFFFFFFFFULL);
    }
    offsets[0] = 0;
    for (int64_t v = 0; v < N; v++) offsets[v + 1] = offsets[v] + deg[v];

    free(out_start); free(keys); free(tmp); free(hist); free(part_start); free(part_kept); free(deg);
    return E;
}

/* ---------------------------------------------------------------- conversions */

static inline uint32_t f32_bits(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static inline float bits_f32(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* float -> IEEE binary16, round to nearest even (Inf/NaN preserved, overflow -> Inf). */
uint16_t synth_f32_to_f16(float f) {
    uint32_t x = f32_bits(f);
    uint16_t sign = (uint16_t)((x >> 16) & 0x8000u);
    uint32_t ax = x & 0x7FFFFFFFu;
    if (ax >= 0x7F800000u) /* Inf or NaN */
        return sign | (uint16_t)(ax > 0x7F800000u ? (0x7E00u | ((ax >> 13) & 0x3FFu)) : 0x7C00u);
    if (ax >= 0x38800000u) { /* |f| >= 2^-14: normal binary16 (or overflow) */
        uint32_t lsb = (ax >> 13) & 1u;
        uint32_t r = ax + 0xFFFu + lsb;           /* round the 13 dropped bits, ties to even */
        r -= (uint32_t)(127 - 15) << 23;          /* rebias the exponent */
        if (r >= (uint32_t)0x1Fu << 23) return sign | 0x7C00u;
        return sign | (uint16_t)(r >> 13);
    }
    /* subnormal binary16 range or zero: value = n * 2^-24, n = round(|f| * 2^24) */
    float af = bits_f32(ax);
    float scaled = af * 16777216.0f;              /* exact: power-of-two scaling */
    /* round to nearest even integer (scaled < 1024, so rint in float is exact) */
    float n = rintf(scaled);
    return sign | (uint16_t)(uint32_t)n;
}

/* float -> bfloat16, round to nearest even (NaN kept quiet). */
uint16_t synth_f32_to_bf16(float f) {
    uint32_t x = f32_bits(f);
    if ((x & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((x >> 16) | 0x40u);
    uint32_t lsb = (x >> 16) & 1u;
    x += 0x7FFFu + lsb;
    return (uint16_t)(x >> 16);
}

void synth_convert_f32(const float* in, int64_t n, int dtype, void* out) {
    /* dtype: 0 = float32 (copy), 1 = float16, 2 = bfloat16 */
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; i++) {
        if (dtype == 0) ((float*)out)[i] = in[i];
        else if (dtype == 1) ((uint16_t*)out)[i] = synth_f32_to_f16(in[i]);
        else ((uint16_t*)out)[i] = synth_f32_to_bf16(in[i]);
    }
}

/* ---------------------------------------------------------------- features */

/*
 * n*dim values ~ N(0,1) by the Box-Muller transform.  Element e uses the pair
 * (e >> 1): u1 from word 2p, u2 from word 2p+1; even e takes the cosine branch,
 * odd e the sine branch.  The value is computed in double, rounded to float, and
 * for dtype 1/2 rounded again (nearest even) to float16/bfloat16.
 */
void synth_features(int64_t n, int64_t dim, int dtype, uint64_t seed, void* out) {
    const uint64_t base = stream_base(seed, TAG_FEAT);
    const int64_t total = n * dim;
    const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for schedule(static)
    for (int64_t p = 0; p < (total + 1) / 2; p++) {
        uint64_t w1 = word_at(base, 2 * (uint64_t)p), w2 = word_at(base, 2 * (uint64_t)p + 1);
        double u1 = ((double)(w1 >> 11) + 1.0) * (1.0 / 9007199254740992.0); /* (0, 1] */
        double u2 = (double)(w2 >> 11) * (1.0 / 9007199254740992.0);         /* [0, 1) */
        double r = sqrt(-2.0 * log(u1));
        float z[2] = {(float)(r * cos(two_pi * u2)), (float)(r * sin(two_pi * u2))};
        for (int s = 0; s < 2; s++) {
            int64_t e = 2 * p + s;
            if (e >= total) break;
            if (dtype == 0) ((float*)out)[e] = z[s];
            else if (dtype == 1) ((uint16_t*)out)[e] = synth_f32_to_f16(z[s]);
            else ((uint16_t*)out)[e] = synth_f32_to_bf16(z[s]);
        }
    }
}

/* ---------------------------------------------------------------- targets */

/* First `count` entries of a partial Fisher-Yates shuffle of [0, n): distinct ids. */
int synth_targets(int64_t n, int64_t count, uint64_t seed, int32_t* out) {
    if (count > n) return -1;
    int32_t* perm = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    if (!perm) return -1;
    for (int64_t i = 0; i < n; i++) perm[i] = (int32_t)i;
    const uint64_t base = stream_base(seed, TAG_TARGET);
    for (int64_t i = 0; i < count; i++) {
        uint64_t j = (uint64_t)i + word_at(base, (uint64_t)i) % (uint64_t)(n - i);
        int32_t t = perm[i]; perm[i] = perm[j]; perm[j] = t;
        out[i] = perm[i];
    }
    free(perm);
    return 0;
}
