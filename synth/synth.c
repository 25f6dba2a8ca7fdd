/*
 * synth.c -- seeded synthetic power traces and operator-interval lists.
 *
 * Shared input generator for the tests, the benchmark and the smoke check.
 * It holds none of the attribution arithmetic: it only draws timestamps,
 * power samples, interval bounds and operator keys.
 *
 * Random numbers: splitmix64 (Steele, Lea & Flood 2014) seeds one
 * xoshiro256** stream (Blackman & Vigna 2018) per purpose and per block of
 * 2^16 draws, so that blocks are drawn in parallel (OpenMP) and the result
 * does not depend on the thread count.  Uniforms are the
 * top 53 bits; normals come from Box-Muller; lognormal(median, sigma) is
 * exp(ln(median) + sigma * Z); exponential(mean) is -mean * ln(1 - U); a
 * Zipf(s, K) rank is found by inverse CDF over the cumulative weights r^-s.
 *
 * Workloads (sizes per side):
 *   1  tiny A/B          n = 10,000 @ 1 ms +-5% jitter, 2,000 packed intervals,
 *                        50 keys Zipf(1.1), random-walk power 100..700 W
 *   2  decode-shaped     n = 2,000,000 @ 100 kHz, 32 layers x 12 ops x 256 steps,
 *                        416 keys (op, layer, shape bucket), per-key mean power
 *   3  multi-stream      n = 100,000,000 @ 1 MHz, 4 streams x 1,000,000 intervals,
 *                        5,000 keys Zipf(1.2), power = base + sum of active loads
 *   4  batched sweep     n = 20,000,000 @ 200 kHz, 1,000,000 intervals, 2,000
 *                        uniform keys, baseline + 8 candidates
 *   5  long run          n = 360,000,000 @ 100 kHz, 50,000,000 intervals,
 *                        20,000 keys Zipf(1.05), random-walk power 100..750 W
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* generators                                                           */
/* ------------------------------------------------------------------ */

static uint64_t splitmix64_next(uint64_t* x)
{
    uint64_t z = (*x += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

uint64_t synth_mix64(uint64_t v)
{
    uint64_t x = v;
    return splitmix64_next(&x);
}

typedef struct {
    uint64_t s[4];
    int has_spare;
    double spare;
} rng_t;

static uint64_t rotl(uint64_t x, int k) { return (x << k) | (x >> (64 - k)); }

static uint64_t rng_next(rng_t* g)
{
    uint64_t* s = g->s;
    uint64_t result = rotl(s[1] * 5, 7) * 9;
    uint64_t t = s[1] << 17;
    s[2] ^= s[0];
    s[3] ^= s[1];
    s[1] ^= s[2];
    s[0] ^= s[3];
    s[2] ^= t;
    s[3] = rotl(s[3], 45);
    return result;
}

static void rng_seed(rng_t* g, uint64_t seed)
{
    uint64_t x = seed;
    int i;
    for (i = 0; i < 4; ++i)
        g->s[i] = splitmix64_next(&x);
    g->has_spare = 0;
    g->spare = 0.0;
}

static double u01(rng_t* g) { return (double)(rng_next(g) >> 11) * 0x1.0p-53; }

static double normal01(rng_t* g)
{
    double u1, u2, r;
    if (g->has_spare) {
        g->has_spare = 0;
        return g->spare;
    }
    u1 = 1.0 - u01(g); /* (0, 1] */
    u2 = u01(g);
    r = sqrt(-2.0 * log(u1));
    g->spare = r * sin(6.283185307179586 * u2);
    g->has_spare = 1;
    return r * cos(6.283185307179586 * u2);
}

static double lognormal(rng_t* g, double median, double sigma)
{
    return exp(log(median) + sigma * normal01(g));
}

static double expo(rng_t* g, double mean) { return -mean * log(1.0 - u01(g)); }

/* purpose-specific stream: ASCII "MAGNETON" salted by workload, side, purpose, seed */
static void rng_for(rng_t* g, int cfg, int side, int purpose, uint64_t seed)
{
    uint64_t v = 0x4D41474E45544F4Eull ^ ((uint64_t)cfg << 16) ^ ((uint64_t)side << 8) ^
                 (uint64_t)purpose ^ (seed * 0x9E3779B97F4A7C15ull);
    rng_seed(g, synth_mix64(v));
}

/* the stream of block b of a purpose */
#define BLK ((int64_t)1 << 16)
static void rng_block(rng_t* g, int cfg, int side, int purpose, uint64_t seed, int64_t b)
{
    uint64_t v = 0x4D41474E45544F4Eull ^ ((uint64_t)cfg << 16) ^ ((uint64_t)side << 8) ^
                 (uint64_t)purpose ^ (seed * 0x9E3779B97F4A7C15ull);
    rng_seed(g, synth_mix64(synth_mix64(v) ^ (uint64_t)(b + 1) * 0xD1B54A32D192ED03ull));
}

enum {
    PU_TIME = 1,
    PU_DUR = 2,
    PU_GAP = 3,
    PU_KEY = 4,
    PU_POWER = 5,
    PU_KEYPARAM = 6,
    PU_NOISE = 7,
    PU_PICK = 8,
    PU_VOCAB = 9
};

/* Zipf(s, K) sampler by inverse CDF */
typedef struct {
    double* cum;
    int64_t K;
} zipf_t;

static int zipf_init(zipf_t* z, double s, int64_t K)
{
    int64_t r;
    double acc = 0.0;
    z->K = K;
    z->cum = (double*)malloc(sizeof(double) * (size_t)K);
    if (!z->cum)
        return -1;
    for (r = 0; r < K; ++r) {
        acc += pow((double)(r + 1), -s);
        z->cum[r] = acc;
    }
    return 0;
}

/* rank in [0, K) */
static int64_t zipf_draw(zipf_t* z, rng_t* g)
{
    double u = u01(g) * z->cum[z->K - 1];
    int64_t lo = 0, hi = z->K - 1;
    while (lo < hi) {
        int64_t mid = (lo + hi) / 2;
        if (z->cum[mid] <= u)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

/* ------------------------------------------------------------------ */
/* workload table                                                       */
/* ------------------------------------------------------------------ */

typedef struct {
    int64_t n, m, K;
    int32_t streams;
} shape_t;

static int shape_of(int cfg, shape_t* sh)
{
    switch (cfg) {
    case 1: sh->n = 10000; sh->m = 2000; sh->K = 50; sh->streams = 1; return 0;
    case 2: sh->n = 2000000; sh->m = 98304; sh->K = 416; sh->streams = 1; return 0;
    case 3: sh->n = 100000000; sh->m = 4000000; sh->K = 5000; sh->streams = 4; return 0;
    case 4: sh->n = 20000000; sh->m = 1000000; sh->K = 2000; sh->streams = 1; return 0;
    case 5: sh->n = 360000000; sh->m = 50000000; sh->K = 20000; sh->streams = 1; return 0;
    default: return -1;
    }
}

/* sizes[4] = {n_samples, n_intervals, n_keys in the vocabulary, n_streams} */
int synth_shape(int cfg, int64_t* sizes)
{
    shape_t sh;
    if (shape_of(cfg, &sh))
        return -1;
    sizes[0] = sh.n;
    sizes[1] = sh.m;
    sizes[2] = sh.K;
    sizes[3] = sh.streams;
    return 0;
}

/* vocabulary: key of rank r = mix64(vocab seed ^ r); unique by check */
static int make_vocab(int cfg, uint64_t seed, int64_t K, uint64_t* vocab)
{
    rng_t g;
    uint64_t base;
    int64_t r;
    rng_for(&g, cfg, 0, PU_VOCAB, seed);
    base = rng_next(&g);
    for (r = 0; r < K; ++r)
        vocab[r] = synth_mix64(base ^ (uint64_t)r);
    return 0;
}

int synth_vocab(int cfg, uint64_t seed, uint64_t* vocab)
{
    shape_t sh;
    if (shape_of(cfg, &sh))
        return -1;
    return make_vocab(cfg, seed, sh.K, vocab);
}

/* decode-shaped key: 64-bit mix of (op type, layer, shape bucket) */
static uint64_t decode_key(uint64_t salt, int op, int layer, int bucket)
{
    return synth_mix64(salt ^ ((uint64_t)op << 40) ^ ((uint64_t)layer << 20) ^ (uint64_t)bucket);
}

/* ------------------------------------------------------------------ */
/* structure: timestamps, intervals, keys                               */
/* ------------------------------------------------------------------ */

/* out[i] = lognormal(median, sigma), drawn block-parallel */
static void draw_lognormal(int cfg, int side, int purpose, uint64_t seed, int64_t m, double median,
                           double sigma, double* out)
{
    int64_t nb = (m + BLK - 1) / BLK, b;
#pragma omp parallel for schedule(static)
    for (b = 0; b < nb; ++b) {
        rng_t g;
        int64_t i, hi = (b + 1) * BLK < m ? (b + 1) * BLK : m;
        rng_block(&g, cfg, side, purpose, seed, b);
        for (i = b * BLK; i < hi; ++i)
            out[i] = lognormal(&g, median, sigma);
    }
}

static void draw_expo(int cfg, int side, int purpose, uint64_t seed, int64_t m, double mean,
                      double* out)
{
    int64_t nb = (m + BLK - 1) / BLK, b;
#pragma omp parallel for schedule(static)
    for (b = 0; b < nb; ++b) {
        rng_t g;
        int64_t i, hi = (b + 1) * BLK < m ? (b + 1) * BLK : m;
        rng_block(&g, cfg, side, purpose, seed, b);
        for (i = b * BLK; i < hi; ++i)
            out[i] = expo(&g, mean);
    }
}

/* keys by Zipf rank (zs > 0) or uniform rank (zs == 0) */
static int draw_keys(int cfg, int side, int purpose, uint64_t seed, int64_t m, double zs,
                     const uint64_t* vocab, int64_t K, uint64_t* key)
{
    zipf_t z = {0, 0};
    int64_t nb = (m + BLK - 1) / BLK, b;
    if (zs > 0 && zipf_init(&z, zs, K))
        return -2;
#pragma omp parallel for schedule(static)
    for (b = 0; b < nb; ++b) {
        rng_t g;
        int64_t i, hi = (b + 1) * BLK < m ? (b + 1) * BLK : m;
        rng_block(&g, cfg, side, purpose, seed, b);
        for (i = b * BLK; i < hi; ++i) {
            int64_t r = (zs > 0) ? zipf_draw(&z, &g) : (int64_t)(u01(&g) * (double)K);
            if (r >= K)
                r = K - 1;
            key[i] = vocab[r];
        }
    }
    free(z.cum);
    return 0;
}

/*
 * synth_structure: fill t[n], s[m], e[m], key[m] and offsets[streams+1] of
 * workload cfg.  'side' selects an independent draw (workload 5's second
 * trace); every other workload shares one structure between its sides.
 */
int synth_structure(int cfg, uint64_t seed, int side, double* t, double* s, double* e,
                    uint64_t* key, int64_t* offsets)
{
    shape_t sh;
    int64_t j, i;
    uint64_t* vocab;
    int rc = 0;
    if (shape_of(cfg, &sh))
        return -1;
    if (cfg != 5)
        side = 0;
    vocab = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)sh.K);
    if (!vocab)
        return -2;
    make_vocab(cfg, seed, sh.K, vocab);

    /* timestamps */
    if (cfg == 1) {
        int64_t nb = (sh.n + BLK - 1) / BLK, b;
#pragma omp parallel for schedule(static)
        for (b = 0; b < nb; ++b) {
            rng_t g;
            int64_t hi = (b + 1) * BLK < sh.n ? (b + 1) * BLK : sh.n, jj;
            rng_block(&g, cfg, side, PU_TIME, seed, b);
            for (jj = b * BLK; jj < hi; ++jj) {
                double jit = (u01(&g) * 2.0 - 1.0) * 5e-5;
                t[jj] = (jj == 0) ? 0.0 : (double)jj * 1e-3 + jit;
            }
        }
    } else {
        double rate = (cfg == 3) ? 1e6 : (cfg == 4) ? 2e5 : 1e5;
#pragma omp parallel for schedule(static)
        for (j = 0; j < sh.n; ++j)
            t[j] = (double)j / rate;
    }

    offsets[0] = 0;
    if (cfg == 1 || cfg == 4 || cfg == 5) {
        double median = (cfg == 1) ? 3e-3 : (cfg == 4) ? 60e-6 : 40e-6;
        double sigma = (cfg == 1) ? 0.8 : 1.0;
        double zs = (cfg == 1) ? 1.1 : (cfg == 4) ? 0.0 : 1.05;
        double cur = 0.0;
        draw_lognormal(cfg, side, PU_DUR, seed, sh.m, median, sigma, e);
        for (i = 0; i < sh.m; ++i) { /* packed back to back from t = 0 */
            s[i] = cur;
            e[i] = cur + e[i];
            cur = e[i];
        }
        rc = draw_keys(cfg, side, PU_KEY, seed, sh.m, zs, vocab, sh.K, key);
        offsets[1] = sh.m;
    } else if (cfg == 2) {
        const int layers = 32, ops = 12, steps = 256;
        rng_t gk;
        uint64_t salt;
        rng_for(&gk, cfg, side, PU_KEY, seed);
        salt = rng_next(&gk);
        draw_lognormal(cfg, side, PU_DUR, seed, sh.m, 20e-6, 1.0, e);
        i = 0;
        for (int st = 0; st < steps; ++st) {
            double cur = (double)st * 0.078125;
            for (int l = 0; l < layers; ++l) {
                for (int o = 0; o < ops; ++o) {
                    int bucket = (o == 4) ? st / 128 : 0;
                    s[i] = cur;
                    e[i] = cur + e[i];
                    cur = e[i];
                    key[i] = decode_key(salt, o, l, bucket);
                    ++i;
                }
            }
        }
        offsets[1] = sh.m;
    } else { /* cfg 3: four streams, an exponential gap before each interval */
        int64_t per = sh.m / sh.streams;
        draw_lognormal(cfg, side, PU_DUR, seed, sh.m, 15e-6, 1.0, e);
        draw_expo(cfg, side, PU_GAP, seed, sh.m, 73e-6, s);
        for (int a = 0; a < sh.streams; ++a) {
            double cur = 0.0;
            for (int64_t u = 0; u < per; ++u) {
                i = (int64_t)a * per + u;
                cur += s[i];
                s[i] = cur;
                e[i] = cur + e[i];
                cur = e[i];
            }
            offsets[a + 1] = (int64_t)(a + 1) * per;
        }
        rc = draw_keys(cfg, side, PU_KEY, seed, sh.m, 1.2, vocab, sh.K, key);
    }
    free(vocab);
    return rc;
}

/* ------------------------------------------------------------------ */
/* power                                                                */
/* ------------------------------------------------------------------ */

/* uniform in [lo, hi) per vocabulary rank, from its own stream */
static void per_key_uniform(int cfg, int side, int purpose, uint64_t seed, int64_t K, double lo,
                            double hi, double* out)
{
    rng_t g;
    int64_t r;
    rng_for(&g, cfg, side, purpose, seed);
    for (r = 0; r < K; ++r)
        out[r] = lo + (hi - lo) * u01(&g);
}

static int cmp_u64(const void* a, const void* b)
{
    uint64_t x = *(const uint64_t*)a, y = *(const uint64_t*)b;
    return (x > y) - (x < y);
}

/* map a key back to its vocabulary rank through a sorted (key, rank) table */
typedef struct {
    uint64_t* keys; /* sorted */
    int64_t* rank;
    int64_t K;
} keyindex_t;

static int keyindex_build(keyindex_t* ki, const uint64_t* vocab, int64_t K)
{
    int64_t r;
    ki->keys = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)K);
    ki->rank = (int64_t*)malloc(sizeof(int64_t) * (size_t)K);
    ki->K = K;
    if (!ki->keys || !ki->rank)
        return -1;
    for (r = 0; r < K; ++r)
        ki->keys[r] = vocab[r];
    qsort(ki->keys, (size_t)K, sizeof(uint64_t), cmp_u64);
    for (r = 0; r < K; ++r) {
        int64_t lo = 0, hi = K - 1;
        while (lo < hi) {
            int64_t mid = (lo + hi) / 2;
            if (ki->keys[mid] < vocab[r])
                lo = mid + 1;
            else
                hi = mid;
        }
        ki->rank[lo] = r;
    }
    return 0;
}

static int64_t keyindex_find(const keyindex_t* ki, uint64_t k)
{
    int64_t lo = 0, hi = ki->K - 1;
    while (lo < hi) {
        int64_t mid = (lo + hi) / 2;
        if (ki->keys[mid] < k)
            lo = mid + 1;
        else
            hi = mid;
    }
    return (ki->keys[lo] == k) ? ki->rank[lo] : -1;
}

static void keyindex_free(keyindex_t* ki)
{
    free(ki->keys);
    free(ki->rank);
}

/* first interval of [lo, hi) whose end is after time x (ends are sorted) */
static int64_t first_ending_after(const double* e, int64_t lo, int64_t hi, double x)
{
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (e[mid] <= x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

/* clamped random walk: P[0] = 400, P[j] = clamp(P[j-1] + 5 N(0,1), 100, hi) */
static void random_walk(int cfg, int side, uint64_t seed, int64_t n, double hi, float* P)
{
    int64_t nb = (n + BLK - 1) / BLK, b, j;
    double x = 400.0;
#pragma omp parallel for schedule(static)
    for (b = 0; b < nb; ++b) {
        rng_t g;
        int64_t jj, top = (b + 1) * BLK < n ? (b + 1) * BLK : n;
        rng_block(&g, cfg, side, PU_POWER, seed, b);
        for (jj = b * BLK; jj < top; ++jj)
            P[jj] = (float)normal01(&g); /* the step, kept in the output for now */
    }
    for (j = 0; j < n; ++j) {
        if (j > 0) {
            x += 5.0 * (double)P[j];
            if (x < 100.0)
                x = 100.0;
            if (x > hi)
                x = hi;
        }
        P[j] = (float)x;
    }
}

/*
 * synth_power: fill P[n] (W, fp32, >= 0) for the given side of workload cfg,
 * from the structure arrays produced by synth_structure for that side.
 *   1: side 0 is a clamped random walk; side 1 multiplies samples whose
 *      active key has vocabulary rank 0, 4 or 19 by 1.15 and adds N(0, 1 W).
 *   2: per-key mean U[200, 750] (idle 100) + N(0, 20); side 1 scales the
 *      mean of 5 drawn keys by 1.3.
 *   3: 100 + sum over active intervals of w[key] + N(0, 20), w ~ U[50, 160];
 *      side 1 uses w * U[0.8, 1.5] per key.
 *   4: base[key] ~ U[200, 750] (idle 100) + N(0, 20); side b >= 1 multiplies
 *      base by U[0.8, 1.5] per key.
 *   5: clamped random walk; each side draws its own.
 * "active key at t_j" is the key of the interval with s <= t_j < e.
 */
int synth_power(int cfg, uint64_t seed, int side, const double* t, const double* s,
                const double* e, const uint64_t* key, const int64_t* offsets, float* P)
{
    shape_t sh;
    uint64_t* vocab = NULL;
    double* level = NULL;
    keyindex_t ki = {0, 0, 0};
    int rc = 0;
    int64_t nb, b;
    if (shape_of(cfg, &sh))
        return -1;
    nb = (sh.n + BLK - 1) / BLK;

    if (cfg == 1 || cfg == 5) {
        random_walk(cfg, (cfg == 5) ? side : 0, seed, sh.n, (cfg == 1) ? 700.0 : 750.0, P);
        if (cfg == 1 && side == 1) {
            uint64_t chosen[3];
            vocab = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)sh.K);
            if (!vocab)
                return -2;
            make_vocab(cfg, seed, sh.K, vocab);
            chosen[0] = vocab[0];
            chosen[1] = vocab[4];
            chosen[2] = vocab[19];
#pragma omp parallel for schedule(static)
            for (b = 0; b < nb; ++b) {
                rng_t g;
                int64_t j, top = (b + 1) * BLK < sh.n ? (b + 1) * BLK : sh.n;
                int64_t i = first_ending_after(e, 0, sh.m, t[b * BLK]);
                rng_block(&g, cfg, side, PU_NOISE, seed, b);
                for (j = b * BLK; j < top; ++j) {
                    double v = (double)P[j];
                    while (i < sh.m && e[i] <= t[j])
                        ++i;
                    if (i < sh.m && s[i] <= t[j] && t[j] < e[i] &&
                        (key[i] == chosen[0] || key[i] == chosen[1] || key[i] == chosen[2]))
                        v *= 1.15;
                    v += normal01(&g);
                    P[j] = (float)(v < 0.0 ? 0.0 : v);
                }
            }
        }
        free(vocab);
        return 0;
    }

    vocab = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)sh.K);
    level = (double*)malloc(sizeof(double) * (size_t)sh.K);
    if (!vocab || !level) {
        rc = -2;
        goto done;
    }
    if (cfg == 2) {
        /* the structure's keys are hashes of (op, layer, bucket): collect them */
        int64_t u = 0, i;
        uint64_t* tmp = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)sh.m);
        if (!tmp) {
            rc = -2;
            goto done;
        }
        memcpy(tmp, key, sizeof(uint64_t) * (size_t)sh.m);
        qsort(tmp, (size_t)sh.m, sizeof(uint64_t), cmp_u64);
        for (i = 0; i < sh.m; ++i)
            if (i == 0 || tmp[i] != tmp[i - 1]) {
                if (u < sh.K)
                    vocab[u] = tmp[i];
                ++u;
            }
        free(tmp);
        if (u != sh.K) {
            rc = -3;
            goto done;
        }
    } else {
        make_vocab(cfg, seed, sh.K, vocab);
    }
    if (keyindex_build(&ki, vocab, sh.K)) {
        rc = -2;
        goto done;
    }

    if (cfg == 2 || cfg == 4) {
        per_key_uniform(cfg, 0, PU_KEYPARAM, seed, sh.K, 200.0, 750.0, level);
        if (cfg == 2 && side == 1) {
            rng_t gp;
            int picked = 0;
            char* seen = (char*)calloc((size_t)sh.K, 1);
            rng_for(&gp, cfg, 1, PU_PICK, seed);
            while (seen && picked < 5) {
                int64_t r = (int64_t)(u01(&gp) * (double)sh.K);
                if (!seen[r]) {
                    seen[r] = 1;
                    level[r] *= 1.3;
                    ++picked;
                }
            }
            free(seen);
        }
        if (cfg == 4 && side >= 1) {
            double* mult = (double*)malloc(sizeof(double) * (size_t)sh.K);
            int64_t r;
            if (!mult) {
                rc = -2;
                goto done;
            }
            per_key_uniform(cfg, side, PU_PICK, seed, sh.K, 0.8, 1.5, mult);
            for (r = 0; r < sh.K; ++r)
                level[r] *= mult[r];
            free(mult);
        }
#pragma omp parallel for schedule(static)
        for (b = 0; b < nb; ++b) {
            rng_t g;
            int64_t j, top = (b + 1) * BLK < sh.n ? (b + 1) * BLK : sh.n;
            int64_t i = first_ending_after(e, 0, sh.m, t[b * BLK]);
            int64_t cur_i = -1, cur_rank = -1;
            rng_block(&g, cfg, side, PU_NOISE, seed, b);
            for (j = b * BLK; j < top; ++j) {
                double v = 100.0;
                while (i < sh.m && e[i] <= t[j])
                    ++i;
                if (i < sh.m && s[i] <= t[j] && t[j] < e[i]) {
                    if (i != cur_i) {
                        cur_i = i;
                        cur_rank = keyindex_find(&ki, key[i]);
                    }
                    if (cur_rank >= 0)
                        v = level[cur_rank];
                }
                v += 20.0 * normal01(&g);
                P[j] = (float)(v < 0.0 ? 0.0 : v);
            }
        }
    } else { /* cfg 3 */
        int S = sh.streams;
        if (S > 64) {
            rc = -1;
            goto done;
        }
        per_key_uniform(cfg, 0, PU_KEYPARAM, seed, sh.K, 50.0, 160.0, level);
        if (side == 1) {
            double* mult = (double*)malloc(sizeof(double) * (size_t)sh.K);
            int64_t r;
            if (!mult) {
                rc = -2;
                goto done;
            }
            per_key_uniform(cfg, 1, PU_PICK, seed, sh.K, 0.8, 1.5, mult);
            for (r = 0; r < sh.K; ++r)
                level[r] *= mult[r];
            free(mult);
        }
#pragma omp parallel for schedule(static)
        for (b = 0; b < nb; ++b) {
            rng_t g;
            int64_t cursor[64], cur_i[64];
            double cur_level[64];
            int a;
            int64_t j, top = (b + 1) * BLK < sh.n ? (b + 1) * BLK : sh.n;
            rng_block(&g, cfg, side, PU_NOISE, seed, b);
            for (a = 0; a < S; ++a) {
                cursor[a] = first_ending_after(e, offsets[a], offsets[a + 1], t[b * BLK]);
                cur_i[a] = -1;
                cur_level[a] = 0.0;
            }
            for (j = b * BLK; j < top; ++j) {
                double v = 100.0;
                for (a = 0; a < S; ++a) {
                    int64_t i = cursor[a];
                    while (i < offsets[a + 1] && e[i] <= t[j])
                        ++i;
                    cursor[a] = i;
                    if (i < offsets[a + 1] && s[i] <= t[j] && t[j] < e[i]) {
                        if (i != cur_i[a]) {
                            int64_t r = keyindex_find(&ki, key[i]);
                            cur_i[a] = i;
                            cur_level[a] = (r >= 0) ? level[r] : 0.0;
                        }
                        v += cur_level[a];
                    }
                }
                v += 20.0 * normal01(&g);
                P[j] = (float)(v < 0.0 ? 0.0 : v);
            }
        }
    }
done:
    keyindex_free(&ki);
    free(vocab);
    free(level);
    return rc;
}
