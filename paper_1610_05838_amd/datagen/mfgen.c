/*
 * mfgen.c -- seeded synthetic rating data for SGD matrix factorisation.
 *
 * Makes stand-ins with the shapes of the paper's Table 2 data sets (which are
 * not available here): a planted low-rank model p*_u . q*_v plus noise,
 * user/item indices drawn uniformly or Zipf-like.  Nothing here performs an
 * SGD step; the module only makes inputs, which both the GPU library and the
 * CPU checker consume.
 *
 * Every random draw is a pure function of (seed, stream, counter), so a
 * sample depends only on its index and generation parallelises with OpenMP
 * without changing the output.  Draws come from SplitMix64 outputs (Steele,
 * Lea, Flood 2014) used in counter mode.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int32_t u;
    int32_t v;
    float r;
} gen_sample;

typedef struct {
    int64_t m, n;
    int32_t k;         /* rank of the planted model (may be below the trained rank) */
    int32_t model;     /* rating model, see gen_rating */
    uint64_t seed;
    double noise_var;  /* variance of the additive Gaussian noise */
    double mean;       /* offset added before rounding (model 1) */
} gen_spec;

enum { GEN_ADDITIVE = 0, GEN_STARS = 1, GEN_PERCENTILE = 2, GEN_REAL = 3 };

enum {
    GEN_S_PSTAR = 101,
    GEN_S_QSTAR = 102,
    GEN_S_DRAW = 103,
    GEN_S_PERM_U = 104,
    GEN_S_PERM_V = 105,
    GEN_S_CELLS = 106
};

static uint64_t gen_hash(uint64_t state0, uint64_t i)
{
    uint64_t z = state0 + (i + 1) * 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static uint64_t gen_stream(uint64_t seed, uint64_t which) { return gen_hash(seed ^ 0xA5A5A5A5DEADBEEFULL, which); }

/* uniform on [0,1) with 53 bits */
static double gen_u01(uint64_t x) { return (double)(x >> 11) * 0x1p-53; }

/* standard normal from one 64-bit draw (Box-Muller on its two 32-bit halves) */
static double gen_normal(uint64_t x)
{
    double u1 = ((double)(x >> 32) + 0.5) * 0x1p-32; /* (0,1) */
    double u2 = (double)(x & 0xffffffffULL) * 0x1p-32;
    return sqrt(-2.0 * log(u1)) * cos(6.283185307179586476925 * u2);
}

/* planted factors: every entry N(0, 1/sqrt(k)) (the second parameter is the variance) */
void gen_planted(const gen_spec* sp, float* Ps, float* Qs)
{
    double sd = sqrt(1.0 / sqrt((double)sp->k));
    uint64_t a = gen_stream(sp->seed, GEN_S_PSTAR), b = gen_stream(sp->seed, GEN_S_QSTAR);
    int64_t nm = sp->m * sp->k, nn = sp->n * sp->k;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < nm; i++)
        Ps[i] = (float)(sd * gen_normal(gen_hash(a, (uint64_t)i)));
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < nn; i++)
        Qs[i] = (float)(sd * gen_normal(gen_hash(b, (uint64_t)i)));
}

/* Zipf-like table over N ranks: P(rank r) proportional to r^-a (r = 1..N),
 * cdf[r-1] = cumulative probability; perm maps rank-1 to an index through a
 * seeded Fisher-Yates permutation, so popularity is not tied to the index.
 * guide[j] (j = 0..G, G = 2^guide_bits) = first r with cdf[r] > j/G, which
 * narrows the search of gen_pick to one bucket (Chen and Asau's guide table);
 * the pick itself is unchanged. */
void gen_zipf_table(int64_t N, double a, uint64_t seed, int which, double* cdf, int32_t* perm)
{
    double acc = 0.0;
    for (int64_t r = 1; r <= N; r++) {
        acc += pow((double)r, -a);
        cdf[r - 1] = acc;
    }
    for (int64_t r = 0; r < N; r++)
        cdf[r] /= acc;
    cdf[N - 1] = 1.0;
    uint64_t st = gen_stream(seed, which ? GEN_S_PERM_V : GEN_S_PERM_U);
    for (int64_t i = 0; i < N; i++)
        perm[i] = (int32_t)i;
    for (int64_t i = N - 1; i >= 1; i--) {
        uint64_t x = gen_hash(st, (uint64_t)(N - 1 - i));
        int64_t j = (int64_t)(((unsigned __int128)x * (unsigned __int128)(i + 1)) >> 64);
        int32_t t = perm[i];
        perm[i] = perm[j];
        perm[j] = t;
    }
}

void gen_zipf_guide(int64_t N, const double* cdf, int guide_bits, int64_t* guide)
{
    const int64_t G = (int64_t)1 << guide_bits;
    int64_t r = 0;
    for (int64_t j = 0; j < G; j++) {
        const double x = ldexp((double)j, -guide_bits);
        while (r < N - 1 && !(cdf[r] > x))
            r++;
        guide[j] = r;
    }
    guide[G] = N - 1;
}

typedef struct {
    const double* cdf;   /* NULL: uniform */
    const int32_t* perm;
    const int64_t* guide; /* NULL: plain binary search */
    int guide_bits;
} gen_table;

static int64_t gen_pick(double x, int64_t N, const gen_table* t)
{
    if (!t->cdf) {
        int64_t i = (int64_t)(x * (double)N);
        return i < N ? i : N - 1;
    }
    const double* cdf = t->cdf;
    int64_t lo = 0, hi = N - 1; /* first r with cdf[r] > x */
    if (t->guide) {
        const int64_t j = (int64_t)ldexp(x, t->guide_bits); /* exact: x < 1 is scaled by a power of two */
        lo = t->guide[j];
        hi = t->guide[j + 1];
    }
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (cdf[mid] > x)
            hi = mid;
        else
            lo = mid + 1;
    }
    return t->perm[lo];
}

static float gen_rating(const gen_spec* sp, const float* Ps, const float* Qs, int64_t u, int64_t v, double z)
{
    const float* p = Ps + u * sp->k;
    const float* q = Qs + v * sp->k;
    double dot = 0.0;
    for (int32_t j = 0; j < sp->k; j++)
        dot += (double)p[j] * (double)q[j];
    double x = dot + sqrt(sp->noise_var) * z;
    switch (sp->model) {
    case GEN_STARS: { /* clamp(round(mean + dot + noise), 1, 5) */
        double s = floor(sp->mean + x + 0.5);
        return (float)(s < 1.0 ? 1.0 : (s > 5.0 ? 5.0 : s));
    }
    case GEN_PERCENTILE: { /* integer 0..100 from the normal CDF, then /20 */
        double c = 0.5 * erfc(-x / sqrt(2.0));
        double s = floor(100.0 * c + 0.5);
        s = s < 0.0 ? 0.0 : (s > 100.0 ? 100.0 : s);
        return (float)(s / 20.0);
    }
    case GEN_REAL:
    case GEN_ADDITIVE:
    default:
        return (float)(sp->mean + x);
    }
}

/* Picks for explicit uniforms (lets a test compare the guided and the plain search). */
void gen_pick_batch(const double* x, int64_t count, int64_t N, const gen_table* t, int64_t* out)
{
    for (int64_t i = 0; i < count; i++)
        out[i] = gen_pick(x[i], N, t);
}

/* Independent draws for counters c0 .. c0+count-1: user and item from the
 * given tables (NULL cdf = uniform), rating from the planted model. */
void gen_draw(const gen_spec* sp, const float* Ps, const float* Qs, const gen_table* tu, const gen_table* tv,
              int64_t c0, int64_t count, gen_sample* out)
{
    uint64_t st = gen_stream(sp->seed, GEN_S_DRAW);
#pragma omp parallel for schedule(static, 4096)
    for (int64_t i = 0; i < count; i++) {
        uint64_t c = (uint64_t)(c0 + i) * 4;
        int64_t u = gen_pick(gen_u01(gen_hash(st, c)), sp->m, tu);
        int64_t v = gen_pick(gen_u01(gen_hash(st, c + 1)), sp->n, tv);
        double z = gen_normal(gen_hash(st, c + 2));
        out[i].u = (int32_t)u;
        out[i].v = (int32_t)v;
        out[i].r = gen_rating(sp, Ps, Qs, u, v, z);
    }
}

/* `total` distinct cells of the m x n grid, uniformly, in random order
 * (partial Fisher-Yates over the cell ids).  Returns 0, or -1 if total > m*n
 * or memory runs out. */
int gen_distinct(const gen_spec* sp, const float* Ps, const float* Qs, int64_t total, gen_sample* out)
{
    int64_t cells = sp->m * sp->n;
    if (total > cells)
        return -1;
    int64_t* id = (int64_t*)malloc(sizeof(int64_t) * (size_t)cells);
    if (!id)
        return -1;
    for (int64_t i = 0; i < cells; i++)
        id[i] = i;
    uint64_t st = gen_stream(sp->seed, GEN_S_CELLS);
    for (int64_t i = 0; i < total; i++) {
        uint64_t x = gen_hash(st, (uint64_t)i);
        int64_t j = i + (int64_t)(((unsigned __int128)x * (unsigned __int128)(cells - i)) >> 64);
        int64_t t = id[i];
        id[i] = id[j];
        id[j] = t;
    }
    uint64_t sd = gen_stream(sp->seed, GEN_S_DRAW);
    for (int64_t i = 0; i < total; i++) {
        int64_t u = id[i] / sp->n, v = id[i] % sp->n;
        out[i].u = (int32_t)u;
        out[i].v = (int32_t)v;
        out[i].r = gen_rating(sp, Ps, Qs, u, v, gen_normal(gen_hash(sd, (uint64_t)i)));
    }
    free(id);
    return 0;
}
