/*
 * mfsgd_oracle.c -- plain, slow, serial CPU oracle for SGD matrix
 * factorisation (Xie, Tan, Fong, Liang: "CuMF_SGD: Fast and Scalable Matrix
 * Factorization", arXiv 1610.05838).
 *
 * TEST INFRASTRUCTURE ONLY.  The test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark are the only code allowed to load or call
 * this library.  It shares no code, header, table or constant generator with
 * the GPU library: every routine here is written from the paper and from the
 * published definitions of the helpers it needs (IEEE 754 binary16,
 * SplitMix64, the Fisher-Yates shuffle).
 *
 * Arithmetic is IEEE binary64 throughout (built with -ffp-contract=off, no
 * fast-math).  A feature value is rounded once, to the storage type
 * (binary32 or binary16, round-to-nearest-even), when it is written back.
 *
 * Storage layout (shared with the GPU library only by specification):
 *   P  : m rows of k values, row-major  (row u is the user vector p_u)
 *   Qt : n rows of k values, row-major  (row v is the item vector q_v, i.e.
 *        the paper's k x n matrix Q stored transposed so that q_v is
 *        contiguous)
 *   a rating sample is {int32 u; int32 v; float r;}, 12 bytes, 0-based.
 *
 * Every function's pins are listed in the tests; the readings of the paper
 * it relies on are marked "Reading:" below.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int32_t u;
    int32_t v;
    float r;
} orc_sample;

enum { ORC_F32 = 0, ORC_F16 = 1 };

/* ------------------------------------------------------------------------ */
/* IEEE 754 binary16, written from the format definition: 1 sign bit, 5       */
/* exponent bits (bias 15), 10 fraction bits; subnormals have exponent field  */
/* 0 and value frac * 2^-24.                                                  */
/* ------------------------------------------------------------------------ */

double orc_half_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int f = h & 0x3ff;
    double mag;
    if (e == 0x1f)
        mag = f ? NAN : INFINITY;
    else if (e == 0)
        mag = ldexp((double)f, -24);
    else
        mag = ldexp((double)(1024 + f), e - 25);
    return sign ? -mag : mag;
}

/* Round a binary64 value to the nearest binary16, ties to even. */
uint16_t orc_double_to_half(double x)
{
    uint16_t sign = signbit(x) ? 0x8000 : 0;
    double a = fabs(x);
    if (isnan(x))
        return (uint16_t)(sign | 0x7e00);
    /* 65504 is the largest finite binary16; 65520 is the midpoint between it
     * and 2^16, and ties go to the even neighbour, which is the overflow. */
    if (a >= 65520.0)
        return (uint16_t)(sign | 0x7c00);
    if (a < ldexp(1.0, -14)) {
        /* subnormal range: multiples of 2^-24 (scaling is exact) */
        double n = nearbyint(ldexp(a, 24)); /* default mode: ties to even */
        return (uint16_t)(sign | (uint16_t)n); /* n == 1024 encodes 2^-14 */
    }
    int E;
    frexp(a, &E);               /* a = f * 2^E, f in [0.5, 1) */
    int e = E - 1;              /* a in [2^e, 2^(e+1)) */
    double n = nearbyint(ldexp(a, 10 - e)); /* 1024 <= n <= 2048 */
    if (n == 2048.0) {
        n = 1024.0;
        e += 1;
    }
    return (uint16_t)(sign | (uint16_t)((e + 15) << 10) | (uint16_t)((int)n - 1024));
}

/* ------------------------------------------------------------------------ */
/* SplitMix64 (Steele, Lea, Flood, OOPSLA 2014): the state advances by the    */
/* golden-ratio increment and each output is the state after that step passed */
/* through the variant-13 finaliser.  Output number i (0-based) of a          */
/* generator whose state starts at state0 is therefore a pure function of     */
/* (state0, i), which is how it is used here.                                 */
/* ------------------------------------------------------------------------ */

uint64_t orc_splitmix64(uint64_t state0, uint64_t i)
{
    uint64_t z = state0 + (i + 1) * 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* Stream keys: the state of stream `tag` is output number `tag` of a
 * SplitMix64 generator seeded with the user seed. */
enum {
    ORC_TAG_P = 1,
    ORC_TAG_Q = 2,
    ORC_TAG_SIGMA_C = 16, /* + 2t for epoch t */
    ORC_TAG_SIGMA_O = 17  /* + 2t for epoch t */
};

static uint64_t orc_stream(uint64_t seed, uint64_t tag) { return orc_splitmix64(seed, tag); }

/* ------------------------------------------------------------------------ */
/* Storage access                                                             */
/* ------------------------------------------------------------------------ */

static double orc_load(const void* base, int dtype, int64_t idx)
{
    if (dtype == ORC_F32)
        return (double)((const float*)base)[idx];
    return orc_half_to_double(((const uint16_t*)base)[idx]);
}

static void orc_store(void* base, int dtype, int64_t idx, double x)
{
    if (dtype == ORC_F32)
        ((float*)base)[idx] = (float)x; /* C cast: round to nearest even */
    else
        ((uint16_t*)base)[idx] = orc_double_to_half(x);
}

/* ------------------------------------------------------------------------ */
/* Initialisation.  The paper does not state one; the feature matrices start  */
/* uniform on [0, 1/sqrt(k)).  Reading: element j of row u of P takes output  */
/* u*k+j of stream (seed, P); Q likewise on stream (seed, Q).  The uniform is */
/* the top 24 bits of the output times 2^-24 (exact in binary64), multiplied  */
/* in binary64 by 1/sqrt(k) and rounded once to the storage type.             */
/* ------------------------------------------------------------------------ */

static double orc_init_value(uint64_t stream, int64_t idx, double inv_sqrt_k)
{
    uint64_t x = orc_splitmix64(stream, (uint64_t)idx);
    double u01 = (double)(x >> 40) * 0x1p-24;
    return u01 * inv_sqrt_k;
}

void orc_init_factors(int64_t m, int64_t n, int32_t k, uint64_t seed, int dtype, void* P, void* Qt)
{
    double inv_sqrt_k = 1.0 / sqrt((double)k);
    uint64_t sp = orc_stream(seed, ORC_TAG_P), sq = orc_stream(seed, ORC_TAG_Q);
    for (int64_t i = 0; i < m * (int64_t)k; i++)
        orc_store(P, dtype, i, orc_init_value(sp, i, inv_sqrt_k));
    for (int64_t i = 0; i < n * (int64_t)k; i++)
        orc_store(Qt, dtype, i, orc_init_value(sq, i, inv_sqrt_k));
}

/* The same initial values for selected rows only (which: 0 = P, 1 = Q^T):
 * out[i][j] = initial value of row rows[i], column j.  Lets a check at a very
 * large m look at the rows a sample prefix touches without building all of P. */
void orc_init_rows(int64_t nrows_total, int32_t k, uint64_t seed, int dtype, int which, const int64_t* rows,
                   int64_t count, void* out)
{
    double inv_sqrt_k = 1.0 / sqrt((double)k);
    uint64_t st = orc_stream(seed, which ? ORC_TAG_Q : ORC_TAG_P);
    (void)nrows_total;
    for (int64_t i = 0; i < count; i++)
        for (int32_t j = 0; j < k; j++)
            orc_store(out, dtype, i * k + j, orc_init_value(st, rows[i] * (int64_t)k + j, inv_sqrt_k));
}

/* ------------------------------------------------------------------------ */
/* One SGD update (section 2.2, the error and the two update equations).      */
/* Reading: both vectors are updated from their values before this step (the */
/* gradient of the per-sample cost at the current point); the factor 2 of the */
/* squared loss is absorbed into the learning rate.                           */
/* p and q are binary64 working copies of p_u and q_v, updated in place.      */
/* ------------------------------------------------------------------------ */

void orc_sgd_step(double* p, double* q, int32_t k, double r, double lr, double lambda_p, double lambda_q)
{
    double dot = 0.0;
    for (int32_t j = 0; j < k; j++)
        dot += p[j] * q[j];
    double err = r - dot;
    for (int32_t j = 0; j < k; j++) {
        double pj = p[j], qj = q[j];
        p[j] = pj + lr * (err * qj - lambda_p * pj);
        q[j] = qj + lr * (err * pj - lambda_q * qj);
    }
}

/* Apply the update for one sample to storage: widen p_u and q_v, step, round
 * both rows back once. */
static void orc_update_sample(void* P, void* Qt, int dtype, int32_t k, const orc_sample* s, double lr,
                              double lambda_p, double lambda_q, double* pbuf, double* qbuf)
{
    int64_t pu = (int64_t)s->u * k, qv = (int64_t)s->v * k;
    for (int32_t j = 0; j < k; j++) {
        pbuf[j] = orc_load(P, dtype, pu + j);
        qbuf[j] = orc_load(Qt, dtype, qv + j);
    }
    orc_sgd_step(pbuf, qbuf, k, (double)s->r, lr, lambda_p, lambda_q);
    for (int32_t j = 0; j < k; j++) {
        orc_store(P, dtype, pu + j, pbuf[j]);
        orc_store(Qt, dtype, qv + j, qbuf[j]);
    }
}

/* ------------------------------------------------------------------------ */
/* Serial epoch: N updates, one per sample, in array order (section 2.3: an   */
/* epoch is N updates one after the other).  Reading: the sample array is    */
/* shuffled once when it is made (section 3.2.2 relies on that shuffle), so   */
/* array order is the serial order.  This is also the order batch-Hogwild!    */
/* reduces to with a single worker.                                           */
/* ------------------------------------------------------------------------ */

int orc_epoch_serial(int32_t k, int dtype, void* P, void* Qt, const orc_sample* S, int64_t nnz, float lr,
                     float lambda_p, float lambda_q)
{
    double* buf = (double*)malloc(2 * sizeof(double) * (size_t)k);
    if (!buf)
        return -2;
    for (int64_t i = 0; i < nnz; i++)
        orc_update_sample(P, Qt, dtype, k, &S[i], lr, lambda_p, lambda_q, buf, buf + k);
    free(buf);
    return 0;
}

/* batch-Hogwild! schedule (section 3.2.2): batches of f consecutive samples.
 * Reading: batch b = samples [b*f, min((b+1)*f, nnz)) goes to worker b mod W
 * and a worker updates its batches in increasing b, each serially.  Writes
 * out[b] = worker of batch b for b < ceil(nnz/f). */
void orc_hogwild_batch_owner(int64_t nnz, int32_t f, int64_t W, int64_t* out)
{
    int64_t nb = (nnz + f - 1) / f;
    for (int64_t b = 0; b < nb; b++)
        out[b] = b % W;
}

/* ------------------------------------------------------------------------ */
/* Wavefront-update (section 3.2.3).                                          */
/* Reading: R is cut into an s x s grid; sample (u,v) is in row block         */
/* floor(u*s/m) and column block floor(v*s/n).  Worker i owns row block i.    */
/* Each worker's column sequence is row i of a Latin square                   */
/*     sigma_i(w) = C[(i + O[w]) mod s]                                       */
/* where C and O are permutations of 0..s-1 drawn afresh each epoch t, so in  */
/* every wave the s workers touch s different columns and each worker visits  */
/* every column once per epoch.  A block's samples keep their array order.    */
/* ------------------------------------------------------------------------ */

int32_t orc_row_block(int64_t u, int64_t m, int32_t s) { return (int32_t)((u * (int64_t)s) / m); }
int32_t orc_col_block(int64_t v, int64_t n, int32_t s) { return (int32_t)((v * (int64_t)s) / n); }

/* Load-balanced alternative to the equal index ranges above (the paper draws
 * equal blocks and does not say how they are cut).  The indices (users if
 * which == 0, items if which == 1) are split into s consecutive ranges so
 * that the largest number of samples in one range is as small as possible.
 * Canonical choice: C = the smallest cap for which filling ranges greedily
 * (a range takes the next index while its count stays <= C) needs at most s
 * ranges; the ranges are those of that greedy fill.  bounds[k] is the first
 * index of range k; unused trailing ranges are empty and start at N. */
static int64_t orc_greedy_ranges(const int64_t* cnt, int64_t N, int64_t cap, int32_t s, int64_t* bounds)
{
    int64_t k = 0, load = 0;
    if (bounds)
        bounds[0] = 0;
    for (int64_t i = 0; i < N; i++) {
        if (load + cnt[i] > cap) {
            k++;
            load = 0;
            if (bounds && k <= s)
                bounds[k] = i;
        }
        load += cnt[i];
    }
    if (bounds)
        for (int64_t j = k + 1; j <= s; j++)
            bounds[j] = N;
    return k + 1;
}

int orc_balanced_bounds(const orc_sample* S, int64_t nnz, int64_t N, int which, int32_t s, int64_t* bounds)
{
    int64_t* cnt = (int64_t*)calloc((size_t)N, sizeof(int64_t));
    if (!cnt)
        return -2;
    int64_t top = 0;
    for (int64_t i = 0; i < nnz; i++)
        cnt[which ? S[i].v : S[i].u]++;
    for (int64_t i = 0; i < N; i++)
        top = cnt[i] > top ? cnt[i] : top;
    int64_t lo = (nnz + s - 1) / s;
    lo = lo > top ? lo : top;
    int64_t hi = nnz > lo ? nnz : lo; /* one range holding everything always fits */
    while (lo < hi) {                 /* smallest feasible cap */
        int64_t mid = lo + (hi - lo) / 2;
        if (orc_greedy_ranges(cnt, N, mid, s, NULL) <= s)
            hi = mid;
        else
            lo = mid + 1;
    }
    orc_greedy_ranges(cnt, N, lo, s, bounds);
    free(cnt);
    return 0;
}

int32_t orc_bounded_block(int64_t i, const int64_t* bounds, int32_t s)
{
    int32_t k = 0;
    for (int32_t j = 0; j < s; j++)
        if (bounds[j] <= i)
            k = j;
    return k;
}

/* Durstenfeld's Fisher-Yates: for i = s-1 down to 1 swap a[i] with a[j],
 * j uniform on 0..i.  Draw number (s-1-i) of the stream gives j as the high
 * 32 bits times (i+1), shifted down 32 (multiply-shift range reduction). */
void orc_fisher_yates(uint64_t stream, int32_t s, int32_t* a)
{
    for (int32_t i = 0; i < s; i++)
        a[i] = i;
    for (int32_t i = s - 1; i >= 1; i--) {
        uint64_t x = orc_splitmix64(stream, (uint64_t)(s - 1 - i));
        int32_t j = (int32_t)(((x >> 32) * (uint64_t)(i + 1)) >> 32);
        int32_t t = a[i];
        a[i] = a[j];
        a[j] = t;
    }
}

/* sigma[i*s + w] = column block worker i processes in wave w of epoch t. */
int orc_wavefront_sigma(uint64_t seed, int64_t t, int32_t s, int32_t* sigma)
{
    int32_t* C = (int32_t*)malloc(sizeof(int32_t) * (size_t)s);
    int32_t* O = (int32_t*)malloc(sizeof(int32_t) * (size_t)s);
    if (!C || !O) {
        free(C);
        free(O);
        return -2;
    }
    orc_fisher_yates(orc_stream(seed, (uint64_t)(ORC_TAG_SIGMA_C + 2 * t)), s, C);
    orc_fisher_yates(orc_stream(seed, (uint64_t)(ORC_TAG_SIGMA_O + 2 * t)), s, O);
    for (int32_t i = 0; i < s; i++)
        for (int32_t w = 0; w < s; w++)
            sigma[(int64_t)i * s + w] = C[(i + O[w]) % s];
    free(C);
    free(O);
    return 0;
}

/* Group sample indices by block (I, J), keeping array order inside a block:
 * order[] receives the sample indices block by block (block id I*s+J
 * ascending), start[b] .. start[b+1] delimits block b.  A counting pass,
 * a prefix sum and an in-order placement. */
static int64_t orc_block_id(const orc_sample* x, int64_t m, int64_t n, int32_t s, const int64_t* rb,
                            const int64_t* cb)
{
    int32_t r = rb ? orc_bounded_block(x->u, rb, s) : orc_row_block(x->u, m, s);
    int32_t c = cb ? orc_bounded_block(x->v, cb, s) : orc_col_block(x->v, n, s);
    return (int64_t)r * s + c;
}

/* rb, cb: balanced bounds (s+1 entries each) or NULL for equal index ranges. */
int orc_block_order(const orc_sample* S, int64_t nnz, int64_t m, int64_t n, int32_t s, const int64_t* rb,
                    const int64_t* cb, int64_t* order, int64_t* start)
{
    int64_t nb = (int64_t)s * s;
    int64_t* fill = (int64_t*)calloc((size_t)nb, sizeof(int64_t));
    if (!fill)
        return -2;
    for (int64_t b = 0; b <= nb; b++)
        start[b] = 0;
    for (int64_t i = 0; i < nnz; i++)
        start[orc_block_id(&S[i], m, n, s, rb, cb) + 1]++;
    for (int64_t b = 0; b < nb; b++)
        start[b + 1] += start[b];
    for (int64_t i = 0; order && i < nnz; i++) { /* order == NULL: block starts only */
        int64_t b = orc_block_id(&S[i], m, n, s, rb, cb);
        order[start[b] + fill[b]++] = i;
    }
    free(fill);
    return 0;
}

/* One deterministic wavefront-update epoch in its serial-equivalent order:
 * waves in sequence; inside a wave, workers 0..s-1 in sequence (their blocks
 * share no row and no column, so any interleaving gives the same result);
 * inside a block, array order. */
int orc_epoch_wavefront(int64_t m, int64_t n, int32_t k, int dtype, void* P, void* Qt, const orc_sample* S,
                        int64_t nnz, float lr, float lambda_p, float lambda_q, int32_t s, uint64_t seed,
                        int64_t t, int balanced)
{
    int64_t nb = (int64_t)s * s;
    int64_t* order = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nnz > 0 ? nnz : 1));
    int64_t* start = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nb + 1));
    int32_t* sigma = (int32_t*)malloc(sizeof(int32_t) * (size_t)nb);
    double* buf = (double*)malloc(2 * sizeof(double) * (size_t)k);
    int64_t* rb = (int64_t*)malloc(sizeof(int64_t) * (size_t)(s + 1));
    int64_t* cb = (int64_t*)malloc(sizeof(int64_t) * (size_t)(s + 1));
    int rc = -2;
    if (balanced && rb && cb &&
        (orc_balanced_bounds(S, nnz, m, 0, s, rb) || orc_balanced_bounds(S, nnz, n, 1, s, cb)))
        balanced = -1;
    if (balanced >= 0 && order && start && sigma && buf && rb && cb &&
        orc_block_order(S, nnz, m, n, s, balanced ? rb : NULL, balanced ? cb : NULL, order, start) == 0 &&
        orc_wavefront_sigma(seed, t, s, sigma) == 0) {
        for (int32_t w = 0; w < s; w++)
            for (int32_t i = 0; i < s; i++) {
                int64_t b = (int64_t)i * s + sigma[(int64_t)i * s + w];
                for (int64_t x = start[b]; x < start[b + 1]; x++)
                    orc_update_sample(P, Qt, dtype, k, &S[order[x]], lr, lambda_p, lambda_q, buf, buf + k);
            }
        rc = 0;
    }
    free(order);
    free(start);
    free(sigma);
    free(buf);
    free(rb);
    free(cb);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Global scheduling table (section 3.2.1): LIBMF's policy, which the paper   */
/* measures on a GPU ("LIBMF-GPU") as the baseline its two schedules replace. */
/* R is cut into an s x s grid of blocks (equal index ranges, as above); one  */
/* table, used by one worker at a time, records which row blocks and column   */
/* blocks are in use, and a free worker is given an idle block that shares    */
/* neither with a block in progress.                                          */
/* Reading: an epoch takes every non-empty block exactly once, and among the  */
/* blocks not yet taken the choice is random (LIBMF's least-updated-first    */
/* rule, with random ties, reduces to this inside one epoch).  The table keeps */
/* the blocks not yet taken in a list, initially the non-empty block ids in   */
/* ascending order.  Decision d of epoch t draws a position uniformly from    */
/* the list (output d of stream (seed, TABLE + t), high 32 bits times the     */
/* list length, shifted down 32), takes the first block at or cyclically     */
/* after that position whose row and column are free, and moves the list's   */
/* last entry into its place.  A single worker finds every block free, so    */
/* its order is the draw order alone, which is what is computed here.        */
/* ------------------------------------------------------------------------ */

#define ORC_TAG_TABLE (1ULL << 40) /* + t for epoch t */

int orc_table_order(uint64_t seed, int64_t t, const int64_t* blocks, int64_t nblocks, int64_t* order)
{
    int64_t* list = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nblocks > 0 ? nblocks : 1));
    if (!list)
        return -2;
    memcpy(list, blocks, sizeof(int64_t) * (size_t)nblocks);
    uint64_t stream = orc_stream(seed, ORC_TAG_TABLE + (uint64_t)t);
    int64_t rem = nblocks;
    for (int64_t d = 0; d < nblocks; d++) {
        uint64_t x = orc_splitmix64(stream, (uint64_t)d);
        int64_t pos = (int64_t)(((x >> 32) * (uint64_t)rem) >> 32);
        order[d] = list[pos];
        list[pos] = list[rem - 1];
        rem--;
    }
    free(list);
    return 0;
}

/* One epoch under the global table with a single worker: the non-empty blocks
 * of the equal-range s x s grid in the order of orc_table_order, each block's
 * samples in array order. */
int orc_epoch_table(int64_t m, int64_t n, int32_t k, int dtype, void* P, void* Qt, const orc_sample* S,
                    int64_t nnz, float lr, float lambda_p, float lambda_q, int32_t s, uint64_t seed, int64_t t)
{
    int64_t nb = (int64_t)s * s;
    int64_t* order = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nnz > 0 ? nnz : 1));
    int64_t* start = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nb + 1));
    int64_t* blocks = (int64_t*)malloc(sizeof(int64_t) * (size_t)nb);
    int64_t* seq = (int64_t*)malloc(sizeof(int64_t) * (size_t)nb);
    double* buf = (double*)malloc(2 * sizeof(double) * (size_t)k);
    int rc = -2;
    if (order && start && blocks && seq && buf && orc_block_order(S, nnz, m, n, s, NULL, NULL, order, start) == 0) {
        int64_t used = 0;
        for (int64_t b = 0; b < nb; b++)
            if (start[b + 1] > start[b])
                blocks[used++] = b;
        if (orc_table_order(seed, t, blocks, used, seq) == 0) {
            for (int64_t d = 0; d < used; d++)
                for (int64_t x = start[seq[d]]; x < start[seq[d] + 1]; x++)
                    orc_update_sample(P, Qt, dtype, k, &S[order[x]], lr, lambda_p, lambda_q, buf, buf + k);
            rc = 0;
        }
    }
    free(order);
    free(start);
    free(blocks);
    free(seq);
    free(buf);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Test RMSE: the square root of the mean squared prediction error over the  */
/* held-out samples (the convergence measure of section 3.2.4), without any  */
/* clamping of the prediction.  ntest == 0 gives 0.                           */
/* ------------------------------------------------------------------------ */

double orc_rmse(int32_t k, int dtype, const void* P, const void* Qt, const orc_sample* T, int64_t ntest)
{
    if (ntest <= 0)
        return 0.0;
    double sum = 0.0;
    for (int64_t i = 0; i < ntest; i++) {
        int64_t pu = (int64_t)T[i].u * k, qv = (int64_t)T[i].v * k;
        double dot = 0.0;
        for (int32_t j = 0; j < k; j++)
            dot += orc_load(P, dtype, pu + j) * orc_load(Qt, dtype, qv + j);
        double e = (double)T[i].r - dot;
        sum += e * e;
    }
    return sqrt(sum / (double)ntest);
}

/* Per-sample squared error for the first `count` samples (for spot checks at
 * sizes where only sampled outputs are compared). */
void orc_sq_errors(int32_t k, int dtype, const void* P, const void* Qt, const orc_sample* T, int64_t count,
                   double* out)
{
    for (int64_t i = 0; i < count; i++) {
        int64_t pu = (int64_t)T[i].u * k, qv = (int64_t)T[i].v * k;
        double dot = 0.0;
        for (int32_t j = 0; j < k; j++)
            dot += orc_load(P, dtype, pu + j) * orc_load(Qt, dtype, qv + j);
        double e = (double)T[i].r - dot;
        out[i] = e * e;
    }
}

/* The section 2.2 objective: sum over samples of the squared error plus the
 * two regularisers, each counted once per sample (diagnostic only). */
double orc_objective(int32_t k, int dtype, const void* P, const void* Qt, const orc_sample* S, int64_t nnz,
                     double lambda_p, double lambda_q)
{
    double sum = 0.0;
    for (int64_t i = 0; i < nnz; i++) {
        int64_t pu = (int64_t)S[i].u * k, qv = (int64_t)S[i].v * k;
        double dot = 0.0, pp = 0.0, qq = 0.0;
        for (int32_t j = 0; j < k; j++) {
            double p = orc_load(P, dtype, pu + j), q = orc_load(Qt, dtype, qv + j);
            dot += p * q;
            pp += p * p;
            qq += q * q;
        }
        double e = (double)S[i].r - dot;
        sum += e * e + lambda_p * pp + lambda_q * qq;
    }
    return sum;
}

/* ------------------------------------------------------------------------ */
/* OpenMP Hogwild! variant -- for CPU timing only, never for parity.          */
/* Threads claim batches of f samples from a shared counter and apply the     */
/* same per-sample update without any locking (races are intended).          */
/* Returns the number of threads used.                                        */
/* ------------------------------------------------------------------------ */

int orc_epoch_hogwild_omp(int32_t k, int dtype, void* P, void* Qt, const orc_sample* S, int64_t nnz, float lr,
                          float lambda_p, float lambda_q, int32_t f, int32_t nthreads)
{
    int used = 1;
    int64_t nb = (nnz + f - 1) / f;
    int64_t next = 0;
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#pragma omp parallel
    {
#pragma omp single
        used = omp_get_num_threads();
        double* buf = (double*)malloc(2 * sizeof(double) * (size_t)k);
        for (;;) {
            int64_t b;
#pragma omp atomic capture
            b = next++;
            if (b >= nb)
                break;
            int64_t hi = (b + 1) * f < nnz ? (b + 1) * f : nnz;
            for (int64_t i = b * f; i < hi; i++)
                orc_update_sample(P, Qt, dtype, k, &S[i], lr, lambda_p, lambda_q, buf, buf + k);
        }
        free(buf);
    }
#else
    (void)nthreads;
    (void)nb;
    (void)next;
    orc_epoch_serial(k, dtype, P, Qt, S, nnz, lr, lambda_p, lambda_q);
#endif
    return used;
}
