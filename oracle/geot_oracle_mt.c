/*
 * Multi-threaded CPU oracle: the serial oracle's definitions, with the output
 * segments split into contiguous ranges, one range per POSIX thread.
 *
 * TEST INFRASTRUCTURE ONLY, like geot_oracle.c: only the test suite and the
 * bench's CPU baseline load it; the GPU library never includes, links or calls
 * it. It exists so that full-size parity checks and the all-core CPU baseline
 * finish in seconds; the serial oracle in geot_oracle.c is the reference it is
 * checked against (bit for bit, on the CPU).
 *
 * What it computes is the same plain definition (GeoT paper, Section II-B,
 * segment reduction; Section IV and V-D, the fused gather-weight form): output
 * row s reduces the terms of the rows (edges) whose sorted index is s, with
 *  - sum and mean accumulated in fp64 in row order and rounded once to fp32
 *    (mean divides the fp64 sum by the count in fp64);
 *  - max the IEEE 754-2019 maximum folded over the members in fp32 (NaN
 *    propagates, +0 ranks above -0);
 *  - a weighted term one fp32 multiply w[e] * x;
 *  - empty segments 0.0f.
 * Each output element is computed by exactly one thread with the same
 * operations in the same order as the serial oracle, so the results are
 * identical bit for bit whatever the thread count. Segments are independent;
 * the split only decides which thread computes which of them.
 *
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off -pthread -shared -fPIC.
 * Error codes as the serial oracle: 0 ok, 1 invalid argument, 2 index not
 * sorted, 3 index (or column) out of range.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>

enum { MT_OK = 0, MT_INVALID = 1, MT_NOT_SORTED = 2, MT_OUT_OF_RANGE = 3 };
enum { MT_SUM = 0, MT_MEAN = 1, MT_MAX = 2 };
#define MT_MAX_THREADS 256

static int check_index(const int64_t *idx, int64_t nnz, int64_t S)
{
    for (int64_t i = 0; i < nnz; ++i) {
        if (idx[i] < 0 || idx[i] >= S) return MT_OUT_OF_RANGE;
        if (i > 0 && idx[i] < idx[i - 1]) return MT_NOT_SORTED;
    }
    return MT_OK;
}

/* start[s] = first row with idx >= s, s = 0..S (one linear walk). */
static void starts_of(const int64_t *idx, int64_t nnz, int64_t S, int64_t *start)
{
    int64_t i = 0;
    for (int64_t s = 0; s <= S; ++s) {
        while (i < nnz && idx[i] < s) ++i;
        start[s] = i;
    }
}

static float term_of(const float *rows, int64_t F, const int64_t *col, const float *w, int64_t e, int64_t f)
{
    if (col == NULL) return rows[e * F + f];
    float x = rows[col[e] * F + f];
    if (w == NULL) return x;
    float t = w[e] * x; /* one fp32 multiply */
    return t;
}

/* IEEE 754-2019 maximum(a, b): NaN when either is NaN; +0 above -0. */
static float max754(float a, float b)
{
    if (isnan(a)) return a;
    if (isnan(b)) return b;
    if (a == b) return signbit(a) ? b : a;
    return a > b ? a : b;
}

typedef struct {
    const float *rows;
    int64_t F;
    const int64_t *col;
    const float *w;
    const int64_t *start;
    int64_t s0, s1; /* this thread's segments [s0, s1) */
    int op;
    int absolute;   /* 1: per element sum of |term| in fp64 (mean: divided by the count) */
    float *out;
    double *out_abs;
} job_t;

static void *run_job(void *arg)
{
    const job_t *j = (const job_t *)arg;
    const int64_t F = j->F;
    for (int64_t s = j->s0; s < j->s1; ++s) {
        const int64_t b = j->start[s], e = j->start[s + 1], count = e - b;
        for (int64_t f = 0; f < F; ++f) {
            if (j->absolute) {
                double acc = 0.0;
                for (int64_t i = b; i < e; ++i) acc += fabs((double)term_of(j->rows, F, j->col, j->w, i, f));
                if (j->op == MT_MEAN && count > 0) acc /= (double)count;
                j->out_abs[s * F + f] = acc;
                continue;
            }
            float result;
            if (count == 0) {
                result = 0.0f;
            } else if (j->op == MT_MAX) {
                float m = term_of(j->rows, F, j->col, j->w, b, f);
                for (int64_t i = b + 1; i < e; ++i) m = max754(m, term_of(j->rows, F, j->col, j->w, i, f));
                result = m;
            } else {
                double acc = 0.0;
                for (int64_t i = b; i < e; ++i) acc += (double)term_of(j->rows, F, j->col, j->w, i, f);
                if (j->op == MT_MEAN) acc = acc / (double)count;
                result = (float)acc;
            }
            j->out[s * F + f] = result;
        }
    }
    return NULL;
}

/* Splits [0, S) into nthreads ranges of about equal work (rows plus one per segment),
 * runs them and joins. */
static int run_split(job_t base, int64_t S, int64_t nnz, int nthreads)
{
    if (nthreads < 1) nthreads = 1;
    if (nthreads > MT_MAX_THREADS) nthreads = MT_MAX_THREADS;
    if ((int64_t)nthreads > S) nthreads = (int)S;
    pthread_t tid[MT_MAX_THREADS];
    job_t jobs[MT_MAX_THREADS];
    const double total = (double)nnz + (double)S;
    int64_t s = 0;
    int started = 0, rc = MT_OK;
    for (int t = 0; t < nthreads; ++t) {
        int64_t s1 = S;
        if (t + 1 < nthreads) {
            const double goal = total * (double)(t + 1) / (double)nthreads;
            s1 = s;
            while (s1 < S && (double)base.start[s1] + (double)s1 < goal) ++s1;
        }
        jobs[t] = base;
        jobs[t].s0 = s;
        jobs[t].s1 = s1;
        s = s1;
        if (pthread_create(&tid[t], NULL, run_job, &jobs[t]) != 0) {
            run_job(&jobs[t]); /* no thread: run this range here */
            tid[t] = 0;
            continue;
        }
        ++started;
    }
    for (int t = 0; t < nthreads; ++t)
        if (tid[t] != 0 && pthread_join(tid[t], NULL) != 0) rc = MT_INVALID;
    (void)started;
    return rc;
}

static int reduce_mt(const float *rows, int64_t n_x, const int64_t *col, const float *w, const int64_t *idx,
                     int64_t nnz, int64_t S, int64_t F, int op, int absolute, float *out, double *out_abs,
                     int nthreads)
{
    if (nnz < 0 || S < 0 || F < 0 || n_x < 0 || op < MT_SUM || op > MT_MAX) return MT_INVALID;
    if (S == 0 || F == 0) return MT_OK;
    int rc = check_index(idx, nnz, S);
    if (rc != MT_OK) return rc;
    if (col)
        for (int64_t e = 0; e < nnz; ++e)
            if (col[e] < 0 || col[e] >= n_x) return MT_OUT_OF_RANGE;
    int64_t *start = (int64_t *)malloc((size_t)(S + 1) * sizeof(int64_t));
    if (!start) return MT_INVALID;
    starts_of(idx, nnz, S, start);
    job_t base = {rows, F, col, w, start, 0, 0, op, absolute, out, out_abs};
    rc = run_split(base, S, nnz, nthreads);
    free(start);
    return rc;
}

/* out[s, :] = op over { src[i, :] : idx[i] == s } (as oracle_segment_reduce). */
int oracle_mt_segment_reduce(const float *src, const int64_t *idx, int64_t nnz, int64_t S, int64_t F, int op,
                             float *out, int nthreads)
{
    return reduce_mt(src, nnz, NULL, NULL, idx, nnz, S, F, op, 0, out, NULL, nthreads);
}

/* out[r, :] = op over { w[e] * X[col[e], :] : row[e] == r } (as oracle_gather_scatter). */
int oracle_mt_gather_scatter(const float *X, int64_t n_x, const int64_t *col, const float *w, const int64_t *row,
                             int64_t nnz, int64_t R, int64_t F, int op, float *out, int nthreads)
{
    return reduce_mt(X, n_x, col, w, row, nnz, R, F, op, 0, out, NULL, nthreads);
}

/* Per output element, the fp64 sum of |term| (as oracle_abs_term_sum); col NULL: plain rows. */
int oracle_mt_abs_term_sum(const float *rows, int64_t n_x, const int64_t *col, const float *w, const int64_t *idx,
                           int64_t nnz, int64_t S, int64_t F, int op, double *out, int nthreads)
{
    return reduce_mt(rows, col ? n_x : nnz, col, w, idx, nnz, S, F, op, 1, NULL, out, nthreads);
}
