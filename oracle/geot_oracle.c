/*
 * CPU oracle for sorted segment reduction and its fused gather-weight form.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the reference the GPU library is
 * checked against. Only the test suite, the smoke check and the bench's CPU
 * baseline load it; the GPU library never includes, links or calls it, and it
 * includes nothing from the GPU library.
 *
 * What it computes is the plain definition of segment reduction (GeoT paper,
 * Section II-B, "Segment Reduction"): Idx is a non-decreasing 1-D array of
 * length M, X is an M x N matrix (N = F features), and output row s of the
 * |V| x N result Y reduces the rows i of X with Idx[i] == s. The aggregate
 * step of message passing (Eq. 2) is the sum case; the reduction may also be
 * mean or max (Fig. "scatter" caption; Section VI, diverse reduction types).
 * The fused form (Section IV and Listing "GeoT solution for fusion"; the
 * weighted variant used as SpMM in Section V-D) reduces the messages
 * w[e] * x[col[e], :] by the sorted destination row of each edge.
 *
 * Readings where the paper is silent (all stated, none derived from a GPU):
 *  - empty segments produce 0.0f for sum, mean and max;
 *  - sum and mean accumulate in fp64 and round once to fp32 at the end;
 *    mean divides the fp64 sum by the row (edge) count in fp64;
 *  - max is the IEEE 754-2019 maximum operation folded over the members, in fp32
 *    (a NaN member makes the result NaN; +0 ranks above -0); a max never rounds,
 *    so it is exact. The paper does not say what max does with NaN or signed
 *    zeros; this operation is order-independent, so every reduction order the
 *    GPU may take has the same answer;
 *  - a weighted term is one fp32 multiply w[e] * x (round to nearest even);
 *    without weights the term is x itself;
 *  - the output is overwritten in full (not accumulated into).
 *
 * Gradients (Section VI names training support as future work; these are the
 * derivatives of the definition above, written out):
 *  - segment reduction w.r.t. src: sum copies grad_out[idx[i]] to row i; mean
 *    divides it by the segment length (fp64 division, rounded once); max
 *    routes grad_out[s, f] to the first row of segment s (lowest index) whose
 *    src[i, f] equals out[s, f] (compared with ==, so either zero matches a zero
 *    maximum and a NaN maximum routes nothing), every other row gets 0;
 *  - fused form w.r.t. X: grad_X[c] = sum over edges e with col[e] == c of
 *    coef(e) * grad_out[row[e]] with coef = w[e] (1 without weights), divided
 *    by the row's edge count for mean; for max only the first edge of each
 *    (row, feature) whose rounded product equals out[row, f] contributes;
 *  - fused form w.r.t. the weights: grad_w[e] = sum over f of
 *    grad_out[row[e], f] * X[col[e], f] (divided by the count for mean;
 *    restricted to the features where e is that first edge for max).
 *  Both accumulate in fp64 and return fp64.
 *
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off -shared -fPIC.
 * Error codes: 0 ok, 1 invalid argument, 2 index not sorted, 3 index (or
 * column) out of range.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_OK = 0, OR_INVALID = 1, OR_NOT_SORTED = 2, OR_OUT_OF_RANGE = 3 };
enum { OR_SUM = 0, OR_MEAN = 1, OR_MAX = 2 };

/* Check the preconditions of the definition: Idx non-decreasing, 0 <= Idx < S. */
int oracle_check_index(const int64_t *idx, int64_t nnz, int64_t S)
{
    if (nnz < 0 || S < 0) return OR_INVALID;
    for (int64_t i = 0; i < nnz; ++i) {
        if (idx[i] < 0 || idx[i] >= S) return OR_OUT_OF_RANGE;
        if (i > 0 && idx[i] < idx[i - 1]) return OR_NOT_SORTED;
    }
    return OR_OK;
}

/* start[s] = first row i with idx[i] >= s, for s = 0..S (start[S] = nnz).
 * Rows of segment s are start[s] .. start[s+1]-1. Computed by one linear walk. */
static void segment_starts(const int64_t *idx, int64_t nnz, int64_t S, int64_t *start)
{
    int64_t i = 0;
    for (int64_t s = 0; s <= S; ++s) {
        while (i < nnz && idx[i] < s) ++i;
        start[s] = i;
    }
}

/* The term a segment reduces for (row or edge) e and feature f. */
static float term(const float *rows, int64_t F, const int64_t *col, const float *w,
                  int64_t e, int64_t f)
{
    if (col == NULL) return rows[e * F + f];
    float x = rows[col[e] * F + f];
    if (w == NULL) return x;
    float t = w[e] * x; /* one fp32 multiply */
    return t;
}

/* IEEE 754-2019 maximum(a, b): NaN when either operand is NaN, otherwise the
 * larger value, with +0 taken as larger than -0. */
static float maximum(float a, float b)
{
    if (isnan(a)) return a;
    if (isnan(b)) return b;
    if (a == b) return signbit(a) ? b : a; /* equal: the same value, or zeros of either sign */
    return a > b ? a : b;
}

/* Shared body of both operations: for each segment s and feature f reduce the
 * terms of rows start[s]..start[s+1]-1 with op. */
static void reduce_segments(const float *rows, int64_t F, const int64_t *col, const float *w,
                            const int64_t *start, int64_t S, int op, float *out)
{
    for (int64_t s = 0; s < S; ++s) {
        int64_t b = start[s], e = start[s + 1];
        int64_t count = e - b;
        for (int64_t f = 0; f < F; ++f) {
            float result;
            if (count == 0) {
                result = 0.0f; /* empty segment */
            } else if (op == OR_MAX) {
                float m = term(rows, F, col, w, b, f);
                for (int64_t i = b + 1; i < e; ++i) {
                    float t = term(rows, F, col, w, i, f);
                    m = maximum(m, t);
                }
                result = m;
            } else {
                double acc = 0.0;
                for (int64_t i = b; i < e; ++i) acc += (double)term(rows, F, col, w, i, f);
                if (op == OR_MEAN) acc = acc / (double)count;
                result = (float)acc;
            }
            out[s * F + f] = result;
        }
    }
}

/* out[s, :] = op over { src[i, :] : idx[i] == s }, s in [0, S). */
int oracle_segment_reduce(const float *src, const int64_t *idx, int64_t nnz, int64_t S,
                          int64_t F, int op, float *out)
{
    if (nnz < 0 || S < 0 || F < 0 || op < OR_SUM || op > OR_MAX) return OR_INVALID;
    if (S == 0 || F == 0) return OR_OK;
    int rc = oracle_check_index(idx, nnz, S);
    if (rc != OR_OK) return rc;
    int64_t *start = (int64_t *)malloc((size_t)(S + 1) * sizeof(int64_t));
    if (!start) return OR_INVALID;
    segment_starts(idx, nnz, S, start);
    reduce_segments(src, F, NULL, NULL, start, S, op, out);
    free(start);
    return OR_OK;
}

/* out[r, :] = op over { w[e] * X[col[e], :] : row[e] == r }, r in [0, R);
 * w == NULL means every weight is 1 (the term is X[col[e], :] itself). */
int oracle_gather_scatter(const float *X, int64_t n_x, const int64_t *col, const float *w,
                          const int64_t *row, int64_t nnz, int64_t R, int64_t F, int op,
                          float *out)
{
    if (nnz < 0 || R < 0 || F < 0 || n_x < 0 || op < OR_SUM || op > OR_MAX) return OR_INVALID;
    if (R == 0 || F == 0) return OR_OK;
    int rc = oracle_check_index(row, nnz, R);
    if (rc != OR_OK) return rc;
    for (int64_t e = 0; e < nnz; ++e)
        if (col[e] < 0 || col[e] >= n_x) return OR_OUT_OF_RANGE;
    int64_t *start = (int64_t *)malloc((size_t)(R + 1) * sizeof(int64_t));
    if (!start) return OR_INVALID;
    segment_starts(row, nnz, R, start);
    reduce_segments(X, F, col, w, start, R, op, out);
    free(start);
    return OR_OK;
}

/* Per output element, the sum of |term| that the element reduces, in fp64
 * (for mean, each term is divided by the count). Used to state the
 * floating-point tolerance of sum and mean; col == NULL selects plain rows. */
int oracle_abs_term_sum(const float *rows, int64_t n_x, const int64_t *col, const float *w,
                        const int64_t *idx, int64_t nnz, int64_t S, int64_t F, int op,
                        double *out)
{
    if (nnz < 0 || S < 0 || F < 0) return OR_INVALID;
    if (S == 0 || F == 0) return OR_OK;
    int rc = oracle_check_index(idx, nnz, S);
    if (rc != OR_OK) return rc;
    if (col)
        for (int64_t e = 0; e < nnz; ++e)
            if (col[e] < 0 || col[e] >= n_x) return OR_OUT_OF_RANGE;
    int64_t *start = (int64_t *)malloc((size_t)(S + 1) * sizeof(int64_t));
    if (!start) return OR_INVALID;
    segment_starts(idx, nnz, S, start);
    for (int64_t s = 0; s < S; ++s) {
        int64_t b = start[s], e = start[s + 1];
        for (int64_t f = 0; f < F; ++f) {
            double acc = 0.0;
            for (int64_t i = b; i < e; ++i) acc += fabs((double)term(rows, F, col, w, i, f));
            if (op == OR_MEAN && e > b) acc /= (double)(e - b);
            out[s * F + f] = acc;
        }
    }
    free(start);
    return OR_OK;
}

/* Segment-length statistics of a sorted index over S segments:
 * mean = nnz / S, var = (1/S) * sum_s (len_s - mean)^2 (population variance),
 * the longest segment, the number of empty segments and sum_s len_s^2. */
int oracle_index_stats(const int64_t *idx, int64_t nnz, int64_t S, double *mean, double *var,
                       int64_t *max_len, int64_t *num_empty, int64_t *sum_len_sq)
{
    if (nnz < 0 || S <= 0) return OR_INVALID;
    int rc = oracle_check_index(idx, nnz, S);
    if (rc != OR_OK) return rc;
    int64_t *start = (int64_t *)malloc((size_t)(S + 1) * sizeof(int64_t));
    if (!start) return OR_INVALID;
    segment_starts(idx, nnz, S, start);
    double m = (double)nnz / (double)S, v = 0.0;
    int64_t mx = 0, ne = 0, sq = 0;
    for (int64_t s = 0; s < S; ++s) {
        int64_t len = start[s + 1] - start[s];
        double d = (double)len - m;
        v += d * d;
        if (len > mx) mx = len;
        if (len == 0) ++ne;
        sq += len * len;
    }
    *mean = m;
    *var = v / (double)S;
    *max_len = mx;
    *num_empty = ne;
    *sum_len_sq = sq;
    free(start);
    return OR_OK;
}

/* Gradient of segment reduction w.r.t. src (see the header). src and out are
 * read for max only. */
int oracle_segment_reduce_backward(const float *grad_out, const int64_t *idx, int64_t nnz,
                                   int64_t S, int64_t F, int op, const float *src,
                                   const float *out, float *grad_src)
{
    if (nnz < 0 || S < 0 || F < 0 || op < OR_SUM || op > OR_MAX) return OR_INVALID;
    if (nnz == 0 || F == 0) return OR_OK;
    int rc = oracle_check_index(idx, nnz, S);
    if (rc != OR_OK) return rc;
    int64_t *start = (int64_t *)malloc((size_t)(S + 1) * sizeof(int64_t));
    if (!start) return OR_INVALID;
    segment_starts(idx, nnz, S, start);
    for (int64_t s = 0; s < S; ++s) {
        int64_t b = start[s], e = start[s + 1];
        for (int64_t f = 0; f < F; ++f) {
            double g = (double)grad_out[s * F + f];
            int found = 0;
            for (int64_t i = b; i < e; ++i) {
                float r;
                if (op == OR_SUM) {
                    r = (float)g;
                } else if (op == OR_MEAN) {
                    r = (float)(g / (double)(e - b));
                } else if (!found && src[i * F + f] == out[s * F + f]) {
                    r = (float)g;
                    found = 1;
                } else {
                    r = 0.0f;
                }
                grad_src[i * F + f] = r;
            }
        }
    }
    free(start);
    return OR_OK;
}

/* Gradients of the fused form w.r.t. X (grad_X, [n_x x F]) and the weights
 * (grad_w, [nnz]); either may be NULL. With absolute != 0 every term is
 * replaced by its absolute value (the sums of |terms| that state the
 * floating-point bound). out is read for max only. */
int oracle_gather_scatter_backward(const float *X, int64_t n_x, const int64_t *col, const float *w,
                                   const int64_t *row, int64_t nnz, int64_t R, int64_t F, int op,
                                   const float *grad_out, const float *out, int absolute,
                                   double *grad_X, double *grad_w)
{
    if (nnz < 0 || R < 0 || F < 0 || n_x < 0 || op < OR_SUM || op > OR_MAX) return OR_INVALID;
    if (grad_X)
        for (int64_t i = 0; i < n_x * F; ++i) grad_X[i] = 0.0;
    if (grad_w)
        for (int64_t e = 0; e < nnz; ++e) grad_w[e] = 0.0;
    if (nnz == 0 || F == 0) return OR_OK;
    int rc = oracle_check_index(row, nnz, R);
    if (rc != OR_OK) return rc;
    for (int64_t e = 0; e < nnz; ++e)
        if (col[e] < 0 || col[e] >= n_x) return OR_OUT_OF_RANGE;
    int64_t *start = (int64_t *)malloc((size_t)(R + 1) * sizeof(int64_t));
    if (!start) return OR_INVALID;
    segment_starts(row, nnz, R, start);
    for (int64_t r = 0; r < R; ++r) {
        int64_t b = start[r], e_end = start[r + 1];
        double cnt = (double)(e_end - b);
        for (int64_t f = 0; f < F; ++f) {
            double g = (double)grad_out[r * F + f];
            int found = 0;
            for (int64_t e = b; e < e_end; ++e) {
                double x = (double)X[col[e] * F + f];
                double coef = w ? (double)w[e] : 1.0;
                int use = 1;
                if (op == OR_MAX) {
                    use = !found && term(X, F, col, w, e, f) == out[r * F + f];
                    if (use) found = 1;
                }
                if (!use) continue;
                double tx = coef * g, tw = g * x;
                if (op == OR_MEAN) {
                    tx /= cnt;
                    tw /= cnt;
                }
                if (absolute) {
                    tx = fabs(tx);
                    tw = fabs(tw);
                }
                if (grad_X) grad_X[col[e] * F + f] += tx;
                if (grad_w) grad_w[e] += tw;
            }
        }
    }
    free(start);
    return OR_OK;
}
