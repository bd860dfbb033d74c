/*
 * fa_oracle.c -- plain, slow, single-threaded fp64 reference for exact
 * softmax attention with grouped / multi-query key-value heads.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, calls or
 * includes this file; only the test suite, the package smoke check and the
 * benchmark's CPU-baseline leg load it.  It shares no source with the GPU
 * path (no common headers, helpers, tables or constants).
 *
 * What it computes (Sec. 2, the scaled-dot-product attention definition;
 * Sec. 1, "exact self-attention"; Sec. 4.1, the problem statement with Q, K,
 * V of shape N x D per head and N = 1 in decode):
 *
 *   for every batch b, query head h, query row i:
 *     g    = h / (Hq / Hkv)                  query head -> key/value head
 *                                             (Sec. 4.1.1: one K/V row is
 *                                             replicated across the query
 *                                             heads sharing it)
 *     last = causal ? i + (Nk - Nq) : Nk - 1 bottom-right causal alignment
 *                                             (the paper only says "check for
 *                                             causal masking", Alg. 1 and
 *                                             Alg. 2; this reading is listed
 *                                             with the others in the design
 *                                             notes)
 *     s_j  = scale * sum_d q[b,i,h,d] * k[b,j,g,d]           j = 0..last
 *     m    = max_j s_j
 *     w_j  = exp(s_j - m),  l = sum_j w_j                     (two-pass softmax)
 *     o[b,i,h,:] = (sum_j w_j * v[b,j,g,:]) / l
 *     lse[b,h,i] = m + ln(l)              natural-log log-sum-exp of the scores
 *
 * This is the plain definition, not the paper's streaming recurrence: the
 * recurrence (Alg. 1) and its blocked form (Alg. 2) reach the same value up to
 * rounding order, which is what the test suite checks independently.
 *
 * Layouts (row-major, D fastest): q, o [B][Nq][Hq][D]; k, v [B][Nk][Hkv][D];
 * lse [B][Hq][Nq].  All arithmetic is IEEE double, summed left to right; build
 * without fast-math and with floating-point contraction off.
 *
 * Return value: 0 on success, -1 on an invalid argument (null pointer,
 * non-positive size, Hq not a multiple of Hkv, causal with Nq > Nk, or a row
 * index out of range).  Nothing is written on error.
 */
#include <math.h>
#include <stddef.h>
#include <stdlib.h>

static int check_args(const void *q, const void *k, const void *v, int B,
                      int Hq, int Hkv, int Nq, int Nk, int D, int causal) {
    if (!q || !k || !v) return -1;
    if (B < 1 || Hq < 1 || Hkv < 1 || Nq < 1 || Nk < 1 || D < 1) return -1;
    if (Hq % Hkv != 0) return -1;
    if (causal && Nq > Nk) return -1;
    return 0;
}

/* One query row (b, h, i): writes D outputs to out_row, the log-sum-exp to
 * *out_lse, and, when w_row is not NULL, the Nk normalised weights (zero for
 * keys the causal mask hides).  scores is caller scratch of Nk doubles. */
static void one_row(const double *q, const double *k, const double *v,
                    int Hq, int Hkv, int Nq, int Nk, int D, int causal,
                    double scale, int b, int h, int i, double *scores,
                    double *out_row, double *out_lse, double *w_row) {
    const int G = Hq / Hkv;
    const int g = h / G;
    const long last = causal ? (long)i + (long)(Nk - Nq) : (long)Nk - 1;
    const double *qrow = q + (((size_t)b * Nq + i) * Hq + h) * (size_t)D;

    /* scores s_j = scale * <q_i, k_j> over the visible keys */
    for (long j = 0; j <= last; ++j) {
        const double *krow = k + (((size_t)b * Nk + j) * Hkv + g) * (size_t)D;
        double dot = 0.0;
        for (int d = 0; d < D; ++d) dot += qrow[d] * krow[d];
        scores[j] = scale * dot;
    }
    /* pass 1: the maximum */
    double m = -INFINITY;
    for (long j = 0; j <= last; ++j)
        if (scores[j] > m) m = scores[j];
    /* pass 2: unnormalised weights and their sum */
    double l = 0.0;
    for (long j = 0; j <= last; ++j) {
        scores[j] = exp(scores[j] - m);
        l += scores[j];
    }
    /* weighted sum of value rows, then one division per element */
    for (int d = 0; d < D; ++d) out_row[d] = 0.0;
    for (long j = 0; j <= last; ++j) {
        const double *vrow = v + (((size_t)b * Nk + j) * Hkv + g) * (size_t)D;
        const double w = scores[j];
        for (int d = 0; d < D; ++d) out_row[d] += w * vrow[d];
    }
    for (int d = 0; d < D; ++d) out_row[d] /= l;
    *out_lse = m + log(l);
    if (w_row) {
        for (long j = 0; j < Nk; ++j) w_row[j] = (j <= last) ? scores[j] / l : 0.0;
    }
}

/* Full attention over every (b, h, i). */
int fa_oracle_f64(const double *q, const double *k, const double *v, double *o,
                  double *lse, int B, int Hq, int Hkv, int Nq, int Nk, int D,
                  int causal, double scale) {
    if (check_args(q, k, v, B, Hq, Hkv, Nq, Nk, D, causal) || !o) return -1;
    double *scores = (double *)malloc(sizeof(double) * (size_t)Nk);
    if (!scores) return -1;
    for (int b = 0; b < B; ++b)
        for (int i = 0; i < Nq; ++i)
            for (int h = 0; h < Hq; ++h) {
                double l_out;
                one_row(q, k, v, Hq, Hkv, Nq, Nk, D, causal, scale, b, h, i,
                        scores, o + (((size_t)b * Nq + i) * Hq + h) * (size_t)D,
                        &l_out, NULL);
                if (lse) lse[((size_t)b * Hq + h) * Nq + i] = l_out;
            }
    free(scores);
    return 0;
}

/* Selected rows only.  rows holds nrows triples (b, h, i); o_rows is
 * [nrows][D] and lse_rows [nrows].  Used to spread the work over processes and
 * to check sampled outputs of shapes too large for a full pass. */
int fa_oracle_rows_f64(const double *q, const double *k, const double *v,
                       int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal,
                       double scale, const int *rows, int nrows, double *o_rows,
                       double *lse_rows) {
    if (check_args(q, k, v, B, Hq, Hkv, Nq, Nk, D, causal) || !o_rows || !lse_rows ||
        (nrows > 0 && !rows) || nrows < 0)
        return -1;
    for (int r = 0; r < nrows; ++r) {
        const int b = rows[3 * r], h = rows[3 * r + 1], i = rows[3 * r + 2];
        if (b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= Nq) return -1;
    }
    double *scores = (double *)malloc(sizeof(double) * (size_t)Nk);
    if (!scores) return -1;
    for (int r = 0; r < nrows; ++r)
        one_row(q, k, v, Hq, Hkv, Nq, Nk, D, causal, scale, rows[3 * r],
                rows[3 * r + 1], rows[3 * r + 2], scores, o_rows + (size_t)r * D,
                lse_rows + r, NULL);
    free(scores);
    return 0;
}

/* Debug entry for tiny inputs: the normalised attention weights
 * w[b][h][i][j] (softmax row of query i over keys j, zero where masked). */
int fa_oracle_weights_f64(const double *q, const double *k, const double *v,
                          double *w, int B, int Hq, int Hkv, int Nq, int Nk, int D,
                          int causal, double scale) {
    if (check_args(q, k, v, B, Hq, Hkv, Nq, Nk, D, causal) || !w) return -1;
    double *scores = (double *)malloc(sizeof(double) * (size_t)Nk);
    double *orow = (double *)malloc(sizeof(double) * (size_t)D);
    if (!scores || !orow) {
        free(scores);
        free(orow);
        return -1;
    }
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < Hq; ++h)
            for (int i = 0; i < Nq; ++i) {
                double l_out;
                one_row(q, k, v, Hq, Hkv, Nq, Nk, D, causal, scale, b, h, i, scores,
                        orow, &l_out,
                        w + (((size_t)b * Hq + h) * Nq + i) * (size_t)Nk);
            }
    free(scores);
    free(orow);
    return 0;
}
