/* Calls the fp64 oracles (attention, rows, weights, Q8_0 product) on small
 * seeded inputs and edge shapes; built with AddressSanitizer and
 * UndefinedBehaviorSanitizer by the CPU test suite, which fails on any report
 * or on a failed sanity check (finite outputs, weight rows summing to 1,
 * rejected invalid arguments). */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int fa_oracle_f64(const double *q, const double *k, const double *v, double *o, double *lse, int B,
                  int Hq, int Hkv, int Nq, int Nk, int D, int causal, double scale);
int fa_oracle_rows_f64(const double *q, const double *k, const double *v, int B, int Hq, int Hkv,
                       int Nq, int Nk, int D, int causal, double scale, const int *rows, int nrows,
                       double *o_rows, double *lse_rows);
int fa_oracle_weights_f64(const double *q, const double *k, const double *v, double *w, int B,
                          int Hq, int Hkv, int Nq, int Nk, int D, int causal, double scale);
int q8_0_gemv_f64(const uint8_t *w, const double *x, double *y, int M, int K);

static unsigned long long state = 12345;
static double rnd(void) {   /* xorshift64*, uniform in [-1, 1) */
    state ^= state >> 12; state ^= state << 25; state ^= state >> 27;
    return (double)((state * 2685821657736338717ULL) >> 11) / 4503599627370496.0 - 1.0;
}
static double *fill(size_t n) {
    double *p = (double *)malloc(n * sizeof(double));
    for (size_t i = 0; i < n; ++i) p[i] = rnd();
    return p;
}

int main(void) {
    /* B, Hq, Hkv, Nq, Nk, D, causal */
    static const int shapes[][7] = {{1, 1, 1, 1, 1, 1, 0}, {1, 2, 1, 1, 1, 8, 1}, {2, 4, 2, 5, 9, 3, 1},
                                    {1, 6, 3, 7, 7, 16, 1}, {3, 8, 1, 4, 33, 5, 0}, {1, 3, 3, 1, 50, 2, 1}};
    int bad = 0;
    for (size_t s = 0; s < sizeof(shapes) / sizeof(shapes[0]); ++s) {
        const int B = shapes[s][0], Hq = shapes[s][1], Hkv = shapes[s][2], Nq = shapes[s][3];
        const int Nk = shapes[s][4], D = shapes[s][5], causal = shapes[s][6];
        const size_t nq = (size_t)B * Nq * Hq * D, nk = (size_t)B * Nk * Hkv * D;
        double *q = fill(nq), *k = fill(nk), *v = fill(nk);
        double *o = fill(nq), *lse = fill((size_t)B * Hq * Nq);
        double *w = fill((size_t)B * Hq * Nq * Nk);
        bad |= fa_oracle_f64(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, 0.7) != 0;
        bad |= fa_oracle_weights_f64(q, k, v, w, B, Hq, Hkv, Nq, Nk, D, causal, 0.7) != 0;
        for (size_t i = 0; i < nq; ++i) bad |= !isfinite(o[i]);
        for (size_t r = 0; r < (size_t)B * Hq * Nq; ++r) {
            double sum = 0.0;
            for (int j = 0; j < Nk; ++j) sum += w[r * Nk + j];
            bad |= fabs(sum - 1.0) > 1e-12;
        }
        int rows[6] = {B - 1, Hq - 1, Nq - 1, 0, 0, 0};
        double orow[2 * 16], lrow[2];
        bad |= fa_oracle_rows_f64(q, k, v, B, Hq, Hkv, Nq, Nk, D, causal, 0.7, rows, 2, orow, lrow) != 0;
        bad |= fa_oracle_rows_f64(q, k, v, B, Hq, Hkv, Nq, Nk, D, causal, 0.7, rows, -1, orow, lrow) != -1;
        rows[0] = B;   /* out of range row: rejected, nothing written */
        bad |= fa_oracle_rows_f64(q, k, v, B, Hq, Hkv, Nq, Nk, D, causal, 0.7, rows, 2, orow, lrow) != -1;
        free(q); free(k); free(v); free(o); free(lse); free(w);
    }
    /* invalid arguments are rejected */
    double x[8] = {0};
    bad |= fa_oracle_f64(NULL, x, x, x, x, 1, 1, 1, 1, 1, 1, 0, 1.0) != -1;
    bad |= fa_oracle_f64(x, x, x, x, x, 1, 3, 2, 1, 1, 1, 0, 1.0) != -1;
    bad |= fa_oracle_f64(x, x, x, x, x, 1, 1, 1, 2, 1, 1, 1, 1.0) != -1;
    /* Q8_0 product: random blocks, including non-finite and subnormal scales */
    const int M = 5, K = 96, nb = K / 32;
    uint8_t *wq = (uint8_t *)malloc((size_t)M * nb * 34);
    for (int i = 0; i < M * nb * 34; ++i) wq[i] = (uint8_t)(rnd() * 127.0 + 128.0);
    wq[0] = 0x00; wq[1] = 0x7c;   /* +inf scale */
    wq[34] = 0x01; wq[35] = 0x00; /* smallest subnormal scale */
    double *xq = fill(K), y[5];
    bad |= q8_0_gemv_f64(wq, xq, y, M, K) != 0;
    for (int m = 1; m < M; ++m) bad |= !isfinite(y[m]);
    bad |= q8_0_gemv_f64(wq, xq, y, M, 33) != -1;
    free(wq); free(xq);
    printf("oracle sanitizer run: %s\n", bad ? "FAILED" : "ok");
    return bad;
}
