/*
 * q8_oracle.c -- plain, slow, single-threaded fp64 reference for the Q8_0
 * matrix-vector product of the decode-time linear layers.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, calls or
 * includes this file; only the test suite, the package smoke check and the
 * benchmark's CPU-baseline leg load it.  It shares no source with the GPU
 * path (no common headers, helpers, tables or constants).
 *
 * What it computes.  In decode the linear projection and feed-forward layers
 * act on a single token, so each is a matrix-vector product (Sec. 4.3).  The
 * weights are in the 8-bit block format Q8_0: a row of K weights is stored as
 * K / 32 blocks, each holding one IEEE binary16 scale d and 32 signed 8-bit
 * values q_0 .. q_31, with weight j of the block equal to d * q_j (symmetric,
 * no zero point; Sec. 4.3).  Sec. 4.3 and Sec. 7 disagree on whether the scale
 * follows or precedes the 32 values; the reading taken (listed with the other
 * readings in the design notes) is Sec. 7's: each 34-byte block is the scale
 * (2 bytes, little-endian) followed by the 32 values.  Then
 *
 *   y[m] = sum_{b = 0}^{K/32 - 1} sum_{j = 0}^{31} (d_{m,b} * q_{m,b,j}) * x[32 b + j]
 *
 * for m = 0 .. M - 1, with W row-major (row m is blocks m * K/32 .. (m+1) *
 * K/32 - 1).  The activations x are used as given (the paper does not
 * quantize them).  All arithmetic is IEEE double, summed left to right;
 * build without fast-math and with floating-point contraction off.
 *
 * The binary16 scale is decoded from its definition (IEEE 754: sign bit,
 * 5-bit exponent with bias 15, 10-bit fraction; exponent 0 encodes zero and
 * subnormals, exponent 31 infinities and NaNs).
 *
 * Return value: 0 on success, -1 on an invalid argument (null pointer,
 * M < 1, K < 32 or K not a multiple of 32).  Nothing is written on error.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>

double q8_half_to_f64(unsigned bits) {
    const unsigned s = (bits >> 15) & 1u, e = (bits >> 10) & 31u, f = bits & 1023u;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);            /* zero and subnormals: f * 2^-24 */
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024u + f), (int)e - 25);   /* (1 + f/1024) * 2^(e - 15) */
    return s ? -v : v;
}

int q8_0_gemv_f64(const uint8_t *w, const double *x, double *y, int M, int K) {
    if (!w || !x || !y || M < 1 || K < 32 || K % 32 != 0) return -1;
    const int nb = K / 32;
    for (int m = 0; m < M; ++m) {
        double acc = 0.0;
        for (int b = 0; b < nb; ++b) {
            const uint8_t *blk = w + ((size_t)m * nb + b) * 34;
            const double d = q8_half_to_f64((unsigned)blk[0] | ((unsigned)blk[1] << 8));
            for (int j = 0; j < 32; ++j) {
                const double q = (double)(int8_t)blk[2 + j];
                acc += (d * q) * x[(size_t)32 * b + j];
            }
        }
        y[m] = acc;
    }
    return 0;
}
