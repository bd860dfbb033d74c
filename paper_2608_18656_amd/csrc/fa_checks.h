// fa_checks.h -- the host-side argument checks of the attention entry points
// (plain C++, no HIP: the library includes it, and a sanitizer build of the
// test suite compiles it with g++ alone).
#pragma once

#include <cmath>
#include <cstddef>
#include <cstdint>

#include "../../include/fa.h"

namespace fa {

inline size_t esize(fa_dtype_t t) { return t == FA_F32 ? 4 : 2; }

// Whether the byte ranges [a, a + na) and [b, b + nb) intersect.
inline bool overlaps(const void *a, size_t na, const void *b, size_t nb) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + nb && y < x + na;
}

// r = a * b for positive a, b, refused (false) when the product would exceed
// INT64_MAX / 4 (element counts that later get multiplied by element sizes).
inline bool mul_ok(long long a, long long b, long long *r) {
    if (a > 0 && b > 0 && a > (long long)(INT64_MAX / 4) / b) return false;
    *r = a * b;
    return true;
}

// The argument checks of every attention entry point.  kv_rows: rows of
// Hkv * D elements that k and v each hold (-1: B * Nk, the contiguous layout).
inline fa_status_t validate_core(const void *q, const void *k, const void *v, const void *o,
                                 const float *lse, int B, int Hq, int Hkv, int Nq, int Nk, int D,
                                 int causal, float scale, fa_dtype_t in, fa_dtype_t out,
                                 long long kv_rows) {
    if (!q || !k || !v || !o) return FA_ERR_NULL;
    if (B < 1 || Hq < 1 || Hkv < 1 || Nq < 1 || Nk < 1 || D < 1) return FA_ERR_DIM;
    if (in != FA_F16 && in != FA_BF16 && in != FA_F32) return FA_ERR_DTYPE;
    if (out != in && out != FA_F32) return FA_ERR_DTYPE;
    if (Hq % Hkv != 0) return FA_ERR_GQA_RATIO;
    if (D % 8 != 0 || D > 256) return FA_ERR_HEAD_DIM;
    if (causal && Nq > Nk) return FA_ERR_CAUSAL_SHAPE;
    if (!std::isfinite(scale)) return FA_ERR_SCALE;
    long long nq, nk, t;
    if (kv_rows < 0) kv_rows = (long long)B * Nk;
    if (!mul_ok((long long)B * Nq, (long long)Hq * D, &nq) ||
        !mul_ok(kv_rows, (long long)Hkv * D, &nk) ||
        !mul_ok((long long)B * Hq, (long long)Nq, &t))
        return FA_ERR_DIM;
    const uintptr_t a16 = 15;
    if ((reinterpret_cast<uintptr_t>(q) & a16) || (reinterpret_cast<uintptr_t>(k) & a16) ||
        (reinterpret_cast<uintptr_t>(v) & a16) || (reinterpret_cast<uintptr_t>(o) & a16) ||
        (reinterpret_cast<uintptr_t>(lse) & 3))
        return FA_ERR_ALIGN;
    const size_t qb = (size_t)nq * esize(in), kb = (size_t)nk * esize(in);
    const size_t ob = (size_t)nq * esize(out), lb = (size_t)t * sizeof(float);
    if (overlaps(o, ob, q, qb) || overlaps(o, ob, k, kb) || overlaps(o, ob, v, kb))
        return FA_ERR_ALIAS;
    if (lse && (overlaps(lse, lb, q, qb) || overlaps(lse, lb, k, kb) ||
                overlaps(lse, lb, v, kb) || overlaps(lse, lb, o, ob)))
        return FA_ERR_ALIAS;
    return FA_OK;
}

}  // namespace fa
