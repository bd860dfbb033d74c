// Exercises the library's host-side argument checks (validate_core) over a
// grid of sizes, scales, dtypes and pointer patterns, including extreme and
// overflowing values; built with AddressSanitizer and UndefinedBehaviorSanitizer
// by the CPU test suite, which fails on any report.  Pointers are fake
// addresses and are never dereferenced (the checks only compare them).
#include <cmath>
#include <climits>
#include <cstdint>
#include <cstdio>
#include <initializer_list>
#include <limits>

#include "../../paper_2608_18656_amd/csrc/fa_checks.h"

static const void *P(uintptr_t x) { return reinterpret_cast<const void *>(x); }

int main() {
    const int sizes[] = {INT_MIN, -1, 0, 1, 2, 3, 7, 8, 64, 128, 255, 256, 264, 65535, 1 << 20,
                         INT_MAX};
    const float scales[] = {0.f, -0.3f, 0.125f, 1e30f, std::numeric_limits<float>::infinity(),
                            -std::numeric_limits<float>::infinity(), std::nanf("")};
    const uintptr_t bases[] = {0, 1u << 20, (uintptr_t)1 << 44, UINTPTR_MAX - 4095};
    const fa_dtype_t dts[] = {FA_F16, FA_BF16, FA_F32, (fa_dtype_t)7};
    long long n = 0, ok = 0;
    int hist[16] = {0};
    for (int B : sizes)
        for (int Hq : sizes)
            for (int Hkv : {1, 2, 3, 8, -4, INT_MAX})
                for (int Nq : sizes)
                    for (int Nk : {1, 77, 4096, INT_MAX, 0})
                        for (int D : {8, 64, 128, 40, 256, 0, 264}) {
                            const int causal = ((unsigned)Nq + (unsigned)Nk + (unsigned)D) & 1u;
                            const float scale = scales[((unsigned)B ^ (unsigned)Nq ^ (unsigned)D) % 7];
                            const fa_dtype_t in = dts[((unsigned)Hq + (unsigned)Nk) % 4];
                            const fa_dtype_t out = ((B ^ Hkv) & 1) ? FA_F32 : in;
                            const uintptr_t base = bases[((unsigned)Nq ^ (unsigned)Hkv) % 4];
                            const uintptr_t step = (uintptr_t)1 << 40;
                            const uintptr_t mis = ((unsigned)B + (unsigned)Hkv) % 5 == 0 ? 2 : 0;
                            const fa_status_t st = fa::validate_core(
                                P(base), P(base + step), P(base + 2 * step + mis), P(base + 3 * step),
                                reinterpret_cast<const float *>(base + 4 * step), B, Hq, Hkv, Nq,
                                Nk, D, causal, scale, in, out, (((unsigned)B + (unsigned)D) & 3u) == 0 ? -1 : (long long)Nk);
                            ++n;
                            if (st == FA_OK) ++ok;
                            if ((int)st >= 0 && (int)st < 16) ++hist[(int)st];
                        }
    // known answers on the plain case and a few single faults
    const void *q = P(1 << 20), *k = P(9 << 20), *v = P(17 << 20), *o = P(25 << 20);
    const float *lse = reinterpret_cast<const float *>((uintptr_t)33 << 20);
    int bad = 0;
    bad |= fa::validate_core(q, k, v, o, lse, 1, 4, 2, 8, 8, 64, 1, 0.125f, FA_F16, FA_F16, -1) != FA_OK;
    bad |= fa::validate_core(q, k, v, o, lse, 1, 4, 2, 9, 8, 64, 1, 0.125f, FA_F16, FA_F16, -1) != FA_ERR_CAUSAL_SHAPE;
    bad |= fa::validate_core(q, k, v, q, lse, 1, 4, 2, 8, 8, 64, 0, 0.125f, FA_F16, FA_F16, -1) != FA_ERR_ALIAS;
    bad |= fa::validate_core(q, k, v, o, lse, INT_MAX, INT_MAX, 1, INT_MAX, 8, 256, 0, 1.f, FA_F16, FA_F16, -1) != FA_ERR_DIM;
    bad |= !fa::overlaps(P(100), 10, P(105), 1) || fa::overlaps(P(100), 10, P(110), 1);
    long long r = 0;
    bad |= fa::mul_ok(LLONG_MAX / 2, 3, &r) || !fa::mul_ok(1 << 20, 1 << 20, &r) || r != (1LL << 40);
    std::printf("checked %lld argument sets, %lld accepted; status histogram:", n, ok);
    for (int i = 0; i < 16; ++i) std::printf(" %d", hist[i]);
    std::printf("\n");
    return bad;
}
