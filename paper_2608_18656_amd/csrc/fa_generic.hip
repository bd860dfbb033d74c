// fa_generic.hip -- vector-ALU attention forward for the cases the matrix-core
// kernels do not take: fp32 inputs, and fp16 / bf16 with a head dimension
// other than 64 or 128 (any D with D % 8 == 0 and D <= 256).
//
// All arithmetic is fp32.  A workgroup of 256 threads owns 256 / TPR query
// rows of one query head; TPR consecutive threads share a row and each holds
// an interleaved 1 / TPR of its D columns (pairs d = 2 TPR i + 2 t + {0, 1}).
// TPR is 4 (64 rows per workgroup), or 16 (16 rows) when a grid of 64-row
// workgroups would leave most CUs idle.  Keys
// are streamed in LDS tiles (the next tile's loads in flight during the
// current one); per tile the scores of all tile keys are formed
// (partial dot products reduced over the four threads of the row), then the
// running maximum / sum / accumulator are updated once for the tile -- the
// blocked form (Alg. 2) of the streaming recurrence of Alg. 1 -- and the
// accumulator is normalised after the last visible tile.
#include "fa_common.h"
#include "fa_internal.h"

namespace fa {
namespace {

struct GenericArgs {
    const void *q, *k, *v;
    void *o;
    float *lse;
    int B, Hq, Hkv, Nq, Nk, D;
    float c;   // scale * log2(e), signed
    int nmb;   // row blocks (of 256 / TPR rows)
    const int *seqlens;   // valid keys per batch element (NULL: Nk for all)
};

template <typename T> struct Scalar { typedef T type; };
template <> struct Scalar<f16_t> { typedef _Float16 type; };
template <> struct Scalar<bf16_t> { typedef __bf16 type; };

template <typename TIN, typename TOUT, int DMAX, bool CAUSAL, int TPR>
__global__ __launch_bounds__(256) void generic_kernel(GenericArgs a) {
    typedef typename Scalar<TIN>::type S;
    constexpr int KT = 16;                       // keys per LDS tile
    constexpr int RW = 256 / TPR;                // query rows per workgroup
    constexpr int NP = DMAX / (2 * TPR);         // column pairs per thread
    static_assert(NP >= 1, "at least one column pair per thread");
    __shared__ __attribute__((aligned(16))) float ks[KT * DMAX];
    __shared__ __attribute__((aligned(16))) float vs[KT * DMAX];

    const int tid = threadIdx.x, row = tid / TPR, part = tid % TPR;
    int bid = blockIdx.x;
    const int mb = a.nmb - 1 - bid % a.nmb;
    bid /= a.nmb;
    const int h = bid % a.Hq;
    const int b = bid / a.Hq;
    const int G = a.Hq / a.Hkv, g = h / G;
    const int D = a.D, Nq = a.Nq;
    // valid keys of this batch element (a.Nk rows per element in K and V)
    const int Nk = a.seqlens ? min(max(a.seqlens[b], 0), a.Nk) : a.Nk;
    const int qi = mb * RW + row;
    const int off = Nk - Nq;
    const int last_blk = min(mb * RW + RW, Nq) - 1;
    const int kend = CAUSAL ? min(Nk, last_blk + off + 1) : Nk;
    const int myend = CAUSAL ? min(Nk, qi + off + 1) : Nk;

    float q0[NP], q1[NP], o0[NP], o1[NP];
    const S *qp = reinterpret_cast<const S *>(a.q) + ((size_t)((size_t)b * Nq + qi) * a.Hq + h) * D;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
        const int d = 2 * TPR * i + 2 * part;
        q0[i] = (qi < Nq && d < D) ? to_f32(qp[d]) : 0.f;
        q1[i] = (qi < Nq && d < D) ? to_f32(qp[d + 1]) : 0.f;
        o0[i] = 0.f;
        o1[i] = 0.f;
    }
    float m = -INFINITY, lsum = 0.f;
    const S *kb_ = reinterpret_cast<const S *>(a.k);
    const S *vb_ = reinterpret_cast<const S *>(a.v);

    // Tile staging: each thread moves CH chunks of 4 consecutive columns of
    // K and of V (chunk e = tid + 256 c: key e / (DMAX / 4), columns
    // 4 (e % (DMAX / 4)) ..), converted to fp32; columns d >= D and keys past
    // the end are zero-filled so the inner loops need no guard.  The next
    // tile's loads are in flight while the current one is used.
    constexpr int CPR4 = DMAX / 4;
    constexpr int CH = (KT * CPR4 + 255) / 256;
    float4_t kr[CH], vr[CH];
    auto load4 = [&](const S *p) {
        if constexpr (sizeof(S) == 4) {
            return *reinterpret_cast<const float4_t *>(p);
        } else {
            typedef S s4 __attribute__((ext_vector_type(4)));
            const s4 u = *reinterpret_cast<const s4 *>(p);
            return float4_t{to_f32(u[0]), to_f32(u[1]), to_f32(u[2]), to_f32(u[3])};
        }
    };
    auto load_tile = [&](int kb) {
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int e = tid + 256 * c, kk = e / CPR4, d = 4 * (e % CPR4), key = kb + kk;
            kr[c] = float4_t{};
            vr[c] = float4_t{};
            if (kk < KT && key < Nk && d < D) {
                const size_t o = ((size_t)((size_t)b * a.Nk + key) * a.Hkv + g) * D + d;
                kr[c] = load4(kb_ + o);
                vr[c] = load4(vb_ + o);
            }
        }
    };
    if (kend > 0) load_tile(0);

    for (int kb = 0; kb < kend; kb += KT) {
        __syncthreads();
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int e = tid + 256 * c, kk = e / CPR4, d = 4 * (e % CPR4);
            if (kk < KT) {
                *reinterpret_cast<float4_t *>(&ks[kk * DMAX + d]) = kr[c];
                *reinterpret_cast<float4_t *>(&vs[kk * DMAX + d]) = vr[c];
            }
        }
        __syncthreads();
        if (kb + KT < kend) load_tile(kb + KT);
        float x[KT];
        float tmax = -INFINITY;
#pragma unroll
        for (int j = 0; j < KT; ++j) {
            float acc = 0.f;
#pragma unroll
            for (int i = 0; i < NP; ++i) {
                const int d = 2 * TPR * i + 2 * part;
                acc += q0[i] * ks[j * DMAX + d] + q1[i] * ks[j * DMAX + d + 1];
            }
#pragma unroll
            for (int off = 1; off < TPR; off <<= 1) acc += __shfl_xor(acc, off);
            const bool vis = kb + j < myend;
            x[j] = vis ? acc * a.c : -INFINITY;
            tmax = __builtin_fmaxf(tmax, x[j]);
        }
        const float m_new = __builtin_fmaxf(m, tmax);
        if (m_new == -INFINITY) continue;   // nothing visible yet for this row
        const float alpha = (m == -INFINITY) ? 0.f : exp2_fast(m - m_new);
        m = m_new;
        lsum *= alpha;
#pragma unroll
        for (int i = 0; i < NP; ++i) {
            o0[i] *= alpha;
            o1[i] *= alpha;
        }
#pragma unroll
        for (int j = 0; j < KT; ++j) {
            const float p = (x[j] == -INFINITY) ? 0.f : exp2_fast(x[j] - m);
            lsum += p;
#pragma unroll
            for (int i = 0; i < NP; ++i) {
                const int d = 2 * TPR * i + 2 * part;
                o0[i] += p * vs[j * DMAX + d];
                o1[i] += p * vs[j * DMAX + d + 1];
            }
        }
    }
    if (qi >= Nq) return;
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;   // no visible key: 0
    TOUT *op = reinterpret_cast<TOUT *>(a.o) + ((size_t)((size_t)b * Nq + qi) * a.Hq + h) * D;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
        const int d = 2 * TPR * i + 2 * part;
        if (d < D) {
            op[d] = from_f32<TOUT>(o0[i] * inv);
            op[d + 1] = from_f32<TOUT>(o1[i] * inv);
        }
    }
    if (a.lse && part == 0)
        a.lse[((size_t)b * a.Hq + h) * Nq + qi] = lsum > 0.f ? (m + log2f(lsum)) * kLn2 : -INFINITY;
}

template <typename TIN, typename TOUT, int DMAX>
hipError_t launch_t(const Problem &p, hipStream_t stream) {
    GenericArgs a;
    a.q = p.q; a.k = p.k; a.v = p.v; a.o = p.o; a.lse = p.lse;
    a.B = p.B; a.Hq = p.Hq; a.Hkv = p.Hkv; a.Nq = p.Nq; a.Nk = p.Nk; a.D = p.D;
    a.seqlens = p.seqlens;
    a.c = p.scale * kLog2e;
    // 16 threads per row (16-row workgroups) when 64-row workgroups would not
    // give every CU of the GPU one
    const bool narrow = (long long)((p.Nq + 63) / 64) * p.B * p.Hq < 256;
    const int RW = narrow ? 16 : 64;
    a.nmb = (p.Nq + RW - 1) / RW;
    const long long nblocks = (long long)a.nmb * p.B * p.Hq;
    if (nblocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)nblocks), block(256);
    if (narrow) {
        if (p.causal)
            hipLaunchKernelGGL((generic_kernel<TIN, TOUT, DMAX, true, 16>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((generic_kernel<TIN, TOUT, DMAX, false, 16>), grid, block, 0, stream, a);
    } else {
        if (p.causal)
            hipLaunchKernelGGL((generic_kernel<TIN, TOUT, DMAX, true, 4>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((generic_kernel<TIN, TOUT, DMAX, false, 4>), grid, block, 0, stream, a);
    }
    return hipGetLastError();
}

template <typename TIN, typename TOUT>
hipError_t launch_d(const Problem &p, hipStream_t s) {
    if (p.D <= 64) return launch_t<TIN, TOUT, 64>(p, s);
    if (p.D <= 128) return launch_t<TIN, TOUT, 128>(p, s);
    return launch_t<TIN, TOUT, 256>(p, s);
}

}  // namespace

hipError_t launch_generic(const Problem &p, hipStream_t stream) {
    switch (p.in) {
    case FA_F32:
        return launch_d<float, float>(p, stream);
    case FA_F16:
        return p.out == FA_F32 ? launch_d<f16_t, float>(p, stream)
                               : launch_d<f16_t, _Float16>(p, stream);
    default:
        return p.out == FA_F32 ? launch_d<bf16_t, float>(p, stream)
                               : launch_d<bf16_t, __bf16>(p, stream);
    }
}

}  // namespace fa
