// fa_prefill.hip -- prefill attention forward on gfx950 matrix cores.
//
// One workgroup = 4 waves.  Each wave owns 32 query rows of one query head
// and walks the key sequence in tiles of 64 keys, carrying the running row
// maximum, running row sum and the unnormalised output accumulator from tile
// to tile (the blocked streaming softmax of Alg. 2, built on the per-key
// recurrence of Alg. 1), and normalises once after its last visible tile.
//
// Head packing (the GPU form of the inter-head packing of Sec. 4.1.1 and the
// GQA reuse of Sec. 4.1.2 (iv)): when the group size G = Hq/Hkv allows, the
// four waves of a workgroup take four query heads of the same key/value group
// at the same query rows, so each K/V tile staged in LDS serves four heads and
// all four waves have the same causal extent.  Otherwise (G = 1 or odd) the
// waves take consecutive row blocks of one head.
//
// Per tile and wave:
//   S^T = K_tile Q^T        32x32x16 MFMA, A = K rows from LDS, B = Q rows
//                           kept in registers for the whole kernel
//   softmax update          scores stay in the MFMA result registers: lane l
//                           owns query row l%32, so the row max needs one
//                           exchange with lane l^32; exp2 with the scale and
//                           log2(e) folded into one multiply-add
//   O^T += V_tile^T P^T     32x32x16 fp16 MFMA; P comes straight from the
//                           score registers (no cross-lane move); V^T operands
//                           come from LDS with transpose reads
// The running maximum used as the exponent base is only raised when a row's
// maximum grows by more than 2^8 (log2 domain), so the accumulator rescale is
// skipped on most tiles; the result is unchanged because the sum and the
// accumulator always share the same base.
#include "fa_common.h"
#include "fa_internal.h"

namespace fa {
namespace {

constexpr int BC = 64;        // keys per tile
constexpr int WR = 32;        // query rows per wave
constexpr int NW = 4;         // waves per workgroup
constexpr float TAU = 8.0f;   // lazy-rescale threshold (log2 units)

struct PrefillArgs {
    const void *q, *k, *v;
    void *o;
    float *lse;
    int B, Hq, Hkv, Nq, Nk;
    float c;      // |scale| * log2(e)
    float scale_zero;  // 1 when scale == 0 (all visible weights equal)
    unsigned qsign;    // 0x80008000 to negate q (scale < 0), else 0
    int HW;       // query heads per workgroup (1, 2 or 4)
    int nmb;      // row blocks of 32 * (4 / HW) rows
    int nhg;      // head groups per key/value head (G / HW)
};

template <int D> struct Smem {
    static constexpr int KS = D + 8;    // K row stride in 16-bit elements
    static constexpr int VS = D + 16;   // V row stride in 16-bit elements
    static constexpr int KSZ = BC * KS;
    static constexpr int VSZ = BC * VS;
    static constexpr int STAGE = KSZ + VSZ;
};

template <typename TIN, typename TOUT, int D, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void prefill_kernel(PrefillArgs a) {
    using S = typename TIN::scalar;
    using V8 = typename TIN::vec8;
    using SM = Smem<D>;
    constexpr int KSTEPS = D / 16;          // QK^T contraction steps
    constexpr int DT = D / 32;              // output column tiles
    constexpr int LOADS = D / 32;           // 16-byte chunks per thread per K (or V) tile
    constexpr int CPR = D / 8;              // 16-byte chunks per row
    constexpr bool IN_BF16 = __is_same(TIN, bf16_t);

    __shared__ __attribute__((aligned(16))) unsigned short smem[2 * SM::STAGE];

    const int tid = threadIdx.x;
    const int w = tid >> 6, l = tid & 63, lq = l & 31, lh = l >> 5;
    const int RB = NW / a.HW;
    const int per_mb = a.B * a.Hkv * a.nhg;
    const int bid = blockIdx.x;
    const int mb = a.nmb - 1 - bid / per_mb;    // latest rows (most keys) first
    int rest = bid % per_mb;
    const int hg = rest % a.nhg;
    rest /= a.nhg;
    const int g = rest % a.Hkv;
    const int b = rest / a.Hkv;
    const int G = a.Hq / a.Hkv;
    const int hs = w % a.HW, rs = w / a.HW;
    const int h = g * G + hg * a.HW + hs;
    const int row0_wg = mb * (WR * RB);
    const int row0 = row0_wg + rs * WR;
    const int qi = row0 + lq;
    const int off = a.Nk - a.Nq;
    const int Nq = a.Nq, Nk = a.Nk;

    // Key extent of the workgroup and of this wave.
    const int last_wg = min(row0_wg + WR * RB, Nq) - 1;
    const int kend_wg = CAUSAL ? min(Nk, last_wg + off + 1) : Nk;
    const bool wave_live = row0 < Nq;
    const int kend_w = !wave_live ? 0 : (CAUSAL ? min(Nk, min(row0 + WR, Nq) - 1 + off + 1) : Nk);
    const int kfree_w = CAUSAL ? min(Nk, row0 + off + 1) : Nk;   // keys visible to all rows
    const int ntiles = (kend_wg + BC - 1) / BC;

    // Q rows of this lane, kept in registers (B operand of S^T = K Q^T).
    V8 qf[KSTEPS];
    {
        const S *qp = reinterpret_cast<const S *>(a.q) +
                      ((size_t)((size_t)b * Nq + qi) * a.Hq + h) * D + 8 * lh;
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            uint4_t u = {0u, 0u, 0u, 0u};
            if (qi < Nq) u = ld16(qp + 16 * ks);
            u ^= a.qsign;
            qf[ks] = as_vec8<V8>(u);
        }
    }

    // Global tile loads: chunk c = tid + 256 i covers key c / CPR, column
    // chunk c % CPR (consecutive threads read consecutive 16-byte pieces).
    const S *kbase = reinterpret_cast<const S *>(a.k);
    const S *vbase = reinterpret_cast<const S *>(a.v);
    uint4_t kr[LOADS], vr[LOADS];
    auto gload = [&](int kb) {
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int c = tid + 256 * i;
            const int key = kb + c / CPR, cc = c % CPR;
            kr[i] = uint4_t{0u, 0u, 0u, 0u};
            vr[i] = uint4_t{0u, 0u, 0u, 0u};
            if (key < Nk) {
                const size_t o = ((size_t)((size_t)b * Nk + key) * a.Hkv + g) * D + 8 * cc;
                kr[i] = ld16(kbase + o);
                vr[i] = ld16(vbase + o);
            }
        }
    };
    auto sstore = [&](int buf) {
        unsigned short *ks = smem + buf * SM::STAGE;
        unsigned short *vs = ks + SM::KSZ;
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int c = tid + 256 * i;
            const int key = c / CPR, cc = c % CPR;
            st16(ks + key * SM::KS + 8 * cc, kr[i]);
            st16(vs + key * SM::VS + 8 * cc, IN_BF16 ? bf16x8_to_f16x8(vr[i]) : vr[i]);
        }
    };

    // Running state of this lane's query row (shared with lane l^32).
    float16_t oacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] = float16_t{};
    float m_run = -INFINITY;   // exponent base (log2 domain)
    float l_run = 0.f;         // this lane's part of the row sum

    // Per-lane offsets into a stage.
    const int k_lane = lq * SM::KS + 8 * lh;
    const int v_lane = ((l & 15) >> 2) * SM::VS + 16 * ((l >> 4) & 1) + 4 * (l & 3) + 4 * lh * SM::VS;

    if (ntiles > 0) {
        gload(0);
        sstore(0);
    }
    __syncthreads();

    for (int t = 0; t < ntiles; ++t) {
        const int kb = t * BC;
        if (t + 1 < ntiles) gload(kb + BC);
        if (kb < kend_w) {
            const unsigned short *ks = smem + (t & 1) * SM::STAGE;
            const _Float16 *vs = reinterpret_cast<const _Float16 *>(ks + SM::KSZ);
            // ---- S^T = K Q^T for two 32-key halves of the tile
            float16_t s0 = float16_t{}, s1 = float16_t{};
#pragma unroll
            for (int kk = 0; kk < KSTEPS; ++kk) {
                V8 a0 = as_vec8<V8>(*reinterpret_cast<const uint4_t *>(ks + k_lane + 16 * kk));
                V8 a1 = as_vec8<V8>(
                    *reinterpret_cast<const uint4_t *>(ks + k_lane + 32 * SM::KS + 16 * kk));
                s0 = mfma32(a0, qf[kk], s0);
                s1 = mfma32(a1, qf[kk], s1);
            }
            // ---- mask (only tiles that reach past the keys every row sees)
            const bool masked = kb + BC > kfree_w;
            if (masked) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key0 = kb + 8 * (r >> 2) + 4 * lh + (r & 3);
                    const int key1 = key0 + 32;
                    const bool v0 = key0 < Nk && (!CAUSAL || key0 <= qi + off);
                    const bool v1 = key1 < Nk && (!CAUSAL || key1 <= qi + off);
                    s0[r] = v0 ? s0[r] : -INFINITY;
                    s1[r] = v1 ? s1[r] : -INFINITY;
                }
            }
            // ---- row maximum of the tile (raw scores; c >= 0)
            float mx = -INFINITY;
#pragma unroll
            for (int r = 0; r < 8; ++r) mx = max3(mx, s0[2 * r], s0[2 * r + 1]);
#pragma unroll
            for (int r = 0; r < 8; ++r) mx = max3(mx, s1[2 * r], s1[2 * r + 1]);
            mx = pair_max(mx);
            const float m_tile = (mx == -INFINITY) ? -INFINITY : mx * a.c;
            // ---- lazy rescale of accumulator and sum
            const float m_new = __builtin_fmaxf(m_run, m_tile);
            const bool need = m_new > m_run + TAU;
            if (__builtin_amdgcn_ballot_w64(need)) {
                const float m_next = need ? m_new : m_run;
                const float alpha = need ? exp2_fast(m_run - m_next) : 1.f;
                m_run = m_next;
                l_run *= alpha;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
            }
            const float base = (m_run == -INFINITY) ? 0.f : m_run;
            // ---- probabilities, row sum, fp16 operands for P V
            float lsum = 0.f;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float p0 = exp2_fast(__builtin_fmaf(s0[r], a.c, -base));
                float p1 = exp2_fast(__builtin_fmaf(s1[r], a.c, -base));
                if (masked) {
                    p0 = (s0[r] == -INFINITY) ? 0.f : p0;
                    p1 = (s1[r] == -INFINITY) ? 0.f : p1;
                }
                s0[r] = p0;
                s1[r] = p1;
                lsum += p0 + p1;
            }
            l_run += lsum;
            half8_t pf[4];
            pf[0] = pack_f16x8(s0[0], s0[1], s0[2], s0[3], s0[4], s0[5], s0[6], s0[7]);
            pf[1] = pack_f16x8(s0[8], s0[9], s0[10], s0[11], s0[12], s0[13], s0[14], s0[15]);
            pf[2] = pack_f16x8(s1[0], s1[1], s1[2], s1[3], s1[4], s1[5], s1[6], s1[7]);
            pf[3] = pack_f16x8(s1[8], s1[9], s1[10], s1[11], s1[12], s1[13], s1[14], s1[15]);
            // ---- O^T += V^T P^T; k-step j covers keys 16 j .. 16 j + 15 of the tile
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const _Float16 *vp = vs + v_lane + 16 * j * SM::VS + 32 * dt;
                    half8_t va = cat_half8(lds_read_tr16(vp), lds_read_tr16(vp + 8 * SM::VS));
                    oacc[dt] = mfma32(va, pf[j], oacc[dt]);
                }
            }
        }
        if (t + 1 < ntiles) sstore((t + 1) & 1);
        __syncthreads();
    }

    if (!wave_live) return;
    // ---- final normalisation and stores
    const float l_tot = pair_sum(l_run);
    const float inv = 1.f / l_tot;
    if (qi < Nq) {
        typedef TOUT OT;
        OT *op = reinterpret_cast<OT *>(a.o) + ((size_t)((size_t)b * Nq + qi) * a.Hq + h) * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int d0 = 32 * dt + 8 * i + 4 * lh;
                OT vals[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) vals[e] = from_f32<OT>(oacc[dt][4 * i + e] * inv);
                if constexpr (sizeof(OT) == 4) {
                    *reinterpret_cast<float4_t *>(op + d0) =
                        float4_t{vals[0], vals[1], vals[2], vals[3]};
                } else {
                    typedef unsigned short us4 __attribute__((ext_vector_type(4)));
                    us4 u;
#pragma unroll
                    for (int e = 0; e < 4; ++e) u[e] = __builtin_bit_cast(unsigned short, vals[e]);
                    *reinterpret_cast<us4 *>(op + d0) = u;
                }
            }
        }
        if (a.lse && lh == 0)
            a.lse[((size_t)b * a.Hq + h) * Nq + qi] = (m_run + log2f(l_tot)) * kLn2;
    }
    (void)a.scale_zero;
}

template <typename TIN, typename TOUT, int D, bool CAUSAL>
hipError_t launch_t(const Problem &p, hipStream_t stream) {
    PrefillArgs a;
    a.q = p.q; a.k = p.k; a.v = p.v; a.o = p.o; a.lse = p.lse;
    a.B = p.B; a.Hq = p.Hq; a.Hkv = p.Hkv; a.Nq = p.Nq; a.Nk = p.Nk;
    a.c = __builtin_fabsf(p.scale) * kLog2e;
    a.scale_zero = p.scale == 0.f ? 1.f : 0.f;
    a.qsign = p.scale < 0.f ? 0x80008000u : 0u;
    const int G = p.Hq / p.Hkv;
    a.HW = (G % 4 == 0) ? 4 : (G % 2 == 0 ? 2 : 1);
    const int RB = NW / a.HW;
    a.nmb = (p.Nq + WR * RB - 1) / (WR * RB);
    a.nhg = G / a.HW;
    const long long nblocks = (long long)a.nmb * p.B * p.Hkv * a.nhg;
    if (nblocks <= 0) return hipSuccess;
    if (nblocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((prefill_kernel<TIN, TOUT, D, CAUSAL>), dim3((unsigned)nblocks),
                       dim3(256), 0, stream, a);
    return hipGetLastError();
}

template <typename TIN, typename TOUT>
hipError_t launch_d(const Problem &p, hipStream_t s) {
    if (p.D == 64) return p.causal ? launch_t<TIN, TOUT, 64, true>(p, s)
                                   : launch_t<TIN, TOUT, 64, false>(p, s);
    return p.causal ? launch_t<TIN, TOUT, 128, true>(p, s) : launch_t<TIN, TOUT, 128, false>(p, s);
}

}  // namespace

bool prefill_supported(int D, fa_dtype_t in) {
    return (D == 64 || D == 128) && (in == FA_F16 || in == FA_BF16);
}

hipError_t launch_prefill(const Problem &p, hipStream_t stream) {
    if (p.in == FA_F16)
        return p.out == FA_F32 ? launch_d<f16_t, float>(p, stream)
                               : launch_d<f16_t, _Float16>(p, stream);
    return p.out == FA_F32 ? launch_d<bf16_t, float>(p, stream) : launch_d<bf16_t, __bf16>(p, stream);
}

}  // namespace fa
