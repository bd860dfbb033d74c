// fa_decode.hip -- decode attention (one query row per head against a long
// key/value cache) on gfx950: split-KV partial kernel plus log-sum-exp merge.
//
// Decode has one query row per head (Sec. 4.1: the operands shrink to 1 x D),
// so the only parallelism inside one (batch, key/value head) is across the
// query heads of its group and along the key sequence.  The G query heads
// that share a key/value head are processed together as the 16 columns of a
// 16x16x32 MFMA (the GPU form of packing several heads into one vector
// register, Sec. 4.1.1, with the K/V row loaded once for the whole group,
// Sec. 4.1.2 (iv)); the key range is cut into splits, one workgroup per
// (batch, key/value head, 16-head query group, split), so that enough
// workgroups stream K/V from HBM to keep every CU busy.
//
// Inside a workgroup each of the 8 waves streams its own 32-key chunks
// (round robin over the split), carrying running max / sum / accumulator as
// in Alg. 1 (tile-wise; the running maximum only moves when a tile's maximum
// exceeds it by more than 8 in the log2 domain).  A chunk's K and V rows are
// loaded whole and staged in the wave's own LDS area, one chunk ahead of the
// arithmetic.  The waves' partial states are merged through LDS and the
// workgroup writes one (unnormalised accumulator, max, sum) triple per query
// head and split.  A second kernel merges the splits of each (batch, query
// head) by their log-sum-exp and applies the final 1/l normalisation.
#include "fa_common.h"
#include "fa_internal.h"

namespace fa {
namespace {

constexpr int KPW = 32;        // keys per wave iteration
constexpr int NW = 8;          // waves per workgroup
constexpr int QG = 16;         // query heads per MFMA column block
constexpr float TAU = 8.0f;    // lazy-rescale threshold (log2 units)
constexpr int MIN_KEYS_PER_SPLIT = 256;
constexpr int TARGET_WORKGROUPS = 256;   // about one workgroup per CU: long splits, few partials

struct DecodeArgs {
    const void *q, *k, *v;
    float *opart, *mpart, *lpart;   // workspace: [B*Hq*S*D], [B*Hq*S], [B*Hq*S]
    int B, Hq, Hkv, Nk;
    int S;          // splits
    int chunk;      // keys per split (multiple of KPW)
    int nqg;        // 16-head query groups per key/value head
    float c;        // |scale| * log2(e)
    unsigned qsign; // sign flip of q for negative scale
    const int *seqlens;   // valid keys per batch element (NULL: Nk for all)
    const int *block_table;   // paged K/V: page of each key block (see Problem)
    int page_size, max_pages, num_pages;
};

template <int D> struct DSmem {
    static constexpr int KS = D + 8;             // K row stride (16-bit elements)
    static constexpr int VS = D + 16;            // V row stride (16-bit elements)
    static constexpr int WAVE = KPW * (KS + VS); // per-wave K and V staging
    static constexpr int MERGE_FLOATS = NW * QG * (D + 2);
    static constexpr int BYTES_STAGE = NW * WAVE * 2;
    static constexpr int BYTES = BYTES_STAGE > MERGE_FLOATS * 4 ? BYTES_STAGE : MERGE_FLOATS * 4;
};

__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <typename TIN, int D, bool PAGED>
__global__ __launch_bounds__(64 * NW, 1) void decode_split_kernel(DecodeArgs a) {
    using S = typename TIN::scalar;
    using V8 = typename TIN::vec8;
    using SM = DSmem<D>;
    constexpr int KST = D / 32;          // QK^T contraction steps (K = 32)
    constexpr int DT = D / 16;           // output row tiles of 16
    constexpr int CPR = D / 8;           // 16-byte chunks per key row
    constexpr int RLOADS = KPW * CPR / 64;   // 16-byte row loads per lane per chunk (K and V each)
    constexpr bool IN_BF16 = __is_same(TIN, bf16_t);

    __shared__ __attribute__((aligned(16))) unsigned char smem[SM::BYTES];

    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    const int lc = l & 15, lg = l >> 4;            // MFMA column (query) and k-group
    int bid = blockIdx.x;
    const int s = bid % a.S;
    bid /= a.S;
    const int qg = bid % a.nqg;
    bid /= a.nqg;
    const int g = bid % a.Hkv;
    const int b = bid / a.Hkv;
    const int G = a.Hq / a.Hkv;
    // valid keys of this batch element (a cache of a.Nk rows per element)
    const int Nk = a.seqlens ? min(max(a.seqlens[b], 0), a.Nk) : a.Nk;
    const int k0 = s * a.chunk;
    const int k1 = min(Nk, k0 + a.chunk);

    // This lane's query head (MFMA column) and its Q operand.
    const int qh = qg * QG + lc;             // index inside the group
    const bool qvalid = qh < G;
    const int h = g * G + qh;
    V8 qf[KST];
    {
        const S *qp = reinterpret_cast<const S *>(a.q) + ((size_t)b * a.Hq + h) * D + 8 * lg;
#pragma unroll
        for (int ks = 0; ks < KST; ++ks) {
            uint4_t u = {0u, 0u, 0u, 0u};
            if (qvalid) u = ld16(qp + 32 * ks);
            u ^= a.qsign;
            qf[ks] = as_vec8<V8>(u);
        }
    }

    const S *kbase = reinterpret_cast<const S *>(a.k);
    const S *vbase = reinterpret_cast<const S *>(a.v);
    const size_t row_stride = (size_t)a.Hkv * D;                  // elements between keys
    const size_t head_off = ((size_t)b * a.Nk * a.Hkv + g) * D;   // key 0 of (b, g)

    unsigned short *kst = reinterpret_cast<unsigned short *>(smem) + w * SM::WAVE;
    unsigned short *vst = kst + KPW * SM::KS;
    const _Float16 *vsth = reinterpret_cast<const _Float16 *>(vst);
    // transpose-read lane offset: rows 4*lg + (lc / 4), columns 4 * (lc % 4)
    const int v_lane = (4 * lg + (lc >> 2)) * SM::VS + 4 * (lc & 3);

    float4_t oacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] = float4_t{};
    float m_run = -INFINITY, l_run = 0.f;

    // A chunk's K and V rows are loaded whole (64 lanes cover 64 / CPR
    // complete rows per instruction, the access pattern that streams from HBM
    // fastest) and staged in the wave's own LDS area: K as is (read back in
    // the MFMA operand layout), V as fp16 (read back transposed).
    uint4_t kr[RLOADS], vr[RLOADS];   // the next chunk's rows, in flight
    auto gload = [&](int kb) {
        // element offset of key kb's row (head g): contiguous, or through the
        // block table (a chunk never crosses a page: chunks start at multiples
        // of 32 keys and pages hold a multiple of 64; page numbers are clamped
        // into the pool)
        size_t rbase;
        if constexpr (PAGED) {
            const int pi = kb / a.page_size;
            const int page = min(max(a.block_table[(size_t)b * a.max_pages + pi], 0), a.num_pages - 1);
            rbase = ((size_t)page * a.page_size + (kb - pi * a.page_size)) * row_stride + (size_t)g * D;
        } else {
            rbase = head_off + (size_t)kb * row_stride;
        }
#pragma unroll
        for (int i = 0; i < RLOADS; ++i) {
            const int c = l + 64 * i;
            const int kc = c / CPR, cc = c % CPR;
            kr[i] = uint4_t{0u, 0u, 0u, 0u};
            vr[i] = uint4_t{0u, 0u, 0u, 0u};
            if (kb + kc < k1) {
                kr[i] = ld16_stream(kbase + rbase + kc * row_stride + 8 * cc);
                vr[i] = ld16_stream(vbase + rbase + kc * row_stride + 8 * cc);
            }
        }
    };
    auto kvstore = [&]() {
#pragma unroll
        for (int i = 0; i < RLOADS; ++i) {
            const int c = l + 64 * i;
            const int key = c / CPR, cc = c % CPR;
            st16(kst + key * SM::KS + 8 * cc, kr[i]);
            st16(vst + key * SM::VS + 8 * cc, IN_BF16 ? bf16x8_to_f16x8(vr[i]) : vr[i]);
        }
    };

    const int nchunks = (k1 > k0) ? (k1 - k0 + KPW - 1) / KPW : 0;
    if (w < nchunks) {
        gload(k0 + w * KPW);
        kvstore();
        wave_lds_fence();
    }
    for (int ch = w; ch < nchunks; ch += NW) {
        const int kb = k0 + ch * KPW;
        const bool more = ch + NW < nchunks;
        if (more) gload(kb + NW * KPW);
        // ---- S^T = K Q^T: two 16-key halves, lane owns query lc, keys 4 lg + r
        float4_t s0 = float4_t{}, s1 = float4_t{};
        const unsigned short *kl = kst + lc * SM::KS + 8 * lg;
#pragma unroll
        for (int ks = 0; ks < KST; ++ks) {
            s0 = mfma16(as_vec8<V8>(*reinterpret_cast<const uint4_t *>(kl + 32 * ks)), qf[ks], s0);
            s1 = mfma16(as_vec8<V8>(*reinterpret_cast<const uint4_t *>(kl + 16 * SM::KS + 32 * ks)),
                        qf[ks], s1);
        }
        const bool masked = kb + KPW > k1;
        if (masked) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                s0[r] = (kb + 4 * lg + r < k1) ? s0[r] : -INFINITY;
                s1[r] = (kb + 16 + 4 * lg + r < k1) ? s1[r] : -INFINITY;
            }
        }
        float mx = max3(max3(s0[0], s0[1], s0[2]), max3(s0[3], s1[0], s1[1]), __builtin_fmaxf(s1[2], s1[3]));
        mx = __builtin_fmaxf(mx, __shfl_xor(mx, 16));
        mx = __builtin_fmaxf(mx, __shfl_xor(mx, 32));
        const float m_tile = (mx == -INFINITY) ? -INFINITY : mx * a.c;
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
        float p[8];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            p[r] = exp2_fast(__builtin_fmaf(s0[r], a.c, -base));
            p[4 + r] = exp2_fast(__builtin_fmaf(s1[r], a.c, -base));
        }
        if (masked) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                p[r] = (s0[r] == -INFINITY) ? 0.f : p[r];
                p[4 + r] = (s1[r] == -INFINITY) ? 0.f : p[4 + r];
            }
        }
        l_run += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
        const half8_t pf = pack_f16x8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
        // ---- O^T += V^T P^T over the 32 keys (k-group lg: keys 4lg..+3, 16+4lg..+3)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const _Float16 *vp = vsth + v_lane + 16 * dt;
            half8_t va = cat_half8(lds_read_tr16(vp), lds_read_tr16(vp + 16 * SM::VS));
            oacc[dt] = mfma16(va, pf, oacc[dt]);
        }
        if (more) {
            wave_lds_fence();   // operand reads of this chunk are done
            kvstore();
            wave_lds_fence();
        }
    }

    // ---- merge the waves' partial states through LDS
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
    __syncthreads();
    float *mf = reinterpret_cast<float *>(smem);     // [NW][QG][D + 2]
    float *mine = mf + (w * QG + lc) * (D + 2);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 4; ++r) mine[16 * dt + 4 * lg + r] = oacc[dt][r];
    if (lg == 0) {
        mine[D] = m_run;
        mine[D + 1] = l_run;
    }
    __syncthreads();
    // the first 256 threads: query column tid / 16, 16 threads per query, D / 16 columns each
    const int mq = tid >> 4, part = tid & 15;
    const int mh = qg * QG + mq;
    if (mq < QG && mh < G) {
        float M = -INFINITY;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) M = __builtin_fmaxf(M, mf[(ww * QG + mq) * (D + 2) + D]);
        float wgt[NW];
        float L = 0.f;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) {
            const float mw = mf[(ww * QG + mq) * (D + 2) + D];
            wgt[ww] = (mw == -INFINITY) ? 0.f : exp2_fast(mw - M);
            L += wgt[ww] * mf[(ww * QG + mq) * (D + 2) + D + 1];
        }
        const size_t slot = ((size_t)b * a.Hq + g * G + mh) * a.S + s;
        float *op = a.opart + slot * D;
#pragma unroll
        for (int j = 0; j < D / 16; ++j) {
            const int d = part + 16 * j;
            float acc = 0.f;
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) acc += wgt[ww] * mf[(ww * QG + mq) * (D + 2) + d];
            op[d] = acc;
        }
        if (part == 0) {
            a.mpart[slot] = M;
            a.lpart[slot] = L;
        }
    }
}

// Merge of the S partial results of one (batch, query head): lse-weighted sum
// of the unnormalised accumulators, final normalisation, log-sum-exp output.
// Splits are taken in groups of 16 whose loads are all issued together (one
// memory round trip per group; the usual split counts fit in one group); the
// running maximum moves once per group.  Every thread of the block handles
// one output column and forms the same maximum and sum.
template <typename TOUT, int D>
__global__ __launch_bounds__(D) void decode_combine_kernel(const float *__restrict__ opart,
                                                          const float *__restrict__ mpart,
                                                          const float *__restrict__ lpart,
                                                          void *o, float *lse, int S) {
    constexpr int CH = 16;
    const int bh = blockIdx.x, t = threadIdx.x;
    const float *mp = mpart + (size_t)bh * S;
    const float *lp = lpart + (size_t)bh * S;
    const float *op = opart + (size_t)bh * S * D + t;
    float M = -INFINITY, L = 0.f, acc = 0.f;
    for (int s0 = 0; s0 < S; s0 += CH) {
        float mv[CH], lv[CH], ov[CH];
#pragma unroll
        for (int j = 0; j < CH; ++j) {
            mv[j] = -INFINITY;
            lv[j] = 0.f;
            ov[j] = 0.f;
            if (s0 + j < S) {
                mv[j] = mp[s0 + j];
                lv[j] = lp[s0 + j];
                ov[j] = op[(size_t)(s0 + j) * D];
            }
        }
        float Mc = M;
#pragma unroll
        for (int j = 0; j < CH; ++j) Mc = __builtin_fmaxf(Mc, mv[j]);
        const float alpha = (M == -INFINITY) ? 0.f : exp2_fast(M - Mc);
        L *= alpha;
        acc *= alpha;
#pragma unroll
        for (int j = 0; j < CH; ++j) {
            const float w = (mv[j] == -INFINITY) ? 0.f : exp2_fast(mv[j] - Mc);
            L = __builtin_fmaf(w, lv[j], L);
            acc = __builtin_fmaf(w, ov[j], acc);
        }
        M = Mc;
    }
    // a sequence with no valid key (per-sequence lengths) gives 0 and -inf
    reinterpret_cast<TOUT *>(o)[(size_t)bh * D + t] = from_f32<TOUT>(L > 0.f ? acc / L : 0.f);
    if (lse && t == 0) lse[bh] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
}

template <typename TIN, typename TOUT, int D>
hipError_t launch_t(const Problem &p, int S, void *ws, hipStream_t stream) {
    DecodeArgs a;
    a.q = p.q; a.k = p.k; a.v = p.v;
    const size_t nslot = (size_t)p.B * p.Hq * S;
    a.opart = reinterpret_cast<float *>(ws);
    a.mpart = a.opart + nslot * D;
    a.lpart = a.mpart + nslot;
    a.B = p.B; a.Hq = p.Hq; a.Hkv = p.Hkv; a.Nk = p.Nk;
    a.S = S;
    const int per = (p.Nk + S - 1) / S;
    a.chunk = (per + KPW - 1) / KPW * KPW;
    const int G = p.Hq / p.Hkv;
    a.nqg = (G + QG - 1) / QG;
    a.c = __builtin_fabsf(p.scale) * kLog2e;
    a.qsign = p.scale < 0.f ? 0x80008000u : 0u;
    a.seqlens = p.seqlens;
    a.block_table = p.block_table;
    a.page_size = p.page_size;
    a.max_pages = p.max_pages;
    a.num_pages = p.num_pages;
    const long long nblocks = (long long)p.B * p.Hkv * a.nqg * S;
    if (nblocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    if (p.block_table)
        hipLaunchKernelGGL((decode_split_kernel<TIN, D, true>), dim3((unsigned)nblocks), dim3(64 * NW), 0,
                           stream, a);
    else
        hipLaunchKernelGGL((decode_split_kernel<TIN, D, false>), dim3((unsigned)nblocks), dim3(64 * NW), 0,
                           stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((decode_combine_kernel<TOUT, D>), dim3((unsigned)(p.B * p.Hq)), dim3(D), 0,
                       stream, a.opart, a.mpart, a.lpart, p.o, p.lse, S);
    return hipGetLastError();
}

template <typename TIN, typename TOUT>
hipError_t launch_d(const Problem &p, int S, void *ws, hipStream_t s) {
    return p.D == 64 ? launch_t<TIN, TOUT, 64>(p, S, ws, s) : launch_t<TIN, TOUT, 128>(p, S, ws, s);
}

}  // namespace

bool decode_supported(int Nq, int D, fa_dtype_t in) {
    return Nq == 1 && (D == 64 || D == 128) && (in == FA_F16 || in == FA_BF16);
}

int decode_default_splits(int B, int Hq, int Hkv, int Nk, int D) {
    (void)D;
    const int G = Hq / Hkv;
    const long long units = (long long)B * Hkv * ((G + QG - 1) / QG);
    long long s = (TARGET_WORKGROUPS + units - 1) / units;
    const long long cap = (Nk + MIN_KEYS_PER_SPLIT - 1) / MIN_KEYS_PER_SPLIT;
    if (s > cap) s = cap;
    if (s < 1) s = 1;
    if (s > FA_MAX_SPLITS) s = FA_MAX_SPLITS;
    return (int)s;
}

size_t decode_workspace_bytes(int B, int Hq, int D, int splits) {
    return (size_t)B * Hq * splits * (size_t)(D + 2) * sizeof(float);
}

hipError_t launch_decode(const Problem &p, int splits, void *ws, hipStream_t stream) {
    if (p.in == FA_F16)
        return p.out == FA_F32 ? launch_d<f16_t, float>(p, splits, ws, stream)
                               : launch_d<f16_t, _Float16>(p, splits, ws, stream);
    return p.out == FA_F32 ? launch_d<bf16_t, float>(p, splits, ws, stream)
                           : launch_d<bf16_t, __bf16>(p, splits, ws, stream);
}

}  // namespace fa
