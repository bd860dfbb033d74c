// fa_unfused.hip -- unfused self-attention forward on gfx950: the path with a
// materialised score matrix that the paper optimises beside FlashAttention-V
// (Sec. 4.2) and measures it against (Sec. 6.2, self-attention against the
// fused kernel in prefill).  Three kernels, each leaving its whole result in
// HBM for the next:
//   scores   S = scale * Q K^T in fp32, [B][Hq][Nq][NkP] (NkP = Nk rounded up
//            to 64 keys); masked entries are -inf.  A workgroup's four waves
//            are four (query head, 32-row block) slots that read one
//            key/value head -- query heads of one group at the same rows when
//            the group size allows, the reuse across heads of Sec. 4.2 (one
//            staged key row serves several heads) -- and it takes a chunk of
//            64-key tiles; tiles past the causal edge are not computed.
//            32x32x16 MFMA, A = the wave's 32 query rows (registers),
//            B = 32 key rows of the tile in LDS.
//   softmax  one wave per query row, or two or four for rows past 4096
//            keys: the row's scores are read once into registers (4096 keys
//            per wave; rows past four waves stream the rest twice), the
//            waves' maxima and sums combined through LDS, then P = 2^(S log2 e - max) /
//            sum in fp16, with zeros from the last visible key up to the end
//            of the last tile the P.V kernel reads for that row, and the
//            row's log-sum-exp.  Loads and stores go through buffer views
//            that end at the row's last visible chunk and at the end of its
//            padding, so no lane needs a bounds branch.
//   pv       O = P V.  A = 16 keys of P per lane, read straight from HBM;
//            B = V from a row-major fp16 copy of the 64-key tile in LDS, read
//            with the transposing LDS load (four keys of one column per
//            read); fp32 accumulation, one rounding to the output type.
// Per visible score the path writes S (4 bytes) and P (2) and reads each
// once: the traffic the fused kernel never makes.
#include "fa_common.h"
#include "fa_internal.h"

namespace fa {
namespace {

constexpr int UR = 32;       // query rows per slot (one wave)
constexpr int USLOT = 4;     // slots per workgroup
constexpr int UKT = 64;      // keys per tile
constexpr int UCHUNK = 8;    // key tiles per scores workgroup
constexpr int UNT = 64 * USLOT;

struct UnfusedArgs {
    const void *q, *k, *v;
    void *o;
    float *lse;
    float *s;           // workspace: scores, [B][Hq][Nq][NkP] fp32
    _Float16 *p;        // workspace: weights, [B][Hq][Nq][NkP] fp16
    int B, Hq, Hkv, Nq, Nk, NkP;
    float scale;
    int HW;             // query heads per workgroup (4, 2 or 1)
    int nmb;            // row blocks of 32 * (4 / HW) rows
    int nhg;            // head groups per key/value head (G / HW)
    int nchunk;         // key-tile chunks per row block (scores)
};

// Slot of wave w of a workgroup whose row block is mb, head group hg, key/value head g.
struct Slot {
    int h, row0, row0_wg, rows_wg;
};
__device__ __forceinline__ Slot slot_of(const UnfusedArgs &a, int w, int mb, int hg, int g) {
    const int G = a.Hq / a.Hkv, RB = USLOT / a.HW;
    Slot s;
    s.h = g * G + hg * a.HW + w % a.HW;
    s.rows_wg = UR * RB;
    s.row0_wg = mb * s.rows_wg;
    s.row0 = s.row0_wg + (w / a.HW) * UR;
    return s;
}

// Visible keys of query row i (bottom-right causal alignment).
__device__ __forceinline__ int kend_row(int i, int Nq, int Nk, bool causal) {
    return causal ? min(Nk, i + Nk - Nq + 1) : Nk;
}

// Copy of one 64-key tile of K or V (keys t0 .. t0 + 63 of head g) into
// registers: chunk c = tid + 256 i is key c / (D / 8), columns 8 (c % (D / 8)).
// Keys past Nk read as zero.
template <typename TIN, int D>
__device__ __forceinline__ void tile_load(const void *base, int b, int g, int Hkv, int Nk, int t0,
                                          int tid, uint4_t (&r)[UKT * D / 8 / UNT]) {
    using S = typename TIN::scalar;
    constexpr int CPR = D / 8;
#pragma unroll
    for (int i = 0; i < UKT * CPR / UNT; ++i) {
        const int c = tid + UNT * i;
        const int key = t0 + c / CPR;
        r[i] = uint4_t{0u, 0u, 0u, 0u};
        if (key < Nk)
            r[i] = ld16(reinterpret_cast<const S *>(base) +
                        ((size_t)((size_t)b * Nk + key) * Hkv + g) * D + 8 * (c % CPR));
    }
}

typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
constexpr int kRsrcFlags = 0x00020000;   // buffer descriptor word 3 for raw 32-bit element access

template <typename TIN, int D, bool CAUSAL>
__global__ __launch_bounds__(UNT) void unfused_scores_kernel(UnfusedArgs a) {
    using S = typename TIN::scalar;
    using V8 = typename TIN::vec8;
    constexpr int KS = D + 8;            // LDS row stride (16-bit elements)
    constexpr int KSTEPS = D / 16;
    constexpr int CPR = D / 8;
    constexpr int NLD = UKT * CPR / UNT;
    __shared__ __attribute__((aligned(16))) unsigned short kt[UKT * KS];

    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l = tid & 63, lq = l & 31, lh = l >> 5;
    int bid = blockIdx.x;
    const int chunk = bid % a.nchunk;
    bid /= a.nchunk;
    const int hg = bid % a.nhg;
    bid /= a.nhg;
    const int g = bid % a.Hkv;
    bid /= a.Hkv;
    const int b = bid % a.B;
    const int mbi = bid / a.B;
    const int mb = CAUSAL ? a.nmb - 1 - mbi : mbi;   // longest rows first
    const Slot sl = slot_of(a, w, mb, hg, g);
    const int Nq = a.Nq, Nk = a.Nk, off = Nk - Nq;

    const int last_wg = min(sl.row0_wg + sl.rows_wg, Nq) - 1;
    const int ntiles = (kend_row(last_wg, Nq, Nk, CAUSAL) + UKT - 1) / UKT;
    const int t0 = chunk * UCHUNK, t1 = min(t0 + UCHUNK, ntiles);
    if (t0 >= t1) return;   // the same for the whole workgroup
    const bool live = sl.row0 < Nq;
    const int kend_w = live ? kend_row(min(sl.row0 + UR, Nq) - 1, Nq, Nk, CAUSAL) : 0;
    // keys every row of the slot sees: tiles below need no mask
    const int kfree_w = live ? kend_row(sl.row0, Nq, Nk, CAUSAL) : 0;

    V8 qf[KSTEPS];
    {
        const int qrow = min(sl.row0 + lq, Nq - 1);
        const S *qp = reinterpret_cast<const S *>(a.q) + ((size_t)((size_t)b * Nq + qrow) * a.Hq + sl.h) * D + 8 * lh;
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) qf[ks] = as_vec8<V8>(ld16(qp + 16 * ks));
    }
    // The slot's 32 rows of S as a buffer view ending after row Nq - 1: stores
    // to rows past the end fall outside it and are dropped.  Lane l stores key
    // (l % 32) of rows 8 (r / 4) + 4 (l / 32) + r % 4 (byte offsets stay below
    // 2^31: Nk <= 2^23).
    const int nrows = live ? min(UR, Nq - sl.row0) : 0;
    const __amdgpu_buffer_rsrc_t srs = __builtin_amdgcn_make_buffer_rsrc(
        a.s + ((size_t)((size_t)b * a.Hq + sl.h) * Nq + (live ? sl.row0 : 0)) * a.NkP, (short)0,
        nrows * a.NkP * 4, kRsrcFlags);
    const int lane_off = (4 * lh * a.NkP + lq) * 4;

    uint4_t kr[NLD];
    tile_load<TIN, D>(a.k, b, g, a.Hkv, Nk, t0 * UKT, tid, kr);
    for (int t = t0; t < t1; ++t) {
        __syncthreads();   // the previous tile's operand reads are done
#pragma unroll
        for (int i = 0; i < NLD; ++i) {
            const int c = tid + UNT * i;
            st16(kt + (c / CPR) * KS + 8 * (c % CPR), kr[i]);
        }
        __syncthreads();
        if (t + 1 < t1) tile_load<TIN, D>(a.k, b, g, a.Hkv, Nk, (t + 1) * UKT, tid, kr);
        if (t * UKT >= kend_w) continue;   // wave-uniform: no row of the slot sees this tile
        const bool masked = t * UKT + UKT > kfree_w;   // wave-uniform
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            float16_t s = float16_t{};
#pragma unroll
            for (int ks = 0; ks < KSTEPS; ++ks)
                s = mfma32(qf[ks], as_vec8<V8>(*reinterpret_cast<const uint4_t *>(kt + (32 * half + lq) * KS + 8 * lh + 16 * ks)), s);
            const int k0 = t * UKT + 32 * half;
            const int voff = lane_off + k0 * 4;
            // causal: key visible to row (row0 + 4 lh + dr) iff key - off - row0 - 4 lh <= dr
            const int kd = k0 + lq - off - sl.row0 - 4 * lh;
            const bool kin = k0 + lq < Nk;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int dr = 8 * (r >> 2) + (r & 3);
                float val = s[r] * a.scale;
                if (masked) val = (kin && (!CAUSAL || kd <= dr)) ? val : -INFINITY;
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(val), srs, voff + dr * a.NkP * 4, 0, 0);
            }
        }
    }
}

template <bool CAUSAL, int WPR>
__global__ __launch_bounds__(UNT) void unfused_softmax_kernel(UnfusedArgs a) {
    constexpr int CH = 16;            // 16-byte chunks per lane held in registers
    constexpr int SEG = CH * 256;     // keys held by one wave (4096)
    constexpr int RPW = USLOT / WPR;  // rows per workgroup (WPR waves per row)
    __shared__ float red[USLOT];
    const int tid = threadIdx.x, l = tid & 63, w = tid >> 6;
    const int seg = w % WPR;
    const long long row = (long long)blockIdx.x * RPW + w / WPR;
    const bool valid = row < (long long)a.B * a.Hq * a.Nq;   // the same for the row's waves
    // rows past the end take part in the workgroup's barriers and store nothing
    const long long rr = valid ? row : 0;
    const int kend = valid ? kend_row((int)(rr % a.Nq), a.Nq, a.Nk, CAUSAL) : 0;
    // the P.V kernel reads whole 64-key tiles up to the extent of the last
    // row of this row's 32-row slot, at most 31 keys past this row's own
    const int zend = valid ? min(a.NkP, ((kend + UKT - 1) / UKT) * UKT + UKT) : 0;
    float *sr = a.s + (size_t)rr * a.NkP;
    _Float16 *pr = a.p + (size_t)rr * a.NkP;
    // this wave's segment of the row: keys k0 .. k0 + SEG - 1, kc of them visible
    const int k0 = seg * SEG;
    const int kc = max(0, min(kend - k0, SEG));
    const int zc = max(0, min(zend - k0, SEG));
    // views of the segment: S up to its last visible chunk (loads past it
    // return zero and read no memory), P up to the end of the zero padding
    const __amdgpu_buffer_rsrc_t srs = __builtin_amdgcn_make_buffer_rsrc(sr + k0, (short)0, ((kc + 3) & ~3) * 4, kRsrcFlags);
    const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(pr + k0, (short)0, zc * 2, kRsrcFlags);

    const int nch = (kc + 255) / 256;   // held chunks with visible keys (wave-uniform)
    float4_t x[CH];
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        x[j] = float4_t{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
        if (j < nch)
            x[j] = __builtin_bit_cast(float4_t, __builtin_amdgcn_raw_buffer_load_b128(srs, (4 * l + 256 * j) * 4, 0, 0));
    }
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        if (j < nch) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float t = (4 * l + 256 * j + e < kc) ? x[j][e] * kLog2e : -INFINITY;
                x[j][e] = t;
                m = __builtin_fmaxf(m, t);
            }
        }
    }
    // keys past the held segments (rows longer than WPR * 4096 keys), in
    // chunks interleaved over the row's waves: running maximum and sum, read
    // again for the weights
    float mt = -INFINITY, st = 0.f;
    for (int c = WPR * SEG + 256 * seg + 4 * l; c < kend; c += 256 * WPR) {
        const float4_t y = *reinterpret_cast<const float4_t *>(sr + c);
        float t[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) t[e] = (c + e < kend) ? y[e] * kLog2e : -INFINITY;
        const float mx = __builtin_fmaxf(__builtin_fmaxf(t[0], t[1]), __builtin_fmaxf(t[2], t[3]));
        if (mx > mt) {
            st = (mt == -INFINITY) ? 0.f : st * exp2_fast(mt - mx);
            mt = mx;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) st += exp2_fast(t[e] - mt);
    }
    float M = __builtin_fmaxf(m, mt);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) M = __builtin_fmaxf(M, __shfl_xor(M, o));
    const int r0 = w - seg;   // first wave of this row
    if constexpr (WPR > 1) {
        if (l == 0) red[w] = M;
        __syncthreads();
#pragma unroll
        for (int k = 0; k < WPR; ++k) M = __builtin_fmaxf(M, red[r0 + k]);
        __syncthreads();
    }
    float sum = (mt == -INFINITY) ? 0.f : st * exp2_fast(mt - M);
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        if (j < nch) {
#pragma unroll
            for (int e = 0; e < 4; ++e) sum += exp2_fast(x[j][e] - M);
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) sum += __shfl_xor(sum, o);
    if constexpr (WPR > 1) {
        if (l == 0) red[w] = sum;
        __syncthreads();
        sum = 0.f;
#pragma unroll
        for (int k = 0; k < WPR; ++k) sum += red[r0 + k];   // fixed order: the same on every wave
    }
    const float inv = 1.f / sum;
    if (valid && a.lse && seg == 0 && l == 0) a.lse[row] = (M + __builtin_log2f(sum)) * kLn2;
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        if (256 * j < zc) {
            half4_t h = {(_Float16)0.f, (_Float16)0.f, (_Float16)0.f, (_Float16)0.f};
            if (j < nch) {
#pragma unroll
                for (int e = 0; e < 4; ++e) h[e] = (_Float16)(exp2_fast(x[j][e] - M) * inv);
            }
            __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2_t, h), prs, (4 * l + 256 * j) * 2, 0, 0);
        }
    }
    for (int c = WPR * SEG + 256 * seg + 4 * l; c < zend; c += 256 * WPR) {
        half4_t h = {(_Float16)0.f, (_Float16)0.f, (_Float16)0.f, (_Float16)0.f};
        if (c < kend) {
            const float4_t y = *reinterpret_cast<const float4_t *>(sr + c);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                h[e] = (c + e < kend) ? (_Float16)(exp2_fast(y[e] * kLog2e - M) * inv) : (_Float16)0.f;
        }
        *reinterpret_cast<half4_t *>(pr + c) = h;
    }
}

// P.V: the workgroup's four slots share each staged V tile (the slot layout
// of the scores kernel, longest rows first).  The next tile's V loads are in
// flight during a tile's products; a tile's P loads go out at the start of
// its step (the wait before the V copy into LDS also covers them).
template <typename TIN, typename TOUT, int D, bool CAUSAL>
__global__ __launch_bounds__(UNT) void unfused_pv_kernel(UnfusedArgs a) {
    constexpr int VS = D + 8;            // LDS row stride (fp16 elements)
    constexpr int CPR = D / 8;
    constexpr int NLD = UKT * CPR / UNT;
    constexpr int DT = D / 32;
    constexpr bool IN_BF16 = __is_same(TIN, bf16_t);
    __shared__ __attribute__((aligned(16))) _Float16 vt[UKT * VS];

    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l = tid & 63, lq = l & 31, lh = l >> 5;
    int bid = blockIdx.x;
    const int hg = bid % a.nhg;
    bid /= a.nhg;
    const int g = bid % a.Hkv;
    bid /= a.Hkv;
    const int b = bid % a.B;
    const int mb = CAUSAL ? a.nmb - 1 - bid / a.B : bid / a.B;   // longest rows first
    const Slot sl = slot_of(a, w, mb, hg, g);
    const int Nq = a.Nq, Nk = a.Nk;

    const int last_wg = min(sl.row0_wg + sl.rows_wg, Nq) - 1;
    const int ntiles = (kend_row(last_wg, Nq, Nk, CAUSAL) + UKT - 1) / UKT;
    const bool live = sl.row0 < Nq;
    const int kend_w = live ? kend_row(min(sl.row0 + UR, Nq) - 1, Nq, Nk, CAUSAL) : 0;
    const int ntiles_w = (kend_w + UKT - 1) / UKT;

    // A operand source: 8 weights of row (row0 + l % 32) at keys 8 (l / 32) + 16 kk
    const _Float16 *prow = a.p + ((size_t)((size_t)b * a.Hq + sl.h) * Nq + min(sl.row0 + lq, Nq - 1)) * a.NkP + 8 * lh;
    // B operand: the transposing read gives lane j of each 16-lane group
    // column c0 + j of four consecutive keys; lane j addresses key (r0 + j / 4),
    // columns c0 + 4 (j % 4) .. + 3
    const int j = l & 15;
    const int vlane = (8 * lh + j / 4) * VS + 16 * ((l >> 4) & 1) + 4 * (j % 4);

    float16_t oacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] = float16_t{};
    uint4_t vr[NLD];
    if (ntiles > 0) tile_load<TIN, D>(a.v, b, g, a.Hkv, Nk, 0, tid, vr);
    for (int t = 0; t < ntiles; ++t) {
        const bool comp = t < ntiles_w;   // wave-uniform
        half8_t pa[4];
        if (comp) {
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) pa[kk] = as_vec8<half8_t>(ld16(prow + t * UKT + 16 * kk));
        }
        __syncthreads();   // the previous tile's operand reads are done
#pragma unroll
        for (int i = 0; i < NLD; ++i) {
            const int c = tid + UNT * i;
            st16(vt + (c / CPR) * VS + 8 * (c % CPR), IN_BF16 ? bf16x8_to_f16x8(vr[i]) : vr[i]);
        }
        __syncthreads();
        if (t + 1 < ntiles) tile_load<TIN, D>(a.v, b, g, a.Hkv, Nk, (t + 1) * UKT, tid, vr);
        if (!comp) continue;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const _Float16 *src = vt + vlane + 16 * kk * VS + 32 * dt;
                const half8_t vb = cat_half8(lds_read_tr16(src), lds_read_tr16(src + 4 * VS));
                oacc[dt] = mfma32(pa[kk], vb, oacc[dt]);
            }
        }
    }
    if (!live) return;
    // lane l holds column 32 dt + l % 32 of rows 8 (r / 4) + 4 (l / 32) + r % 4
    TOUT *o = reinterpret_cast<TOUT *>(a.o);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int row = sl.row0 + 8 * (r >> 2) + 4 * lh + (r & 3);
        if (row < Nq) {
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
                o[((size_t)((size_t)b * Nq + row) * a.Hq + sl.h) * D + 32 * dt + lq] = from_f32<TOUT>(oacc[dt][r]);
        }
    }
}

template <typename TIN, typename TOUT, int D, bool CAUSAL>
hipError_t launch_t(const UnfusedArgs &a, hipStream_t s) {
    const long long nsc = (long long)a.nmb * a.B * a.Hkv * a.nhg * a.nchunk;
    const long long nrow = ((long long)a.B * a.Hq * a.Nq + USLOT - 1) / USLOT;   // one wave per row
    const long long nrow4 = (long long)a.B * a.Hq * a.Nq;                          // four waves per row
    const long long npv = (long long)a.nmb * a.B * a.Hkv * a.nhg;
    if (nsc > 0x7fffffffLL || nrow4 > 0x7fffffffLL || npv > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((unfused_scores_kernel<TIN, D, CAUSAL>), dim3((unsigned)nsc), dim3(UNT), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // rows longer than one wave's 4096 held keys take two or four waves
    if (a.Nk <= 4096)
        hipLaunchKernelGGL((unfused_softmax_kernel<CAUSAL, 1>), dim3((unsigned)nrow), dim3(UNT), 0, s, a);
    else if (a.Nk <= 8192)
        hipLaunchKernelGGL((unfused_softmax_kernel<CAUSAL, 2>), dim3((unsigned)((nrow4 + 1) / 2)), dim3(UNT), 0, s, a);
    else
        hipLaunchKernelGGL((unfused_softmax_kernel<CAUSAL, 4>), dim3((unsigned)nrow4), dim3(UNT), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((unfused_pv_kernel<TIN, TOUT, D, CAUSAL>), dim3((unsigned)npv), dim3(UNT), 0, s, a);
    return hipGetLastError();
}

template <typename TIN, typename TOUT>
hipError_t launch_d(const Problem &p, const UnfusedArgs &a, hipStream_t s) {
    if (p.D == 64)
        return p.causal ? launch_t<TIN, TOUT, 64, true>(a, s) : launch_t<TIN, TOUT, 64, false>(a, s);
    return p.causal ? launch_t<TIN, TOUT, 128, true>(a, s) : launch_t<TIN, TOUT, 128, false>(a, s);
}

}  // namespace

size_t unfused_workspace_bytes(long long B, long long Hq, long long Nq, long long Nk) {
    if (B < 1 || Hq < 1 || Nq < 1 || Nk < 1) return 0;
    const long long nkp = (Nk + UKT - 1) / UKT * UKT;
    const long long lim = 0x7fffffffffffffffLL / 8;
    if (B > lim / Hq) return 0;
    const long long bh = B * Hq;
    if (bh > lim / Nq) return 0;
    const long long rows = bh * Nq;
    if (rows > lim / nkp) return 0;
    const long long n = rows * nkp;
    if (n > lim / 6) return 0;
    return (size_t)(n * 6);   // fp32 scores, then fp16 weights
}

bool unfused_supported(int D, fa_dtype_t in) { return (D == 64 || D == 128) && in != FA_F32; }

hipError_t launch_unfused(const Problem &p, void *workspace, hipStream_t stream) {
    UnfusedArgs a;
    a.q = p.q; a.k = p.k; a.v = p.v; a.o = p.o; a.lse = p.lse;
    a.B = p.B; a.Hq = p.Hq; a.Hkv = p.Hkv; a.Nq = p.Nq; a.Nk = p.Nk;
    a.NkP = (p.Nk + UKT - 1) / UKT * UKT;
    a.s = reinterpret_cast<float *>(workspace);
    a.p = reinterpret_cast<_Float16 *>(reinterpret_cast<char *>(workspace) +
                                       (size_t)p.B * p.Hq * p.Nq * a.NkP * sizeof(float));
    a.scale = p.scale;
    const int G = p.Hq / p.Hkv;
    a.HW = G % 4 == 0 ? 4 : (G % 2 == 0 ? 2 : 1);
    const int rows_wg = UR * (USLOT / a.HW);
    a.nmb = (p.Nq + rows_wg - 1) / rows_wg;
    a.nhg = G / a.HW;
    a.nchunk = (a.NkP / UKT + UCHUNK - 1) / UCHUNK;
    if (p.in == FA_BF16)
        return p.out == FA_F32 ? launch_d<bf16_t, float>(p, a, stream) : launch_d<bf16_t, __bf16>(p, a, stream);
    return p.out == FA_F32 ? launch_d<f16_t, float>(p, a, stream) : launch_d<f16_t, _Float16>(p, a, stream);
}

}  // namespace fa
