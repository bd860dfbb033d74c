// fa_prefill.hip -- prefill attention forward on gfx950 matrix cores.
//
// Work split.  A workgroup owns NS (query head, 32-row block) slots that read
// the same key/value head: four, or at D = 64 eight on grids large enough to
// give every CU two or more eight-slot workgroups (1 and 2 exist for the
// packing ablation).  When the group size G = Hq/Hkv allows, up to four of the slots
// are query heads of one key/value group at the same rows -- the GPU form of
// the inter-head packing of Sec. 4.1.1 and the GQA reuse of Sec. 4.1.2 (iv):
// every K/V tile staged in LDS serves all slots of the workgroup, and slots
// of different heads share one causal extent; the other slots are
// consecutive row blocks.  Every wave handles 32 rows and 32 keys of each
// tile.  At D = 64 a slot has two waves (64-key tiles; wave kh takes keys
// 32 kh .. 32 kh + 31) whose states are merged through LDS at the end; at
// D = 128 one wave (32-key tiles).
//
// Per wave and tile, the blocked streaming softmax (Alg. 2 state carry over
// the per-key recurrence of Alg. 1):
//   S^T = K Q^T        32x32x16 MFMA; A = 32 K rows from LDS, B = the wave's
//                      32 query rows, kept in registers for the whole kernel
//   softmax            scores stay in the MFMA result registers; lane l owns
//                      query row l%32 (a row maximum needs one exchange with
//                      lane l^32); scale and log2(e) fold into one
//                      multiply-add ahead of exp2; weights packed to fp16
//   O^T += V^T P^T     32x32x16 fp16 MFMA; P straight from the score registers,
//                      V^T operands read from a transposed copy of the V tile
//                      that the staging step writes into LDS (a transposing
//                      LDS read is slower than the plain 16-byte read on
//                      gfx950, so the transpose is paid once per tile in the
//                      copy instead of once per wave)
// The exponent base only moves when a tile's weights against the current base
// grow too large (see the softmax step below), so the accumulator rescale is
// skipped on most tiles; sum and accumulator always share the base, so the
// result is unchanged.
// A wave's steps run in order; latency is hidden by the other waves of the
// SIMD (four-slot layouts: two 8-wave workgroups per CU at D = 64, four waves
// per SIMD within 128 VGPRs; three 4-wave ones at D = 128, three waves per
// SIMD within 168 VGPRs; their barriers are independent).  Matrix
// instructions are issued at raised wave priority.
// Masked scores are -inf and give exactly 0 (the exponent factor is kept
// strictly positive, also for scale = 0).  Keys past the end read as zero
// (buffer loads with the tensor's extent as the range) and are masked.
// Normalisation happens once, after the last tile.
#include <atomic>
#include <type_traits>

#include "fa_common.h"
#include "fa_internal.h"

namespace fa {
namespace {

constexpr int WR = 32;        // query rows per slot
constexpr int NSLOT = 4;      // slots per workgroup (the default; 1, 2 and 8 also exist)
constexpr float kMaxLaneSum = 4096.0f;   // largest 16-weight lane sum kept without a rescale

struct PrefillArgs {
    const void *q, *k, *v;
    void *o;
    float *lse;
    int B, Hq, Hkv, Nq, Nk;
    float c;          // max(|scale|, tiny) * log2(e), > 0
    unsigned qsign;   // 0x80008000 to negate q (scale < 0), else 0
    int HW;           // query heads per workgroup (1, 2, 4 or 8)
    int nmb;          // row blocks of 32 * (slots / HW) rows
    int nhg;          // head groups per key/value head (G / HW)
    int pair;         // 1: every workgroup is resident at once; order heavy/light pairs
    const int *seqlens;   // valid keys per batch element (NULL: Nk for all)
    const int *block_table;   // paged K/V: page of each key block (see Problem)
    int page_size, max_pages, num_pages;
};

// Tile shape per head size.  Every wave handles 32 query rows and 32 keys of
// a tile.  D = 64: two waves per slot (64-key tiles, key halves merged at the
// end), 8-wave workgroups of at most 128 VGPRs, two per CU (four waves per
// SIMD).  D = 128: the accumulator (64 VGPRs) and Q (32) leave no room for
// that, so one wave per slot (32-key tiles) and 4-wave workgroups, three per
// CU (three waves per SIMD, from independent workgroups; operands are read
// from LDS in small groups to fit 168 VGPRs).  Two LDS stages in both.
// NS, the slots per workgroup (all reading one key/value head, each staged
// tile serving all of them), is 4 or, at D = 64 on large grids, 8; 1 and 2
// exist for the packing ablation (fewer slots stage more per thread, so they
// hold fewer waves per SIMD).
template <int D, int NS = NSLOT> struct Cfg {
    static constexpr int NQ = D == 64 ? 2 : 1;       // waves per slot
    // waves per SIMD (what the registers allow; fewer slots stage more per thread)
    static constexpr int WPE = D == 64 ? (NS >= 4 ? 4 : NS == 2 ? 3 : 2) : (NS >= 4 ? 3 : NS == 2 ? 2 : 1);
    static constexpr int NWG = NS * NQ;              // waves per workgroup
    static constexpr int WPC = NWG >= 4 * WPE ? 1 : 4 * WPE / NWG;   // workgroups per CU (registers)
    static constexpr int BC = 32 * NQ;               // keys per tile
    static constexpr int NT = 64 * NWG;              // threads per workgroup
    static constexpr int NSTAGE = 2;                 // LDS tile stages
    static constexpr int KS = D + 8;                 // K row stride in 16-bit elements
    static constexpr int VTS = BC + 8;               // V^T row stride: BC key positions + pad
    static constexpr int KSZ = BC * KS;
    static constexpr int VSZ = D * VTS;
    static constexpr int STAGE = KSZ + VSZ;
    static constexpr int MERGE = NQ > 1 ? NS * (NQ / 2) * ((D / 32) * 16 + 2) * 64 : 0;  // floats
    static constexpr int WORDS = (NSTAGE * STAGE) > (2 * MERGE) ? NSTAGE * STAGE : 2 * MERGE;
    // Staging split.  KCH 16-byte K chunks and VUN V key-pair units (two
    // 16-byte loads each) per tile.  With two or more waves the upper half of
    // the workgroup stages K and the lower half V (SH threads each); a
    // one-wave workgroup stages both itself.
    static constexpr int KCH = BC * (D / 8);
    static constexpr int VUN = (BC / 2) * (D / 8);
    static constexpr bool BOTH = NT < 128;
    static constexpr int SH = BOTH ? NT : NT / 2;
    static constexpr int KPT = KCH / SH;                      // K chunks per staging thread
    static constexpr int VPT = VUN >= SH ? VUN / SH : 1;      // V units per staging thread
    static constexpr bool VPART = VUN < SH;                   // only the first VUN V threads stage
    static constexpr int SL = BOTH ? KPT + 2 * VPT : (KPT > 2 * VPT ? KPT : 2 * VPT);   // loads in flight
    static_assert(KCH % SH == 0 && (VUN % SH == 0 || SH % VUN == 0), "staging split");
};

template <typename TIN, typename TOUT, int D, int NS, bool CAUSAL, bool PAGED>
__global__ __launch_bounds__((Cfg<D, NS>::NT)) __attribute__((amdgpu_waves_per_eu((Cfg<D, NS>::WPE), (Cfg<D, NS>::WPE)))) void prefill_kernel(PrefillArgs a) {
    using S = typename TIN::scalar;
    using V8 = typename TIN::vec8;
    using SM = Cfg<D, NS>;
    constexpr int NSLOT = NS;
    constexpr int NQ = SM::NQ, BC = SM::BC, NT = SM::NT, NSTAGE = SM::NSTAGE;
    constexpr int KSTEPS = D / 16;          // QK^T contraction steps
    constexpr int DT = D / 32;              // output column tiles
    constexpr int CPR = D / 8;              // 16-byte chunks per row
    constexpr bool IN_BF16 = __is_same(TIN, bf16_t);

    __shared__ __attribute__((aligned(16))) unsigned short smem[SM::WORDS];

    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l = tid & 63, lq = l & 31, lh = l >> 5;
    const int kh = w / NSLOT, slot = w % NSLOT;   // kh: the wave's 32 keys of a tile
    const int RB = NSLOT / a.HW;
    const int per_mb = a.B * a.Hkv * a.nhg;
    const int bid = blockIdx.x;
    // Row block of this workgroup.  Latest rows (most keys) first, so that
    // the short causal blocks fill the tail; when the whole grid is resident
    // at once (two workgroups per CU), the first half of the grid takes the
    // long blocks in decreasing and the second half the short ones in
    // increasing length, so that the two workgroups sharing a CU carry about
    // the same total work.
    const int q_ = bid / per_mb, half_ = (a.nmb + 1) / 2;
    const int mb = (!a.pair || q_ < half_) ? a.nmb - 1 - q_ : q_ - half_;
    int rest = bid % per_mb;
    const int hg = rest % a.nhg;
    rest /= a.nhg;
    const int g = rest % a.Hkv;
    const int b = rest / a.Hkv;
    const int G = a.Hq / a.Hkv;
    const int hs = slot % a.HW, rs = slot / a.HW;
    const int h = g * G + hg * a.HW + hs;
    const int row0_wg = mb * (WR * RB);
    const int row0 = row0_wg + rs * WR;
    const int qi = row0 + lq;
    const int Nq = a.Nq;
    // Valid keys of this batch element: with per-sequence lengths the K/V
    // tensors hold a.Nk rows per batch element of which the first seqlens[b]
    // are valid, and the queries are the sequence's last Nq positions.
    const int Nk = a.seqlens ? min(max(a.seqlens[b], 0), a.Nk) : a.Nk;
    const int off = Nk - Nq;

    // Key extents: workgroup, this slot, and keys every row of the slot sees.
    const int last_wg = min(row0_wg + WR * RB, Nq) - 1;
    const int kend_wg = CAUSAL ? min(Nk, last_wg + off + 1) : Nk;
    const bool live = row0 < Nq;
    const int kfree_w = CAUSAL ? min(Nk, row0 + off + 1) : Nk;
    const int ntiles = (kend_wg + BC - 1) / BC;

    // Q rows of this lane (B operand of S^T = K Q^T).
    V8 qf[KSTEPS];
    {
        const int qrow = min(qi, Nq - 1);
        const S *qp = reinterpret_cast<const S *>(a.q) +
                      ((size_t)((size_t)b * Nq + qrow) * a.Hq + h) * D + 8 * lh;
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            uint4_t u = ld16(qp + 16 * ks);
            u ^= a.qsign;
            qf[ks] = as_vec8<V8>(u);
        }
    }

    // Tile staging.  The second half of the workgroup copies K rows (chunk
    // c = st + SH i: key c / CPR, 16-byte column chunk c % CPR); the first
    // half stages V transposed: unit u holds keys 2p, 2p+1 (p = u % KP) of
    // column chunk u / KP and writes eight 32-bit words, each the (2p, 2p+1)
    // pair of one column d, into row d of V^T (as fp16).  Within every 16 keys
    // the V^T positions swap bits 2 and 3 of the key index, so that the eight
    // keys one MFMA lane needs are contiguous.  (A one-wave workgroup stages
    // both: its loads 0 .. KPT-1 are K chunks, the rest V units.)  Loads are
    // buffer loads: the tile's first key row is the (scalar) base and each
    // lane keeps a fixed byte offset, so a step spends no vector instructions
    // on addresses.
    constexpr int SL = SM::SL;                  // 16-byte loads in flight per thread
    constexpr int KPT = SM::KPT, VPT = SM::VPT, SH = SM::SH;
    constexpr bool BOTH = SM::BOTH;
    constexpr int KP = BC / 2;                  // key pairs per tile
    static_assert(!(BOTH && PAGED), "paged K/V takes the default slots");
    // second half of the workgroup: K (wave-uniform).  The older wave of each
    // SIMD wins issue priority and finishes its softmax first, so it takes the
    // heavier V staging (the bf16 conversion) and the later one the K copy.
    const bool kgroup = !BOTH && w >= NT / 128;
    // the tensor this thread's loads read: K for the K half (and for the
    // K loads of a one-wave workgroup, whose V loads use vnext below)
    const S *kvbase = reinterpret_cast<const S *>((kgroup || BOTH) ? a.k : a.v) +
                      ((size_t)b * a.Nk * a.Hkv + g) * D;
    const int st = kgroup ? tid - NT / 2 : tid;
    // loads this thread issues per tile (wave-uniform; FULL: SL for every thread)
    constexpr bool FULL = !BOTH && KPT == 2 * VPT && !SM::VPART;
    const int nload = BOTH ? SL : kgroup ? KPT : (SM::VPART && st >= SM::VUN ? 0 : 2 * VPT);
    const size_t row_elems = (size_t)a.Hkv * D;      // elements between consecutive keys
    auto isk = [&](int i) __attribute__((always_inline)) { return BOTH ? i < KPT : kgroup; };
    // tile-relative key and column of load i of this thread
    auto lkey = [&](int i) __attribute__((always_inline)) {
        if (isk(i)) return (st + SH * i) / CPR;
        const int j = BOTH ? i - KPT : i;
        return 2 * ((st + SH * (j >> 1)) % KP) + (j & 1);
    };
    auto lcol = [&](int i) __attribute__((always_inline)) {
        if (isk(i)) return 8 * ((st + SH * i) % CPR);
        const int j = BOTH ? i - KPT : i;
        return 8 * ((st + SH * (j >> 1)) / KP);
    };
    int goff[SL];                                    // tile-relative byte offsets
#pragma unroll
    for (int i = 0; i < SL; ++i) goff[i] = (int)((lkey(i) * row_elems + lcol(i)) * sizeof(S));
    uint4_t sr[SL];   // the next tile, in flight during a step
    // Scalar state of the next tile to load: its first key row, and the bytes
    // from there to the end of the last key row (the buffer view, so that
    // keys past the end read as zero); both advance by one tile per load.
    const S *tnext = kvbase;
    // a one-wave workgroup: the first key row of the next V tile
    const S *vnext = reinterpret_cast<const S *>(a.v) + ((size_t)b * a.Nk * a.Hkv + g) * D;
    long long rem = (long long)(Nk - 1) * (long long)row_elems * (long long)sizeof(S) +
                    (long long)D * (long long)sizeof(S);
    // paged K/V: the pool of pages, at head g.  Tiles are loaded in order
    // and a page holds a whole number of tiles, so the page index and the
    // offset inside the page advance without a division.  The table entry of
    // the following page is read ahead with a vector load through a view of
    // this sequence's row of the table (entries past the row read as zero),
    // so it has arrived when the page is reached, and no scalar load (whose
    // counter the LDS reads share) is in flight during a step.
    const S *kvpool = reinterpret_cast<const S *>(kgroup ? a.k : a.v) + (size_t)g * D;
    const __amdgpu_buffer_rsrc_t trs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int *>(PAGED ? a.block_table + (size_t)b * a.max_pages : nullptr), (short)0,
        PAGED ? a.max_pages * 4 : 0, 0x00020000);
    const size_t page_elems = (size_t)a.page_size * row_elems;
    const int row_bytes = (int)(row_elems * sizeof(S));                 // paged: one key row of the pool
    const int tile_bytes = (BC - 1) * row_bytes + D * (int)sizeof(S);    // paged: view of a full tile
    int pidx = 0, poff = 0;   // page index and key offset of the next tile
    int tcur = 0, tnx = 0;    // table entries of pages pidx and pidx + 1
    if constexpr (PAGED) {
        tcur = __builtin_amdgcn_raw_buffer_load_b32(trs, 0, 0, 0);
        tnx = __builtin_amdgcn_raw_buffer_load_b32(trs, 4, 0, 0);
    }
    auto gload = [&](int kt) __attribute__((always_inline)) {   // the next tile (tiles are loaded in order; the argument is its first key)
        int nrec;
        if constexpr (PAGED) {
            // the tile's rows sit in one page (pages hold a multiple of 64
            // keys, tiles start at multiples of BC): at the start of a page
            // the base comes from the table (page numbers clamped into the
            // pool), within it the base advances by one tile per load; the
            // view ends after the last valid key of the tile (one tile's
            // extent, which fits 31 bits)
            if (poff == 0) {
                const int page = min(max(__builtin_amdgcn_readfirstlane(tcur), 0), a.num_pages - 1);
                tnext = kvpool + (size_t)page * page_elems;
            }
            const int left = Nk - kt;
            nrec = left >= BC ? tile_bytes : (left - 1) * row_bytes + D * (int)sizeof(S);
        } else {
            // view range, clamped to 31 bits (the tile's own extent always
            // fits); the halves are opaque so that the test stays two 32-bit
            // scalar compares instead of one 64-bit vector compare
            unsigned rlo = (unsigned)rem, rhi = (unsigned)(rem >> 32);
            asm volatile("" : "+s"(rlo), "+s"(rhi));
            nrec = (int)(rhi != 0u ? 0x7fffffffu : __builtin_elementwise_min(rlo, 0x7fffffffu));
        }
        const __amdgpu_buffer_rsrc_t rs =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<S *>(tnext), (short)0, nrec, 0x00020000);
        if constexpr (BOTH) {
            const __amdgpu_buffer_rsrc_t rv =
                __builtin_amdgcn_make_buffer_rsrc(const_cast<S *>(vnext), (short)0, nrec, 0x00020000);
#pragma unroll
            for (int i = 0; i < SL; ++i)
                sr[i] = __builtin_bit_cast(uint4_t, __builtin_amdgcn_raw_buffer_load_b128(i < KPT ? rs : rv, goff[i], 0, 0));
            vnext += (size_t)BC * row_elems;
        } else {
#pragma unroll
            for (int i = 0; i < SL; ++i)
                if (FULL || i < nload)
                    sr[i] = __builtin_bit_cast(uint4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, goff[i], 0, 0));
        }
        if constexpr (!PAGED) {
            tnext += (size_t)BC * row_elems;
            rem -= (long long)BC * (long long)row_elems * (long long)sizeof(S);
        } else {
            tnext += (size_t)BC * row_elems;
            poff += BC;
            const bool cross = poff == a.page_size;   // wave-uniform
            tcur = cross ? tnx : tcur;
            poff = cross ? 0 : poff;
            pidx += cross ? 1 : 0;
            tnx = __builtin_amdgcn_raw_buffer_load_b32(trs, (pidx + 1) * 4, 0, 0);
        }
    };
    // LDS destination (element offset inside a stage) of load i
    auto sdst = [&](int i) __attribute__((always_inline)) {
        if (isk(i)) return lkey(i) * SM::KS + lcol(i);
        const int key = lkey(i) & ~1;
        const int pos = (key & ~12) | ((key & 4) << 1) | ((key & 8) >> 1);
        return SM::KSZ + lcol(i) * SM::VTS + pos;   // row d = lcol + e, position pos
    };
    auto sstore_v = [&](unsigned short *stage, int i0) __attribute__((always_inline)) {   // the V unit of loads i0, i0 + 1
        unsigned *vt = reinterpret_cast<unsigned *>(stage + sdst(i0));
        const uint4_t x = sr[i0], y = sr[i0 + 1];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const unsigned xe = x[e >> 1], ye = y[e >> 1];
            unsigned w;
            if constexpr (IN_BF16) {
                const float fx = __uint_as_float((e & 1) ? (xe & 0xffff0000u) : (xe << 16));
                const float fy = __uint_as_float((e & 1) ? (ye & 0xffff0000u) : (ye << 16));
                w = pack_f16x2(fx, fy);
            } else {
                w = (e & 1) ? __builtin_amdgcn_perm(ye, xe, 0x07060302u)
                            : __builtin_amdgcn_perm(ye, xe, 0x05040100u);
            }
            vt[e * (SM::VTS / 2)] = w;
        }
    };
    auto sstore = [&](unsigned short *stage) __attribute__((always_inline)) {
        if constexpr (BOTH) {
#pragma unroll
            for (int i = 0; i < KPT; ++i) st16(stage + sdst(i), sr[i]);
#pragma unroll
            for (int u = 0; u < VPT; ++u) sstore_v(stage, KPT + 2 * u);
        } else if (kgroup) {
#pragma unroll
            for (int i = 0; i < KPT; ++i) st16(stage + sdst(i), sr[i]);
        } else if (FULL || nload > 0) {
#pragma unroll
            for (int u = 0; u < VPT; ++u) sstore_v(stage, 2 * u);
        }
    };

    float16_t oacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] = float16_t{};
    float m_run = -INFINITY;   // exponent base (log2 domain), same in lanes l and l^32
    float l_run = 0.f;         // this lane's part of the row sum
    float nbase = 0.f;         // -m_run, or 0 while the row has no base
    bool fresh = true;         // some row of the wave has no base yet (wave-uniform)

    const int k_lane = (32 * kh + lq) * SM::KS + 8 * lh;
    const int v_lane = SM::KSZ + lq * SM::VTS + 32 * kh + 8 * lh;
    auto stage_at = [&](int r) { return smem + r * SM::STAGE; };

    // K operands of this wave's 32 keys of the tile held in `stage`
    auto kread = [&](const unsigned short *stage, V8 (&ka)[KSTEPS]) {
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk)
            ka[kk] = as_vec8<V8>(*reinterpret_cast<const uint4_t *>(stage + k_lane + 16 * kk));
    };
    // S^T = K Q^T.  Matrix instructions are issued at raised wave priority:
    // the SIMD then starts a wave's next MFMA as soon as the matrix core is
    // free and fills the gaps with the other waves' vector work.
    auto qk = [&](const V8 (&ka)[KSTEPS]) {
        float16_t s = float16_t{};
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk) s = mfma32(ka[kk], qf[kk], s);
        __builtin_amdgcn_s_setprio(0);
        return s;
    };
    auto scores = [&](const unsigned short *stage) {
        V8 ka[KSTEPS];
        kread(stage, ka);
        return qk(ka);
    };

    // V^T operands of one tile for this wave (k-step order: dt, j)
    auto vread = [&](const unsigned short *stage, half8_t (&va)[KSTEPS]) {
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk)
            va[kk] = as_vec8<half8_t>(*reinterpret_cast<const uint4_t *>(
                stage + v_lane + 32 * (kk >> 1) * SM::VTS + 16 * (kk & 1)));
    };
    // O^T += V^T P^T with the weights of one tile (k-step j = keys 16 j .. 16 j
    // + 15 of the wave's half)
    auto pv = [&](const half8_t &p0, const half8_t &p1, const half8_t (&va)[KSTEPS]) {
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            oacc[dt] = mfma32(va[2 * dt], p0, oacc[dt]);
            oacc[dt] = mfma32(va[2 * dt + 1], p1, oacc[dt]);
        }
        __builtin_amdgcn_s_setprio(0);
    };

    // Grouped operand reads for D = 128: two k-steps per group, the next
    // group read from LDS while the current one multiplies, so that at most
    // four operand words are live instead of one per k-step (this keeps the
    // kernel within the 168 VGPRs of three waves per SIMD).
    auto scores_jit = [&](const unsigned short *stage) {
        float16_t s = float16_t{};
        V8 cur0, cur1, nxt0, nxt1;
        cur0 = as_vec8<V8>(*reinterpret_cast<const uint4_t *>(stage + k_lane));
        cur1 = as_vec8<V8>(*reinterpret_cast<const uint4_t *>(stage + k_lane + 16));
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int g = 0; g < KSTEPS / 2; ++g) {
            if (g + 1 < KSTEPS / 2) {
                nxt0 = as_vec8<V8>(*reinterpret_cast<const uint4_t *>(stage + k_lane + 32 * (g + 1)));
                nxt1 = as_vec8<V8>(*reinterpret_cast<const uint4_t *>(stage + k_lane + 32 * (g + 1) + 16));
            }
            s = mfma32(cur0, qf[2 * g], s);
            s = mfma32(cur1, qf[2 * g + 1], s);
            __builtin_amdgcn_sched_barrier(0);
            cur0 = nxt0;
            cur1 = nxt1;
        }
        __builtin_amdgcn_s_setprio(0);
        return s;
    };
    auto pv_jit = [&](const half8_t &p0, const half8_t &p1, const unsigned short *stage) {
        half8_t cur0, cur1, nxt0, nxt1;
        cur0 = as_vec8<half8_t>(*reinterpret_cast<const uint4_t *>(stage + v_lane));
        cur1 = as_vec8<half8_t>(*reinterpret_cast<const uint4_t *>(stage + v_lane + 16));
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            if (dt + 1 < DT) {
                nxt0 = as_vec8<half8_t>(*reinterpret_cast<const uint4_t *>(stage + v_lane + 32 * (dt + 1) * SM::VTS));
                nxt1 = as_vec8<half8_t>(*reinterpret_cast<const uint4_t *>(stage + v_lane + 32 * (dt + 1) * SM::VTS + 16));
            }
            oacc[dt] = mfma32(cur0, p0, oacc[dt]);
            oacc[dt] = mfma32(cur1, p1, oacc[dt]);
            __builtin_amdgcn_sched_barrier(0);
            cur0 = nxt0;
            cur1 = nxt1;
        }
        __builtin_amdgcn_s_setprio(0);
    };

    // hide keys of tile t that some row of the wave must not see
    auto mask = [&](float16_t &s, int t) {
        const int kw = t * BC + 32 * kh;        // first key of this wave's half
        if (kw + 32 > kfree_w) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int key = kw + 8 * (r >> 2) + 4 * lh + (r & 3);
                const bool vis = key < Nk && (!CAUSAL || key <= qi + off);
                s[r] = vis ? s[r] : -INFINITY;
            }
        }
    };

    // p = 2^(s c + nbase) for the 16 scores of the lane, packed to f16 in the
    // key order of the two PV k-steps
    auto exp_pack = [&](const float16_t &s, float nbase, half8_t &p0, half8_t &p1) {
        float p[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) p[r] = exp2_fast(__builtin_fmaf(s[r], a.c, nbase));
        p0 = pack_f16x8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
        p1 = pack_f16x8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
    };

    // row sum += the 16 f16 weights of the lane, in fp32 (dot products with (1, 1))
    auto add_sum = [&](float l, const half8_t &p0, const half8_t &p1) {
        const half2_t one = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
        for (int i = 0; i < 4; ++i)
            l = __builtin_amdgcn_fdot2(half2_t{p0[2 * i], p0[2 * i + 1]}, one, l, false);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            l = __builtin_amdgcn_fdot2(half2_t{p1[2 * i], p1[2 * i + 1]}, one, l, false);
        return l;
    };
    // Online softmax of one tile.  The weights are first formed against the
    // current base and kept if the lane's 16 weights add at most 4096 to its
    // row sum (every weight then fits f16 with room to spare and no rescale is
    // due; the row maximum is never formed).  Only when some row outgrows its
    // base that far (or a row has no base yet) is the row maximum taken, the
    // accumulator and row sum rescaled to it and the weights recomputed.  The
    // row sum adds, in fp32, the f16 weights that also feed the matrix product.
    auto softmax = [&](const float16_t &s, half8_t &p0, half8_t &p1) {
        exp_pack(s, nbase, p0, p1);
        const float l_old = l_run;
        l_run = add_sum(l_run, p0, p1);
        const bool over = !(l_run <= l_old + kMaxLaneSum);
        if (fresh || __builtin_amdgcn_ballot_w64(over) != 0) {
            float mx = max3(s[0], s[1], s[2]);
            mx = max3(mx, s[3], s[4]);
            mx = max3(mx, s[5], s[6]);
            mx = max3(mx, s[7], s[8]);
            mx = max3(mx, s[9], s[10]);
            mx = max3(mx, s[11], s[12]);
            mx = max3(mx, s[13], s[14]);
            mx = __builtin_fmaxf(mx, s[15]);
            mx = pair_max(mx);
            const float m_new = __builtin_fmaxf(m_run, mx * a.c);
            const float alpha = (m_new == -INFINITY) ? 1.f : exp2_fast(m_run - m_new);
            m_run = m_new;
            nbase = (m_new == -INFINITY) ? 0.f : -m_new;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
            exp_pack(s, nbase, p0, p1);
            l_run = add_sum(l_old * alpha, p0, p1);
            fresh = __builtin_amdgcn_ballot_w64(m_run == -INFINITY) != 0;
        }
    };

    // Tile loop: one tile per step, in order -- scores, softmax, PV.  The next
    // tile's global loads are in flight during the step, and it is written
    // to the other LDS stage at the end of the step.  The latencies of a
    // step are hidden by the waves of the other workgroups on the CU, whose
    // barriers are independent of this one's.
    if (ntiles > 0) {
        gload(0);
        sstore(stage_at(0));
    }
    __syncthreads();
    auto step = [&](int i, auto R) {   // R: stage of tile i (i % 2)
        constexpr int r = decltype(R)::value;
        const bool more = i + 1 < ntiles;
        // the next tile's loads are issued after the K operand reads (their
        // scalar set-up then overlaps the LDS latency, and at D = 128 their
        // registers are not live across the QK^T product)
        float16_t s = D == 128 ? scores_jit(stage_at(r)) : scores(stage_at(r));
        if (more) gload((i + 1) * BC);
        mask(s, i);
        half8_t p0, p1;
        half8_t va[KSTEPS];
        // D = 64: the V operands are read before the softmax, so that their
        // LDS latency is not on the step's critical path
        if constexpr (D == 64) vread(stage_at(r), va);
        softmax(s, p0, p1);
        if constexpr (D == 128) {
            pv_jit(p0, p1, stage_at(r));
        } else {
            pv(p0, p1, va);
        }
        if (more) sstore(stage_at(r ^ 1));
        __syncthreads();
    };
    int i = 0;
    for (; i + 2 <= ntiles; i += 2) {   // unrolled by two: stage offsets are constants
        step(i, std::integral_constant<int, 0>{});
        step(i + 1, std::integral_constant<int, 1>{});
    }
    if (i < ntiles) step(i, std::integral_constant<int, 0>{});
    __syncthreads();   // the merge below reuses the stage memory

    // ---- merge the two key halves of each slot through LDS
    float *mf = reinterpret_cast<float *>(smem);
    constexpr int NV = DT * 16 + 2;
    float *mine = mf + (slot * NV) * 64 + l;
    if (NQ == 2 && kh == 1) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int r = 0; r < 16; ++r) mine[(dt * 16 + r) * 64] = oacc[dt][r];
        mine[(DT * 16) * 64] = m_run;
        mine[(DT * 16 + 1) * 64] = l_run;
    }
    if (NQ == 2) __syncthreads();
    if (kh != 0 || !live) return;
    if (NQ == 2) {
        const float m1 = mine[(DT * 16) * 64];
        const float l1 = mine[(DT * 16 + 1) * 64];
        const float M = __builtin_fmaxf(m_run, m1);
        const float a0 = (m_run == -INFINITY) ? 0.f : exp2_fast(m_run - M);
        const float a1 = (m1 == -INFINITY) ? 0.f : exp2_fast(m1 - M);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                oacc[dt][r] = a0 * oacc[dt][r] + a1 * mine[(dt * 16 + r) * 64];
        l_run = a0 * l_run + a1 * l1;
        m_run = M;
    }
    const float l_tot = pair_sum(l_run);
    // a row with no visible key (only with per-sequence lengths) gives 0 and
    // a log-sum-exp of -inf
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    if (qi < Nq) {
        TOUT *op = reinterpret_cast<TOUT *>(a.o) + ((size_t)((size_t)b * Nq + qi) * a.Hq + h) * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int d0 = 32 * dt + 8 * i + 4 * lh;
                if constexpr (sizeof(TOUT) == 4) {
                    *reinterpret_cast<float4_t *>(op + d0) =
                        float4_t{oacc[dt][4 * i] * inv, oacc[dt][4 * i + 1] * inv,
                                 oacc[dt][4 * i + 2] * inv, oacc[dt][4 * i + 3] * inv};
                } else {
                    typedef TOUT t4 __attribute__((ext_vector_type(4)));
                    t4 u;
#pragma unroll
                    for (int e = 0; e < 4; ++e) u[e] = from_f32<TOUT>(oacc[dt][4 * i + e] * inv);
                    *reinterpret_cast<t4 *>(op + d0) = u;
                }
            }
        }
        if (a.lse && lh == 0)
            a.lse[((size_t)b * a.Hq + h) * Nq + qi] = l_tot > 0.f ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
    }
}

// Compute units of the current device (cached per device; 0 if unknown).
int cu_count() {
    static std::atomic<int> cached[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    int n = cached[dev].load(std::memory_order_relaxed);
    if (n == 0 && hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess)
        cached[dev].store(n, std::memory_order_relaxed);
    return n;
}

template <typename TIN, typename TOUT, int D, int NS, bool CAUSAL>
hipError_t launch_t(const Problem &p, hipStream_t stream) {
    using SM = Cfg<D, NS>;
    PrefillArgs a;
    a.q = p.q; a.k = p.k; a.v = p.v; a.o = p.o; a.lse = p.lse;
    a.B = p.B; a.Hq = p.Hq; a.Hkv = p.Hkv; a.Nq = p.Nq; a.Nk = p.Nk;
    a.seqlens = p.seqlens;
    a.block_table = p.block_table;
    a.page_size = p.page_size;
    a.max_pages = p.max_pages;
    a.num_pages = p.num_pages;
    // A zero scale keeps a tiny positive factor: every visible exponent is then
    // exactly 0 in fp32, and masked (-inf) scores still give 0.
    a.c = __builtin_fmaxf(__builtin_fabsf(p.scale), 1e-30f) * kLog2e;
    a.qsign = p.scale < 0.f ? 0x80008000u : 0u;
    const int G = p.Hq / p.Hkv;
    // query heads per workgroup: the requested packing, else the most heads
    // of one key/value group (up to 4) that fill the slots evenly
    int hw = 1;
    for (int c = 2; c <= (NS < 4 ? NS : 4); c *= 2)
        if (NS % c == 0 && G % c == 0) hw = c;
    a.HW = p.hw > 0 ? p.hw : hw;
    const int RB = NS / a.HW;
    a.nmb = (p.Nq + WR * RB - 1) / (WR * RB);
    a.nhg = G / a.HW;
    a.pair = 0;
    const long long nblocks = (long long)a.nmb * p.B * p.Hkv * a.nhg;
    if (nblocks <= 0) return hipSuccess;
    if (nblocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    if (p.causal) a.pair = nblocks <= (long long)SM::WPC * cu_count() ? 1 : 0;
    if constexpr (NS == NSLOT) {
        if (p.block_table) {
            hipLaunchKernelGGL((prefill_kernel<TIN, TOUT, D, NS, CAUSAL, true>), dim3((unsigned)nblocks),
                               dim3(SM::NT), 0, stream, a);
            return hipGetLastError();
        }
    } else if (p.block_table) {
        return hipErrorInvalidValue;   // paged K/V takes the default slots
    }
    hipLaunchKernelGGL((prefill_kernel<TIN, TOUT, D, NS, CAUSAL, false>), dim3((unsigned)nblocks),
                       dim3(SM::NT), 0, stream, a);
    return hipGetLastError();
}

// Default slots per workgroup: 8 at D = 64 when the grid of 8-slot
// workgroups (the default heads, up to 4, times 2 row blocks) still gives
// every CU at least two of them -- each staged tile then serves twice the
// rows (MQA prefill, 16 heads on one K/V head, 16384 rows: 578 against
// 602 us); 4 otherwise: on a small grid (the 32-head, 2048-row GQA prefill:
// 39 against 31.5 us), at D = 128 (the eight-slot workgroup holds two waves
// per SIMD instead of three; on the 32-head, 4096-row prefill it ran from
// 2 % faster to 3 % slower depending on the box), for paged K/V and when the
// caller fixed the heads per workgroup.
int default_slots(const Problem &p) {
    if (p.D != 64 || p.block_table || p.hw > 0) return NSLOT;
    const int G = p.Hq / p.Hkv;
    const int hw = G % 4 == 0 ? 4 : G % 2 == 0 ? 2 : 1;
    const int rows = WR * (8 / hw);
    const long long nblocks = (long long)((p.Nq + rows - 1) / rows) * p.B * p.Hkv * (G / hw);
    const int cus = cu_count();
    return cus > 0 && nblocks >= 2LL * cus ? 8 : NSLOT;
}

template <typename TIN, typename TOUT, int D, bool CAUSAL>
hipError_t launch_s(const Problem &p, hipStream_t s) {
    switch (p.slots > 0 ? p.slots : default_slots(p)) {
    case 1: return launch_t<TIN, TOUT, D, 1, CAUSAL>(p, s);
    case 2: return launch_t<TIN, TOUT, D, 2, CAUSAL>(p, s);
    case 8: return launch_t<TIN, TOUT, D, 8, CAUSAL>(p, s);
    default: return launch_t<TIN, TOUT, D, NSLOT, CAUSAL>(p, s);
    }
}

template <typename TIN, typename TOUT>
hipError_t launch_d(const Problem &p, hipStream_t s) {
    if (p.D == 64) return p.causal ? launch_s<TIN, TOUT, 64, true>(p, s)
                                   : launch_s<TIN, TOUT, 64, false>(p, s);
    return p.causal ? launch_s<TIN, TOUT, 128, true>(p, s) : launch_s<TIN, TOUT, 128, false>(p, s);
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
