// fa_q8.hip -- Q8_0 matrix-vector product y = W x for the decode-time linear
// layers (Sec. 4.3: one token turns the projections into matrix-vector
// products; Q8_0 blocks of one binary16 scale followed by 32 int8 values,
// the layout of Sec. 7) on gfx950.
//
// The product is bound by HBM: every weight byte (34 per 32 weights) is read
// once, 2 flops per weight.  Each row is taken by L consecutive lanes of a
// wave (R = 64 / L rows per wave at a time; L of 16, 32 or 64, the one that
// leaves the fewest lanes idle in a row's last round).  When a row has an even number of blocks, every row and
// every pair of blocks (68 bytes) starts on a 4-byte boundary, and a lane's
// unit of work is one pair: four 16-byte loads and one 4-byte load
// (consecutive lanes take consecutive pairs, so a row streams contiguously).
// The two scales sit in the 16-bit halves of the first and ninth words; the
// first block's 32 values start 2 bytes into the pair and are realigned with
// funnel shifts.  Rows with an odd number of blocks take one block per lane:
// a 2-byte load of the scale and two 16-byte loads of the values at 2-byte
// aligned offsets (the unaligned access mode of the HSA runtime serves
// those).  All weight loads go through a buffer view of W that begins at the
// wave's current row group, so that rows past M and lanes without a unit
// read zeros without a branch and move no data.
//
// x is staged once per workgroup in LDS as fp32 (16-byte loads, all in flight
// together; four floats of padding after every 64, so that lanes reading x
// at a stride of 64 elements hit different banks); rows of more than 15168
// weights use 16-wave workgroups whose x takes up to the 160 KB of LDS a
// workgroup may hold, and for longer rows a lane loads the slice of x its
// unit needs.  Products are accumulated in
// fp32: each int8 value is widened exactly (one sign-extending convert),
// multiplied by x and summed per block, then scaled and added to the lane's
// sum; the L lanes of a row are summed with DPP row shifts and broadcasts.
//
// Latency decides the time of a matrix of a few MB, so a wave issues the
// loads of its first unit before the workgroup stages x, and the loads of
// its next unit before it computes the current one; no load sits behind a
// branch, so each wait covers exactly the unit it needs.  Finished rows go to
// a small LDS buffer and are written out in bursts.  The grid is capped at
// 1024 four-wave (or 512 sixteen-wave) workgroups and strides over row groups.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "fa_internal.h"

namespace fa {
namespace {

constexpr int Q8_NT = 256;              // threads per workgroup (4 waves)
constexpr int Q8_NT_WIDE = 1024;        // threads per workgroup for long rows (16 waves)
constexpr int Q8_XLDS_MAX = 15168;      // largest K staged in LDS by a 4-wave workgroup ((K + K/16)
                                        // floats and the result buffers within 64 KB)
constexpr int Q8_XLDS_WIDE_MAX = 37568; // largest K staged by a 16-wave workgroup (within the
                                        // 160 KB of LDS a workgroup may hold on gfx950)
constexpr int Q8_DEPTH = 2;             // units in flight per lane
constexpr int Q8_MAX_WG = 256 * 4;      // grid cap: workgroups (rows are strided beyond it)

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// LDS slot of x[k]: 4 floats of padding after every 64
__device__ __forceinline__ int xslot(int k) { return k + 4 * (k >> 6); }

__device__ __forceinline__ float half_bits_to_f32(unsigned bits) {
    return (float)__builtin_bit_cast(_Float16, (unsigned short)bits);
}

// 16 bytes of x (8 halves or 4 floats) -> fp32
template <typename TX> __device__ __forceinline__ void widen16(const u32x4 &v, float *o);
template <> __device__ __forceinline__ void widen16<float>(const u32x4 &v, float *o) {
#pragma unroll
    // the element is copied out first: bit-casting the vector element
    // expression itself has compiled to element 0 for every i
    for (int i = 0; i < 4; ++i) {
        const unsigned e = v[i];
        o[i] = __builtin_bit_cast(float, e);
    }
}
template <> __device__ __forceinline__ void widen16<_Float16>(const u32x4 &v, float *o) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        o[2 * i] = half_bits_to_f32(v[i] & 0xffffu);
        o[2 * i + 1] = half_bits_to_f32(v[i] >> 16);
    }
}
template <> __device__ __forceinline__ void widen16<__bf16>(const u32x4 &v, float *o) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        o[2 * i] = __builtin_bit_cast(float, v[i] << 16);
        o[2 * i + 1] = __builtin_bit_cast(float, v[i] & 0xffff0000u);
    }
}

// sum_j q_j * x_j over one block: four int8 values per word, x as fp32
__device__ __forceinline__ float block_dot(const unsigned *qw, const float *xs) {
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int w = (int)qw[i];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float q = (float)((w << (24 - 8 * e)) >> 24);   // sign-extended byte e
            acc = __builtin_fmaf(q, xs[4 * i + e], acc);
        }
    }
    return acc;
}

// One unit of work in registers: a pair of blocks (PAIR) or one block.
template <bool PAIR> struct Unit {
    unsigned u[PAIR ? 17 : 9];   // the pair's 17 words, or a block's 8 value words and its scale
};

// Loads of one unit through a buffer view (offsets past the view read as
// zero and move no data, so lanes without work load without branching).
// A pair is four 16-byte and one 4-byte load at a 4-byte aligned offset; a
// block is a 2-byte load of the scale and two 16-byte loads of the values at
// 2-byte aligned offsets.
template <bool PAIR>
__device__ __forceinline__ void load_unit(__amdgpu_buffer_rsrc_t rs, unsigned off, Unit<PAIR> &t) {
    if constexpr (PAIR) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16 * i, 0, 0));
            t.u[4 * i] = v[0];
            t.u[4 * i + 1] = v[1];
            t.u[4 * i + 2] = v[2];
            t.u[4 * i + 3] = v[3];
        }
        t.u[16] = __builtin_amdgcn_raw_buffer_load_b32(rs, off + 64, 0, 0);
    } else {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 2 + 16 * i, 0, 0));
            t.u[4 * i] = v[0];
            t.u[4 * i + 1] = v[1];
            t.u[4 * i + 2] = v[2];
            t.u[4 * i + 3] = v[3];
        }
        t.u[8] = __builtin_amdgcn_raw_buffer_load_b16(rs, off, 0, 0);
    }
}

template <bool PAIR>
__device__ __forceinline__ float unit_dot(const Unit<PAIR> &t, const float *x0) {
    if constexpr (PAIR) {
        // block 0: scale in bytes 0-1, values in bytes 2-33; block 1: scale in
        // bytes 34-35, values in bytes 36-67
        unsigned q0[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) q0[i] = __builtin_amdgcn_alignbit(t.u[i + 1], t.u[i], 16);
        const float d0 = half_bits_to_f32(t.u[0] & 0xffffu);
        const float d1 = half_bits_to_f32(t.u[8] >> 16);
        return __builtin_fmaf(d1, block_dot(t.u + 9, x0 + 32), d0 * block_dot(q0, x0));
    } else {
        return half_bits_to_f32(t.u[8]) * block_dot(t.u, x0);
    }
}

// x[k0 .. k0 + N) from global memory as fp32 (k0 a multiple of N; x 16-byte aligned)
template <typename TX, int N>
__device__ __forceinline__ void load_x_slice(const TX *x, int k0, float *o) {
    constexpr int E = 16 / sizeof(TX);
    const u32x4 *src = reinterpret_cast<const u32x4 *>(x + k0);
#pragma unroll
    for (int c = 0; c < N / E; ++c) widen16<TX>(src[c], o + c * E);
}

constexpr int Q8_YB = 64;   // per-wave LDS buffer of finished rows' results

// Where a lane finds x for its unit: staged once per workgroup in LDS, or
// loaded from global memory with each unit (K too large for LDS).  (Keeping
// each lane's slice of x in registers instead was slower: the slices are read
// by every lane, which doubles the requests a wave sends to L2.)
enum XMode { X_LDS = 0, X_GLOBAL = 1 };

// Sum of `v` over each run of L consecutive lanes (L = 16, 32 or 64, a
// wave-uniform value); the sum lands in the last lane of the run.  Rows of
// 16 lanes are summed by shifts within the row, then rows are joined by
// broadcasts of their last lane.
template <int CTRL, int ROWS, bool BOUND>
__device__ __forceinline__ float dpp_f32(float a) {   // lane value moved by a DPP pattern (0 where none)
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, a), CTRL, ROWS,
                                                                 0xf, BOUND));
}
__device__ __forceinline__ float segment_sum(float v, int L) {
    v += dpp_f32<0x111, 0xf, true>(v);   // row_shr:1
    v += dpp_f32<0x112, 0xf, true>(v);   // row_shr:2
    v += dpp_f32<0x114, 0xf, true>(v);   // row_shr:4
    v += dpp_f32<0x118, 0xf, true>(v);   // row_shr:8  (lane 15 of each row: the row's sum)
    if (L >= 32) v += dpp_f32<0x142, 0xa, false>(v);   // row_bcast:15 into rows 1 and 3
    if (L == 64) v += dpp_f32<0x143, 0xc, false>(v);   // row_bcast:31 into rows 2 and 3
    return v;
}

// Rows are taken in groups of R consecutive rows; the wave with global index
// wv takes groups wv, wv + NW, wv + 2 NW, ... (NW waves in the grid), and each
// group in `rounds` rounds of its lanes.  A lane keeps DEPTH units in flight:
// the loads of the unit DEPTH - 1 rounds ahead are issued before the current
// unit is computed.  Results of finished rows go to a per-wave LDS buffer and
// are written to y in bursts, so that stores seldom stand between loads.
// Launch constants, computed on the host (so that a wave starts its loads
// without integer divisions): L lanes per row (a power of two, 2^lgL), R =
// 64 / L = 2^lgR rows per group, units per row, rounds = ceil(units / L) and
// the number of row groups.
struct Q8Args {
    int M, K, L, lgL, lgR, units, rounds, groups;
};

template <typename TX, typename TY, bool PAIR, int XM, int DEPTH, int NT>
__global__ __launch_bounds__(NT) void q8_gemv_kernel(const unsigned char *__restrict__ w,
                                                        const TX *__restrict__ x, TY *__restrict__ y,
                                                        Q8Args a) {
    extern __shared__ __align__(16) float smem[];
    constexpr int UW = PAIR ? 64 : 32;                     // weights per unit
    constexpr unsigned UB = PAIR ? 68 : 34;                // bytes per unit
    constexpr int WAVES = NT / 64;
    const int M = a.M, K = a.K, L = a.L, units = a.units, rounds = a.rounds, groups = a.groups;
    const int nb = K / 32;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: the view lives in SGPRs
    const int R = 1 << a.lgR;
    const int sub = lane >> a.lgL, sl = lane & (L - 1);
    const int NW = (int)gridDim.x * WAVES;                  // waves in the grid
    const int wv = (int)blockIdx.x * WAVES + wave;          // this wave's index
    const int my_groups = wv < groups ? (int)((unsigned)(groups - 1 - wv) / (unsigned)NW) + 1 : 0;
    const int steps = my_groups * rounds;
    const unsigned row_bytes = (unsigned)nb * 34u;           // R rows fit in 2^31 - 1 bytes (host)
    const long long group_bytes = (long long)R * row_bytes;
    float *xs = smem;
    float *ybuf = smem + (XM == X_LDS ? K + K / 16 : 0) + wave * Q8_YB;

    // fetch cursor: the group's first byte and the bytes from there to the
    // end of W (the view, clamped to 31 bits), and the round within the group
    const unsigned char *fbase = w + (size_t)wv * (size_t)group_bytes;
    long long frem = (long long)M * row_bytes - (long long)wv * group_bytes;
    int fr = 0;
    auto fetch = [&](Unit<PAIR> &t) {
        unsigned rlo = (unsigned)frem, rhi = (unsigned)(frem >> 32);
        asm volatile("" : "+s"(rlo), "+s"(rhi));
        const int nrec = (int)((int)rhi < 0 ? 0u : rhi != 0u ? 0x7fffffffu
                                                            : __builtin_elementwise_min(rlo, 0x7fffffffu));
        const __amdgpu_buffer_rsrc_t rs =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned char *>(fbase), (short)0, nrec, 0x00020000);
        const int idx = sl + fr * L;
        const unsigned off = idx < units ? (unsigned)sub * row_bytes + UB * (unsigned)idx : 0x80000000u;
        load_unit<PAIR>(rs, off, t);
        if (++fr == rounds) {
            fr = 0;
            fbase += (size_t)NW * (size_t)group_bytes;
            frem -= (long long)NW * group_bytes;
        }
    };

    // x is staged in batches of 4 x NT 16-byte chunks.  The first batch's
    // loads are issued before the first unit's (the wait for an older load
    // does not cover a newer one, so x can be staged while W is in flight);
    // loads past the end of x read zero (a buffer view of x), so none sits
    // behind a branch.
    constexpr int E = 16 / sizeof(TX);
    const int C = K / E;                                    // 16-byte chunks of x
    const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<TX *>(x), (short)0, XM == X_LDS ? C * 16 : 0, 0x00020000);
    u32x4 xv[4];
    auto xload = [&](int c0) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            xv[i] = __builtin_bit_cast(
                u32x4, __builtin_amdgcn_raw_buffer_load_b128(xrs, (unsigned)(c0 + tid + i * NT) * 16u, 0, 0));
    };
    auto xstore = [&](int c0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = c0 + tid + i * NT;
            if (c < C) {
                float f[E];
                widen16<TX>(xv[i], f);
                float *dst = xs + xslot(c * E);             // E consecutive slots, 16-byte aligned
#pragma unroll
                for (int j = 0; j < E; j += 4)
                    *reinterpret_cast<f32x4 *>(dst + j) = f32x4{f[j], f[j + 1], f[j + 2], f[j + 3]};
            }
        }
    };
    if constexpr (XM == X_LDS) xload(0);

    Unit<PAIR> b[DEPTH];
#pragma unroll
    for (int i = 0; i < DEPTH - 1; ++i) fetch(b[i]);

    if constexpr (XM == X_LDS) {
        xstore(0);
        for (int c0 = 4 * NT; c0 < C; c0 += 4 * NT) {       // long rows: the further batches
            xload(c0);
            xstore(c0);
        }
        __syncthreads();
    }

    // compute cursor
    int g_done = 0;                // groups of this wave finished
    int g_flushed = 0;             // of which written to y
    int cr = 0;
    float acc = 0.f;
    auto flush = [&]() {
        const int n = (g_done - g_flushed) * R;            // entries in the buffer
        __builtin_amdgcn_wave_barrier();
        if (lane < n) {
            const long long g = wv + (long long)(g_flushed + (lane >> a.lgR)) * NW;
            const long long m = g * R + (lane & (R - 1));
            if (m < M) y[m] = (TY)ybuf[lane];
        }
        __builtin_amdgcn_wave_barrier();
        g_flushed = g_done;
    };
    auto compute = [&](const Unit<PAIR> &t) {
        const int idx = sl + cr * L;
        const bool valid = idx < units;                      // rows past M hold zeros
        const int k0 = (valid ? idx : units - 1) * UW;
        float part;
        if constexpr (XM == X_LDS) {
            part = unit_dot<PAIR>(t, (const float *)__builtin_assume_aligned(xs + xslot(k0), 16));
        } else {
            float xg[UW];
            load_x_slice<TX, UW>(x, k0, xg);
            part = unit_dot<PAIR>(t, xg);
        }
        acc += valid ? part : 0.f;
        if (++cr == rounds) {
            cr = 0;
            // group done: each row's sum over its L lanes lands in its last lane
            acc = segment_sum(acc, L);
            if (sl == L - 1) ybuf[(g_done - g_flushed) * R + sub] = acc;
            acc = 0.f;
            ++g_done;
            if ((g_done - g_flushed) * R == Q8_YB) flush();
        }
    };

    int t = 0;
    for (; t + DEPTH <= steps; t += DEPTH) {
#pragma unroll
        for (int s = 0; s < DEPTH; ++s) {
            fetch(b[(s + DEPTH - 1) % DEPTH]);
            compute(b[s]);
        }
    }
    // the last steps: their units are already in flight
#pragma unroll
    for (int s = 0; s < DEPTH - 1; ++s) {
        if (t < steps) {
            compute(b[s]);
            ++t;
        }
    }
    if (g_done > g_flushed) flush();
}

template <typename TX, typename TY, bool PAIR>
hipError_t launch_q8_t(const void *w, const void *x, void *y, int M, int K, hipStream_t s) {
    Q8Args a;
    a.M = M;
    a.K = K;
    a.units = PAIR ? K / 64 : K / 32;                   // lane work items per row
    a.L = 64;
    a.lgL = 6;
    {   // lanes per row: the fewest idle lanes in a row's last round (more
        // lanes per row on ties); rows short of work share a wave, as long as
        // the 64 / L rows of a group fit the 31-bit view a wave loads through
        const long long row_bytes = (long long)(K / 32) * 34;
        int best = 64, least = 1 << 30;
        for (int Lc = 64; Lc >= 16; Lc /= 2) {
            if ((64 / Lc) * row_bytes > 0x7fffffffLL) continue;
            const int idle = (a.units + Lc - 1) / Lc * Lc - a.units;
            if (idle < least) {
                least = idle;
                best = Lc;
            }
        }
        while (a.L > best) {
            a.L /= 2;
            --a.lgL;
        }
    }
    a.lgR = 6 - a.lgL;
    a.rounds = (a.units + a.L - 1) / a.L;
    a.groups = (int)(((long long)M + (1 << a.lgR) - 1) >> a.lgR);
    const long long waves_needed = a.groups;            // one wave per row group at most
    const auto *wp = reinterpret_cast<const unsigned char *>(w);
    const auto *xp = reinterpret_cast<const TX *>(x);
    auto *yp = reinterpret_cast<TY *>(y);
    const size_t xlds = (size_t)(K + K / 16) * sizeof(float);
    if (K <= Q8_XLDS_MAX || K > Q8_XLDS_WIDE_MAX) {
        long long blocks = (waves_needed + Q8_NT / 64 - 1) / (Q8_NT / 64);
        if (blocks > Q8_MAX_WG) blocks = Q8_MAX_WG;
        const dim3 grid((unsigned)blocks), block(Q8_NT);
        const size_t ylds = (size_t)(Q8_NT / 64) * Q8_YB * sizeof(float);
        if (K <= Q8_XLDS_MAX)
            hipLaunchKernelGGL((q8_gemv_kernel<TX, TY, PAIR, X_LDS, Q8_DEPTH, Q8_NT>), grid, block, xlds + ylds, s,
                               wp, xp, yp, a);
        else
            hipLaunchKernelGGL((q8_gemv_kernel<TX, TY, PAIR, X_GLOBAL, Q8_DEPTH, Q8_NT>), grid, block, ylds, s,
                               wp, xp, yp, a);
    } else {
        // long rows: x of more than 64 KB, staged once by a 16-wave workgroup
        // (one or two per CU, as the LDS allows)
        long long blocks = (waves_needed + Q8_NT_WIDE / 64 - 1) / (Q8_NT_WIDE / 64);
        if (blocks > Q8_MAX_WG / 2) blocks = Q8_MAX_WG / 2;
        const size_t ylds = (size_t)(Q8_NT_WIDE / 64) * Q8_YB * sizeof(float);
        hipLaunchKernelGGL((q8_gemv_kernel<TX, TY, PAIR, X_LDS, Q8_DEPTH, Q8_NT_WIDE>), dim3((unsigned)blocks),
                           dim3(Q8_NT_WIDE), xlds + ylds, s, wp, xp, yp, a);
    }
    return hipGetLastError();
}

template <typename TX, typename TY>
hipError_t launch_q8_xy(const void *w, const void *x, void *y, int M, int K, hipStream_t s) {
    return (K / 32) % 2 == 0 ? launch_q8_t<TX, TY, true>(w, x, y, M, K, s)
                             : launch_q8_t<TX, TY, false>(w, x, y, M, K, s);
}

}  // namespace

hipError_t launch_q8_gemv(const void *w, const void *x, void *y, int M, int K, fa_dtype_t xt,
                          fa_dtype_t yt, hipStream_t s) {
    if (xt == FA_F32) return launch_q8_xy<float, float>(w, x, y, M, K, s);
    if (xt == FA_F16)
        return yt == FA_F32 ? launch_q8_xy<_Float16, float>(w, x, y, M, K, s)
                            : launch_q8_xy<_Float16, _Float16>(w, x, y, M, K, s);
    return yt == FA_F32 ? launch_q8_xy<__bf16, float>(w, x, y, M, K, s)
                        : launch_q8_xy<__bf16, __bf16>(w, x, y, M, K, s);
}

}  // namespace fa
