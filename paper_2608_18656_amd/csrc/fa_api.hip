// fa_api.hip -- the exported C entry points: argument validation, dispatch to
// the prefill / decode / generic / unfused kernels, and the decode workspace.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <mutex>
#include <vector>

#include "../../include/fa.h"
#include "fa_checks.h"
#include "fa_internal.h"

namespace {

using fa::esize;
using fa::overlaps;
using fa::validate_core;

// Device workspace for the split-KV partial results.  Library-owned buffers
// are kept per (device, stream), so that calls on different streams never
// share one; a buffer that is outgrown is retired, not freed (an earlier call
// or a captured graph may still use it) until fa_release_workspace().  No
// buffer is allocated while the stream is being captured.  A caller-owned
// workspace set with fa_set_workspace() replaces them for its device.
struct OwnedWs {
    int dev;
    hipStream_t stream;
    void *ptr;
    size_t bytes;
};
struct Retired {
    int dev;
    void *ptr;
};
constexpr int kMaxDevices = 64;
struct UserWs {
    void *ptr = nullptr;
    size_t bytes = 0;
};
UserWs g_user[kMaxDevices];
std::vector<OwnedWs> g_owned;
std::vector<Retired> g_retired;
std::mutex g_ws_mu;

fa_status_t get_workspace(size_t need, hipStream_t stream, void **out, bool *user) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return FA_ERR_HIP;
    std::lock_guard<std::mutex> lk(g_ws_mu);
    *user = g_user[dev].ptr != nullptr;
    if (*user) {
        if (g_user[dev].bytes < need) return FA_ERR_WORKSPACE;
        *out = g_user[dev].ptr;
        return FA_OK;
    }
    OwnedWs *cur = nullptr;
    for (OwnedWs &w : g_owned)
        if (w.dev == dev && w.stream == stream) cur = &w;
    if (cur && cur->bytes >= need) {
        *out = cur->ptr;
        return FA_OK;
    }
    // a new buffer is needed: never inside stream capture (the allocation
    // would invalidate it)
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &cs) != hipSuccess) {
        (void)hipGetLastError();
        return FA_ERR_WORKSPACE;
    }
    if (cs != hipStreamCaptureStatusNone) return FA_ERR_WORKSPACE;
    const size_t sz = need < ((size_t)1 << 20) ? ((size_t)1 << 20) : need;
    void *ptr = nullptr;
    if (hipMalloc(&ptr, sz) != hipSuccess) {
        (void)hipGetLastError();
        return FA_ERR_WORKSPACE;
    }
    if (cur) {
        g_retired.push_back(Retired{dev, cur->ptr});
        cur->ptr = ptr;
        cur->bytes = sz;
    } else {
        g_owned.push_back(OwnedWs{dev, stream, ptr, sz});
    }
    *out = ptr;
    return FA_OK;
}

// A caller-owned workspace passed with one call (the *_ws entry points).
struct CallWs {
    void *ptr;
    size_t bytes;
};

// Fixed device scratch of fa_fwd_splitkv_noalloc: the split-KV partial results
// of its calls live here (each GPU holds its own copy until the process
// ends).  Host code never passes `scratch` itself to a kernel (on the host
// that name is a stand-in, not a device address): the address of the
// device's copy is read once per device with hipGetSymbolAddress and kept.
constexpr size_t kScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
void *g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of the current device's scratch (read on the first call per
// device, with that device current).
fa_status_t scratch_address(void **out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return FA_ERR_HIP;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) {
            (void)hipGetLastError();
            return FA_ERR_HIP;
        }
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return FA_OK;
}

struct Paging {
    const int *block_table = nullptr;
    int page_size = 0, max_pages = 0, num_pages = 0;
};

fa_status_t run(const void *q, const void *k, const void *v, void *o, float *lse, int B, int Hq,
                int Hkv, int Nq, int Nk, int D, int causal, float scale, void *stream,
                fa_dtype_t in, fa_dtype_t out, int splits_req, int hw_req = 0,
                const int *seqlens = nullptr, const Paging &pg = Paging(),
                const CallWs *cws = nullptr, int slots_req = 0) {
    const long long kv_rows = pg.block_table ? (long long)pg.num_pages * pg.page_size : -1;
    fa_status_t st = validate_core(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, in, out, kv_rows);
    if (st != FA_OK) return st;
    if (splits_req < 0 || splits_req > FA_MAX_SPLITS) return FA_ERR_SPLITS;
    const int slots = slots_req > 0 ? slots_req : 4;
    if (!(slots_req == 0 || slots_req == 1 || slots_req == 2 || slots_req == 4 || slots_req == 8) ||
        !(hw_req == 0 || hw_req == 1 || hw_req == 2 || hw_req == 4 || hw_req == 8) ||
        (hw_req > 0 && ((Hq / Hkv) % hw_req != 0 || slots % hw_req != 0)))
        return FA_ERR_PACKING;
    fa::Problem p{q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, in, out, hw_req, slots_req, seqlens,
                  pg.block_table, pg.page_size, pg.max_pages, pg.num_pages};
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipError_t e;
    if (fa::decode_supported(Nq, D, in)) {
        const int S = splits_req > 0 ? splits_req : fa::decode_default_splits(B, Hq, Hkv, Nk, D);
        const size_t need = fa::decode_workspace_bytes(B, Hq, D, S);
        void *ws = nullptr;
        bool user = false;
        if (cws) {   // this call's own workspace: checked here, never allocated
            if (!cws->ptr) return FA_ERR_NULL;
            if (reinterpret_cast<uintptr_t>(cws->ptr) & 15) return FA_ERR_ALIGN;
            if (cws->bytes < need) return FA_ERR_WORKSPACE;
            ws = cws->ptr;
            user = true;
        } else {
            st = get_workspace(need, s, &ws, &user);
            if (st != FA_OK) return st;
        }
        if (user) {   // a caller-owned workspace must not overlap the call's tensors
            const size_t qb = (size_t)B * Nq * Hq * D * esize(in);
            const size_t kb = (size_t)(kv_rows < 0 ? (long long)B * Nk : kv_rows) * Hkv * D * esize(in);
            const size_t ob = (size_t)B * Nq * Hq * D * esize(out), lb = (size_t)B * Hq * Nq * sizeof(float);
            if (overlaps(ws, need, q, qb) || overlaps(ws, need, k, kb) || overlaps(ws, need, v, kb) ||
                overlaps(ws, need, o, ob) || (lse && overlaps(ws, need, lse, lb)))
                return FA_ERR_ALIAS;
        }
        e = fa::launch_decode(p, S, ws, s);
    } else if (fa::prefill_supported(D, in)) {
        e = fa::launch_prefill(p, s);
    } else {
        e = fa::launch_generic(p, s);
    }
    return e == hipSuccess ? FA_OK : FA_ERR_HIP;
}

}  // namespace

extern "C" {

const char *fa_status_string(fa_status_t s) {
    switch (s) {
    case FA_OK: return "FA_OK";
    case FA_ERR_NULL: return "FA_ERR_NULL: q, k, v or o is NULL";
    case FA_ERR_DIM: return "FA_ERR_DIM: a size is < 1 or the tensors are too large";
    case FA_ERR_GQA_RATIO: return "FA_ERR_GQA_RATIO: Hq is not a multiple of Hkv";
    case FA_ERR_HEAD_DIM: return "FA_ERR_HEAD_DIM: D must be a multiple of 8 and at most 256";
    case FA_ERR_CAUSAL_SHAPE: return "FA_ERR_CAUSAL_SHAPE: causal requires Nq <= Nk";
    case FA_ERR_SCALE: return "FA_ERR_SCALE: scale is NaN or infinite";
    case FA_ERR_ALIGN: return "FA_ERR_ALIGN: a tensor pointer is misaligned";
    case FA_ERR_ALIAS: return "FA_ERR_ALIAS: o or lse overlaps another tensor";
    case FA_ERR_DTYPE: return "FA_ERR_DTYPE: unsupported dtype combination";
    case FA_ERR_WORKSPACE:
        return "FA_ERR_WORKSPACE: workspace allocation failed or not allowed during stream capture, or a caller-owned workspace is too small";
    case FA_ERR_HIP: return "FA_ERR_HIP: HIP runtime or launch error";
    case FA_ERR_SPLITS: return "FA_ERR_SPLITS: num_splits out of range";
    case FA_ERR_PACKING:
        return "FA_ERR_PACKING: slots_per_workgroup must be 0, 1, 2, 4 or 8; heads_per_workgroup 0, 1, 2, 4 or "
               "8, dividing Hq / Hkv and the slots";
    }
    return "unknown fa_status_t";
}

int fa_version(void) { return (0 << 16) | (1 << 8) | 0; }

fa_status_t fa_validate(const void *q, const void *k, const void *v, const void *o,
                        const float *lse, int B, int Hq, int Hkv, int Nq, int Nk, int D,
                        int causal, float scale, fa_dtype_t in, fa_dtype_t out) {
    return validate_core(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, in, out, -1);
}

fa_status_t fa_fwd(const void *q, const void *k, const void *v, void *o, float *lse, int B,
                   int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale, void *stream,
                   fa_dtype_t in_dtype, fa_dtype_t out_dtype) {
    return run(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, in_dtype, out_dtype,
               0);
}

fa_status_t fa_fwd_f16(const void *q, const void *k, const void *v, void *o, float *lse, int B,
                       int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale,
                       void *stream) {
    return run(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, FA_F16, FA_F16, 0);
}

fa_status_t fa_fwd_bf16(const void *q, const void *k, const void *v, void *o, float *lse, int B,
                        int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale,
                        void *stream) {
    return run(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, FA_BF16, FA_BF16,
               0);
}

fa_status_t fa_fwd_f32(const void *q, const void *k, const void *v, void *o, float *lse, int B,
                       int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale,
                       void *stream) {
    return run(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, FA_F32, FA_F32, 0);
}

fa_status_t fa_fwd_splitkv(const void *q, const void *k, const void *v, void *o, float *lse,
                           int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale,
                           void *stream, fa_dtype_t in_dtype, fa_dtype_t out_dtype,
                           int num_splits) {
    return run(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, in_dtype, out_dtype,
               num_splits);
}

fa_status_t fa_fwd_packed(const void *q, const void *k, const void *v, void *o, float *lse,
                          int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale,
                          void *stream, fa_dtype_t in_dtype, fa_dtype_t out_dtype,
                          int heads_per_workgroup) {
    return run(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, in_dtype, out_dtype,
               0, heads_per_workgroup);
}

}  // extern "C"

namespace {

fa_status_t kvcache(const void *q, const void *k, const void *v, void *o, float *lse,
                    const int *seqlens_k, int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal,
                    float scale, void *stream, fa_dtype_t in_dtype, fa_dtype_t out_dtype,
                    const CallWs *cws) {
    if (!seqlens_k) return FA_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(seqlens_k) & 3) return FA_ERR_ALIGN;
    if (B >= 1 && o && Hq >= 1 && Nq >= 1 && D >= 1) {
        const size_t ob = (size_t)B * Nq * Hq * D * esize(out_dtype);
        if (overlaps(o, ob, seqlens_k, (size_t)B * sizeof(int)) ||
            (lse && overlaps(lse, (size_t)B * Hq * Nq * sizeof(float), seqlens_k, (size_t)B * sizeof(int))))
            return FA_ERR_ALIAS;
    }
    return run(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, in_dtype, out_dtype, 0,
               0, seqlens_k, Paging(), cws);
}

fa_status_t kvcache_paged(const void *q, const void *k_pages, const void *v_pages, void *o,
                          float *lse, const int *seqlens_k, const int *block_table, int B, int Hq,
                          int Hkv, int Nq, int D, int page_size, int max_pages, int num_pages,
                          int causal, float scale, void *stream, fa_dtype_t in_dtype,
                          fa_dtype_t out_dtype, const CallWs *cws) {
    if (!seqlens_k || !block_table) return FA_ERR_NULL;
    if (page_size < 64 || page_size % 64 != 0 || max_pages < 1 || num_pages < 1 ||
        (long long)page_size * max_pages > 0x7fffffffLL || (long long)B * max_pages > 0x7fffffffLL)
        return FA_ERR_DIM;
    if ((reinterpret_cast<uintptr_t>(seqlens_k) & 3) || (reinterpret_cast<uintptr_t>(block_table) & 3))
        return FA_ERR_ALIGN;
    const int Nk = page_size * max_pages;
    // only the matrix-core kernels read pages
    if (in_dtype != FA_F16 && in_dtype != FA_BF16) {
        const fa_status_t st = validate_core(q, k_pages, v_pages, o, lse, B, Hq, Hkv, Nq, Nk, D, causal,
                                             scale, in_dtype, out_dtype, (long long)num_pages * page_size);
        return st != FA_OK ? st : FA_ERR_DTYPE;
    }
    if (D != 64 && D != 128) {
        const fa_status_t st = validate_core(q, k_pages, v_pages, o, lse, B, Hq, Hkv, Nq, Nk, D, causal,
                                             scale, in_dtype, out_dtype, (long long)num_pages * page_size);
        return st != FA_OK ? st : FA_ERR_HEAD_DIM;
    }
    if (B >= 1 && o && Hq >= 1 && Nq >= 1) {
        const size_t ob = (size_t)B * Nq * Hq * D * esize(out_dtype);
        const size_t lb = (size_t)B * Hq * Nq * sizeof(float);
        const size_t sb = (size_t)B * sizeof(int), tb = (size_t)B * max_pages * sizeof(int);
        if (overlaps(o, ob, seqlens_k, sb) || overlaps(o, ob, block_table, tb) ||
            (lse && (overlaps(lse, lb, seqlens_k, sb) || overlaps(lse, lb, block_table, tb))))
            return FA_ERR_ALIAS;
    }
    Paging pg;
    pg.block_table = block_table;
    pg.page_size = page_size;
    pg.max_pages = max_pages;
    pg.num_pages = num_pages;
    return run(q, k_pages, v_pages, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, in_dtype,
               out_dtype, 0, 0, seqlens_k, pg, cws);
}

}  // namespace

extern "C" {

fa_status_t fa_fwd_slots(const void *q, const void *k, const void *v, void *o, float *lse, int B,
                         int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale, void *stream,
                         fa_dtype_t in_dtype, fa_dtype_t out_dtype, int slots_per_workgroup,
                         int heads_per_workgroup) {
    return run(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, in_dtype, out_dtype, 0,
               heads_per_workgroup, nullptr, Paging(), nullptr, slots_per_workgroup);
}

fa_status_t fa_fwd_kvcache(const void *q, const void *k, const void *v, void *o, float *lse,
                           const int *seqlens_k, int B, int Hq, int Hkv, int Nq, int Nk, int D,
                           int causal, float scale, void *stream, fa_dtype_t in_dtype,
                           fa_dtype_t out_dtype) {
    return kvcache(q, k, v, o, lse, seqlens_k, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, in_dtype,
                   out_dtype, nullptr);
}

fa_status_t fa_fwd_kvcache_paged(const void *q, const void *k_pages, const void *v_pages, void *o,
                                 float *lse, const int *seqlens_k, const int *block_table, int B,
                                 int Hq, int Hkv, int Nq, int D, int page_size, int max_pages,
                                 int num_pages, int causal, float scale, void *stream,
                                 fa_dtype_t in_dtype, fa_dtype_t out_dtype) {
    return kvcache_paged(q, k_pages, v_pages, o, lse, seqlens_k, block_table, B, Hq, Hkv, Nq, D,
                         page_size, max_pages, num_pages, causal, scale, stream, in_dtype, out_dtype,
                         nullptr);
}

fa_status_t fa_fwd_ws(const void *q, const void *k, const void *v, void *o, float *lse, int B,
                      int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale, void *stream,
                      fa_dtype_t in_dtype, fa_dtype_t out_dtype, int num_splits, void *workspace,
                      size_t workspace_bytes) {
    const CallWs cws{workspace, workspace_bytes};
    return run(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, in_dtype, out_dtype,
               num_splits, 0, nullptr, Paging(), &cws);
}

fa_status_t fa_fwd_splitkv_noalloc(const void *q, const void *k, const void *v, void *o, float *lse,
                                   int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal,
                                   float scale, void *stream, fa_dtype_t in_dtype,
                                   fa_dtype_t out_dtype, int num_splits) {
    // the argument checks of fa_fwd_splitkv, then the size of the partial
    // results against the scratch, all before any HIP call
    fa_status_t st = validate_core(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, in_dtype,
                                   out_dtype, -1);
    if (st != FA_OK) return st;
    if (num_splits < 0 || num_splits > FA_MAX_SPLITS) return FA_ERR_SPLITS;
    CallWs cws{nullptr, 0};
    if (fa::decode_supported(Nq, D, in_dtype)) {
        const int S = num_splits > 0 ? num_splits : fa::decode_default_splits(B, Hq, Hkv, Nk, D);
        if (fa::decode_workspace_bytes(B, Hq, D, S) > kScratchBytes) return FA_ERR_WORKSPACE;
        st = scratch_address(&cws.ptr);
        if (st != FA_OK) return st;
        cws.bytes = kScratchBytes;
    }
    return run(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, in_dtype, out_dtype,
               num_splits, 0, nullptr, Paging(), &cws);
}

fa_status_t fa_fwd_kvcache_ws(const void *q, const void *k, const void *v, void *o, float *lse,
                              const int *seqlens_k, int B, int Hq, int Hkv, int Nq, int Nk, int D,
                              int causal, float scale, void *stream, fa_dtype_t in_dtype,
                              fa_dtype_t out_dtype, void *workspace, size_t workspace_bytes) {
    const CallWs cws{workspace, workspace_bytes};
    return kvcache(q, k, v, o, lse, seqlens_k, B, Hq, Hkv, Nq, Nk, D, causal, scale, stream, in_dtype,
                   out_dtype, &cws);
}

fa_status_t fa_fwd_kvcache_paged_ws(const void *q, const void *k_pages, const void *v_pages, void *o,
                                    float *lse, const int *seqlens_k, const int *block_table, int B,
                                    int Hq, int Hkv, int Nq, int D, int page_size, int max_pages,
                                    int num_pages, int causal, float scale, void *stream,
                                    fa_dtype_t in_dtype, fa_dtype_t out_dtype, void *workspace,
                                    size_t workspace_bytes) {
    const CallWs cws{workspace, workspace_bytes};
    return kvcache_paged(q, k_pages, v_pages, o, lse, seqlens_k, block_table, B, Hq, Hkv, Nq, D,
                         page_size, max_pages, num_pages, causal, scale, stream, in_dtype, out_dtype,
                         &cws);
}

size_t fa_workspace_bytes(int B, int Hq, int Hkv, int Nq, int Nk, int D, fa_dtype_t in_dtype,
                          int num_splits) {
    if (B < 1 || Hq < 1 || Hkv < 1 || Nk < 1 || Hq % Hkv != 0) return 0;
    if (!fa::decode_supported(Nq, D, in_dtype)) return 0;
    if (num_splits < 0 || num_splits > FA_MAX_SPLITS) return 0;
    const int S = num_splits > 0 ? num_splits : fa::decode_default_splits(B, Hq, Hkv, Nk, D);
    return fa::decode_workspace_bytes(B, Hq, D, S);
}

fa_status_t fa_set_workspace(void *dev_ptr, size_t bytes) {
    if ((dev_ptr == nullptr) != (bytes == 0)) return FA_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(dev_ptr) & 15) return FA_ERR_ALIGN;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return FA_ERR_HIP;
    std::lock_guard<std::mutex> lk(g_ws_mu);
    g_user[dev].ptr = dev_ptr;
    g_user[dev].bytes = bytes;
    return FA_OK;
}

fa_status_t fa_q8_0_gemv(const void *w, const void *x, void *y, int M, int K, fa_dtype_t x_dtype,
                         fa_dtype_t y_dtype, void *stream) {
    if (!w || !x || !y) return FA_ERR_NULL;
    if (M < 1 || K < 32 || K % 32 != 0 || K > (1 << 30)) return FA_ERR_DIM;
    const bool xt_ok = x_dtype == FA_F16 || x_dtype == FA_BF16 || x_dtype == FA_F32;
    if (!xt_ok || !(y_dtype == x_dtype || y_dtype == FA_F32)) return FA_ERR_DTYPE;
    const size_t xe = esize(x_dtype), ye = esize(y_dtype);
    if ((reinterpret_cast<uintptr_t>(w) & 3) || (reinterpret_cast<uintptr_t>(x) & 15) ||
        (reinterpret_cast<uintptr_t>(y) & (ye - 1)))
        return FA_ERR_ALIGN;
    const size_t wb = (size_t)M * (size_t)(K / 32) * 34;
    if (overlaps(y, (size_t)M * ye, w, wb) || overlaps(y, (size_t)M * ye, x, (size_t)K * xe))
        return FA_ERR_ALIAS;
    const hipError_t e =
        fa::launch_q8_gemv(w, x, y, M, K, x_dtype, y_dtype, reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? FA_OK : FA_ERR_HIP;
}

size_t fa_unfused_workspace_bytes(int B, int Hq, int Nq, int Nk) {
    return fa::unfused_workspace_bytes(B, Hq, Nq, Nk);
}

fa_status_t fa_fwd_unfused(const void *q, const void *k, const void *v, void *o, float *lse, int B,
                           int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale,
                           void *stream, fa_dtype_t in_dtype, fa_dtype_t out_dtype,
                           void *workspace, size_t workspace_bytes) {
    fa_status_t st = validate_core(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, in_dtype,
                                   out_dtype, -1);
    if (st != FA_OK) return st;
    if (in_dtype == FA_F32) return FA_ERR_DTYPE;
    if (!fa::unfused_supported(D, in_dtype)) return FA_ERR_HEAD_DIM;
    if (Nk > (1 << 23)) return FA_ERR_DIM;   // 32-bit offsets within a 32-row block of scores
    if ((long long)B * Hq * Nq > 0x7fffffffLL) return FA_ERR_DIM;   // one softmax workgroup per row at most
    if (!workspace) return FA_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(workspace) & 255) return FA_ERR_ALIGN;
    const size_t need = fa::unfused_workspace_bytes(B, Hq, Nq, Nk);
    if (need == 0) return FA_ERR_DIM;
    if (workspace_bytes < need) return FA_ERR_WORKSPACE;
    const size_t qb = (size_t)B * Nq * Hq * D * esize(in_dtype), kb = (size_t)B * Nk * Hkv * D * esize(in_dtype);
    const size_t ob = (size_t)B * Nq * Hq * D * esize(out_dtype), lb = (size_t)B * Hq * Nq * sizeof(float);
    if (overlaps(workspace, need, q, qb) || overlaps(workspace, need, k, kb) ||
        overlaps(workspace, need, v, kb) || overlaps(workspace, need, o, ob) ||
        (lse && overlaps(workspace, need, lse, lb)))
        return FA_ERR_ALIAS;
    fa::Problem p{q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, in_dtype, out_dtype, 0, 0,
                  nullptr, nullptr, 0, 0, 0};
    const hipError_t e = fa::launch_unfused(p, workspace, reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? FA_OK : FA_ERR_HIP;
}

fa_status_t fa_release_workspace(void) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return FA_ERR_HIP;
    std::lock_guard<std::mutex> lk(g_ws_mu);
    bool any = false;
    for (const OwnedWs &w : g_owned) any = any || w.dev == dev;
    for (const Retired &r : g_retired) any = any || r.dev == dev;
    if (!any) return FA_OK;
    // calls queued on any stream may still use these buffers
    if (hipDeviceSynchronize() != hipSuccess) return FA_ERR_HIP;
    fa_status_t st = FA_OK;
    std::vector<OwnedWs> keep;
    for (const OwnedWs &w : g_owned) {
        if (w.dev != dev) keep.push_back(w);
        else if (hipFree(w.ptr) != hipSuccess) st = FA_ERR_HIP;
    }
    g_owned.swap(keep);
    std::vector<Retired> keep_r;
    for (const Retired &r : g_retired) {
        if (r.dev != dev) keep_r.push_back(r);
        else if (hipFree(r.ptr) != hipSuccess) st = FA_ERR_HIP;
    }
    g_retired.swap(keep_r);
    return st;
}

}  // extern "C"
