// fa_internal.h -- host-side launcher declarations shared by the library's
// translation units (not part of the public interface in include/fa.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

#include "../../include/fa.h"

namespace fa {

struct Problem {
    const void *q, *k, *v;
    void *o;
    float *lse;
    int B, Hq, Hkv, Nq, Nk, D;
    int causal;
    float scale;
    fa_dtype_t in, out;
    int hw;   // prefill query heads per workgroup (0: the default choice)
    int slots;   // prefill 32-row query slots per workgroup (0: the default, 4)
    const int *seqlens;   // device [B]: valid keys per batch element (NULL: Nk for all)
    // Paged K/V (block_table != NULL): k and v are [num_pages][page_size][Hkv][D];
    // key j of batch element b is row j % page_size of page
    // block_table[b * max_pages + j / page_size]; Nk = page_size * max_pages.
    const int *block_table;
    int page_size, max_pages, num_pages;
};

// Each launcher enqueues its kernels on `stream` and returns the first HIP
// error (hipSuccess when the launch was accepted).
hipError_t launch_prefill(const Problem &p, hipStream_t stream);
hipError_t launch_generic(const Problem &p, hipStream_t stream);
hipError_t launch_decode(const Problem &p, int splits, void *workspace, hipStream_t stream);
hipError_t launch_unfused(const Problem &p, void *workspace, hipStream_t stream);
hipError_t launch_q8_gemv(const void *w, const void *x, void *y, int M, int K, fa_dtype_t x_dtype,
                          fa_dtype_t y_dtype, hipStream_t stream);

// Decode split planning (shared by the dispatcher and fa_workspace_bytes).
bool decode_supported(int Nq, int D, fa_dtype_t in);
bool prefill_supported(int D, fa_dtype_t in);
int decode_default_splits(int B, int Hq, int Hkv, int Nk, int D);
size_t decode_workspace_bytes(int B, int Hq, int D, int splits);

// Unfused path: supported shapes and the workspace it needs (0 when a size is
// < 1 or the product overflows).
bool unfused_supported(int D, fa_dtype_t in);
size_t unfused_workspace_bytes(long long B, long long Hq, long long Nq, long long Nk);

}  // namespace fa
