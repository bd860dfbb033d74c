/*
 * c_client.c -- a plain C caller of the library (no PyTorch): reads a problem
 * and its inputs from a file, copies them to device memory, calls fa_fwd,
 * fa_q8_0_gemv and (fp16 / bf16 inputs) fa_fwd_unfused with a workspace of
 * its own through the C ABI on the null stream, and writes the outputs to a
 * file.  Used by tests/test_c_client_gpu.py; built by __graft_entry__.build().
 *
 * Input file (little-endian):
 *   int32  B, Hq, Hkv, Nq, Nk, D, causal, in_dtype   then float32 scale
 *   q, k, v as raw elements of in_dtype
 *   int32  M, K   then M * K / 32 * 34 bytes of Q8_0 weights and K float32 x
 * Output file:
 *   o (float32, B*Nq*Hq*D), lse (float32, B*Hq*Nq), y (float32, M), then for
 *   fp16 / bf16 inputs the unfused path's o and lse (float32, same shapes)
 * Exit status 0 on success; otherwise the failing call is printed.
 */
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>

#include "fa.h"

#define HIP_OK(call)                                                              \
    do {                                                                          \
        hipError_t e_ = (call);                                                   \
        if (e_ != hipSuccess) {                                                   \
            fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));     \
            return 2;                                                             \
        }                                                                         \
    } while (0)

static int read_all(FILE *f, void *p, size_t n) { return fread(p, 1, n, f) == n; }

int main(int argc, char **argv) {
    if (argc != 3) {
        fprintf(stderr, "usage: %s input output\n", argv[0]);
        return 1;
    }
    FILE *in = fopen(argv[1], "rb");
    if (!in) return 1;
    int hdr[8];
    float scale;
    if (!read_all(in, hdr, sizeof hdr) || !read_all(in, &scale, sizeof scale)) return 1;
    const int B = hdr[0], Hq = hdr[1], Hkv = hdr[2], Nq = hdr[3], Nk = hdr[4], D = hdr[5];
    const int causal = hdr[6];
    const fa_dtype_t dt = (fa_dtype_t)hdr[7];
    const size_t es = dt == FA_F32 ? 4 : 2;
    const size_t nq = (size_t)B * Nq * Hq * D, nk = (size_t)B * Nk * Hkv * D, nl = (size_t)B * Hq * Nq;
    void *hq = malloc(nq * es), *hk = malloc(nk * es), *hv = malloc(nk * es);
    if (!hq || !hk || !hv || !read_all(in, hq, nq * es) || !read_all(in, hk, nk * es) ||
        !read_all(in, hv, nk * es))
        return 1;
    int mk[2];
    if (!read_all(in, mk, sizeof mk)) return 1;
    const int M = mk[0], K = mk[1];
    const size_t wb = (size_t)M * (K / 32) * 34;
    void *hw = malloc(wb);
    float *hx = (float *)malloc((size_t)K * 4);
    if (!hw || !hx || !read_all(in, hw, wb) || !read_all(in, hx, (size_t)K * 4)) return 1;
    fclose(in);

    void *dq, *dk, *dv, *dw, *dx;
    float *dout, *dlse, *dy;
    HIP_OK(hipMalloc(&dq, nq * es));
    HIP_OK(hipMalloc(&dk, nk * es));
    HIP_OK(hipMalloc(&dv, nk * es));
    HIP_OK(hipMalloc((void **)&dout, nq * 4));
    HIP_OK(hipMalloc((void **)&dlse, nl * 4));
    HIP_OK(hipMalloc(&dw, wb));
    HIP_OK(hipMalloc(&dx, (size_t)K * 4));
    HIP_OK(hipMalloc((void **)&dy, (size_t)M * 4));
    HIP_OK(hipMemcpy(dq, hq, nq * es, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dk, hk, nk * es, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dv, hv, nk * es, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dw, hw, wb, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dx, hx, (size_t)K * 4, hipMemcpyHostToDevice));

    /* an argument error comes back before any launch */
    if (fa_fwd(dq, dk, dv, dout, dlse, B, Hq, Hkv + 1000, Nq, Nk, D, causal, scale, NULL, dt,
               FA_F32) == FA_OK) {
        fprintf(stderr, "a bad head ratio was accepted\n");
        return 3;
    }
    fa_status_t st = fa_fwd(dq, dk, dv, dout, dlse, B, Hq, Hkv, Nq, Nk, D, causal, scale, NULL, dt,
                            FA_F32);
    if (st != FA_OK) {
        fprintf(stderr, "fa_fwd: %s\n", fa_status_string(st));
        return 3;
    }
    st = fa_q8_0_gemv(dw, dx, dy, M, K, FA_F32, FA_F32, NULL);
    if (st != FA_OK) {
        fprintf(stderr, "fa_q8_0_gemv: %s\n", fa_status_string(st));
        return 3;
    }
    /* the unfused path into a second pair of outputs, workspace from hipMalloc */
    float *dout2 = NULL, *dlse2 = NULL;
    void *dws = NULL;
    const int unfused = dt != FA_F32;
    if (unfused) {
        const size_t wsb = fa_unfused_workspace_bytes(B, Hq, Nq, Nk);
        if (wsb == 0) {
            fprintf(stderr, "fa_unfused_workspace_bytes returned 0\n");
            return 3;
        }
        HIP_OK(hipMalloc((void **)&dout2, nq * 4));
        HIP_OK(hipMalloc((void **)&dlse2, nl * 4));
        HIP_OK(hipMalloc(&dws, wsb));
        if (fa_fwd_unfused(dq, dk, dv, dout2, dlse2, B, Hq, Hkv, Nq, Nk, D, causal, scale, NULL, dt,
                           FA_F32, dws, wsb - 1) != FA_ERR_WORKSPACE) {
            fprintf(stderr, "a short workspace was accepted\n");
            return 3;
        }
        st = fa_fwd_unfused(dq, dk, dv, dout2, dlse2, B, Hq, Hkv, Nq, Nk, D, causal, scale, NULL, dt,
                            FA_F32, dws, wsb);
        if (st != FA_OK) {
            fprintf(stderr, "fa_fwd_unfused: %s\n", fa_status_string(st));
            return 3;
        }
    }
    HIP_OK(hipDeviceSynchronize());

    float *ho = (float *)malloc(nq * 4), *hl = (float *)malloc(nl * 4), *hy = (float *)malloc((size_t)M * 4);
    if (!ho || !hl || !hy) return 1;
    HIP_OK(hipMemcpy(ho, dout, nq * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hl, dlse, nl * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hy, dy, (size_t)M * 4, hipMemcpyDeviceToHost));
    FILE *out = fopen(argv[2], "wb");
    if (!out || fwrite(ho, 4, nq, out) != nq || fwrite(hl, 4, nl, out) != nl ||
        fwrite(hy, 4, (size_t)M, out) != (size_t)M)
        return 1;
    if (unfused) {
        HIP_OK(hipMemcpy(ho, dout2, nq * 4, hipMemcpyDeviceToHost));
        HIP_OK(hipMemcpy(hl, dlse2, nl * 4, hipMemcpyDeviceToHost));
        if (fwrite(ho, 4, nq, out) != nq || fwrite(hl, 4, nl, out) != nl) return 1;
    }
    fclose(out);
    fa_release_workspace();
    printf("c_client: fa_fwd, fa_q8_0_gemv%s done\n", unfused ? " and fa_fwd_unfused" : "");
    return 0;
}
