"""Minimal runs for profilers (rocprofv3): one workload's attention call a few
times, or a plain device copy of known size (the reference for scaling the
HBM byte counters).

    python3 paper_2608_18656_amd/profile_run.py gqa_prefill_bf16 5
    python3 paper_2608_18656_amd/profile_run.py copy 268435456 5
    python3 paper_2608_18656_amd/profile_run.py q8_gate_up 5

``q8_<name>`` runs the Q8_0 matrix-vector product of one TinyLlama-shaped
projection (qkv, o, gate_up or down; bf16 activations); ``paged_<workload>
<page_size>`` runs a decode workload against its K/V scattered over pages
of that size in a seeded random order.

    python3 paper_2608_18656_amd/profile_run.py paged_gqa_decode_bf16 256 5

``unfused_<workload>`` runs the unfused self-attention path (scores,
softmax and P.V kernels through a workspace) on a prefill workload.

    python3 paper_2608_18656_amd/profile_run.py unfused_gqa_prefill_bf16 5

``chunked_prefill`` runs the chunked prefill of the benchmark (512 new
tokens per sequence against caches of 4096, 3072, 2048 and 1024 keys, 32/8
heads, D = 64, bf16, causal) on the contiguous cache, then on the same cache
in shuffled pages of 256 keys.

    python3 paper_2608_18656_amd/profile_run.py chunked_prefill 20
"""
from __future__ import annotations

import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))


def main(argv):
    import torch

    what = argv[1] if len(argv) > 1 else "gqa_prefill_bf16"
    if what == "copy":
        nbytes = int(argv[2]) if len(argv) > 2 else 1 << 28
        reps = int(argv[3]) if len(argv) > 3 else 5
        src = torch.ones(nbytes // 2, dtype=torch.float16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(reps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"copied {nbytes} bytes x {reps}", flush=True)
        return
    import paper_2608_18656_amd as fa
    from paper_2608_18656_amd.inputs import Q8_LAYER_SHAPES, WORKLOADS, make_q8_0, make_workload

    if what.startswith("paged_"):
        w = WORKLOADS[what[len("paged_"):]]
        ps = int(argv[2]) if len(argv) > 2 else 256
        reps = int(argv[3]) if len(argv) > 3 else 5
        q, k, v = make_workload(w)
        npg = w.B * (w.Nk // ps)
        perm = torch.randperm(npg, generator=torch.Generator().manual_seed(4000))
        kp = torch.empty((npg, ps, w.Hkv, w.D), dtype=k.dtype)
        vp = torch.empty_like(kp)
        kp[perm] = k.reshape(npg, ps, w.Hkv, w.D)
        vp[perm] = v.reshape(npg, ps, w.Hkv, w.D)
        table = perm.reshape(w.B, -1).to(torch.int32).cuda()
        sl = torch.full((w.B,), w.Nk, dtype=torch.int32, device="cuda")
        qd, kp, vp = q.cuda(), kp.cuda(), vp.cuda()
        for _ in range(reps):
            fa.fwd_kvcache_paged(qd, kp, vp, table, sl, scale=w.softmax_scale)
        torch.cuda.synchronize()
        print(f"ran {what} pages of {ps} x {reps}", flush=True)
        return
    reps = int(argv[2]) if len(argv) > 2 else 5
    if what.startswith("q8_"):
        shape = {n: (M, K) for n, M, K in Q8_LAYER_SHAPES}[what[3:]]
        w, x = make_q8_0(*shape, seed=2000, x_dtype="bf16")
        w, x = w.cuda(), x.cuda()
        for _ in range(reps):
            fa.q8_0_gemv(w, x)
        torch.cuda.synchronize()
        print(f"ran {what} {shape} x {reps}", flush=True)
        return
    if what == "chunked_prefill":
        from paper_2608_18656_amd.inputs import make_qkv

        B, Hq, Hkv, Nq, Nk, D, ps = 4, 32, 8, 512, 4096, 64, 256
        q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, "bf16", seed=5000)
        sl = torch.tensor([4096, 3072, 2048, 1024], dtype=torch.int32, device="cuda")
        npg = B * (Nk // ps)
        perm = torch.randperm(npg, generator=torch.Generator().manual_seed(5001))
        kp = torch.empty((npg, ps, Hkv, D), dtype=k.dtype)
        vp = torch.empty_like(kp)
        kp[perm] = k.reshape(npg, ps, Hkv, D)
        vp[perm] = v.reshape(npg, ps, Hkv, D)
        table = perm.reshape(B, -1).to(torch.int32).cuda()
        qd, kd, vd, kp, vp = q.cuda(), k.cuda(), v.cuda(), kp.cuda(), vp.cuda()
        for _ in range(reps):
            fa.fwd_kvcache(qd, kd, vd, sl, causal=True, scale=D ** -0.5)
        torch.cuda.synchronize()
        for _ in range(reps):
            fa.fwd_kvcache_paged(qd, kp, vp, table, sl, causal=True, scale=D ** -0.5)
        torch.cuda.synchronize()
        print(f"ran {what} x {reps} (contiguous, then paged)", flush=True)
        return
    if what.startswith("unfused_"):
        w = WORKLOADS[what[len("unfused_"):]]
        q, k, v = (t.cuda() for t in make_workload(w))
        ws = torch.empty(fa.unfused_workspace_bytes(w.B, w.Hq, w.Nq, w.Nk), dtype=torch.uint8,
                         device="cuda")
        for _ in range(reps):
            fa.fwd_unfused(q, k, v, causal=w.causal, scale=w.softmax_scale, workspace=ws)
        torch.cuda.synchronize()
        print(f"ran {what} x {reps}", flush=True)
        return
    w = WORKLOADS[what]
    q, k, v = (t.cuda() for t in make_workload(w))
    for _ in range(reps):
        fa.fwd(q, k, v, causal=w.causal, scale=w.softmax_scale)
    torch.cuda.synchronize()
    print(f"ran {what} x {reps}", flush=True)


if __name__ == "__main__":
    main(sys.argv)
