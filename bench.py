#!/usr/bin/env python3
"""One-GPU benchmark of the MI355X attention forward.

A timed step is one call of the attention forward on the headline workload
(default: GQA causal prefill, B=1, Hq=32, Hkv=8, Nq=Nk=2048, D=64, bf16) with
its inputs already resident in HBM; the value is algorithmic TFLOP/s
(4 * D FLOPs per visible query-key pair per head).  The decode path (split-KV
plus log-sum-exp merge) is timed in the same run on the GQA decode workload
(B=16, Hq=32, Hkv=8, Nk=8192, D=128, bf16) as KV-read GB/s, and the other
workloads are reported alongside.  The fp64 CPU oracle is timed on the host
cores on the headline workload as a baseline (not a target), and the GPU
output of the benchmark is checked against it.  The Q8_0 matrix-vector
products of a decode step (the linear layers of a TinyLlama-1.1B shaped
model) are reported under "q8_0_gemv" as weight GB/s.  Also reported: the
inter-head packing ablation ("packing_ablation"), the fused kernel against
the unfused self-attention path with its materialised score matrix
("unfused_ablation"), decode against a paged cache ("paged_decode") and a
chunked prefill against caches of per-sequence lengths, contiguous and
paged ("chunked_prefill").  ``--only WHAT`` instead makes a minimal run of one
thing for a profiler (see profile_only).

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_MFMA_TFLOPS = {"bf16": 2500.0, "f16": 2500.0, "f32": 157.3}   # dense, MI355X
PEAK_HBM_GBS = 8000.0
METRIC = "prefill attention TFLOP/s (% MFMA peak); decode KV GB/s (% HBM peak)"
PREFILL_SOURCES = ["paper_2608_18656_amd/csrc/fa_prefill.hip",
                   "paper_2608_18656_amd/csrc/fa_common.h"]
DECODE_SOURCES = ["paper_2608_18656_amd/csrc/fa_decode.hip",
                  "paper_2608_18656_amd/csrc/fa_common.h"]
Q8_SOURCES = ["paper_2608_18656_amd/csrc/fa_q8.hip"]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_hash(paths):
    """sha256 over the kernel sources with comments and blank space removed,
    so that the stored counters stay valid across comment-only edits."""
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def stored_traffic(kernel: str, workload: str, paths):
    """HBM bytes per launch from the committed rocprofv3 counter runs, or None
    when they were taken on a different version of the kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f).get(kernel, {}).get(workload)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_sha256") != source_hash(paths):
        return None
    return rec.get("hbm_bytes_per_launch")


def time_calls(torch, fns, steps, warmup):
    """Mean ms per call over ``steps`` back-to-back calls (cycling through
    ``fns``), bracketed by device synchronisation; HIP events recorded on the
    current stream, which is the stream the kernels are launched on."""
    stream = torch.cuda.current_stream()
    for i in range(warmup):
        fns[i % len(fns)]()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for i in range(steps):
        fns[i % len(fns)]()
    t1.record(stream)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def loaded_sclk_mhz(torch, call, seconds=2.0):
    """Shader clock (MHz, mean over the XCDs and two samples) read with amd-smi
    right after `call` has been queued back to back for about `seconds`
    (replayed from a HIP graph; queueing a replay takes about as long as the
    GPU takes to run it, so the samples fall while work is still queued);
    None when amd-smi is missing or its output cannot be read."""
    import shutil
    import subprocess

    if shutil.which("amd-smi") is None:
        return None
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for _ in range(2):
            call()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for _ in range(20):
            call()
    clocks = []
    try:
        t_end = time.time() + seconds
        while time.time() < t_end:
            g.replay()
        for _ in range(2):
            out = subprocess.run(["amd-smi", "metric", "--clock", "--json"], capture_output=True,
                                 text=True, timeout=20).stdout
            data = json.loads(out[out.index("{"):])
            gpus = data.get("gpu_data", data) if isinstance(data, dict) else data
            for gpu in (gpus if isinstance(gpus, list) else [gpus])[:1]:
                for name, blk in gpu.get("clock", {}).items():
                    if name.lower().startswith("gfx") and isinstance(blk, dict):
                        clocks.append(float(blk["clk"]["value"]))
    except (OSError, subprocess.SubprocessError, ValueError, KeyError, TypeError):
        clocks = []
    torch.cuda.synchronize()
    del g
    return round(sum(clocks) / len(clocks), 1) if clocks else None


# Workgroup layouts of the packing ablation: (label, query slots per
# workgroup, query heads among them).  Every staged K/V tile serves all slots
# of its workgroup: one slot (no sharing), four row blocks of one head, four
# heads of one K/V group (the default for small grids), eight slots of four
# heads (the default for large D = 64 grids), eight heads of an MQA group.
LAYOUTS = {
    "gqa_prefill_bf16": [("unshared", 1, 1), ("per_head", 4, 1), ("packed", 4, 4)],
    "gqa_prefill_d128_f16": [("unshared", 1, 1), ("per_head", 4, 1), ("packed", 4, 4), ("eight_slots", 8, 4)],
    "mqa_prefill_f16": [("unshared", 1, 1), ("packed", 4, 4), ("eight_slots", 8, 4), ("packed_wide", 8, 8)],
}


def staged_kv_bytes(w, slots: int, heads: int) -> int:
    """K and V bytes the workgroups of one prefill launch copy into LDS with
    this layout: each workgroup (slots / heads row blocks of 32 rows, heads
    query heads of one K/V head) stages every tile of keys its causal extent
    reaches once, K and V (tiles of 64 keys at D = 64, 32 at D = 128)."""
    bc = 64 if w.D == 64 else 32
    rows = 32 * (slots // heads)
    tiles = 0
    for mb in range((w.Nq + rows - 1) // rows):
        last = min((mb + 1) * rows, w.Nq) - 1
        kend = min(w.Nk, last + w.Nk - w.Nq + 1) if w.causal else w.Nk
        tiles += (kend + bc - 1) // bc
    groups = w.B * w.Hkv * ((w.Hq // w.Hkv) // heads)
    return tiles * groups * bc * w.D * 2 * 2


def run_workload(torch, fa, w, steps, warmup, kv_sets=1, num_splits=None, packing=None, slots=None):
    from paper_2608_18656_amd.inputs import make_workload

    q, k, v = make_workload(w)
    sets = [(q.cuda(), k.cuda(), v.cuda())]
    for extra in range(1, kv_sets):   # more K/V copies so every call streams from HBM
        q2, k2, v2 = make_workload(w, seed=w.seed + 1000 * extra)
        sets.append((q2.cuda(), k2.cuda(), v2.cuda()))
    del q, k, v
    outs = [torch.empty_like(s[0]) for s in sets]
    lses = [torch.empty((w.B, w.Hq, w.Nq), dtype=torch.float32, device="cuda") for _ in sets]

    def make(i):
        qd, kd, vd = sets[i]
        return lambda: fa.fwd(qd, kd, vd, causal=w.causal, scale=w.softmax_scale, out=outs[i],
                              lse=lses[i], num_splits=num_splits, heads_per_workgroup=packing,
                              slots_per_workgroup=slots)

    ms = time_calls(torch, [make(i) for i in range(len(sets))], steps, warmup)
    return ms, sets[0], outs[0], lses[0]


def unfused_vs_fused(torch, fa, w, steps):
    """Fused kernel against the unfused path on one workload.  The unfused
    path's minimum HBM traffic: per visible score, S written (4 B) and read
    (4 B) and P written (2 B) and read (2 B); Q, K, V and O once."""
    from paper_2608_18656_amd.inputs import DTYPES, make_workload

    q, k, v = (t.cuda() for t in make_workload(w))
    out = torch.empty_like(q)
    lse = torch.empty((w.B, w.Hq, w.Nq), dtype=torch.float32, device="cuda")
    ws = torch.empty(fa.unfused_workspace_bytes(w.B, w.Hq, w.Nq, w.Nk), dtype=torch.uint8,
                     device="cuda")
    fused_ms = time_calls(torch, [lambda: fa.fwd(q, k, v, causal=w.causal, scale=w.softmax_scale,
                                                 out=out, lse=lse)], steps, 2)
    unf_ms = time_calls(torch, [lambda: fa.fwd_unfused(q, k, v, causal=w.causal,
                                                       scale=w.softmax_scale, out=out, lse=lse,
                                                       workspace=ws)], steps, 2)
    es = torch.finfo(DTYPES[w.dtype]).bits // 8
    nbytes = unfused_min_bytes(w.B, w.Hq, w.Hkv, w.Nq, w.Nk, w.D, w.visible_pairs(), es)
    del ws
    return {"workload": w.name, "fused_us": round(fused_ms * 1e3, 2),
            "unfused_us": round(unf_ms * 1e3, 2), "fused_speedup": round(unf_ms / fused_ms, 2),
            "fused_tflops": round(w.flops() / (fused_ms * 1e-3) / 1e12, 1),
            "unfused_tflops": round(w.flops() / (unf_ms * 1e-3) / 1e12, 1),
            "unfused_min_hbm_bytes": nbytes,
            "unfused_gbs": round(nbytes / (unf_ms * 1e-3) / 1e9, 1),
            "unfused_frac_hbm": round(nbytes / (unf_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "steps": steps}


MANT_BITS = {"f16": 10, "bf16": 7, "f32": 23}
MIN_NORMAL_EXP = {"f16": -14, "bf16": -126, "f32": -126}


def half_ulp(x, dtype: str):
    """Half the spacing of the ``dtype`` format at magnitude |x| (fp64 array in,
    fp64 array out; subnormal-aware)."""
    import numpy as np

    e = np.floor(np.log2(np.maximum(np.abs(x), 2.0 ** MIN_NORMAL_EXP[dtype])))
    return 0.5 * np.exp2(e - MANT_BITS[dtype])


def cpu_model() -> str | None:
    """The host CPU's model name (from /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def parity_report(torch, fa, w, inputs, o_dev, lse_dev, o_ref, l_ref):
    """The benchmark's GPU output against the oracle, read the three ways the
    tests check it: raw max|o - o_ref| of the shipped output; T1, the same
    kernel asked for fp32 output (verify mode: its result before the final
    rounding); T2, the part of the shipped error beyond half a unit in the
    last place of the output format; plus the rounding floor max|rne(o_ref) -
    o_ref|, the error that correctly rounding the exact result to the output
    format already has."""
    import numpy as np

    import oracle
    from paper_2608_18656_amd.inputs import DTYPES

    og = oracle.to_f64(o_dev)
    diff = np.abs(og - o_ref)
    qd, kd, vd = inputs
    o32, l32 = fa.fwd(qd, kd, vd, causal=w.causal, scale=w.softmax_scale, out_dtype=torch.float32)
    torch.cuda.synchronize()
    t1 = float(np.abs(oracle.to_f64(o32) - o_ref).max())
    t1_lse = float(np.abs(oracle.to_f64(l32) - l_ref).max())
    rep = {"max_abs_err_vs_oracle": float(diff.max()),
           "lse_max_abs_err": float(np.abs(oracle.to_f64(lse_dev) - l_ref).max()),
           "t1_verify_max_abs": t1, "t1_verify_lse_max_abs": t1_lse, "tolerance": 2e-3}
    if w.dtype in ("f16", "bf16"):
        rep["t2_adjusted_max_abs"] = float(np.max(diff - half_ulp(np.maximum(np.abs(og), np.abs(o_ref)), w.dtype)))
        rounded = torch.from_numpy(o_ref).to(DTYPES[w.dtype]).double().numpy()
        rep["rounding_floor"] = float(np.abs(rounded - o_ref).max())
    else:
        rep["t2_adjusted_max_abs"] = float(diff.max())
        rep["rounding_floor"] = 0.0
    rep["pass"] = bool(t1 <= 2e-3 and t1_lse <= 2e-3 and rep["t2_adjusted_max_abs"] <= 2e-3
                       and rep["lse_max_abs_err"] <= 2e-3)
    del o32, l32
    return rep


def cpu_baseline(torch, fa, w, inputs, o_dev, lse_dev):
    """The oracle as it stands, on the host cores, over the whole workload;
    also the parity of the benchmark's GPU output against it."""
    import oracle

    q, k, v = (t.cpu() for t in inputs)
    stats = {}
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        affinity = os.cpu_count()
    t0 = time.perf_counter()
    o_ref, l_ref = oracle.attention_parallel(q, k, v, w.causal, w.softmax_scale,
                                             workers=oracle.default_workers(), stats=stats)
    wall = time.perf_counter() - t0
    parity = parity_report(torch, fa, w, inputs, o_dev, lse_dev, o_ref, l_ref)
    return ({"value": w.flops() / wall / 1e12, "unit": "TFLOP/s", "cores": stats["workers"],
             "kind": "oracle", "cpu_model": cpu_model(), "cpus_available": affinity,
             "cpu_seconds": round(stats["cpu_s"], 2), "wall_seconds": round(wall, 2),
             "sample": f"whole {w.name} workload ({w.B * w.Hq * w.Nq} query rows), fp64 C, "
                       f"one thread per worker process (workers: the CPUs this process may use, "
                       f"within the CPU share OMP_NUM_THREADS gives)"},
            parity)


def paged_decode(torch, fa, w, steps, warmup, page_size):
    """Decode of workload ``w`` against a paged cache: the K/V rows of each
    sequence scattered over pages of ``page_size`` keys in a seeded random
    order (two pools alternated, so that every call streams from HBM); every
    sequence full.  Returns us per call and K+V GB/s."""
    from paper_2608_18656_amd.inputs import make_workload

    q, k, v = make_workload(w)
    max_pages = w.Nk // page_size
    npg = w.B * max_pages
    sets = []
    for r in range(2):
        gen = torch.Generator().manual_seed(4000 + r)
        perm = torch.randperm(npg, generator=gen)
        table = perm.reshape(w.B, max_pages).to(torch.int32)
        kp = torch.empty((npg, page_size, w.Hkv, w.D), dtype=k.dtype)
        vp = torch.empty_like(kp)
        kp[perm] = k.reshape(npg, page_size, w.Hkv, w.D)
        vp[perm] = v.reshape(npg, page_size, w.Hkv, w.D)
        sets.append((kp.cuda(), vp.cuda(), table.cuda()))
    qd = q.cuda()
    sl = torch.full((w.B,), w.Nk, dtype=torch.int32, device="cuda")
    out = torch.empty_like(qd)
    lse = torch.empty((w.B, w.Hq, 1), dtype=torch.float32, device="cuda")
    fns = [(lambda s=s: fa.fwd_kvcache_paged(qd, s[0], s[1], s[2], sl, scale=w.softmax_scale, out=out,
                                             lse=lse)) for s in sets]
    ms = time_calls(torch, fns, steps, warmup)
    del sets
    torch.cuda.empty_cache()
    return ms * 1e3, w.kv_bytes() / (ms * 1e-3) / 1e9


def chunked_visible_pairs(Nq, lens):
    """Visible (query, key) pairs per head of a causal chunked prefill: the
    Nq queries of a sequence of length L are its last positions, so query i
    sees L - Nq + i + 1 keys (L >= Nq)."""
    return sum(Nq * (L - Nq + 1) + Nq * (Nq - 1) // 2 for L in lens)


def unfused_min_bytes(B, Hq, Hkv, Nq, Nk, D, vis_per_head, esize):
    """Minimum HBM bytes of the unfused path: per visible score, S written and
    read in fp32 and P written and read in fp16; Q, K, V and O once."""
    vis = B * Hq * vis_per_head
    return 12 * vis + (2 * B * Nq * Hq * D + 2 * B * Nk * Hkv * D) * esize


def chunked_prefill(torch, fa, steps, warmup):
    """Chunked prefill: 512 new query tokens per sequence against K/V caches
    whose valid lengths are 4096, 3072, 2048 and 1024 (the headline model's
    heads: 32 query / 8 key-value heads, D = 64, bf16, causal, bottom-right
    per sequence), on the contiguous cache and on the same cache in shuffled
    pages of 256 keys.  FLOPs: 4 D per visible (query, key) pair per head."""
    from paper_2608_18656_amd.inputs import make_qkv

    B, Hq, Hkv, Nq, Nk, D, ps = 4, 32, 8, 512, 4096, 64, 256
    lens = [4096, 3072, 2048, 1024]
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, "bf16", seed=5000)
    vis = chunked_visible_pairs(Nq, lens)
    flops = 4 * D * Hq * vis
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    sl = torch.tensor(lens, dtype=torch.int32, device="cuda")
    out = torch.empty_like(qd)
    lse = torch.empty((B, Hq, Nq), dtype=torch.float32, device="cuda")
    scale = D ** -0.5
    ms_c = time_calls(torch, [lambda: fa.fwd_kvcache(qd, kd, vd, sl, causal=True, scale=scale, out=out,
                                                     lse=lse)], steps, warmup)
    npg = B * (Nk // ps)
    perm = torch.randperm(npg, generator=torch.Generator().manual_seed(5001))
    kp = torch.empty((npg, ps, Hkv, D), dtype=k.dtype)
    vp = torch.empty_like(kp)
    kp[perm] = k.reshape(npg, ps, Hkv, D)
    vp[perm] = v.reshape(npg, ps, Hkv, D)
    table = perm.reshape(B, -1).to(torch.int32).cuda()
    kp, vp = kp.cuda(), vp.cuda()
    ms_p = time_calls(torch, [lambda: fa.fwd_kvcache_paged(qd, kp, vp, table, sl, causal=True, scale=scale,
                                                           out=out, lse=lse)], steps, warmup)
    res = {"metric": "chunked prefill TFLOP/s (4 D FLOPs per visible pair per head)",
           "shape": {"B": B, "Hq": Hq, "Hkv": Hkv, "Nq": Nq, "Nk": Nk, "D": D, "seqlens": lens,
                     "dtype": "bf16", "causal": True},
           "flops": flops}
    for label, ms in (("contiguous", ms_c), ("paged256", ms_p)):
        tf = flops / (ms * 1e-3) / 1e12
        res[label] = {"us_per_call": round(ms * 1e3, 2), "tflops": round(tf, 1),
                      "frac": round(tf / PEAK_MFMA_TFLOPS["bf16"], 4)}
    return res


def q8_decode_step(torch, fa, steps, warmup, with_cpu):
    """The Q8_0 matrix-vector products of one decode step of a TinyLlama-1.1B
    shaped model (22 layers; per layer the fused q/k/v projection, the output
    projection, the fused gate/up projection and the down projection, each
    with its own weights, 1.03 GB in all), launched in order on one stream and
    replayed from a HIP graph; the value is weight GB/s (34 bytes per 32
    weights, read once).  Also the average time of each launch shape, and one
    launch over 22 stacked gate/up matrices (539 MB) as the streaming rate."""
    from paper_2608_18656_amd.inputs import Q8_LAYER_SHAPES, Q8_LAYERS, make_q8_0

    base = [make_q8_0(M, K, seed=2000 + i, x_dtype="bf16") for i, (_, M, K) in enumerate(Q8_LAYER_SHAPES)]
    W = [[b[0].cuda() for b in base]]
    for _ in range(1, Q8_LAYERS):
        W.append([t.clone() for t in W[0]])
    X = [b[1].cuda() for b in base]
    Y = [torch.empty(M, dtype=torch.bfloat16, device="cuda") for _, M, _ in Q8_LAYER_SHAPES]
    total = sum(t.numel() for layer in W for t in layer)

    def launch(l, i):
        fa.q8_0_gemv(W[l][i], X[i], out=Y[i])

    def graph_of(calls):
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            for c in calls:
                c()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for c in calls:
                c()
        return g

    def time_graph(g, n):
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(n):
            g.replay()
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / n

    # eager reference of the last layer's outputs, then the graph, replayed
    # several times and checked bitwise against it
    for i in range(len(Q8_LAYER_SHAPES)):
        launch(Q8_LAYERS - 1, i)
    torch.cuda.synchronize()
    eager = [y.clone() for y in Y]
    step = graph_of([(lambda l=l, i=i: launch(l, i)) for l in range(Q8_LAYERS)
                     for i in range(len(Q8_LAYER_SHAPES))])
    for _ in range(3):
        step.replay()
        torch.cuda.synchronize()
        if not all(torch.equal(a, b) for a, b in zip(eager, Y)):
            raise RuntimeError("graph replay of the Q8_0 products differs from the eager result")
    ms = time_graph(step, steps)
    gbs = total / (ms * 1e-3) / 1e9
    per_shape = []
    for i, (name, M, K) in enumerate(Q8_LAYER_SHAPES):
        g = graph_of([(lambda l=l, i=i: launch(l, i)) for l in range(Q8_LAYERS)])
        sms = time_graph(g, steps) / Q8_LAYERS
        nbytes = W[0][i].numel()
        per_shape.append({"name": name, "M": M, "K": K, "bytes": nbytes, "us": round(sms * 1e3, 2),
                          "GB_s": round(nbytes / (sms * 1e-3) / 1e9, 1)})
        del g
    dom = max(per_shape, key=lambda r: r["bytes"])   # the largest launch dominates the step
    # one large launch: the gate/up matrices of all layers stacked
    Mbig, Kbig = Q8_LAYER_SHAPES[2][1] * Q8_LAYERS, Q8_LAYER_SHAPES[2][2]
    wbig = torch.cat([W[l][2] for l in range(Q8_LAYERS)], dim=0)
    ybig = torch.empty(Mbig, dtype=torch.bfloat16, device="cuda")
    bms = time_calls(torch, [lambda: fa.q8_0_gemv(wbig, X[2], out=ybig)], max(5, steps // 2), 2)
    out = {
        "workload": "tinyllama-1.1b-shaped Q8_0 decode linear layers (22 layers x "
                    "{qkv 2560x2048, o 2048x2048, gate_up 11264x2048, down 2048x5632}), bf16 x",
        "metric": "weight GB/s (Q8_0 bytes read once per step)",
        "us_per_step": round(ms * 1e3, 1), "bytes_per_step": total,
        "value": round(gbs, 1), "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
        "launches_per_step": Q8_LAYERS * len(Q8_LAYER_SHAPES), "graph": True,
        "per_shape": per_shape,
        "roofline": {"bound": "hbm", "kernel": "q8_gemv_kernel (" + dom["name"] + ")",
                     "achieved": dom["GB_s"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(dom["GB_s"] / PEAK_HBM_GBS, 4),
                     "traffic": stored_traffic("q8_gemv_kernel", dom["name"], Q8_SOURCES),
                     "algorithmic_per_launch": dom["bytes"]},
        "streaming": {"M": Mbig, "K": Kbig, "bytes": wbig.numel(), "us": round(bms * 1e3, 1),
                      "GB_s": round(wbig.numel() / (bms * 1e-3) / 1e9, 1),
                      "frac": round(wbig.numel() / (bms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)},
    }
    log(f"[bench] q8_0 decode step: {ms * 1e3:.1f} us, {gbs:.0f} GB/s ({100 * gbs / PEAK_HBM_GBS:.1f}%); "
        f"streaming {out['streaming']['GB_s']} GB/s")
    if with_cpu:
        from oracle import q8 as oracle_q8

        wc = [b[0].numpy() for b in base]
        xc = [b[1].float().numpy() for b in base]
        t0 = time.perf_counter()
        for wi, xi in zip(wc, xc):
            oracle_q8.gemv(wi, xi)
        wall = time.perf_counter() - t0
        nbytes = sum(wi.size for wi in wc)
        out["cpu_baseline"] = {"value": round(nbytes / wall / 1e9, 3), "unit": "GB/s", "cores": 1,
                               "kind": "oracle",
                               "sample": "one layer's four matrices (46.8 MB), fp64 C, one thread"}
    del W, wbig
    torch.cuda.empty_cache()
    return out


def profile_only(torch, fa, what: str, reps: int, copy_bytes: int, page_size: int,
                 slots: int | None = None, heads: int | None = None):
    """A minimal run for a profiler (rocprofv3 kernel traces and counters):
    ``reps`` calls of one thing and nothing else.  ``what`` is a workload name
    (the attention forward on it), ``copy`` (a plain device copy of
    ``copy_bytes``, the reference that scales the HBM byte counters),
    ``q8_<qkv|o|gate_up|down>`` (one TinyLlama-shaped Q8_0 projection, bf16
    x), ``paged_<workload>`` (decode against its K/V in shuffled pages of
    ``page_size`` keys), ``unfused_<workload>`` (the unfused path) or
    ``chunked_prefill`` (the benchmark's chunked prefill, contiguous cache then
    paged).  ``slots`` and ``heads`` set a prefill workload's workgroup layout
    (fa_fwd_slots).  Returns a description of what ran."""
    from paper_2608_18656_amd.inputs import Q8_LAYER_SHAPES, WORKLOADS, make_q8_0, make_qkv, make_workload

    def done(desc):
        torch.cuda.synchronize()
        return {"only": what, "reps": reps, "ran": desc}

    if what == "copy":
        src = torch.ones(copy_bytes // 2, dtype=torch.float16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(reps):
            dst.copy_(src)
        return done(f"device copy of {copy_bytes} bytes")
    if what.startswith("paged_"):
        w = WORKLOADS[what[len("paged_"):]]
        q, k, v = make_workload(w)
        npg = w.B * (w.Nk // page_size)
        perm = torch.randperm(npg, generator=torch.Generator().manual_seed(4000))
        kp = torch.empty((npg, page_size, w.Hkv, w.D), dtype=k.dtype)
        vp = torch.empty_like(kp)
        kp[perm] = k.reshape(npg, page_size, w.Hkv, w.D)
        vp[perm] = v.reshape(npg, page_size, w.Hkv, w.D)
        table = perm.reshape(w.B, -1).to(torch.int32).cuda()
        sl = torch.full((w.B,), w.Nk, dtype=torch.int32, device="cuda")
        qd, kp, vp = q.cuda(), kp.cuda(), vp.cuda()
        for _ in range(reps):
            fa.fwd_kvcache_paged(qd, kp, vp, table, sl, scale=w.softmax_scale)
        return done(f"{w.name} against pages of {page_size} keys in shuffled order")
    if what.startswith("q8_"):
        shape = {n: (M, K) for n, M, K in Q8_LAYER_SHAPES}[what[3:]]
        wq, x = make_q8_0(*shape, seed=2000, x_dtype="bf16")
        wq, x = wq.cuda(), x.cuda()
        for _ in range(reps):
            fa.q8_0_gemv(wq, x)
        return done(f"Q8_0 product {shape[0]}x{shape[1]}")
    if what == "chunked_prefill":
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
        return done("chunked prefill, contiguous cache then pages of 256")
    if what.startswith("unfused_"):
        w = WORKLOADS[what[len("unfused_"):]]
        q, k, v = (t.cuda() for t in make_workload(w))
        ws = torch.empty(fa.unfused_workspace_bytes(w.B, w.Hq, w.Nq, w.Nk), dtype=torch.uint8, device="cuda")
        for _ in range(reps):
            fa.fwd_unfused(q, k, v, causal=w.causal, scale=w.softmax_scale, workspace=ws)
        return done(f"unfused path on {w.name}")
    w = WORKLOADS[what]
    q, k, v = (t.cuda() for t in make_workload(w))
    for _ in range(reps):
        fa.fwd(q, k, v, causal=w.causal, scale=w.softmax_scale, slots_per_workgroup=slots,
               heads_per_workgroup=heads)
    return done(f"attention forward on {w.name}" +
                (f" ({slots} slots, {heads} heads per workgroup)" if slots else ""))


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="gqa_prefill_bf16")
    ap.add_argument("--no-extras", action="store_true", help="headline workload only")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sclk", action="store_true",
                    help="skip the shader-clock reading under load (a burst of headline calls)")
    ap.add_argument("--no-ablation", action="store_true",
                    help="skip the inter-head packing and unfused ablations and the chunked-prefill leg "
                         "(e.g. under a kernel trace)")
    ap.add_argument("--only", metavar="WHAT",
                    help="profiler run: REPS calls of one thing only (a workload name, copy, q8_<shape>, "
                         "paged_<workload>, unfused_<workload> or chunked_prefill); prints what ran")
    ap.add_argument("--reps", type=int, default=5, help="calls for --only")
    ap.add_argument("--copy-bytes", type=int, default=1 << 28, help="bytes of the --only copy run")
    ap.add_argument("--page-size", type=int, default=256, help="page size of the --only paged run")
    ap.add_argument("--slots", type=int, default=None, help="--only prefill run: query slots per workgroup")
    ap.add_argument("--heads", type=int, default=None, help="--only prefill run: query heads per workgroup")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE "
              f"{world}); this attention forward is built and measured on a single MI355X",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2608_18656_amd as fa
    from paper_2608_18656_amd.inputs import WORKLOADS

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.only:
        print(json.dumps(profile_only(torch, fa, args.only, args.reps, args.copy_bytes, args.page_size,
                                      args.slots, args.heads)), flush=True)
        return
    w = WORKLOADS[args.workload]
    decode_main = w.Nq == 1
    log(f"[bench] headline {w.name}: steps {args.steps} warmup {args.warmup}")
    ms, inputs, out, lse = run_workload(torch, fa, w, args.steps, args.warmup,
                                        kv_sets=2 if decode_main else 1)
    if decode_main:
        value, unit = w.kv_bytes() / (ms * 1e-3) / 1e9, "GB/s"
        peak, bound, runit = PEAK_HBM_GBS, "hbm", "GB/s"
        algo = w.kv_bytes()
        kname, ksrc = "decode_split_kernel", DECODE_SOURCES
    else:
        value, unit = w.flops() / (ms * 1e-3) / 1e12, "TFLOP/s"
        peak, bound, runit = PEAK_MFMA_TFLOPS[w.dtype], "mfma", "TFLOP/s"
        algo = w.flops()
        kname, ksrc = "prefill_kernel", PREFILL_SOURCES
    log(f"[bench] {w.name}: {ms * 1e3:.1f} us/call, {value:.1f} {unit}")
    # shader clock under this workload's load, against the 2.4 GHz the peaks assume
    qd, kd, vd = inputs
    sclk = None if args.no_sclk else loaded_sclk_mhz(
        torch, lambda: fa.fwd(qd, kd, vd, causal=w.causal, scale=w.softmax_scale, out=out, lse=lse))
    log(f"[bench] shader clock under load: {sclk} MHz (peaks assume 2400)")
    result = {
        "metric": METRIC, "value": round(value, 3), "unit": unit, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic (seeded i.i.d. inputs shaped like the paper's SLM layers)",
        "config": {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "Nq": w.Nq,
                   "Nk": w.Nk, "D": w.D, "causal": w.causal, "scale": w.softmax_scale,
                   "parallelism": "single GPU"},
        "roofline": {"bound": bound, "achieved": round(value, 3), "peak": peak, "unit": runit,
                     "frac": round(value / peak, 4),
                     "traffic": stored_traffic(kname, w.name, ksrc),
                     "kernel": kname, "algorithmic_per_launch": algo,
                     "launch_us": round(ms * 1e3, 3),
                     "sclk_mhz_under_load": sclk,
                     "frac_at_measured_sclk": (round(value / (peak * sclk / 2400.0), 4)
                                               if sclk and bound == "mfma" else None)},
    }
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline: oracle on host cores")
        base, parity = cpu_baseline(torch, fa, w, inputs, out, lse)
        result["cpu_baseline"] = base
        result["parity"] = parity
        log(f"[bench] oracle {base['wall_seconds']} s wall on {base['cores']} cores ({base['cpu_model']}); "
            f"gpu raw max err {parity['max_abs_err_vs_oracle']:.3e}, T1 {parity['t1_verify_max_abs']:.3e}, "
            f"T2 {parity['t2_adjusted_max_abs']:.3e}, rounding floor {parity['rounding_floor']:.3e}")
    del inputs, out, lse
    torch.cuda.empty_cache()

    if not args.no_extras:
        extras = []
        for name in ("gqa_decode_bf16", "mqa_decode_f16", "gqa_prefill_d128_f16",
                     "mqa_prefill_f16", "gqa_prefill_bf16", "tiny_mha_f32"):
            if name == w.name:
                continue
            x = WORKLOADS[name]
            steps = max(5, min(args.steps, 30))
            xms, *_ = run_workload(torch, fa, x, steps, 3, kv_sets=2 if x.Nq == 1 else 1)
            if x.Nq == 1:
                val, u, pk = x.kv_bytes() / (xms * 1e-3) / 1e9, "GB/s", PEAK_HBM_GBS
            else:
                val, u = x.flops() / (xms * 1e-3) / 1e12, "TFLOP/s"
                pk = PEAK_MFMA_TFLOPS[x.dtype]
            extras.append({"workload": name, "us_per_call": round(xms * 1e3, 2),
                           "value": round(val, 2), "unit": u, "frac": round(val / pk, 4),
                           "steps": steps})
            if name == "gqa_decode_bf16":
                result["decode"] = {
                    "workload": name, "metric": "decode KV GB/s (K+V bytes read once)",
                    "value": round(val, 1), "unit": "GB/s", "us_per_call": round(xms * 1e3, 2),
                    "roofline": {"bound": "hbm", "achieved": round(val, 1), "peak": PEAK_HBM_GBS,
                                 "unit": "GB/s", "frac": round(val / PEAK_HBM_GBS, 4),
                                 "traffic": stored_traffic("decode_split_kernel", name,
                                                           DECODE_SOURCES),
                                 "kernel": "decode_split_kernel + decode_combine_kernel",
                                 "algorithmic_per_launch": x.kv_bytes()}}
            log(f"[bench] {name}: {xms * 1e3:.1f} us/call, {val:.1f} {u} ({100 * val / pk:.1f}%)")
            torch.cuda.empty_cache()
        # inter-head packing ablation: workgroup layouts that differ in how many
        # query slots (heads or row blocks) each staged K/V tile serves
        ablation = []
        for name in (() if args.no_ablation else tuple(LAYOUTS)):
            x = WORKLOADS[name]
            steps = max(5, min(args.steps, 20))
            row = {"workload": name, "layouts": []}
            for label, ns, hw in LAYOUTS[name]:
                xms, *_ = run_workload(torch, fa, x, steps, 3, packing=hw, slots=ns)
                row["layouts"].append({
                    "layout": label, "slots_per_workgroup": ns, "heads_per_workgroup": hw,
                    "us": round(xms * 1e3, 2), "tflops": round(x.flops() / (xms * 1e-3) / 1e12, 1),
                    "staged_kv_bytes": staged_kv_bytes(x, ns, hw),
                    "hbm_fetch_bytes": stored_traffic("prefill_kernel", f"{name}_slots{ns}_heads{hw}",
                                                      PREFILL_SOURCES)})
                torch.cuda.empty_cache()
            base = row["layouts"][0]["us"]
            for lay in row["layouts"]:
                lay["speedup_vs_unshared"] = round(base / lay["us"], 3)
            ablation.append(row)
            log(f"[bench] packing {name}: " + ", ".join(
                f"{lay['layout']} {lay['us']} us ({lay['staged_kv_bytes'] / 1e6:.0f} MB staged)"
                for lay in row["layouts"]))
        if ablation:
            result["packing_ablation"] = ablation
        # fused against unfused self-attention (score matrix S in fp32 and
        # weights P in fp16 through HBM), the comparison of the paper's
        # evaluation of its optimised self-attention
        unfused = []
        for name in (() if args.no_ablation else
                     ("gqa_prefill_bf16", "gqa_prefill_d128_f16", "mqa_prefill_f16")):
            x = WORKLOADS[name]
            steps = max(3, min(args.steps, 10))
            row = unfused_vs_fused(torch, fa, x, steps)
            unfused.append(row)
            log(f"[bench] unfused {name}: {row['unfused_us']} us against fused {row['fused_us']} us "
                f"({row['fused_speedup']}x); S/P traffic {row['unfused_gbs']} GB/s")
            torch.cuda.empty_cache()
        if unfused:
            result["unfused_ablation"] = unfused
        # decode against a paged K/V cache (pages of 64 and 256 keys, shuffled)
        xw = WORKLOADS["gqa_decode_bf16"]
        paged = {"workload": xw.name, "metric": "decode KV GB/s, K/V in shuffled pages", "pages": []}
        for ps in (64, 256):
            pus, pgbs = paged_decode(torch, fa, xw, max(5, min(args.steps, 30)), 3, ps)
            paged["pages"].append({"page_size": ps, "us_per_call": round(pus, 2), "value": round(pgbs, 1),
                                   "unit": "GB/s", "frac": round(pgbs / PEAK_HBM_GBS, 4),
                                   "traffic": stored_traffic("decode_split_kernel",
                                                             f"{xw.name}_paged{ps}", DECODE_SOURCES)})
            log(f"[bench] paged decode, pages of {ps}: {pus:.1f} us/call, {pgbs:.0f} GB/s")
        result["paged_decode"] = paged
        if not args.no_ablation:   # same kernel instance as the headline: kept out of its traces
            cp = chunked_prefill(torch, fa, max(5, min(args.steps, 30)), 3)
            result["chunked_prefill"] = cp
            log(f"[bench] chunked prefill 4 x 512 new tokens: {cp['contiguous']['us_per_call']} us "
                f"({cp['contiguous']['tflops']} TFLOP/s), paged 256: {cp['paged256']['us_per_call']} us")
        result["q8_0_gemv"] = q8_decode_step(torch, fa, max(5, min(args.steps, 20)), 3,
                                             not args.no_cpu_baseline)
        # achievable HBM bandwidth for context: a plain 1 GiB device copy
        src = torch.empty(1 << 29, dtype=torch.float16, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        cms = time_calls(torch, [lambda: dst.copy_(src)], 20, 3)
        extras.append({"workload": "device_copy_1GiB", "us_per_call": round(cms * 1e3, 2),
                       "value": round(2 * src.numel() * 2 / (cms * 1e-3) / 1e9, 1),
                       "unit": "GB/s (read + write)"})
        result["workloads"] = extras
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
