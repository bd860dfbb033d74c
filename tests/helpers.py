"""Shared helpers for the GPU parity tests: run the HIP path through the
Python binding of the C ABI, run the fp64 oracle on the same input bits, and
apply the tolerance rules.

Tolerance (the 2e-3 max-abs bound on fp16 / bf16 inputs with fp32
accumulation):
  T1  verify mode (fp32 output of the same kernels): max |o - o_ref| <= 2e-3
      and max |lse - lse_ref| <= 2e-3.
  T2  shipped fp16 / bf16 output: the part of |o - o_ref| beyond half a unit
      in the last place of the output format, max(|o - o_ref| - ulp/2), is
      <= 2e-3 -- i.e. within 2e-3 of a correctly rounded answer.  (Rounding
      the exact result to bf16 alone can move it by up to 7.8e-3 where
      |o| is near 4, so a literal 2e-3 on bf16 storage cannot be met.)
fp32 inputs: max |o - o_ref| <= 2e-3 as well, plus a 1e-4 quality bound.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle
import paper_2608_18656_amd as fa

TOL = 2e-3
MANT = {torch.float16: 10, torch.bfloat16: 7, torch.float32: 23}
MIN_EXP = {torch.float16: -14, torch.bfloat16: -126, torch.float32: -126}


def to_dev(*ts, device="cuda"):
    return [t.to(device) for t in ts]


def gpu_attention(q, k, v, causal, scale, out_dtype=None, num_splits=None):
    """Run the HIP path on CPU input tensors; returns float64 numpy (o, lse)."""
    qd, kd, vd = to_dev(q, k, v)
    o, lse = fa.fwd(qd, kd, vd, causal=causal, scale=scale, out_dtype=out_dtype,
                    num_splits=num_splits)
    torch.cuda.synchronize()
    return o, lse


def to_np(t):
    return oracle.to_f64(t)


def half_ulp(x: np.ndarray, dtype) -> np.ndarray:
    """Half the spacing of ``dtype`` at magnitude |x| (subnormal-aware)."""
    ax = np.abs(x)
    e = np.floor(np.log2(np.maximum(ax, 2.0 ** MIN_EXP[dtype])))
    return 0.5 * np.exp2(e - MANT[dtype])


def errors(o_gpu, lse_gpu, o_ref, lse_ref, dtype):
    """(raw max-abs, rounding-adjusted max-abs, lse max-abs)."""
    og = to_np(o_gpu)
    diff = np.abs(og - o_ref)
    raw = float(diff.max())
    adj = raw
    if dtype in (torch.float16, torch.bfloat16):
        hu = half_ulp(np.maximum(np.abs(og), np.abs(o_ref)), dtype)
        adj = float(np.max(diff - hu))
    le = float(np.abs(to_np(lse_gpu) - lse_ref).max()) if lse_gpu is not None else 0.0
    return raw, adj, le


def check_against(o_gpu, lse_gpu, o_ref, lse_ref, dtype, verify: bool, label=""):
    raw, adj, le = errors(o_gpu, lse_gpu, o_ref, lse_ref, dtype)
    assert np.all(np.isfinite(to_np(o_gpu))), f"{label}: non-finite output"
    if verify or dtype == torch.float32:
        assert raw <= TOL, f"{label}: T1 max|o-ref| = {raw:.3e}"
        if dtype == torch.float32:
            assert raw <= 1e-4, f"{label}: fp32 path max|o-ref| = {raw:.3e}"
    else:
        assert adj <= TOL, f"{label}: T2 max(|o-ref| - ulp/2) = {adj:.3e} (raw {raw:.3e})"
    assert le <= TOL, f"{label}: max|lse-ref| = {le:.3e}"
    return raw, adj, le


def oracle_full(q, k, v, causal, scale, workers=None):
    workers = workers or oracle.default_workers()
    if q.numel() * k.shape[1] < 2e7:
        return oracle.attention(q, k, v, causal, scale)
    return oracle.attention_parallel(q, k, v, causal, scale, workers=workers)


def sample_rows(B, Hq, Nq, n, seed):
    """Row triples (b, h, i): first and last rows of every head plus random ones."""
    r = np.random.default_rng(seed)
    rows = set()
    for b in range(B):
        for h in range(Hq):
            for i in (0, Nq - 1):
                rows.add((b, h, i))
    while len(rows) < n + 2 * B * Hq:
        rows.add((int(r.integers(B)), int(r.integers(Hq)), int(r.integers(Nq))))
    return np.array(sorted(rows), dtype=np.int32)


def default_scale(D):
    return 1.0 / math.sqrt(D)
