"""Seeded random sweeps of the GPU paths against the fp64 oracles, beside the
hand-picked cases: shapes, dtypes, masks, scales, head ratios, cache lengths,
page sizes, Q8_0 matrix sizes and unfused-path shapes drawn from fixed seeds (the draw is printed
with each case so that a failure names it).

Attention: every output and lse compared in verify mode (fp32 output of the
same kernels) within 2e-3, and the shipped output within 2e-3 of the
correctly rounded answer (the tolerance rules of helpers.py).  Paged cache:
equal bit for bit to the contiguous cache path.  Q8_0: within the derived fp32
bound of test_q8_gpu.py.
"""
import random

import numpy as np
import pytest
import torch

import paper_2608_18656_amd as fa
from paper_2608_18656_amd.inputs import DTYPES, make_q8_0, make_qkv

from helpers import check_against, oracle_full

pytestmark = pytest.mark.gpu


def _attention_case(seed):
    r = random.Random(seed)
    dt = r.choice(["bf16", "f16", "f16", "bf16", "f32"])
    D = r.choice([64, 64, 128, 128, 32, 96]) if dt != "f32" else r.choice([64, 32, 128])
    Hkv = r.choice([1, 2, 4, 8])
    G = r.choice([1, 2, 3, 4, 8, 16])
    Hq = Hkv * G
    B = r.choice([1, 1, 2, 3])
    decode = r.random() < 0.35
    Nk = r.randint(1, 1500) if decode else r.randint(1, 700)
    causal = r.random() < 0.6
    Nq = 1 if decode else (r.randint(1, Nk) if causal else r.randint(1, 700))
    scale = r.choice([None, None, 0.5, -0.3, 2.0])
    return B, Hq, Hkv, Nq, Nk, D, causal, dt, scale


@pytest.mark.parametrize("seed", range(40))
def test_random_attention_against_oracle(seed):
    B, Hq, Hkv, Nq, Nk, D, causal, dt, scale = _attention_case(seed)
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    # keep the oracle fast: bound the work of one case
    while B * Hq * Nq * Nk * D > 6e7 and Hq > Hkv:
        Hq -= Hkv
    label = f"seed {seed}: B{B} Hq{Hq} Hkv{Hkv} Nq{Nq} Nk{Nk} D{D} causal={causal} {dt} scale={scale}"
    print(label, flush=True)
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, dt, seed=10_000 + seed)
    o_ref, l_ref = oracle_full(q, k, v, causal, scale)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    verify = dt != "f32"
    o, lse = fa.fwd(qd, kd, vd, causal=causal, scale=scale,
                    out_dtype=torch.float32 if verify else None)
    torch.cuda.synchronize()
    check_against(o, lse, o_ref, l_ref, DTYPES[dt], verify, label)
    if verify:
        o2, lse2 = fa.fwd(qd, kd, vd, causal=causal, scale=scale)
        torch.cuda.synchronize()
        check_against(o2, lse2, o_ref, l_ref, DTYPES[dt], False, label + " shipped")


@pytest.mark.parametrize("seed", range(12))
def test_random_paged_equals_contiguous(seed):
    r = random.Random(500 + seed)
    dt = r.choice(["bf16", "f16"])
    D = r.choice([64, 128])
    Hkv = r.choice([1, 2, 8])
    Hq = Hkv * r.choice([1, 4, 16])
    B = r.randint(1, 4)
    ps = r.choice([64, 128, 256])
    max_pages = r.randint(1, 12)
    Nk = ps * max_pages
    decode = r.random() < 0.5
    causal = (not decode) and r.random() < 0.7
    Nq = 1 if decode else r.randint(1, min(Nk, 200))
    seqlens = [r.randint(0, Nk) for _ in range(B)]
    label = f"seed {seed}: B{B} Hq{Hq} Hkv{Hkv} Nq{Nq} D{D} {dt} page {ps} x {max_pages} lens {seqlens}"
    print(label, flush=True)
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, dt, seed=20_000 + seed)
    num_pages = B * max_pages + r.randint(0, 5)
    perm = torch.randperm(num_pages, generator=torch.Generator().manual_seed(seed))
    table = perm[: B * max_pages].reshape(B, max_pages).to(torch.int32)
    kp = torch.full((num_pages, ps, Hkv, D), float("nan"), dtype=k.dtype)
    vp = torch.full_like(kp, float("nan"))
    kp[table.reshape(-1).long()] = k.reshape(B * max_pages, ps, Hkv, D)
    vp[table.reshape(-1).long()] = v.reshape(B * max_pages, ps, Hkv, D)
    sl = torch.tensor(seqlens, dtype=torch.int32, device="cuda")
    qd = q.cuda()
    o_p, l_p = fa.fwd_kvcache_paged(qd, kp.cuda(), vp.cuda(), table.cuda(), sl, causal=causal,
                                    out_dtype=torch.float32)
    o_c, l_c = fa.fwd_kvcache(qd, k.cuda(), v.cuda(), sl, causal=causal, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(o_p, o_c) and torch.equal(l_p, l_c), label


@pytest.mark.parametrize("seed", range(16))
def test_random_q8_gemv_against_oracle(seed):
    from oracle import q8 as oracle_q8

    r = random.Random(900 + seed)
    M = r.choice([1, 7, 64, 300, 1000, 4099])
    K = 32 * r.choice([1, 2, 3, 17, 64, 65, 130, 176, 331, 480, 512])
    xdt = r.choice(["f16", "bf16", "f32"])
    ydt = r.choice([xdt, "f32"])
    label = f"seed {seed}: M{M} K{K} {xdt}->{ydt}"
    print(label, flush=True)
    w, x = make_q8_0(M, K, seed=30_000 + seed, x_dtype=xdt)
    y = fa.q8_0_gemv(w.cuda(), x.cuda(), out_dtype=DTYPES[ydt])
    torch.cuda.synchronize()
    wn = w.numpy()
    xn = x.float().numpy().astype(np.float64)
    ref = oracle_q8.gemv(wn, xn)
    nb = K // 32
    d = np.abs(np.ascontiguousarray(wn[:, :, 0:2]).view(np.float16).reshape(M, nb).astype(np.float64))
    qa = np.abs(np.ascontiguousarray(wn[:, :, 2:]).view(np.int8).astype(np.float64))
    S = (d * (qa * np.abs(xn).reshape(1, nb, 32)).sum(axis=2)).sum(axis=1)
    bound = (2 * nb + 64) * 2.0 ** -24 * S
    if ydt == "bf16":
        bound = bound + 2.0 ** -8 * (np.abs(ref) + bound)
    elif ydt == "f16":
        bound = bound + 2.0 ** -11 * (np.abs(ref) + bound) + 2.0 ** -25
    err = np.abs(y.float().cpu().numpy().astype(np.float64) - ref)
    assert np.all(err <= bound), label


@pytest.mark.parametrize("seed", range(12))
def test_random_unfused_against_oracle(seed):
    """The unfused path (fa_fwd_unfused) on drawn shapes, every output and lse
    against the oracle in verify mode and as shipped."""
    r = random.Random(1200 + seed)
    dt = r.choice(["bf16", "f16"])
    D = r.choice([64, 128])
    Hkv = r.choice([1, 2, 4])
    Hq = Hkv * r.choice([1, 2, 3, 4, 8])
    B = r.choice([1, 2])
    Nk = r.randint(1, 600)
    causal = r.random() < 0.6
    Nq = r.randint(1, Nk) if causal else r.randint(1, 600)
    scale = r.choice([None, 0.5, -0.3])
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    label = f"seed {seed}: unfused B{B} Hq{Hq} Hkv{Hkv} Nq{Nq} Nk{Nk} D{D} causal={causal} {dt} scale={scale}"
    print(label, flush=True)
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, dt, seed=40_000 + seed)
    o_ref, l_ref = oracle_full(q, k, v, causal, scale)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    o, lse = fa.fwd_unfused(qd, kd, vd, causal=causal, scale=scale, out_dtype=torch.float32)
    torch.cuda.synchronize()
    check_against(o, lse, o_ref, l_ref, DTYPES[dt], True, label)
    o2, lse2 = fa.fwd_unfused(qd, kd, vd, causal=causal, scale=scale)
    torch.cuda.synchronize()
    check_against(o2, lse2, o_ref, l_ref, DTYPES[dt], False, label + " shipped")
