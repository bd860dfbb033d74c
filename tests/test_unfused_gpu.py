"""GPU parity of the unfused self-attention path (fa_fwd_unfused: scores,
softmax and P.V kernels through an HBM workspace) against the fp64 oracle,
on the same seeded inputs as the fused path.

Output and lse: every element within the tolerance rules of helpers.py (verify
mode: fp32 output within 2e-3; shipped output within 2e-3 beyond its half
ulp), on edge shapes (ragged rows and keys, Nk < 64, causal with Nq < Nk, Nq >
Nk without a mask, group sizes 1, 2, 3, 4 and 16, both head sizes, rows
held by one, two and four softmax waves and rows longer than that, negative
and zero scales) and on the three prefill workloads at reduced sizes and at
full size (in the launch configuration the benchmark times), every element.
Intermediate results: the materialised weights P equal the oracle's
normalised weights to fp16 rounding, with exact zeros past each row's visible
keys up to the last tile the P.V kernel reads; the materialised scores S give
the oracle's weights under an fp64 softmax.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_18656_amd as fa
from paper_2608_18656_amd.inputs import DTYPES, WORKLOADS, make_qkv, make_workload, shrink

from helpers import check_against, oracle_full

pytestmark = pytest.mark.gpu

EDGE = [
    # B, Hq, Hkv, Nq, Nk, D, causal, dtype
    (1, 8, 2, 200, 200, 64, 1, "bf16"),     # G = 4: four heads per workgroup, ragged tail
    (2, 4, 4, 130, 250, 128, 1, "f16"),     # MHA (four row blocks per workgroup), Nq < Nk
    (1, 6, 2, 70, 70, 64, 0, "f16"),        # G = 3
    (1, 4, 2, 33, 1000, 64, 1, "bf16"),     # G = 2, a long cache
    (2, 16, 1, 100, 300, 128, 0, "bf16"),   # MQA, G = 16
    (1, 2, 1, 1, 500, 64, 1, "f16"),        # one query row
    (3, 2, 1, 5, 3, 64, 0, "bf16"),         # Nq > Nk without a mask, Nk < 64
    (1, 2, 2, 1, 1, 128, 1, "f16"),         # one key
    (1, 8, 8, 64, 64, 64, 1, "bf16"),       # exact tiles
    (1, 4, 1, 129, 129, 128, 1, "bf16"),    # one row past a 128-row workgroup
    (1, 2, 1, 3, 6000, 64, 1, "f16"),       # softmax: two waves per row
    (1, 2, 2, 40, 9000, 128, 1, "bf16"),    # softmax: four waves per row, one segment partly visible
    (1, 2, 1, 2, 20000, 64, 0, "bf16"),     # softmax: four waves per row and a streamed tail
]


def _workspace(B, Hq, Nq, Nk):
    return torch.empty(fa.unfused_workspace_bytes(B, Hq, Nq, Nk), dtype=torch.uint8, device="cuda")


def _check_shape(B, Hq, Hkv, Nq, Nk, D, causal, dt, scale, seed):
    label = f"unfused B{B} Hq{Hq} Hkv{Hkv} Nq{Nq} Nk{Nk} D{D} causal={causal} {dt} scale={scale}"
    print(label, flush=True)
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, dt, seed=seed)
    o_ref, l_ref = oracle_full(q, k, v, bool(causal), scale)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    ws = _workspace(B, Hq, Nq, Nk)
    o, lse = fa.fwd_unfused(qd, kd, vd, causal=bool(causal), scale=scale, out_dtype=torch.float32,
                            workspace=ws)
    torch.cuda.synchronize()
    check_against(o, lse, o_ref, l_ref, DTYPES[dt], True, label)
    o2, lse2 = fa.fwd_unfused(qd, kd, vd, causal=bool(causal), scale=scale, workspace=ws)
    torch.cuda.synchronize()
    check_against(o2, lse2, o_ref, l_ref, DTYPES[dt], False, label + " shipped")
    return q, k, v, ws


def _views(ws, B, Hq, Nq, Nk):
    NkP = (Nk + 63) // 64 * 64
    n = B * Hq * Nq * NkP
    S = ws[: 4 * n].view(torch.float32).reshape(B, Hq, Nq, NkP).cpu().numpy().astype(np.float64)
    P = ws[4 * n: 6 * n].view(torch.float16).reshape(B, Hq, Nq, NkP).cpu().numpy().astype(np.float64)
    return S, P, NkP


@pytest.mark.parametrize("shape", EDGE, ids=lambda s: "x".join(map(str, s)))
def test_unfused_edge_shapes_and_intermediates(shape):
    B, Hq, Hkv, Nq, Nk, D, causal, dt = shape
    scale = D ** -0.5
    q, k, v, ws = _check_shape(B, Hq, Hkv, Nq, Nk, D, causal, dt, scale, seed=700 + Nq + Nk)
    S, P, NkP = _views(ws, B, Hq, Nq, Nk)
    w = oracle.weights(q, k, v, bool(causal), scale)            # [B, Hq, Nq, Nk]
    for i in range(Nq):
        kend = min(Nk, i + Nk - Nq + 1) if causal else Nk
        zend = min(NkP, (kend + 63) // 64 * 64 + 64)
        wi, pi, si = w[:, :, i, :kend], P[:, :, i, :kend], S[:, :, i, :kend]
        # P: the oracle's weights rounded to fp16 (half an ulp, subnormals
        # included), plus the fp32 error of the score and the exponential
        assert np.all(np.abs(pi - wi) <= 2.0 ** -11 * wi + 2.0 ** -25 + 1e-5 * wi), f"P row {i}"
        assert np.all(P[:, :, i, kend:zend] == 0.0), f"P padding row {i}"
        # S: its fp64 softmax gives the oracle's weights
        e = np.exp(si - si.max(axis=-1, keepdims=True))
        sm = e / e.sum(axis=-1, keepdims=True)
        assert np.all(np.abs(sm - wi) <= 1e-4 * wi + 1e-9), f"S row {i}"


@pytest.mark.parametrize("scale", [-0.3, 0.0, 2.0])
def test_unfused_negative_zero_and_large_scale(scale):
    _check_shape(1, 4, 2, 90, 150, 64, 1, "f16", scale, seed=731)


@pytest.mark.parametrize("name", ["gqa_prefill_bf16", "gqa_prefill_d128_f16", "mqa_prefill_f16"])
def test_unfused_prefill_workloads_reduced_every_element(name):
    w = shrink(WORKLOADS[name], Nq=333, Nk=333)
    _check_shape(w.B, w.Hq, w.Hkv, w.Nq, w.Nk, w.D, int(w.causal), w.dtype, w.softmax_scale,
                 seed=w.seed)


@pytest.mark.parametrize("name", ["gqa_prefill_bf16", "gqa_prefill_d128_f16", "mqa_prefill_f16"])
def test_unfused_prefill_full_size_every_element(name):
    w = WORKLOADS[name]
    q, k, v = make_workload(w)
    scale = w.softmax_scale
    print(f"unfused {name} full size, every element", flush=True)
    o_r, l_r = oracle.attention_parallel(q, k, v, w.causal, scale, workers=oracle.default_workers())
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    ws = _workspace(w.B, w.Hq, w.Nq, w.Nk)
    for verify in (True, False):
        o, lse = fa.fwd_unfused(qd, kd, vd, causal=w.causal, scale=scale,
                                out_dtype=torch.float32 if verify else None, workspace=ws)
        torch.cuda.synchronize()
        check_against(o, lse, o_r, l_r, DTYPES[w.dtype], verify,
                      f"unfused {name} full every element verify={verify}")
    del ws
    torch.cuda.empty_cache()


def test_unfused_workspace_reused_across_shapes_and_deterministic():
    """One workspace serves calls of different shapes in order; repeated calls
    give the same bits."""
    big = _workspace(2, 8, 300, 300)
    for B, Hq, Hkv, Nq, Nk, D, causal, dt in [(2, 8, 2, 300, 300, 64, 1, "bf16"),
                                              (1, 4, 1, 50, 700, 128, 0, "f16"),
                                              (2, 8, 4, 120, 120, 64, 1, "f16")]:
        q, k, v = (t.cuda() for t in make_qkv(B, Hq, Hkv, Nq, Nk, D, dt, seed=740 + Nk))
        o1, l1 = fa.fwd_unfused(q, k, v, causal=bool(causal), workspace=big)
        o2, l2 = fa.fwd_unfused(q, k, v, causal=bool(causal), workspace=big)
        torch.cuda.synchronize()
        assert torch.equal(o1, o2) and torch.equal(l1, l2)
        o_ref, l_ref = oracle.attention(q.cpu(), k.cpu(), v.cpu(), bool(causal), D ** -0.5)
        check_against(o1, l1, o_ref, l_ref, DTYPES[dt], False, f"reuse {B}x{Hq}x{Nq}x{Nk}")


def test_unfused_refuses_small_workspace_and_fp32():
    q, k, v = (t.cuda() for t in make_qkv(1, 2, 1, 64, 64, 64, "f16", seed=750))
    small = torch.empty(fa.unfused_workspace_bytes(1, 2, 64, 64) - 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(fa.FaError) as e:
        fa.fwd_unfused(q, k, v, workspace=small)
    assert e.value.status == 10
    with pytest.raises(fa.FaError) as e:
        fa.fwd_unfused(q.float(), k.float(), v.float())
    assert e.value.status == 9
