"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the
same seeded input bits, element by element.  Tolerance rules in helpers.py.

Coverage: the six benchmark workloads at sizes the oracle finishes in seconds
(spanning several tiles and a ragged tail) with every output compared; the
two decode workloads at full size with every output compared; the three
prefill workloads at full size on sampled rows and with every output
compared (the oracle fanned out over the host's cores); edge shapes (Nk = 1, ragged
tiles, causal with Nq < Nk, group sizes 1 to 32, odd group sizes, negative
and zero scale, the vector-ALU path for fp32 and other head dimensions);
forced split counts including empty splits; determinism; error reporting;
a caller-owned decode workspace; the prefill query-head packings (bitwise
agreement); K/V caches with per-sequence lengths (decode, chunked prefill,
rows with no visible key); tensors of more than 2^31 elements.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2608_18656_amd as fa
from paper_2608_18656_amd.inputs import DTYPES, WORKLOADS, make_qkv, make_workload, shrink

from helpers import (check_against, default_scale, errors, gpu_attention, oracle_full,
                     sample_rows, to_np)

pytestmark = pytest.mark.gpu

# Reduced sizes: same heads / D / dtype / mask / distributions as the full
# workloads, sequence lengths cut to ragged values that span several tiles.
REDUCED = {
    "tiny_mha_f32": {},
    "gqa_prefill_bf16": dict(Nq=333, Nk=333),
    "gqa_prefill_d128_f16": dict(Nq=300, Nk=300),
    "gqa_decode_bf16": dict(Nk=1000),
    "mqa_decode_f16": dict(B=8, Nk=3001),
    "mqa_prefill_f16": dict(Nq=517, Nk=517),
}


def _run_and_check(w, verify, label, num_splits=None):
    q, k, v = make_workload(w)
    scale = w.softmax_scale
    o_ref, l_ref = oracle_full(q, k, v, w.causal, scale)
    out_dtype = torch.float32 if verify else None
    o, lse = gpu_attention(q, k, v, w.causal, scale, out_dtype=out_dtype, num_splits=num_splits)
    raw, adj, le = check_against(o, lse, o_ref, l_ref, DTYPES[w.dtype], verify, label)
    print(f"[parity] {label}: raw {raw:.3e} adjusted {adj:.3e} lse {le:.3e}", flush=True)


@pytest.mark.parametrize("verify", [True, False], ids=["fp32out", "shipped"])
@pytest.mark.parametrize("name", list(REDUCED))
def test_workloads_reduced_every_element(name, verify):
    w = shrink(WORKLOADS[name], **REDUCED[name])
    if verify and w.dtype == "f32":
        pytest.skip("fp32 inputs already produce fp32 output")
    _run_and_check(w, verify, f"{name} reduced {w.Nq}x{w.Nk}")


@pytest.mark.parametrize("verify", [True, False], ids=["fp32out", "shipped"])
@pytest.mark.parametrize("name", ["gqa_decode_bf16", "mqa_decode_f16"])
def test_decode_full_size_every_element(name, verify):
    _run_and_check(WORKLOADS[name], verify, f"{name} full")


@pytest.mark.parametrize("name", ["gqa_prefill_bf16", "gqa_prefill_d128_f16", "mqa_prefill_f16"])
def test_prefill_full_size_sampled_rows(name):
    w = WORKLOADS[name]
    q, k, v = make_workload(w)
    scale = w.softmax_scale
    rows = sample_rows(w.B, w.Hq, w.Nq, 192, seed=w.seed)
    o_r, l_r = oracle.attention_rows(q, k, v, w.causal, scale, rows,
                                     workers=oracle.default_workers())
    for verify in (True, False):
        o, lse = gpu_attention(q, k, v, w.causal, scale,
                               out_dtype=torch.float32 if verify else None)
        b_i, h_i, q_i = (torch.from_numpy(rows[:, j]).long().to(o.device) for j in range(3))
        og = o[b_i, q_i, h_i].cpu()
        lg = lse[b_i, h_i, q_i].cpu()
        raw, adj, le = check_against(og, lg, o_r, l_r, DTYPES[w.dtype], verify,
                                     f"{name} full sampled verify={verify}")
        print(f"[parity] {name} full sampled ({len(rows)} rows) verify={verify}: raw {raw:.3e} "
              f"adjusted {adj:.3e} lse {le:.3e}", flush=True)
    # a property that holds at any size: every output element is finite
    assert torch.isfinite(o.float()).all()


# Large D = 64 grids (more two-part workgroups than two per CU: the prefill
# kernel's two-key-part layout), bf16 and fp16, causal with ragged rows and
# keys and non-causal, sampled rows against the oracle.
LARGE_D64 = [(2, 64, 8, 4100, 4100, True, "bf16"), (1, 32, 8, 3000, 3100, False, "bf16"),
             (3, 16, 2, 2000, 2333, True, "f16")]


@pytest.mark.parametrize("shape", LARGE_D64, ids=lambda s: "x".join(map(str, s)))
def test_prefill_large_d64_grids_sampled_rows(shape):
    B, Hq, Hkv, Nq, Nk, causal, dt = shape
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, 64, dt, seed=zlib.crc32(repr(shape).encode()))
    scale = default_scale(64)
    rows = sample_rows(B, Hq, Nq, 160, seed=7)
    o_r, l_r = oracle.attention_rows(q, k, v, causal, scale, rows, workers=oracle.default_workers())
    for verify in (True, False):
        o, lse = gpu_attention(q, k, v, causal, scale, out_dtype=torch.float32 if verify else None)
        b_i, h_i, q_i = (torch.from_numpy(rows[:, j]).long().to(o.device) for j in range(3))
        check_against(o[b_i, q_i, h_i].cpu(), lse[b_i, h_i, q_i].cpu(), o_r, l_r, DTYPES[dt], verify,
                      f"large D=64 {shape} verify={verify}")
    assert torch.isfinite(o.float()).all()


@pytest.mark.parametrize("name", ["gqa_prefill_bf16", "gqa_prefill_d128_f16", "mqa_prefill_f16"])
def test_prefill_full_size_every_element(name):
    """Every output element and lse of the three prefill workloads at full
    size (the launch configuration the benchmark times), in verify mode and as
    shipped, against the fp64 oracle fanned out over the host's cores (at most
    16 processes; a few seconds per workload on the GPU host)."""
    w = WORKLOADS[name]
    q, k, v = make_workload(w)
    scale = w.softmax_scale
    print(f"[parity] {name} full size, every element: oracle on {oracle.default_workers()} processes",
          flush=True)
    o_ref, l_ref = oracle.attention_parallel(q, k, v, w.causal, scale, workers=oracle.default_workers())
    for verify in (True, False):
        o, lse = gpu_attention(q, k, v, w.causal, scale, out_dtype=torch.float32 if verify else None)
        raw, adj, le = check_against(o, lse, o_ref, l_ref, DTYPES[w.dtype], verify,
                                     f"{name} full every element verify={verify}")
        print(f"[parity] {name} full, every element, verify={verify}: raw {raw:.3e} adjusted {adj:.3e} "
              f"lse {le:.3e}", flush=True)


EDGE = [
    # B, Hq, Hkv, Nq, Nk, D, causal, dtype
    (1, 2, 2, 1, 1, 64, 0, "f16"),        # decode, one key
    (2, 8, 1, 1, 77, 128, 0, "bf16"),     # MQA decode, ragged chunk
    (1, 4, 4, 1, 5000, 64, 1, "f16"),     # causal decode == non-causal
    (1, 48, 3, 1, 300, 64, 0, "f16"),     # G = 16
    (1, 64, 2, 1, 300, 128, 0, "bf16"),   # G = 32: two 16-head column blocks
    (1, 6, 2, 1, 129, 64, 0, "f16"),      # G = 3
    (1, 2, 1, 1, 1, 64, 1, "bf16"),       # Nq = Nk = 1
    (1, 4, 4, 65, 65, 64, 1, "f16"),      # MHA, ragged rows and keys
    (2, 6, 3, 100, 130, 128, 1, "bf16"),  # G = 2, causal with Nq < Nk
    (1, 3, 1, 37, 200, 64, 1, "f16"),     # G = 3, causal with Nq < Nk
    (1, 8, 2, 2, 1000, 128, 1, "f16"),    # two query rows against a long cache
    (1, 32, 1, 129, 129, 64, 0, "bf16"),  # MQA prefill, G = 32
    (1, 8, 8, 64, 64, 128, 1, "bf16"),    # exact tiles
    (3, 4, 2, 31, 31, 64, 0, "f16"),      # fewer rows than one wave block
    (1, 2, 2, 33, 47, 40, 1, "f16"),      # vector-ALU path, D = 40
    (1, 2, 1, 20, 20, 256, 0, "bf16"),    # vector-ALU path, D = 256
    (1, 4, 2, 9, 9, 8, 1, "f32"),         # vector-ALU path, D = 8
    (1, 2, 2, 70, 70, 128, 1, "f32"),     # fp32, D = 128
    (2, 4, 1, 1, 300, 64, 0, "f32"),      # fp32 decode shape
]


@pytest.mark.parametrize("shape", EDGE, ids=lambda s: "x".join(map(str, s)))
def test_edge_shapes(shape):
    B, Hq, Hkv, Nq, Nk, D, causal, dt = shape
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, dt, seed=zlib.crc32(repr(shape).encode()))
    scale = default_scale(D)
    o_ref, l_ref = oracle.attention(q, k, v, bool(causal), scale)
    for verify in ([True, False] if dt != "f32" else [False]):
        o, lse = gpu_attention(q, k, v, bool(causal), scale,
                               out_dtype=torch.float32 if verify else None)
        check_against(o, lse, o_ref, l_ref, DTYPES[dt], verify, f"edge {shape} verify={verify}")


@pytest.mark.parametrize("scale", [-0.3, 0.0, 2.0])
@pytest.mark.parametrize("Nq", [1, 70])
def test_negative_zero_and_large_scale(scale, Nq):
    q, k, v = make_qkv(1, 8, 2, Nq, 150, 64, "f16", seed=77)
    o_ref, l_ref = oracle.attention(q, k, v, Nq > 1, scale)
    o, lse = gpu_attention(q, k, v, Nq > 1, scale, out_dtype=torch.float32)
    check_against(o, lse, o_ref, l_ref, torch.float16, True, f"scale {scale} Nq {Nq}")


@pytest.mark.parametrize("splits", [1, 3, 64, 256])
def test_forced_split_counts_including_empty_splits(splits):
    q, k, v = make_qkv(2, 16, 4, 1, 1000, 128, "bf16", seed=5)
    scale = default_scale(128)
    o_ref, l_ref = oracle.attention(q, k, v, False, scale)
    o, lse = gpu_attention(q, k, v, False, scale, out_dtype=torch.float32, num_splits=splits)
    check_against(o, lse, o_ref, l_ref, torch.bfloat16, True, f"splits {splits}")


def test_deterministic_bitwise():
    for shape in [(1, 32, 8, 300, 300, 64, True, "bf16"), (4, 32, 8, 1, 3000, 128, False, "bf16")]:
        B, Hq, Hkv, Nq, Nk, D, causal, dt = shape
        q, k, v = [t.cuda() for t in make_qkv(B, Hq, Hkv, Nq, Nk, D, dt, seed=9)]
        o1, l1 = fa.fwd(q, k, v, causal=causal)
        o2, l2 = fa.fwd(q, k, v, causal=causal)
        torch.cuda.synchronize()
        assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
        assert torch.equal(l1, l2)


def test_side_stream_lse_optional_and_output_buffer_reuse():
    q, k, v = [t.cuda() for t in make_qkv(1, 8, 2, 200, 200, 64, "f16", seed=3)]
    o_ref, l_ref = oracle.attention(q.cpu(), k.cpu(), v.cpu(), True, 0.125)
    s = torch.cuda.Stream()
    out = torch.empty_like(q)
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        o, lse = fa.fwd(q, k, v, causal=True, scale=0.125, out=out, return_lse=False)
    s.synchronize()
    assert lse is None and o.data_ptr() == out.data_ptr()
    _, adj, _ = errors(o, None, o_ref, l_ref, torch.float16)
    assert adj <= 2e-3


def test_errors_are_reported():
    q, k, v = [t.cuda() for t in make_qkv(1, 6, 4, 8, 8, 64, "f16", seed=1)]
    with pytest.raises(fa.FaError) as e:
        fa.fwd(q, k, v)
    assert e.value.status == 3
    q, k, v = [t.cuda() for t in make_qkv(1, 4, 4, 9, 8, 64, "f16", seed=1)]
    with pytest.raises(fa.FaError) as e:
        fa.fwd(q, k, v, causal=True)
    assert e.value.status == 5
    q, k, v = [t.cuda() for t in make_qkv(1, 4, 4, 1, 8, 64, "f16", seed=1)]
    with pytest.raises(fa.FaError) as e:
        fa.fwd(q, k, v, num_splits=300)
    assert e.value.status == 12


def test_values_near_fp16_range_in_bf16_inputs():
    """bf16 values are converted to fp16 for the probability x value product;
    values up to 6e4 stay finite and accurate."""
    q, k, v = make_qkv(1, 4, 1, 40, 40, 64, "bf16", seed=12)
    v = (v.float() * 1e4).to(torch.bfloat16)
    o_ref, l_ref = oracle.attention(q, k, v, True, 0.125)
    o, lse = gpu_attention(q, k, v, True, 0.125, out_dtype=torch.float32)
    og = to_np(o)
    rel = np.abs(og - o_ref).max() / np.abs(o_ref).max()
    assert np.isfinite(og).all() and rel < 1e-3


def test_decode_calls_with_changing_shapes():
    """Consecutive decode calls with different batch / head layouts and split
    counts share the library's buffers; each must still match the oracle."""
    shapes = [(16, 32, 8, 1000, 128, "bf16", 4), (8, 16, 1, 3001, 64, "f16", 8),
              (2, 64, 2, 700, 128, "bf16", 3), (16, 32, 8, 1000, 128, "bf16", 4),
              (1, 16, 16, 2000, 64, "f16", 0), (8, 16, 1, 3001, 64, "f16", 8)]
    for i, (B, Hq, Hkv, Nk, D, dt, S) in enumerate(shapes):
        q, k, v = make_qkv(B, Hq, Hkv, 1, Nk, D, dt, seed=500 + i)
        o_ref, l_ref = oracle.attention(q, k, v, False, default_scale(D))
        o, lse = gpu_attention(q, k, v, False, default_scale(D), out_dtype=torch.float32,
                               num_splits=S)
        check_against(o, lse, o_ref, l_ref, DTYPES[dt], True, f"call {i} {B}x{Hq}x{Hkv}")


def test_caller_owned_workspace():
    """fa_set_workspace: a caller buffer of exactly fa_workspace_bytes gives
    bitwise the same result as the library-owned workspace; a smaller one is
    refused with FA_ERR_WORKSPACE before any launch; one overlapping an
    input is refused with FA_ERR_ALIAS; clearing returns to the library's."""
    B, Hq, Hkv, Nk, D, S = 4, 32, 8, 1000, 128, 4
    q, k, v = make_qkv(B, Hq, Hkv, 1, Nk, D, "bf16", seed=77)
    qd, kd, vd = (t.cuda() for t in (q, k, v))
    scale = default_scale(D)
    o_lib, l_lib = fa.fwd(qd, kd, vd, scale=scale, num_splits=S, out_dtype=torch.float32)
    need = fa.workspace_bytes(B, Hq, Hkv, 1, Nk, D, "bf16", S)
    assert need > 0
    buf = torch.empty(need, dtype=torch.uint8, device="cuda")
    try:
        fa.set_workspace(buf)
        o_usr, l_usr = fa.fwd(qd, kd, vd, scale=scale, num_splits=S, out_dtype=torch.float32)
        torch.cuda.synchronize()
        assert torch.equal(o_usr, o_lib) and torch.equal(l_usr, l_lib)
        fa.set_workspace(buf[: need - 16])
        with pytest.raises(fa.FaError) as e:
            fa.fwd(qd, kd, vd, scale=scale, num_splits=S)
        assert e.value.status == 10
        fa.set_workspace(kd.view(torch.uint8)[:need])
        with pytest.raises(fa.FaError) as e:
            fa.fwd(qd, kd, vd, scale=scale, num_splits=S)
        assert e.value.status == 8
    finally:
        fa.set_workspace(None)
    o_again, _ = fa.fwd(qd, kd, vd, scale=scale, num_splits=S, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(o_again, o_lib)
    o_ref, l_ref = oracle.attention(q, k, v, False, scale)
    check_against(o_usr, l_usr, o_ref, l_ref, DTYPES["bf16"], True, "caller workspace")


def _layouts(G):
    """Every (slots, heads) workgroup layout fa_fwd_slots takes for group size G."""
    return [(s, h) for s in (1, 2, 4, 8) for h in (1, 2, 4, 8) if h <= s and s % h == 0 and G % h == 0]


@pytest.mark.parametrize("full", [False, True], ids=["reduced", "full_size"])
@pytest.mark.parametrize("name", ["gqa_prefill_bf16", "gqa_prefill_d128_f16", "mqa_prefill_f16"])
def test_head_packing_schedules_agree_bitwise(name, full):
    """Every workgroup layout -- 1, 2, 4 or 8 query slots sharing each staged
    K/V tile, 1 to 8 of them query heads of one K/V group (the inter-head
    packing) -- against the default one: every row's arithmetic is the same,
    so the outputs agree bit for bit (as shipped and in verify mode), and the
    unshared one-slot layout matches the oracle on the reduced shapes."""
    w = WORKLOADS[name] if full else shrink(WORKLOADS[name], **REDUCED[name])
    q, k, v = make_workload(w)
    qd, kd, vd = (t.cuda() for t in (q, k, v))
    G = w.Hq // w.Hkv
    for odt in (torch.float32, None):
        ref_o, ref_l = fa.fwd(qd, kd, vd, causal=w.causal, scale=w.softmax_scale, out_dtype=odt)
        torch.cuda.synchronize()
        outs = {}
        for slots, hw in _layouts(G):
            o, lse = fa.fwd(qd, kd, vd, causal=w.causal, scale=w.softmax_scale, out_dtype=odt,
                            slots_per_workgroup=slots, heads_per_workgroup=hw)
            torch.cuda.synchronize()
            assert torch.equal(o, ref_o) and torch.equal(lse, ref_l), f"{slots} slots, {hw} heads"
            outs[(slots, hw)] = (o, lse)
        for hw in (1, 2, 4):   # fa_fwd_packed: the default four slots
            if G % hw == 0:
                o, lse = fa.fwd(qd, kd, vd, causal=w.causal, scale=w.softmax_scale, out_dtype=odt,
                                heads_per_workgroup=hw)
                torch.cuda.synchronize()
                assert torch.equal(o, ref_o) and torch.equal(lse, ref_l), f"packed {hw}"
        if odt is torch.float32 and not full:
            o_ref, l_ref = oracle_full(q, k, v, w.causal, w.softmax_scale)
            check_against(outs[(1, 1)][0], outs[(1, 1)][1], o_ref, l_ref, DTYPES[w.dtype], True,
                          f"{name} one slot")


@pytest.mark.parametrize("shape", [(1, 16, 2, 70, 70, 64, 1, "bf16"), (2, 6, 3, 100, 130, 128, 1, "f16"),
                                   (1, 16, 1, 45, 200, 64, 0, "f16"), (1, 8, 8, 33, 33, 128, 1, "bf16")],
                         ids=lambda s: "x".join(map(str, s)))
def test_workgroup_layouts_against_oracle(shape):
    """The one-, two- and eight-slot layouts on ragged rows and keys, causal
    with Nq < Nk and MHA, each against the oracle (as shipped and in verify
    mode)."""
    B, Hq, Hkv, Nq, Nk, D, causal, dt = shape
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, dt, seed=zlib.crc32(repr(shape).encode()))
    scale = default_scale(D)
    o_ref, l_ref = oracle.attention(q, k, v, bool(causal), scale)
    qd, kd, vd = (t.cuda() for t in (q, k, v))
    for slots, hw in _layouts(Hq // Hkv):
        if slots == 4:
            continue
        for verify in (True, False):
            o, lse = fa.fwd(qd, kd, vd, causal=bool(causal), scale=scale,
                            out_dtype=torch.float32 if verify else None,
                            slots_per_workgroup=slots, heads_per_workgroup=hw)
            torch.cuda.synchronize()
            check_against(o, lse, o_ref, l_ref, DTYPES[dt], verify, f"{shape} {slots} slots {hw} heads")


def _kvcache_check(q, k, v, seqlens, causal, scale, dt, label):
    """fa_fwd_kvcache against the oracle run on each sequence's valid cache
    rows; query rows that see no key must give 0 and lse -inf."""
    qd, kd, vd = (t.cuda() for t in (q, k, v))
    sl = torch.tensor(seqlens, dtype=torch.int32, device="cuda")
    o, lse = fa.fwd_kvcache(qd, kd, vd, sl, causal=causal, scale=scale, out_dtype=torch.float32)
    torch.cuda.synchronize()
    Nq = q.shape[1]
    for b, L in enumerate(seqlens):
        first = max(Nq - L, 0) if causal else (Nq if L == 0 else 0)   # first row with a key
        if first > 0:
            assert torch.all(o[b, :first] == 0), f"{label} b={b}: keyless rows not 0"
            assert torch.all(torch.isneginf(lse[b, :, :first])), f"{label} b={b}: keyless lse"
        if first < Nq:
            o_ref, l_ref = oracle.attention(q[b:b + 1, first:].contiguous(), k[b:b + 1, :L].contiguous(),
                                            v[b:b + 1, :L].contiguous(), causal, scale)
            check_against(o[b:b + 1, first:].contiguous(), lse[b:b + 1, :, first:].contiguous(),
                          o_ref, l_ref, DTYPES[dt], True, f"{label} b={b} L={L}")
    return o, lse


@pytest.mark.parametrize("case", [
    # decode against caches of different fill, including an empty one
    (4, 32, 8, 1, 3000, 128, "bf16", False, [3000, 1, 1777, 0]),
    (3, 16, 1, 1, 2500, 64, "f16", True, [2500, 33, 1024]),
    # chunked prefill: Nq new tokens at the end of each sequence
    (3, 8, 2, 70, 600, 64, "f16", True, [600, 70, 333]),
    (2, 32, 8, 64, 512, 128, "bf16", True, [512, 200]),
    # grids large enough for eight-slot workgroups (the default at D = 64)
    (4, 64, 8, 512, 1200, 64, "bf16", True, [1200, 512, 700, 1000]),
    (4, 64, 8, 512, 1200, 64, "f16", True, [1200, 0, 700, 37]),   # and keyless rows
    (4, 64, 8, 512, 1100, 128, "f16", True, [1100, 512, 640, 900]),
    # a chunk longer than its sequence: the first rows see no key
    (2, 4, 4, 100, 256, 128, "bf16", True, [40, 256]),
    # the vector-ALU kernel (fp32)
    (2, 2, 2, 20, 150, 64, "f32", False, [150, 17]),
], ids=lambda c: f"B{c[0]}Hq{c[1]}Hkv{c[2]}Nq{c[3]}Nk{c[4]}D{c[5]}{c[6]}{'c' if c[7] else ''}")
def test_kvcache_per_sequence_lengths(case):
    B, Hq, Hkv, Nq, Nk, D, dt, causal, seqlens = case
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, dt, seed=900 + B * Nq)
    _kvcache_check(q, k, v, seqlens, causal, default_scale(D), dt, "kvcache")


@pytest.mark.parametrize("shape", [(2, 32, 8, 1, 2000, 128, "bf16", False),
                                   (1, 32, 8, 333, 333, 64, "bf16", True),
                                   (1, 16, 1, 200, 260, 64, "f16", True),
                                   (4, 64, 8, 600, 600, 64, "f16", True)])
def test_kvcache_full_lengths_equal_fa_fwd_bitwise(shape):
    B, Hq, Hkv, Nq, Nk, D, dt, causal = shape
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, dt, seed=950 + Nq)
    qd, kd, vd = (t.cuda() for t in (q, k, v))
    sl = torch.full((B,), Nk, dtype=torch.int32, device="cuda")
    o1, l1 = fa.fwd(qd, kd, vd, causal=causal, out_dtype=torch.float32)
    o2, l2 = fa.fwd_kvcache(qd, kd, vd, sl, causal=causal, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


@pytest.mark.parametrize("Nq,causal", [(1, False), (64, False), (64, True)],
                         ids=["decode", "prefill", "prefill_causal"])
def test_offsets_beyond_2_31_elements(Nq, causal):
    """K and V of 2 x 2^31 elements (about 8.6 GB each): batch element 1
    starts past 2^31, so any 32-bit index arithmetic would wrap.  Its output
    must equal, bit for bit, a call on that element alone (whose indices are
    small; the decode call gets a fixed split count, since the default one
    depends on B)."""
    B, Hq, Hkv, Nk, D = 2, 32, 8, 1 << 21, 128
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2024)
    k = torch.randn((B, Nk, Hkv, D), generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    v = torch.randn((B, Nk, Hkv, D), generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    q = torch.randn((B, Nq, Hq, D), generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    assert k[1].numel() >= 1 << 31
    S = 16 if Nq == 1 else None   # the same decode split count for both calls
    o, lse = fa.fwd(q, k, v, causal=causal, out_dtype=torch.float32, num_splits=S)
    o1, lse1 = fa.fwd(q[1:2], k[1:2], v[1:2], causal=causal, out_dtype=torch.float32, num_splits=S)
    torch.cuda.synchronize()
    assert torch.isfinite(o).all()
    assert torch.equal(o[1:2], o1) and torch.equal(lse[1:2], lse1)
    del k, v
    torch.cuda.empty_cache()
