"""Seeded input generators: determinism, shapes, dtypes, distributions."""
import torch

from paper_2608_18656_amd.inputs import WORKLOADS, make_qkv, shrink


def test_same_seed_same_bits_and_dtype():
    a = make_qkv(1, 4, 2, 5, 7, 8, "bf16", 123)
    b = make_qkv(1, 4, 2, 5, 7, 8, "bf16", 123)
    c = make_qkv(1, 4, 2, 5, 7, 8, "bf16", 124)
    for x, y in zip(a, b):
        assert x.dtype == torch.bfloat16
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))
    assert not torch.equal(a[0], c[0])
    assert a[0].shape == (1, 5, 4, 8) and a[1].shape == (1, 7, 2, 8)


def test_rounding_is_nearest_even_from_float32():
    gen = torch.Generator().manual_seed(9)
    q32 = torch.randn((1, 5, 4, 8), generator=gen)
    q16, _, _ = make_qkv(1, 4, 2, 5, 7, 8, "f16", 9)
    assert torch.equal(q16, q32.to(torch.float16))


def test_value_distributions():
    q, k, v = make_qkv(1, 2, 1, 64, 4096, 64, "f16", 5, v_uniform=True)
    assert float(v.abs().max()) <= 1.0 and float(v.float().mean().abs()) < 0.02
    q, k, v = make_qkv(1, 2, 1, 64, 4096, 64, "f32", 5, qk_mult=0.5)
    assert abs(float(k.std()) - 0.5) < 0.01


def test_workload_table_counts():
    w = WORKLOADS["gqa_prefill_bf16"]
    assert w.G == 4 and w.causal and w.visible_pairs() == 2048 * 2049 // 2
    assert w.flops() == 4 * 32 * 64 * (2048 * 2049 // 2)
    assert WORKLOADS["gqa_decode_bf16"].kv_bytes() == 536870912
    assert WORKLOADS["mqa_decode_f16"].kv_bytes() == 536870912
    s = shrink(w, Nq=100, Nk=100)
    assert s.Nq == 100 and s.Hq == 32 and s.visible_pairs() == 5050


def test_q8_inputs_deterministic_and_laid_out():
    """make_q8_0: same seed, same bytes; scale little-endian in bytes 0-1 of
    each block, the 32 values in bytes 2-33; values within [-127, 127] with a
    +-127 in every block; positive scales of weights about 0.02 in size."""
    import numpy as np

    from paper_2608_18656_amd.inputs import Q8_LAYER_SHAPES, make_q8_0, pack_q8_0

    w1, x1 = make_q8_0(40, 256, seed=3)
    w2, x2 = make_q8_0(40, 256, seed=3)
    w3, _ = make_q8_0(40, 256, seed=4)
    assert torch.equal(w1, w2) and torch.equal(x1.view(torch.int16), x2.view(torch.int16))
    assert not torch.equal(w1, w3)
    assert w1.shape == (40, 8, 34) and w1.dtype == torch.uint8 and x1.dtype == torch.bfloat16
    wn = w1.numpy()
    d = wn[:, :, 0].astype(np.uint16) | (wn[:, :, 1].astype(np.uint16) << 8)
    dv = d.view(np.float16).astype(np.float64)
    q = np.ascontiguousarray(wn[:, :, 2:]).view(np.int8).astype(np.int64)
    assert np.all(dv > 0) and 1e-4 <= float(np.median(dv)) <= 5e-4
    assert q.min() >= -127 and q.max() <= 127
    assert np.all(np.abs(q).max(axis=2) == 127)
    wstd = float((dv[:, :, None] * q).std())
    assert 0.005 < wstd < 0.05
    # pack_q8_0 is the inverse of this decoding
    back = pack_q8_0(torch.from_numpy(dv.astype(np.float16)), torch.from_numpy(q.astype(np.int8)))
    assert torch.equal(back, w1)
    assert [s[0] for s in Q8_LAYER_SHAPES] == ["qkv", "o", "gate_up", "down"]


def test_tolerance_rules():
    """The parity checks: fp32 (verify) output within 2e-3 of the oracle; a
    shipped fp16 / bf16 output within 2e-3 of the correctly rounded answer
    (so the exact result rounded to bf16 passes even where bf16 spacing is
    above 2e-3, and 3e-3 beyond that rounding fails); lse within 2e-3."""
    import numpy as np
    import pytest

    import helpers

    rng = np.random.default_rng(0)
    o_ref = rng.uniform(-4, 4, size=(1, 8, 2, 16))
    l_ref = rng.uniform(0, 5, size=(1, 2, 8))
    lse = torch.from_numpy(l_ref.astype(np.float32))
    rounded = torch.from_numpy(o_ref).to(torch.bfloat16)
    assert float(np.abs(rounded.double().numpy() - o_ref).max()) > 2e-3   # bf16 spacing at 2-4
    helpers.check_against(rounded, lse, o_ref, l_ref, torch.bfloat16, False, "rounded")
    worse = rounded.double().numpy().copy()
    worse[0, 3, 1, 5] += 3e-3 + float(helpers.half_ulp(np.array([worse[0, 3, 1, 5]]), torch.bfloat16)[0]) * 2
    with pytest.raises(AssertionError):
        helpers.check_against(torch.from_numpy(worse), lse, o_ref, l_ref, torch.bfloat16, False, "worse")
    f32 = torch.from_numpy(o_ref.astype(np.float32))
    helpers.check_against(f32, lse, o_ref, l_ref, torch.bfloat16, True, "verify")
    off = f32.clone()
    off[0, 0, 0, 0] += 2.5e-3
    with pytest.raises(AssertionError):
        helpers.check_against(off, lse, o_ref, l_ref, torch.bfloat16, True, "verify off")
    with pytest.raises(AssertionError):
        helpers.check_against(f32, lse + 3e-3, o_ref, l_ref, torch.bfloat16, True, "lse off")
