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
