"""Seeded synthetic inputs shared by the GPU path's tests/benchmark and the oracle.

This module holds only random draws, shapes and dtype casts -- none of the
attention arithmetic.  Values are drawn in float32 with a CPU
``torch.Generator`` in the order q, k, v and then rounded to the storage dtype
with round-to-nearest-even (``Tensor.to``), so every consumer sees the same bits.

The shapes stand in for the small-language-model layers of the paper's
evaluation (Table 3: TinyLlama 32/4/64, Llama 3.2 32/8/64, Qwen2.5 16/2/128,
Pythia-410M 16/16/64 as Hq/Hkv/D); the paper measures on model activations,
which are replaced here by i.i.d. draws.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch

DTYPES = {"f16": torch.float16, "bf16": torch.bfloat16, "f32": torch.float32}


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    Nq: int
    Nk: int
    D: int
    causal: bool
    dtype: str
    seed: int
    qk_mult: float = 1.0       # q and k (and v when normal) are N(0,1) * qk_mult
    v_uniform: bool = False    # v ~ U[-1, 1) instead of the normal draw
    scale: float = field(default=float("nan"))

    @property
    def softmax_scale(self) -> float:
        return 1.0 / math.sqrt(self.D) if math.isnan(self.scale) else self.scale

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    def visible_pairs(self) -> int:
        """Number of (query, key) pairs the mask leaves visible, per (b, h)."""
        if not self.causal:
            return self.Nq * self.Nk
        off = self.Nk - self.Nq
        return sum(i + off + 1 for i in range(self.Nq))

    def flops(self) -> int:
        """Algorithmic FLOPs: 2*D for q.k plus 2*D for p*v per visible pair."""
        return 4 * self.B * self.Hq * self.D * self.visible_pairs()

    def kv_bytes(self) -> int:
        """K and V read once, in the storage dtype."""
        esize = torch.finfo(DTYPES[self.dtype]).bits // 8
        return 2 * self.B * self.Nk * self.Hkv * self.D * esize


# The five benchmark configurations (the fifth has a decode and a prefill half).
WORKLOADS = {
    "tiny_mha_f32": Workload("tiny_mha_f32", 1, 2, 2, 128, 128, 64, False, "f32", 1001),
    "gqa_prefill_bf16": Workload("gqa_prefill_bf16", 1, 32, 8, 2048, 2048, 64, True, "bf16",
                                 1002),
    "gqa_prefill_d128_f16": Workload("gqa_prefill_d128_f16", 2, 32, 8, 4096, 4096, 128, True,
                                     "f16", 1003, qk_mult=0.5),
    "gqa_decode_bf16": Workload("gqa_decode_bf16", 16, 32, 8, 1, 8192, 128, False, "bf16",
                                1004),
    "mqa_decode_f16": Workload("mqa_decode_f16", 64, 16, 1, 1, 32768, 64, False, "f16", 1005,
                               v_uniform=True),
    "mqa_prefill_f16": Workload("mqa_prefill_f16", 1, 16, 1, 16384, 16384, 64, True, "f16",
                                1006, v_uniform=True),
}


def make_qkv(B: int, Hq: int, Hkv: int, Nq: int, Nk: int, D: int, dtype: str, seed: int,
             qk_mult: float = 1.0, v_uniform: bool = False):
    """Seeded q [B,Nq,Hq,D], k, v [B,Nk,Hkv,D] on the CPU in ``dtype``."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(int(seed))
    q = torch.randn((B, Nq, Hq, D), generator=gen, dtype=torch.float32)
    k = torch.randn((B, Nk, Hkv, D), generator=gen, dtype=torch.float32)
    if v_uniform:
        v = torch.rand((B, Nk, Hkv, D), generator=gen, dtype=torch.float32) * 2.0 - 1.0
    else:
        v = torch.randn((B, Nk, Hkv, D), generator=gen, dtype=torch.float32)
    if qk_mult != 1.0:
        q.mul_(qk_mult)
        k.mul_(qk_mult)
        if not v_uniform:
            v.mul_(qk_mult)
    t = DTYPES[dtype]
    return q.to(t), k.to(t), v.to(t)


def make_workload(w: Workload, seed: int | None = None):
    return make_qkv(w.B, w.Hq, w.Hkv, w.Nq, w.Nk, w.D, w.dtype,
                    w.seed if seed is None else seed, w.qk_mult, w.v_uniform)


def shrink(w: Workload, **over) -> Workload:
    """A copy of ``w`` with some sizes replaced (smaller parity cases)."""
    d = {f: getattr(w, f) for f in w.__dataclass_fields__}
    d.update(over)
    return Workload(**d)


# Q8_0 weights for the decode-time linear layers.  Shapes of the TinyLlama-1.1B
# projections the paper runs with Q8_0 weights (Table 3: 32 query heads and
# 4 key/value heads of 64; hidden size 2048, feed-forward size 5632, 22
# layers), with the projections that share an input stored as one matrix:
# (name, M rows, K columns).
Q8_LAYER_SHAPES = (
    ("qkv", 2048 + 2 * 256, 2048),
    ("o", 2048, 2048),
    ("gate_up", 2 * 5632, 2048),
    ("down", 2048, 5632),
)
Q8_LAYERS = 22


def make_q8_0(M: int, K: int, seed: int, x_dtype: str = "bf16"):
    """Seeded Q8_0 weights and activations on the CPU.

    Returns (w, x): w uint8 [M, K/32, 34], each block a binary16 scale (bytes
    0-1, little-endian) then 32 int8 values; x [K] in ``x_dtype``.  Values are
    drawn directly in the stored form (no quantisation step): the int8 values
    are N(0, 40^2) rounded and clipped to [-127, 127] with one entry per block
    set to +-127 (a block quantised from its largest magnitude has one), the
    scales |N(0, 1)| * 2e-4 + 1e-4 rounded to binary16 (weights of standard
    deviation about 0.02), and x N(0, 1) rounded to ``x_dtype``."""
    if K % 32 != 0 or K < 32 or M < 1:
        raise ValueError("need M >= 1 and K a positive multiple of 32")
    nb = K // 32
    gen = torch.Generator(device="cpu")
    gen.manual_seed(int(seed))
    q = torch.randn((M, nb, 32), generator=gen, dtype=torch.float32).mul_(40.0).round_()
    q.clamp_(-127.0, 127.0)
    pos = torch.randint(0, 32, (M, nb, 1), generator=gen)
    sgn = torch.randint(0, 2, (M, nb, 1), generator=gen).to(torch.float32).mul_(254.0).sub_(127.0)
    q.scatter_(2, pos, sgn)
    d = torch.randn((M, nb), generator=gen, dtype=torch.float32).abs_().mul_(2e-4).add_(1e-4)
    x = torch.randn((K,), generator=gen, dtype=torch.float32)
    return pack_q8_0(d.to(torch.float16), q.to(torch.int8)), x.to(DTYPES[x_dtype])


def pack_q8_0(d: torch.Tensor, q: torch.Tensor) -> torch.Tensor:
    """Byte layout of Q8_0 rows: d float16 [M, nb] and q int8 [M, nb, 32] ->
    uint8 [M, nb, 34] (scale bytes first, little-endian, then the 32 values)."""
    M, nb = d.shape
    w = torch.empty((M, nb, 34), dtype=torch.uint8)
    w[:, :, 0:2] = d.contiguous().view(torch.uint8).reshape(M, nb, 2)
    w[:, :, 2:] = q.contiguous().view(torch.uint8)
    return w
