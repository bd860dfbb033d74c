"""GPU tests of attention against a paged K/V cache (fa_fwd_kvcache_paged):
pools of fixed-size pages addressed through a per-sequence block table, for
decode and chunked prefill.

Each case scatters a contiguous cache [B, Nk, Hkv, D] over a pool of pages in
a seeded random order (pages no sequence owns are filled with NaN, so a read
of a wrong page cannot go unnoticed) and checks that the paged call gives bit
for bit what fa_fwd_kvcache gives on the contiguous cache (same kernels, same
key order), and that the result matches the fp64 oracle on each sequence's
valid rows (rows that see no key: 0 and lse -inf).  Also: the pages of every
sequence in order (a pool that is the contiguous cache itself), page sizes
64 to 512, block table entries outside the pool (clamped into it), and
argument errors.
"""
import pytest
import torch

import oracle
import paper_2608_18656_amd as fa
from paper_2608_18656_amd.inputs import DTYPES, make_qkv

from helpers import check_against, default_scale

pytestmark = pytest.mark.gpu


def _paginate(k, v, page_size, seed, extra_pages=3):
    """Scatter k, v [B, Nk, Hkv, D] (Nk a multiple of page_size) over a pool of
    B * Nk / page_size + extra_pages pages in a random order.  Returns the two
    pools [num_pages, page_size, Hkv, D] and the block table [B, max_pages]."""
    B, Nk, Hkv, D = k.shape
    max_pages = Nk // page_size
    num_pages = B * max_pages + extra_pages
    gen = torch.Generator().manual_seed(seed)
    perm = torch.randperm(num_pages, generator=gen)
    table = perm[: B * max_pages].reshape(B, max_pages).to(torch.int32)
    kp = torch.full((num_pages, page_size, Hkv, D), float("nan"), dtype=k.dtype)
    vp = torch.full_like(kp, float("nan"))
    kp[table.reshape(-1).long()] = k.reshape(B * max_pages, page_size, Hkv, D)
    vp[table.reshape(-1).long()] = v.reshape(B * max_pages, page_size, Hkv, D)
    return kp, vp, table


def _check_case(B, Hq, Hkv, Nq, Nk, D, dt, causal, seqlens, page_size, seed, out_dtype=torch.float32):
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, dt, seed=seed)
    kp, vp, table = _paginate(k, v, page_size, seed)
    scale = default_scale(D)
    sl = torch.tensor(seqlens, dtype=torch.int32, device="cuda")
    qd = q.cuda()
    o_p, l_p = fa.fwd_kvcache_paged(qd, kp.cuda(), vp.cuda(), table.cuda(), sl, causal=causal, scale=scale,
                                    out_dtype=out_dtype)
    o_c, l_c = fa.fwd_kvcache(qd, k.cuda(), v.cuda(), sl, causal=causal, scale=scale, out_dtype=out_dtype)
    torch.cuda.synchronize()
    assert torch.equal(o_p, o_c), "paged and contiguous outputs differ"
    assert torch.equal(l_p, l_c), "paged and contiguous lse differ"
    if out_dtype != torch.float32:
        return
    for b, L in enumerate(seqlens):
        first = max(Nq - L, 0) if causal else (Nq if L == 0 else 0)
        if first > 0:
            assert torch.all(o_p[b, :first] == 0) and torch.all(torch.isneginf(l_p[b, :, :first]))
        if first < Nq:
            o_ref, l_ref = oracle.attention(q[b:b + 1, first:].contiguous(), k[b:b + 1, :L].contiguous(),
                                            v[b:b + 1, :L].contiguous(), causal, scale)
            check_against(o_p[b:b + 1, first:].contiguous(), l_p[b:b + 1, :, first:].contiguous(),
                          o_ref, l_ref, DTYPES[dt], True, f"paged b={b} L={L}")


CASES = [
    # decode: GQA D=128 bf16, pages of 64; lengths include 0, 1, a page edge and the full cache
    (5, 32, 8, 1, 2560, 128, "bf16", False, [2560, 1, 64, 0, 1777], 64),
    # decode: MQA D=64 f16, pages of 128
    (3, 16, 1, 1, 4096, 64, "f16", False, [4096, 129, 2000], 128),
    # chunked prefill, causal, D=64, pages of 64: a chunk longer than one sequence
    (3, 8, 2, 70, 640, 64, "bf16", True, [640, 70, 33], 64),
    # chunked prefill, causal, D=128 f16, pages of 256
    (2, 32, 8, 96, 1024, 128, "f16", True, [1024, 500], 256),
    # non-causal prefill against the cache, pages of 512
    (2, 4, 4, 50, 1024, 64, "f16", False, [1000, 512], 512),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"B{c[0]}Hq{c[1]}Hkv{c[2]}Nq{c[3]}Nk{c[4]}D{c[5]}"
                                                      f"{c[6]}{'c' if c[7] else ''}p{c[9]}")
def test_paged_equals_contiguous_and_oracle(case):
    B, Hq, Hkv, Nq, Nk, D, dt, causal, seqlens, ps = case
    _check_case(B, Hq, Hkv, Nq, Nk, D, dt, causal, seqlens, ps, seed=3000 + Nk + Nq)


@pytest.mark.parametrize("Nq,causal", [(1, False), (40, True)])
def test_paged_shipped_output_equals_contiguous(Nq, causal):
    _check_case(2, 16, 4, Nq, 1024, 64, "bf16", causal, [1024, 300], 128, seed=77, out_dtype=None)


def test_pages_in_order_equal_the_contiguous_cache():
    """Identity block table over a pool that is the contiguous cache itself."""
    B, Hq, Hkv, Nq, Nk, D, ps = 3, 32, 8, 1, 2048, 128, 256
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, "bf16", seed=91)
    kd, vd = k.cuda(), v.cuda()
    table = torch.arange(B * (Nk // ps), dtype=torch.int32, device="cuda").reshape(B, Nk // ps)
    sl = torch.tensor([2048, 1500, 7], dtype=torch.int32, device="cuda")
    o_p, l_p = fa.fwd_kvcache_paged(q.cuda(), kd.reshape(-1, ps, Hkv, D), vd.reshape(-1, ps, Hkv, D), table, sl,
                                    out_dtype=torch.float32)
    o_c, l_c = fa.fwd_kvcache(q.cuda(), kd, vd, sl, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(o_p, o_c) and torch.equal(l_p, l_c)


@pytest.mark.parametrize("Nq,causal", [(1, False), (64, True)], ids=["decode", "prefill"])
def test_block_table_entries_outside_the_pool_are_clamped(Nq, causal):
    """Entries below 0 or past the pool read the first or last page: the
    result equals a call with the table clamped on the host."""
    B, Hq, Hkv, Nk, D, ps = 2, 8, 2, 512, 64, 64
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, "f16", seed=5)
    kp, vp, table = _paginate(k, v, ps, seed=5, extra_pages=0)
    num_pages = kp.shape[0]
    bad = table.clone()
    bad[0, 1] = -7
    bad[1, 2] = num_pages + 1000
    clamped = bad.clamp(0, num_pages - 1)
    sl = torch.tensor([Nk, Nk], dtype=torch.int32, device="cuda")
    args = (q.cuda(), kp.cuda(), vp.cuda())
    o1, l1 = fa.fwd_kvcache_paged(*args, bad.cuda(), sl, causal=causal, out_dtype=torch.float32)
    o2, l2 = fa.fwd_kvcache_paged(*args, clamped.cuda(), sl, causal=causal, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_paged_argument_errors():
    q, k, v = make_qkv(1, 4, 4, 1, 128, 64, "f16", seed=1)
    kp, vp, table = _paginate(k, v, 64, seed=1)
    qd, kpd, vpd, td = q.cuda(), kp.cuda(), vp.cuda(), table.cuda()
    sl = torch.tensor([128], dtype=torch.int32, device="cuda")
    with pytest.raises(fa.FaError) as e:   # pages of 32 keys
        fa.fwd_kvcache_paged(qd, kpd.reshape(-1, 32, 4, 64), vpd.reshape(-1, 32, 4, 64), td, sl)
    assert e.value.status == 2
    q32, kp32, vp32 = qd.float(), kpd.float(), vpd.float()
    with pytest.raises(fa.FaError) as e:   # fp32 data
        fa.fwd_kvcache_paged(q32, kp32, vp32, td, sl)
    assert e.value.status == 9
