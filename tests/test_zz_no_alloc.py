"""fa_fwd_splitkv_noalloc through the C ABI: two decode calls in a row, the
second on a smaller input, each equal bit for bit to fa_fwd_splitkv on the
same input and split count and within tolerance of the oracle; no device
memory is allocated by the calls; partial results larger than the fixed
scratch are refused with FA_ERR_WORKSPACE before any launch."""
import ctypes

import pytest
import torch

import oracle
from paper_2608_18656_amd import _lib
from paper_2608_18656_amd.inputs import DTYPES, make_qkv

from helpers import check_against, default_scale

pytestmark = pytest.mark.gpu

CODE = {"f16": _lib.FA_F16, "bf16": _lib.FA_BF16}
# B, Hq, Hkv, Nk, D, dtype, splits: a larger call, then a smaller one
CALLS = [(8, 32, 8, 5000, 128, "bf16", 6), (2, 16, 1, 1000, 64, "f16", 0)]


def _call(fn, q, k, v, o, lse, B, Hq, Hkv, Nk, D, dt, S):
    return fn(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), B, Hq, Hkv, 1, Nk, D, 0,
              default_scale(D), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream), CODE[dt], _lib.FA_F32,
              S)


def test_noalloc_matches_splitkv_on_two_calls_in_a_row():
    lib = _lib.load()
    cases = []
    for i, (B, Hq, Hkv, Nk, D, dt, S) in enumerate(CALLS):
        q, k, v = make_qkv(B, Hq, Hkv, 1, Nk, D, dt, seed=400 + i)
        dev = tuple(t.cuda() for t in (q, k, v))
        o_ref = torch.empty((B, 1, Hq, D), dtype=torch.float32, device="cuda")
        l_ref = torch.empty((B, Hq, 1), dtype=torch.float32, device="cuda")
        assert _call(lib.fa_fwd_splitkv, *dev, o_ref, l_ref, B, Hq, Hkv, Nk, D, dt, S) == 0
        o = torch.full_like(o_ref, float("nan"))
        lse = torch.full_like(l_ref, float("nan"))
        cases.append(((q, k, v), dev, o_ref, l_ref, o, lse))
    # set-up: the first call on the device reads the scratch array's address,
    # which makes the runtime place that array in device memory
    (B, Hq, Hkv, Nk, D, dt, S), (_, dev, _, _, o, lse) = CALLS[1], cases[1]
    assert _call(lib.fa_fwd_splitkv_noalloc, *dev, o, lse, B, Hq, Hkv, Nk, D, dt, S) == 0
    torch.cuda.synchronize()
    o.fill_(float("nan"))
    lse.fill_(float("nan"))
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    for (B, Hq, Hkv, Nk, D, dt, S), (_, dev, _, _, o, lse) in zip(CALLS, cases):
        assert _call(lib.fa_fwd_splitkv_noalloc, *dev, o, lse, B, Hq, Hkv, Nk, D, dt, S) == 0
        torch.cuda.synchronize()
    free1 = torch.cuda.mem_get_info()[0]
    assert free0 - free1 < (1 << 20), (free0, free1)   # no workspace allocated by the calls
    for (B, Hq, Hkv, Nk, D, dt, S), (cpu, _, o_ref, l_ref, o, lse) in zip(CALLS, cases):
        assert torch.equal(o, o_ref) and torch.equal(lse, l_ref), (B, Hq, Nk, D)
        o_or, l_or = oracle.attention(*cpu, False, default_scale(D))
        check_against(o, lse, o_or, l_or, DTYPES[dt], True, f"noalloc B{B} Hq{Hq} Nk{Nk} D{D}")


def test_noalloc_refuses_partials_beyond_the_scratch():
    lib = _lib.load()
    far = [ctypes.c_void_p(k << 40) for k in range(1, 6)]   # never dereferenced: refused before launch
    B, Hq, Hkv, Nk, D, S = 256, 64, 8, 65536, 128, 16       # 256 * 64 * 16 * 130 * 4 B = 136 MB
    st = lib.fa_fwd_splitkv_noalloc(*far, B, Hq, Hkv, 1, Nk, D, 0, 0.088, None, _lib.FA_BF16, _lib.FA_BF16, S)
    assert st == 10
