"""GPU parity of the Q8_0 matrix-vector product (fa_q8_0_gemv, the decode-time
linear layers of Sec. 4.3) against the fp64 oracle (oracle/q8.py) on the same
seeded bytes, every output element compared.

Tolerance (derived from the kernel's arithmetic).  The kernel forms each
block's sum of q_j * x_j with fp32 multiply-adds (the int8 values and the
binary16 scale are exact in fp32; x is exact after widening), multiplies by
the block's scale with one more multiply-add into a per-lane fp32 sum, and
adds the lanes' sums in a tree of at most 6 levels.  Every rounding is
relative with unit 2^-24, so with S[m] = sum_b |d_b| sum_j |q_bj x_j| the
error is at most n * 2^-24 * S[m] to first order, n = 32 + 2 nb + 6 bounding
the number of roundings on any path (nb blocks per row).  The test uses
n = 2 nb + 64.  The shipped fp16 / bf16 output adds its own round-to-nearest
(half an ulp: 2^-11 |y|, plus 2^-25 below fp16's normal range, or 2^-8 |y|
for bf16).

Coverage: every input/output dtype pair; K of one block, odd block counts
(the 16-bit load path), even counts with a ragged last round of lanes, the
largest K each workgroup size stages in LDS and the first K beyond it; grid-stride
row counts; the four TinyLlama-shaped projection matrices at full size;
extreme scales (largest binary16, subnormal, zero, negative) and int8 -128;
determinism; a non-default stream; a weight matrix of more than 2^31 bytes.
"""
import numpy as np
import pytest
import torch

import paper_2608_18656_amd as fa
from oracle import q8 as oracle_q8
from paper_2608_18656_amd.inputs import DTYPES, Q8_LAYER_SHAPES, make_q8_0, pack_q8_0

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
U32 = 2.0 ** -24


def _abs_terms(w: np.ndarray, x: np.ndarray) -> np.ndarray:
    """S[m] = sum_b |d_b| sum_j |q_bj| |x_j| (numpy's own int8 / float16 views)."""
    M, nb, _ = w.shape
    d = np.abs(np.ascontiguousarray(w[:, :, 0:2]).view(np.float16).reshape(M, nb).astype(np.float64))
    q = np.abs(np.ascontiguousarray(w[:, :, 2:]).view(np.int8).astype(np.float64))
    ax = np.abs(x).reshape(1, nb, 32)
    return (d * (q * ax).sum(axis=2)).sum(axis=1)


def _check(w_cpu: torch.Tensor, x_cpu: torch.Tensor, y_gpu: torch.Tensor, label: str,
           rows=None):
    w = w_cpu.numpy()
    x = x_cpu.float().numpy().astype(np.float64)
    if rows is not None:
        w = w[rows]
    nb = w.shape[1]
    ref = oracle_q8.gemv(w, x)
    got = y_gpu.float().cpu().numpy().astype(np.float64)
    if rows is not None:
        got = got[rows]
    bound = (2 * nb + 64) * U32 * _abs_terms(w, x)
    if y_gpu.dtype == torch.bfloat16:
        bound = bound + 2.0 ** -8 * (np.abs(ref) + bound)
    elif y_gpu.dtype == torch.float16:
        bound = bound + 2.0 ** -11 * (np.abs(ref) + bound) + 2.0 ** -25
    err = np.abs(got - ref)
    ratio = float(np.max(err / np.maximum(bound, 1e-300)))
    print(f"[q8] {label}: max err {err.max():.3e}, max err/bound {ratio:.3f}", flush=True)
    assert np.all(np.isfinite(got)), label
    assert np.all(err <= bound), (label, int(np.argmax(err / np.maximum(bound, 1e-300))))


def _run(w_cpu, x_cpu, out_dtype=None):
    w = w_cpu.to(DEV)
    x = x_cpu.to(DEV)
    y = fa.q8_0_gemv(w, x, out_dtype=out_dtype)
    torch.cuda.synchronize()
    return y


DTYPE_PAIRS = [("f16", None), ("f16", "f32"), ("bf16", None), ("bf16", "f32"), ("f32", None)]

SHAPES = [
    (1, 32),             # one block: odd path, one lane of work per row
    (3, 96),             # odd block count
    (2, 64),             # one pair of blocks
    (257, 2048),         # 64 blocks: 32 lanes per row, two rows per wave
    (100, 5632),         # feed-forward width (176 blocks)
    (64, 4160),          # 130 blocks: 65 pairs, a ragged second round of lanes
    (9, 32 * 131),       # odd, several rounds of lanes
    (33, 15168),         # largest K staged in LDS by a 4-wave workgroup
    (17, 15200),         # first K staged by a 16-wave workgroup (LDS beyond 64 KB)
    (6, 16384),
    (5, 32 * 1001),      # odd, 16-wave workgroup
    (3, 37568),          # largest K staged in LDS
    (2, 37600),          # first K whose x is read from global memory
    (2, 32 * 1201),      # odd, x from global memory
]


@pytest.mark.parametrize("xdt,ydt", DTYPE_PAIRS, ids=[f"{a}-{b or a}" for a, b in DTYPE_PAIRS])
@pytest.mark.parametrize("M,K", SHAPES, ids=[f"{m}x{k}" for m, k in SHAPES])
def test_q8_gemv_matches_oracle(M, K, xdt, ydt):
    w, x = make_q8_0(M, K, seed=7000 + M + K, x_dtype=xdt)
    y = _run(w, x, out_dtype=DTYPES[ydt] if ydt else None)
    assert y.dtype == (DTYPES[ydt] if ydt else DTYPES[xdt])
    _check(w, x, y, f"{M}x{K} {xdt}->{ydt or xdt}")


@pytest.mark.parametrize("M,K", [(70001, 32), (100003, 64), (40000, 2048)])
def test_q8_gemv_grid_stride_row_counts(M, K):
    """More rows than one sweep of the grid covers."""
    w, x = make_q8_0(M, K, seed=M, x_dtype="bf16")
    y = _run(w, x, out_dtype=torch.float32)
    _check(w, x, y, f"{M}x{K} grid-stride")


@pytest.mark.parametrize("i", range(len(Q8_LAYER_SHAPES)), ids=[s[0] for s in Q8_LAYER_SHAPES])
def test_q8_gemv_tinyllama_projections_full_size(i):
    name, M, K = Q8_LAYER_SHAPES[i]
    w, x = make_q8_0(M, K, seed=9000 + i, x_dtype="bf16")
    y32 = _run(w, x, out_dtype=torch.float32)
    _check(w, x, y32, f"{name} {M}x{K} fp32 out")
    y = _run(w, x)
    _check(w, x, y, f"{name} {M}x{K} bf16 out")


def test_q8_gemv_extreme_scales_and_values():
    M, K = 48, 256
    nb = K // 32
    gen = torch.Generator().manual_seed(11)
    specials = torch.tensor([65504.0, -65504.0, 2.0 ** -24, -(2.0 ** -24), 0.0, -0.0, 6.1e-5,
                             1.0, -1.0, 0.5], dtype=torch.float32)
    d = specials[torch.randint(0, len(specials), (M, nb), generator=gen)].to(torch.float16)
    q = torch.randint(-128, 128, (M, nb, 32), generator=gen, dtype=torch.int32)
    q[0::3] = -128                                         # the one value with no positive twin
    q[1::3, :, ::2] = 127
    w = pack_q8_0(d, q.to(torch.int8))
    for xdt in ("f16", "bf16", "f32"):
        x = (torch.randn((K,), generator=gen) * 8).to(DTYPES[xdt])
        _check(w, x, _run(w, x, out_dtype=torch.float32), f"specials x={xdt} fp32 out")
        if xdt == "bf16":   # fp16 outputs would overflow at these scales
            _check(w, x, _run(w, x), f"specials x={xdt}")


def test_q8_gemv_zero_weights_give_exact_zero():
    M, K = 20, 512
    w = pack_q8_0(torch.zeros((M, K // 32), dtype=torch.float16),
                  torch.ones((M, K // 32, 32), dtype=torch.int8))
    x = torch.randn((K,), generator=torch.Generator().manual_seed(3)).to(torch.bfloat16)
    y = _run(w, x, out_dtype=torch.float32)
    assert torch.equal(y.cpu(), torch.zeros(M))


def test_q8_gemv_deterministic_and_stream_ordered():
    M, K = 4099, 2048
    w_cpu, x_cpu = make_q8_0(M, K, seed=5, x_dtype="f16")
    w, x = w_cpu.to(DEV), x_cpu.to(DEV)
    a = fa.q8_0_gemv(w, x, out_dtype=torch.float32)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        out = torch.empty(M, dtype=torch.float32, device=DEV)
        b = fa.q8_0_gemv(w, x, out=out, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    _check(w_cpu, x_cpu, a, "4099x2048 f16")


def test_q8_gemv_weights_beyond_2_31_bytes():
    """1,000,000 rows of 2176 bytes (2.18 GB): rows whose bytes lie past 2^31
    (and the row that straddles it) are checked against the oracle."""
    M, K = 1_000_000, 2048
    nb = K // 32
    row_bytes = nb * 34
    straddle = (1 << 31) // row_bytes
    pattern, x_cpu = make_q8_0(512, K, seed=77, x_dtype="bf16")
    w = pattern.to(DEV).repeat((M + 511) // 512, 1, 1)[:M].contiguous()
    rows = np.array([0, 1, 511, 512, straddle - 1, straddle, straddle + 1, M // 2, M - 2, M - 1])
    fresh, _ = make_q8_0(len(rows), K, seed=78)
    w[torch.from_numpy(rows).to(DEV)] = fresh.to(DEV)
    x = x_cpu.to(DEV)
    y = fa.q8_0_gemv(w, x, out_dtype=torch.float32)
    torch.cuda.synchronize()
    got = y.cpu()[torch.from_numpy(rows)]
    _check(fresh, x_cpu, got, "2.18 GB weights, sampled rows")
    # rows not overwritten repeat the pattern: spot-check a stretch past 2^31 bytes
    tail = y[straddle + 2: straddle + 2 + 512].cpu()
    idx = (np.arange(straddle + 2, straddle + 2 + 512)) % 512
    _check(torch.from_numpy(pattern.numpy()[idx]), x_cpu, tail, "pattern rows past 2^31 bytes")
    del w
    torch.cuda.empty_cache()


def test_q8_gemv_errors_reported():
    w, x = make_q8_0(4, 64, seed=1)
    w, x = w.to(DEV), x.to(DEV)
    lib_err = fa.FaError
    with pytest.raises(lib_err) as e:
        fa.q8_0_gemv(w, x, out_dtype=torch.float16)       # bf16 x, f16 y
    assert e.value.status == 9
    with pytest.raises(ValueError):
        fa.q8_0_gemv(w, x[:32])                            # K mismatch
