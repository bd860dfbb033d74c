"""Pins of the Q8_0 matrix-vector oracle (oracle/q8_oracle.c) against what
fixes it independently of its own code: numpy's IEEE binary16 decoding of
every 16-bit pattern, numpy's float64 matrix-vector product on the weights
dequantized with numpy's int8 and float16 views, exact values for one-hot and
all-ones blocks, the byte order of the scale, and linearity.  CPU only."""
import numpy as np
import pytest

from oracle import q8


def _blocks(rng, M, K, scale_bits=None):
    """Random Q8_0 rows: uint8 [M, K/32, 34] with varied binary16 scales."""
    nb = K // 32
    w = np.zeros((M, nb, 34), dtype=np.uint8)
    q = rng.integers(-128, 128, size=(M, nb, 32)).astype(np.int8)
    if scale_bits is None:
        d = (rng.standard_normal((M, nb)) * 0.02).astype(np.float16)
        d.reshape(-1)[::7] = np.float16(-3.0e-5)     # a negative subnormal scale
        d.reshape(-1)[::11] = np.float16(1024.0)     # a large one
        scale_bits = d.view(np.uint16)
    w[:, :, 0] = scale_bits & 0xFF
    w[:, :, 1] = scale_bits >> 8
    w[:, :, 2:] = q.view(np.uint8)
    return w


def _numpy_reference(w, x):
    """Dequantize with numpy's own float16 / int8 decoding, then np.dot."""
    M, nb, _ = w.shape
    d = np.ascontiguousarray(w[:, :, 0:2]).view(np.float16).reshape(M, nb).astype(np.float64)
    q = np.ascontiguousarray(w[:, :, 2:]).view(np.int8).astype(np.float64)
    dense = (d[:, :, None] * q).reshape(M, nb * 32)
    return dense @ np.asarray(x, dtype=np.float64)


def test_half_decoding_matches_numpy_for_every_pattern():
    bits = np.arange(1 << 16, dtype=np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([q8.half_to_f64(int(b)) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


@pytest.mark.parametrize("M,K", [(1, 32), (7, 64), (33, 2048), (5, 4096)])
def test_gemv_matches_numpy_dequantized_matvec(M, K):
    rng = np.random.default_rng(M * 1000 + K)
    w = _blocks(rng, M, K)
    x = rng.standard_normal(K)
    ref = _numpy_reference(w, x)
    got = q8.gemv(w, x)
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_one_hot_blocks_select_exact_values():
    K = 96
    x = np.arange(1, K + 1, dtype=np.float64) * 0.5
    w = np.zeros((3, K // 32, 34), dtype=np.uint8)
    # row 0: scale 1.0 (0x3C00) in block 1, value +1 at position 5 -> x[37]
    w[0, 1, 0], w[0, 1, 1] = 0x00, 0x3C
    w[0, 1, 2 + 5] = 1
    # row 1: scale -2^-10 (0x9400) in block 2, value -128 at position 31 -> 0.125 * x[95]
    w[1, 2, 0], w[1, 2, 1] = 0x00, 0x94
    w[1, 2, 2 + 31] = np.uint8(256 - 128)
    # row 2: a zero scale with non-zero values contributes nothing
    w[2, 0, 2:] = 77
    y = q8.gemv(w, x)
    assert y[0] == x[37]
    assert y[1] == 0.125 * x[95]
    assert y[2] == 0.0


def test_scale_is_little_endian_and_precedes_the_values():
    K = 32
    w = np.zeros((2, 1, 34), dtype=np.uint8)
    w[:, 0, 2:] = 1                                   # all values +1
    w[0, 0, 0], w[0, 0, 1] = 0x00, 0x3C               # 1.0 little-endian
    w[1, 0, 0], w[1, 0, 1] = 0x3C, 0x00               # the swapped bytes: 0x003C, a subnormal
    x = np.ones(K)
    y = q8.gemv(w, x)
    assert y[0] == 32.0
    assert y[1] == 32.0 * 60 * 2.0 ** -24


def test_two_blocks_with_different_scales():
    K = 64
    w = np.zeros((1, 2, 34), dtype=np.uint8)
    w[0, 0, 0:2] = np.frombuffer(np.float16(0.5).tobytes(), dtype=np.uint8)
    w[0, 1, 0:2] = np.frombuffer(np.float16(-4.0).tobytes(), dtype=np.uint8)
    w[0, :, 2:] = 3
    x = np.ones(K)
    assert q8.gemv(w, x)[0] == 32 * 3 * 0.5 + 32 * 3 * (-4.0)


def test_linear_in_x():
    rng = np.random.default_rng(5)
    w = _blocks(rng, 9, 256)
    x1, x2 = rng.standard_normal(256), rng.standard_normal(256)
    lhs = q8.gemv(w, 2.0 * x1 - 0.5 * x2)
    rhs = 2.0 * q8.gemv(w, x1) - 0.5 * q8.gemv(w, x2)
    assert np.allclose(lhs, rhs, rtol=1e-12, atol=1e-12 * np.abs(rhs).max())


def test_rejects_k_not_multiple_of_32():
    with pytest.raises(ValueError):
        q8.gemv(np.zeros((1, 34 + 16), dtype=np.uint8), np.ones(48))
