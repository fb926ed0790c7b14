"""Pins for the oracle's W4A16 product (MXFP4 weights dequantized to bfloat16,
bfloat16 activations; CPU only), against numpy's matmul of independently
decoded operands (golden E2M1 table, torch's E8M0 and bfloat16 conversions)."""
import numpy as np
import pytest

import oracle
from paper_2606_15682_amd import workloads as wl
from tests import indep


def _weights(N, K, seed, lo=110, hi=140):
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, 256, (N, K // 2), dtype=np.uint8)
    scales = rng.integers(lo, hi, (N, K // 32), dtype=np.uint8)
    return codes, scales


def _w_bf16_indep(codes, scales):
    """RN_bf16 of the exact dequantized weights, via torch's float64 -> bfloat16."""
    return indep.bf16_values(indep.to_bf16_bits(indep.dequant_indep(1, codes, scales, 1.0)))


@pytest.mark.parametrize("M,N,K", [(4, 8, 64), (16, 40, 256), (3, 17, 1024)])
def test_matches_numpy_matmul(M, N, K):
    x = wl.bf16_bits(wl.random_bf16(M, K, 3 + M, 1.0, "student_t")).copy()
    codes, scales = _weights(N, K, N)
    ms, ns = np.arange(M).repeat(N), np.tile(np.arange(N), M)
    y, ay = oracle.gemm_w4a16_points(x, codes, scales, ms, ns)
    xv, wv = indep.bf16_values(x), _w_bf16_indep(codes, scales)
    ref = (xv @ wv.T).reshape(-1)
    aref = (np.abs(xv) @ np.abs(wv).T).reshape(-1)
    assert np.all(np.abs(y - ref) <= 1e-12 * aref + 1e-300)
    assert np.allclose(ay, aref, rtol=1e-12, atol=0)


def test_extreme_scale_bytes_follow_bfloat16_rounding():
    K = 64
    x = np.full((1, K), 0x3F80, np.uint16)                       # ones
    codes = np.full((4, K // 2), 0x11, np.uint8)                 # every element code 1 (0.5)
    scales = np.array([[0, 0], [1, 1], [253, 253], [0xFF, 127]], np.uint8)
    y, _ = oracle.gemm_w4a16_points(x, codes, scales, np.zeros(4, np.int64), np.arange(4))
    assert y[0] == 64 * 2.0 ** -128                               # 0.5 * 2^-127, a bfloat16 subnormal
    assert y[1] == 64 * 2.0 ** -127
    assert y[2] == 64 * 2.0 ** 125
    assert np.isnan(y[3])                                         # NaN scale poisons the row
    codes[2] = 0x77                                               # code 7 = 6: 6 * 2^126 overflows bfloat16
    y, _ = oracle.gemm_w4a16_points(x, codes, scales, np.array([0]), np.array([2]))
    assert np.isinf(y[0])


def test_zero_activation_row_gives_zero():
    K = 128
    x = np.zeros((2, K), np.uint16)
    codes, scales = _weights(3, K, 5)
    y, ay = oracle.gemm_w4a16_points(x, codes, scales, np.array([0, 1, 1]), np.array([0, 1, 2]))
    assert np.all(y == 0) and np.all(ay == 0)
