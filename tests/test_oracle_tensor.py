"""Pins for the oracle's tensor operations: quantize (scales, codes, packing),
fake-quant and the FP64 block-scaled product (CPU only)."""
import numpy as np
import pytest

import oracle
from oracle import FMT_MXFP4, FMT_NVFP4
from paper_2606_15682_amd import workloads as wl
from tests import indep

FMTS = [FMT_NVFP4, FMT_MXFP4]


def _x(rows, cols, seed, std=1.0, dist="normal"):
    return wl.bf16_bits(wl.random_bf16(rows, cols, seed, std, dist))


def _check_quantize_props(fmt, x, codes, scales, g):
    """Scale minimality + invariant, and codes = brute-force nearest, per block."""
    B = oracle.BLOCK[fmt]
    v = indep.bf16_values(x)
    R, C = v.shape
    stab = indep.e8m0_table() if fmt == FMT_MXFP4 else indep.e4m3_table()
    c = indep.unpack_codes(codes)
    for r in range(R):
        for b in range(C // B):
            blk = v[r, b * B:(b + 1) * B]
            sb = scales[r, b]
            if not np.all(np.isfinite(blk)):
                assert sb == (0xFF if fmt == FMT_MXFP4 else 0x7F)
                assert np.all(c[r, b * B:(b + 1) * B] == 0)
                continue
            a = np.max(np.abs(blk))
            gg = g if fmt == FMT_NVFP4 else 1.0
            s = stab[sb]
            if a == 0:
                assert sb == 0
            elif fmt == FMT_NVFP4 and a > 6.0 * 448.0 * gg:
                assert sb == 0x7E                               # caller's g too small: saturate
            else:
                assert a <= 6.0 * s * gg                        # invariant: amax/scale <= 6
                if fmt == FMT_MXFP4:
                    assert sb == 0 or a > 6.0 * stab[sb - 1]     # minimal
                else:
                    assert sb == 1 or a > 6.0 * stab[sb - 1] * gg
            S = s * gg
            want = indep.nearest_code_brute(np.abs(blk), S) | (np.signbit(blk).astype(np.uint8) << 3)
            assert np.array_equal(c[r, b * B:(b + 1) * B], want), (r, b)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("dist", ["normal", "student_t"])
def test_quantize_random_matches_brute_force(fmt, dist):
    x = _x(7, 256, 11 + fmt, dist=dist)
    codes, scales, g = oracle.quantize(fmt, x)
    _check_quantize_props(fmt, x, codes, scales, g)


def test_quantize_with_outliers_and_given_scale():
    x = _x(5, 512, 12, std=0.02)
    x[:, [3, 100]] = indep.to_bf16_bits(indep.bf16_values(x[:, [3, 100]]) * 400.0)
    for g in [None, 1.0 / 3.0, 2.0 ** -9, 1e-3]:
        codes, scales, gg = oracle.quantize(FMT_NVFP4, x, g)
        _check_quantize_props(FMT_NVFP4, x, codes, scales, gg)


def test_packing_order_hand_worked():
    """One MXFP4 block worked by hand: amax 6 -> scale 2^0 (byte 127);
    elements 6, 1, -0.5, 0.25(tie->0), 0.75(tie->1.0), -3, 5(tie->4), 1.75(tie->2),
    then zeros.  Codes 7,2,9,0,2,13,6,4 pack low nibble first."""
    vals = np.zeros((1, 32))
    vals[0, :8] = [6, 1, -0.5, 0.25, 0.75, -3, 5, 1.75]
    x = indep.to_bf16_bits(vals)
    codes, scales, _ = oracle.quantize(FMT_MXFP4, x)
    assert scales.tolist() == [[127]]
    assert codes[0, :4].tolist() == [0x27, 0x09, 0xD2, 0x46]
    assert np.all(codes[0, 4:] == 0)
    # NVFP4 with g = 1: same block in two halves; first half amax 6 -> s = 1.0 (0x38)
    codes, scales, g = oracle.quantize(FMT_NVFP4, x, 1.0)
    assert scales.tolist() == [[0x38, 0x00]]
    assert codes[0, :4].tolist() == [0x27, 0x09, 0xD2, 0x46]


def test_grid_aligned_inputs_round_trip():
    """x = V[c] * S with an element at 6 per block quantizes back to (c, S)."""
    rng = np.random.default_rng(5)
    for fmt in FMTS:
        B = oracle.BLOCK[fmt]
        R, C = 6, 4 * B
        c = rng.integers(0, 16, (R, C)).astype(np.uint8)
        c[:, ::B] = 7                                  # one 6.0 per block
        if fmt == FMT_MXFP4:
            sb = rng.integers(100, 150, (R, C // B)).astype(np.uint8)
            S = indep.e8m0_table()[sb]
            g = 1.0
        else:
            sb = rng.integers(0x08, 0x70, (R, C // B)).astype(np.uint8)
            g = 2.0 ** -5
            S = indep.e4m3_table()[sb] * g
        vals = indep.e2m1_table()[c] * np.repeat(S, B, axis=1)
        x = indep.to_bf16_bits(vals)
        assert np.array_equal(indep.bf16_values(x), vals)   # exactly representable
        codes, scales, _ = oracle.quantize(fmt, x, g if fmt == FMT_NVFP4 else None)
        assert np.array_equal(scales, sb)
        # -0 codes stay -0 (sign copied)
        assert np.array_equal(indep.unpack_codes(codes), c)


@pytest.mark.parametrize("fmt", FMTS)
def test_error_bound_half_spacing(fmt):
    """|x - x^| <= half the local grid spacing times the block scale."""
    x = _x(9, 320 if fmt == FMT_NVFP4 else 320, 21 + fmt, dist="student_t")
    codes, scales, g = oracle.quantize(fmt, x)
    xh = oracle.dequantize(fmt, codes, scales, g)
    v = indep.bf16_values(x)
    B = oracle.BLOCK[fmt]
    st = (indep.e8m0_table() if fmt == FMT_MXFP4 else indep.e4m3_table() * g)[scales]
    S = np.repeat(st, B, axis=1)
    r = np.abs(xh) / S
    # a value that rounds to grid point r lies within half the wider of the two
    # spacings around r: 0.25 below 2; 0.5 at 2 and 3; 1 at 4 and 6
    half = np.where(r < 2.0, 0.25, np.where(r < 4.0, 0.5, 1.0))
    assert np.all(np.abs(v - xh) <= half * S)
    # and the bound is attained somewhere only at ties, never exceeded


def test_special_blocks():
    """Zero block, negative zeros, NaN/Inf blocks, bf16 subnormals, bf16 max."""
    for fmt in FMTS:
        B = oracle.BLOCK[fmt]
        x = np.zeros((4, 2 * B), np.uint16)
        x[0, :] = 0x8000                      # all -0
        x[1, 0] = 0x7FC0                      # NaN in block 0
        x[1, B] = 0x3F80                      # 1.0 in block 1
        x[2, 3] = 0xFF80                      # -inf
        x[2, B:] = np.arange(1, B + 1)        # bf16 subnormals
        x[3, :B] = 0x7F7F                     # bf16 max
        x[3, B] = 0x0001                      # min subnormal
        codes, scales, g = oracle.quantize(fmt, x)
        c = indep.unpack_codes(codes)
        nan_s = 0xFF if fmt == FMT_MXFP4 else 0x7F
        assert np.all(c[0] == 8) and np.all(scales[0] == 0)
        assert scales[1, 0] == nan_s and np.all(c[1, :B] == 0)
        assert scales[2, 0] == nan_s
        # the tensor amax ignores non-finite values
        assert oracle.tensor_amax(x) == indep.bf16_values(np.array([0x7F7F], np.uint16))[0]
        _check_quantize_props(fmt, x, codes, scales, g)


@pytest.mark.parametrize("fmt", FMTS)
def test_fakequant_is_bf16_rounding_of_dequantized(fmt):
    x = _x(6, 256, 31 + fmt, dist="student_t")
    for g in ([None] if fmt == FMT_MXFP4 else [None, 0.7, 2.0 ** -130 / 3]):
        y, gg = oracle.fakequant(fmt, x, g)
        codes, scales, _ = oracle.quantize(fmt, x, g)
        deq = indep.dequant_indep(fmt, codes, scales, gg)
        with np.errstate(over="ignore"):
            f32 = np.float32(deq)
        exact32 = np.float64(f32) == deq
        want = indep.to_bf16_bits(deq)
        # values that are float32-exact are rounded once by torch; compare all of them
        assert np.array_equal(y[exact32], want[exact32])
        # every output is the bf16 value nearest the dequantized value
        yv = indep.bf16_values(y)
        assert np.all(np.abs(yv - deq) <= np.abs(deq) * 2.0 ** -8 + 2.0 ** -134)


def test_fakequant_nan_block():
    x = np.zeros((1, 32), np.uint16)
    x[0, 5] = 0x7FC0
    x[0, 20] = 0x3F80
    y, _ = oracle.fakequant(FMT_NVFP4, x)
    assert np.all(y[0, :16] == 0x7FC0)
    # the other block is ordinary: amax 1 -> g = 2^-11, s = 352 (smallest E4M3
    # >= 2^11/6), so 1.0 / (352 * 2^-11) = 5.82 rounds to 6 and comes back as 1.03125
    assert indep.bf16_values(y[0, 20:21])[0] == 1.03125
    assert np.all(y[0, 16:20] == 0) and np.all(y[0, 21:] == 0)


# ---------------------------------------------------------------- GEMM

@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("M,N,K", [(1, 1, 32), (3, 4, 64), (4, 3, 128), (5, 7, 96)])
def test_gemm_tiny_matches_numpy_of_independent_dequant(fmt, M, N, K):
    B = oracle.BLOCK[fmt]
    if K % B:
        pytest.skip("K must be a multiple of the block")
    xa = _x(M, K, 41 + M, dist="student_t")
    xb = _x(N, K, 51 + N, std=0.5)
    ac, as_, ga = oracle.quantize(fmt, xa)
    bc, bs, gb = oracle.quantize(fmt, xb)
    y = oracle.gemm(fmt, ac, as_, ga, bc, bs, gb)
    A = indep.dequant_indep(fmt, ac, as_, ga)
    Bm = indep.dequant_indep(fmt, bc, bs, gb)
    ref = A @ Bm.T
    assert y.shape == (M, N)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-300)
    # the transposed product is a different matrix unless symmetric by chance
    if M == N and M > 1:
        assert not np.allclose(y, (Bm @ A.T))
    yp, ayp = oracle.gemm_points(fmt, ac, as_, ga, bc, bs, gb,
                                 np.arange(M).repeat(N), np.tile(np.arange(N), M))
    np.testing.assert_allclose(yp.reshape(M, N), ref, rtol=1e-12, atol=1e-300)
    np.testing.assert_allclose(ayp.reshape(M, N), np.abs(A) @ np.abs(Bm).T, rtol=1e-12)


def test_gemm_closed_forms():
    K = 128
    for fmt in FMTS:
        B = oracle.BLOCK[fmt]
        one = 0x22                                          # two codes of 1.0
        unit = 127 if fmt == FMT_MXFP4 else 0x38            # scale 1.0
        ac = np.full((3, K // 2), one, np.uint8)
        as_ = np.full((3, K // B), unit, np.uint8)
        y = oracle.gemm(fmt, ac, as_, 1.0, ac, as_, 1.0)
        assert np.all(y == K)                               # sum of K ones
        # global scales multiply (NVFP4); MXFP4 has none
        if fmt == FMT_NVFP4:
            y = oracle.gemm(fmt, ac, as_, 0.5, ac, as_, 0.25)
            assert np.all(y == K * 0.125)
        # one-hot rows of A select the matching column of B
        bc = np.zeros((2, K // 2), np.uint8)
        bc[0, 5] = 0x70                                     # element 11 = 6.0
        bc[1, 5] = 0x0D                                     # element 10 = -3.0
        bs = np.full((2, K // B), unit, np.uint8)
        oh = np.zeros((2, K // 2), np.uint8)
        oh[0, 5] = 0x20                                     # element 11 = 1.0
        oh[1, 5] = 0x02                                     # element 10 = 1.0
        y = oracle.gemm(fmt, oh, as_[:2], 1.0, bc, bs, 1.0)
        assert y.tolist() == [[6.0, 0.0], [0.0, -3.0]]


def test_gemm_nan_scale_propagates():
    K = 64
    ac = np.full((2, K // 2), 0x22, np.uint8)
    as_ = np.full((2, K // 32), 127, np.uint8)
    as_[1, 1] = 0xFF
    y = oracle.gemm(FMT_MXFP4, ac, as_, 1.0, ac, as_[:1], 1.0)
    assert y[0, 0] == K and np.isnan(y[1, 0])
