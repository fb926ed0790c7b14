"""Pins for the oracle's block rotation before MXFP4 quantization (CPU only).

The rotation is y = H_32 D x / sqrt(32) per 32-element block (Sec. 4.3,
App. C.2), taken as the exact real value and quantized as an MXFP4 block.
Pinned here against statements that share none of the oracle's arithmetic:
an exact reference in Python integers and fractions built on scipy's
Hadamard matrix and the golden E2M1 table, closed forms (a block that
rotates to a single spike, a constant block), blocks whose decisions hinge
on bits far below FP64 precision, the clamp of the scale at 2^127, and the
half-spacing error bound evaluated in 120-digit decimal arithmetic.
"""
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np
import pytest
import scipy.linalg

import oracle
from paper_2606_15682_amd import workloads as wl
from tests import indep

H32 = scipy.linalg.hadamard(32).astype(np.int64)


def _signs_vec(signs):
    return np.array([-1 if (signs >> j) & 1 else 1 for j in range(32)], np.int64)


def _check_against_reference(x, signs):
    codes, scales = oracle.quantize_mx_rht(x, signs)
    c = indep.unpack_codes(codes)
    for r in range(x.shape[0]):
        for b in range(x.shape[1] // 32):
            sb, cc = indep.rht_block_reference(x[r, 32 * b:32 * (b + 1)], signs)
            assert scales[r, b] == sb, (r, b)
            assert np.array_equal(c[r, 32 * b:32 * (b + 1)], cc), (r, b)


def test_sylvester_matrix_convention():
    i = np.arange(32)
    pop = np.array([[bin(a & b).count("1") for b in i] for a in i])
    assert np.array_equal(H32, np.where(pop % 2 == 0, 1, -1))
    assert np.array_equal(H32 @ H32, 32 * np.eye(32, dtype=np.int64))      # orthogonal up to 32


@pytest.mark.parametrize("dist,signs", [("normal", 0), ("normal", 0x9E3779B9), ("student_t", 0x2545F491),
                                        ("student_t", 0xFFFFFFFF)])
def test_exact_rotation_matches_integer_reference(dist, signs):
    x = wl.bf16_bits(wl.random_bf16(12, 128, 5 + signs % 7, 0.3, dist)).copy()
    x[:, 17] = indep.to_bf16_bits(indep.bf16_values(x[:, 17]) * 25.0)     # an outlier channel
    x[3, 40:50] = 0                                                       # zeros inside a block
    _check_against_reference(x, signs)


def test_special_blocks():
    x = np.zeros((8, 64), np.uint16)
    x[0, :] = 0x8000                               # all -0: y == 0, scale byte 0, codes +0
    x[1, 0] = 0x0001                               # the smallest subnormal alone
    x[1, 32:] = 0x8001                             # subnormals of one sign
    x[2, 0] = x[2, 1] = 0x7F7F                     # two bfloat16 maxima (their FP32 sum overflows)
    x[3, :] = 0x7F7F                               # max|y| = sqrt(32) * 3.39e38 > 6 * 2^127: clamped, saturates
    x[4, 5] = 0x7FC0                               # NaN
    x[4, 40] = 0xFF80                              # -Inf in the second block
    x[5, :] = 0x3F80                               # constant 1.0
    x[6, ::2] = 0x0080                             # smallest normals
    x[6, 1::2] = 0x7F00                            # with 2^127: an exponent spread of 253 bits
    x[7, :] = indep.to_bf16_bits(np.linspace(-3, 3, 64))
    _check_against_reference(x, 0)
    _check_against_reference(x, 0x5A5AC3C3)
    codes, scales = oracle.quantize_mx_rht(x, 0)
    c = indep.unpack_codes(codes)
    assert scales[0, 0] == 0 and np.all(c[0] == 0)
    assert scales[4, 0] == 0xFF and scales[4, 1] == 0xFF and np.all(c[4] == 0)
    assert scales[3, 0] == 254 and (c[3, 0] & 7) == 7
    assert scales[2, 0] != 0xFF
    y = oracle.fakequant_mx_rht(x, 0)
    assert np.all(y[4] == 0x7FC0) and np.all(y[0] == 0)


def test_constant_block_and_spike_closed_forms():
    # x = v * (column j of H D) makes H D x = 32 v e_j: y_j = sqrt(32) v, every other y_i = 0
    for signs, v, j in ((0x0F0F0F0F, 3.0, 0), (0x0F0F0F0F, 3.0, 7), (0x80000001, -0.375, 31),
                        (0, 2.0 ** -100, 9)):
        xv = v * _signs_vec(signs) * H32[:, j]
        codes, scales = oracle.quantize_mx_rht(indep.to_bf16_bits(xv.astype(np.float64)).reshape(1, 32), signs)
        y = np.sqrt(32.0) * abs(v)                  # |y_j|, irrational in units of 2^e
        e = int(np.ceil(np.log2(y / 6.0)))         # smallest e with y <= 6 * 2^e (never equal)
        q = y / 2.0 ** e
        mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
        m3 = int(np.sum(q > mids))                  # q is never a midpoint
        want = np.zeros(32, np.uint8)
        want[j] = m3 | (8 if v < 0 else 0)
        assert scales[0, 0] == e + 127
        assert np.array_equal(indep.unpack_codes(codes)[0], want)
    # the constant block 1.0: y_0 = sqrt(32) = 5.657, scale 2^0, code 6 (|y| between 5 and 6)
    codes, scales = oracle.quantize_mx_rht(np.full((1, 32), 0x3F80, np.uint16), 0)
    assert scales[0, 0] == 127 and indep.unpack_codes(codes)[0, 0] == 7
    assert np.all(indep.unpack_codes(codes)[0, 1:] == 0)


# (t, e, big): y_0 near t * 2^e.  Without `big` y_0 is the block maximum, so t is the
# scale bound 6 or one of the midpoints 3.5 and 5 its ratio to 2^e can reach; with
# big = 9 * 2^e the odd outputs (about 18 * 2^e / sqrt(32)) set the scale 2^e and y_0
# probes the lower midpoints.
NEAR = [(Fraction(6), 0, None), (Fraction(6), -40, None), (Fraction(6), 100, None),
        (Fraction(5), -3, None), (Fraction(7, 2), 10, None), (Fraction(7, 2), -120, None),
        (Fraction(1, 4), 2, 9), (Fraction(3, 4), -20, 9), (Fraction(5, 4), 0, 9),
        (Fraction(7, 4), 5, 9), (Fraction(5, 2), -7, 9)]


@pytest.mark.parametrize("t,e,big", NEAR)
@pytest.mark.parametrize("chunks", [6, 12, 16])
def test_decisions_far_below_fp64_precision(t, e, big, chunks):
    """y_0 within about 2^(-8 chunks) (relative) of a threshold, on either side: each side
    is decided as the integer reference decides it, and the two sides differ."""
    for signs in (0, 0x13579BDF):
        got = []
        for above in (False, True):
            bigv = None if big is None else Fraction(big) * Fraction(2) ** e
            x = indep.rht_near_threshold_block(t, e, above, chunks, signs, bigv).reshape(1, 32)
            _check_against_reference(x, signs)
            codes, scales = oracle.quantize_mx_rht(x, signs)
            got.append((int(scales[0, 0]), int(indep.unpack_codes(codes)[0, 0])))
        assert got[0] != got[1], got
        if big is not None:
            assert got[0][0] == got[1][0] == e + 127          # the odd outputs set the scale


def test_quantization_error_within_half_spacing():
    """|y - y^| <= half the local grid spacing times 2^e (nothing clips under the ceil scale),
    with y in 120-digit decimal arithmetic."""
    getcontext().prec = 120
    x = wl.bf16_bits(wl.random_bf16(4, 256, 17, 1.0, "student_t"))
    signs = 0xC001D00D
    codes, scales = oracle.quantize_mx_rht(x, signs)
    deq = indep.dequant_indep(1, codes, scales, 1.0)
    r32 = Decimal(32).sqrt()
    d = _signs_vec(signs)
    for r in range(x.shape[0]):
        xv = [Decimal(float(v)) for v in indep.bf16_values(x[r])]
        for b in range(x.shape[1] // 32):
            S = 2.0 ** (int(scales[r, b]) - 127)
            for i in range(32):
                y = sum(int(H32[i, j]) * int(d[j]) * xv[32 * b + j] for j in range(32)) / r32
                q = abs(y) / Decimal(S)
                assert q <= 6
                half = Decimal("0.25") if q < 2 else Decimal("0.5") if q < 4 else Decimal(1)
                assert abs(y - Decimal(float(deq[r, 32 * b + i]))) <= half * Decimal(S)


@pytest.mark.parametrize("signs", [0, 0xC001D00D])
def test_fakequant_is_the_dequantized_rotation(signs):
    x = wl.bf16_bits(wl.random_bf16(16, 96, 8, 1.0, "normal")).copy()
    x[2, :32] = 0x7F7F
    codes, scales = oracle.quantize_mx_rht(x, signs)
    want = indep.to_bf16_bits(indep.dequant_indep(1, codes, scales, 1.0))
    assert np.array_equal(oracle.fakequant_mx_rht(x, signs), want)
