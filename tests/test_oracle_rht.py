"""Pins for the oracle's block rotation before MXFP4 quantization (CPU only).

The rotation is y = H_32 D x / sqrt(32) per 32-element block (Sec. 4.3,
App. C.2), evaluated in FP32 by the fast Walsh-Hadamard transform.  Pinned
here against statements that do not reuse the oracle's arithmetic: scipy's
Sylvester Hadamard matrix on inputs where FP32 is exact, the involution
H H = 32 I, a correctly rounded 1/sqrt(32) from decimal arithmetic, the FP32
error bound of a depth-5 summation tree against FP64, and brute-force scale
and nearest-code searches for the quantization that follows.
"""
from decimal import Decimal, getcontext

import numpy as np
import pytest
import scipy.linalg

import oracle
from paper_2606_15682_amd import workloads as wl
from tests import indep

H32 = scipy.linalg.hadamard(32).astype(np.int64)
U = 2.0 ** -24


def _signs_vec(signs):
    return np.array([-1 if (signs >> j) & 1 else 1 for j in range(32)], np.int64)


def test_sylvester_matrix_convention():
    i = np.arange(32)
    pop = np.array([[bin(a & b).count("1") for b in i] for a in i])
    assert np.array_equal(H32, np.where(pop % 2 == 0, 1, -1))


def test_norm_constant_is_correctly_rounded():
    getcontext().prec = 60
    exact = Decimal(1) / Decimal(32).sqrt()
    f = np.float32(float(exact))
    cands = [np.nextafter(f, np.float32(0)), f, np.nextafter(f, np.float32(1))]
    dist = [abs(Decimal(float(c)) - exact) for c in cands]
    best = cands[int(np.argmin(dist))]
    assert np.float32(oracle.rht_norm()) == best
    ulp = Decimal(float(cands[2])) - Decimal(float(cands[1]))
    assert min(dist) < ulp * Decimal("0.45")        # far from a rounding tie


@pytest.mark.parametrize("seed", range(4))
def test_fwht_equals_matrix_product_on_exact_inputs(seed):
    rng = np.random.default_rng(seed)
    v = rng.integers(-2000, 2001, 32)
    got = oracle.fwht32_f32(v.astype(np.float32))
    assert np.array_equal(got.astype(np.int64), H32 @ v)          # |H v| < 2^17: exact in FP32


def test_fwht_is_an_involution_up_to_32():
    rng = np.random.default_rng(9)
    v = rng.integers(-500, 501, 32).astype(np.float32)
    assert np.array_equal(oracle.fwht32_f32(oracle.fwht32_f32(v)), 32 * v)


@pytest.mark.parametrize("signs", [0, 0xFFFFFFFF, 0x1, 0x80000000, 0x9E3779B9])
def test_rotation_signs_and_order_on_exact_inputs(signs):
    rng = np.random.default_rng(signs & 0xFFFF)
    xi = rng.integers(-100, 101, 32)
    xb = indep.to_bf16_bits(xi.astype(np.float64))
    s = H32 @ (_signs_vec(signs) * xi)                             # exact
    want = np.float32(s.astype(np.float32)) * np.float32(oracle.rht_norm())   # one FP32 product
    assert np.array_equal(oracle.rht32(xb, signs), want)


@pytest.mark.parametrize("seed", range(3))
def test_rotation_within_fp32_error_bound(seed):
    x = wl.bf16_bits(wl.random_bf16(64, 32, 70 + seed, 1.0, "student_t")).copy()
    x[:, 3] = indep.to_bf16_bits(indep.bf16_values(x[:, 3]) * 40.0)          # an outlier channel
    signs = 0x5A5AC3C3 ^ seed
    d = _signs_vec(signs).astype(np.float64)
    c = float(np.float32(oracle.rht_norm()))
    for r in range(x.shape[0]):
        xv = indep.bf16_values(x[r])
        exact = (H32.astype(np.float64) @ (d * xv)) / np.sqrt(32.0)
        y = oracle.rht32(x[r], signs).astype(np.float64)
        g5 = 5 * U / (1 - 5 * U)
        bound = c * g5 * np.sum(np.abs(xv)) + 2.01 * U * np.abs(exact) + 1e-300
        assert np.all(np.abs(y - exact) <= bound * 1.0001)


def _brute_quantize(y):
    """Smallest E8M0 scale with max|y| <= 6 s, then nearest-even codes (brute force)."""
    e8 = indep.e8m0_table()
    a = np.max(np.abs(y))
    if a == 0:
        sb = 0
    else:
        ok = [b for b in range(255) if a <= 6.0 * e8[b]]
        sb = min(ok, key=lambda b: e8[b])
    S = e8[sb]
    mag = indep.nearest_code_brute(np.abs(y), S)
    return sb, mag | np.where(np.signbit(y), 8, 0).astype(np.uint8)


@pytest.mark.parametrize("dist", ["normal", "student_t"])
def test_quantize_matches_brute_force_on_the_rotated_values(dist):
    x = wl.bf16_bits(wl.random_bf16(24, 128, 5, 0.3, dist)).copy()
    x[:, 17] = indep.to_bf16_bits(indep.bf16_values(x[:, 17]) * 25.0)
    signs = 0x2545F491
    codes, scales = oracle.quantize_mx_rht(x, signs)
    c = indep.unpack_codes(codes)
    for r in range(x.shape[0]):
        for b in range(x.shape[1] // 32):
            y = oracle.rht32(x[r, 32 * b:32 * (b + 1)], signs).astype(np.float64)
            sb, cc = _brute_quantize(y)
            assert scales[r, b] == sb
            assert np.array_equal(c[r, 32 * b:32 * (b + 1)], cc)


def test_nonfinite_inputs_and_overflow_give_nan_blocks():
    x = np.zeros((4, 64), np.uint16)
    x[0, 5] = 0x7FC0                    # NaN
    x[1, 40] = 0xFF80                   # -Inf
    x[2, 0] = x[2, 1] = 0x7F7F          # 2 * 3.39e38: the first butterfly overflows
    x[3, :] = 0x3F80                    # finite control row
    codes, scales = oracle.quantize_mx_rht(x, 0)
    assert scales[0, 0] == 0xFF and scales[0, 1] != 0xFF
    assert scales[1, 1] == 0xFF and scales[1, 0] != 0xFF
    assert scales[2, 0] == 0xFF
    assert np.all(scales[3] != 0xFF)
    c = indep.unpack_codes(codes)
    assert np.all(c[0, :32] == 0) and np.all(c[1, 32:] == 0) and np.all(c[2, :32] == 0)
    y = oracle.fakequant_mx_rht(x, 0)
    assert np.all(y[0, :32] == 0x7FC0) and np.all(y[2, :32] == 0x7FC0)


@pytest.mark.parametrize("signs", [0, 0xC001D00D])
def test_fakequant_is_the_rounded_dequantized_rotation(signs):
    x = wl.bf16_bits(wl.random_bf16(16, 96, 8, 1.0, "normal")).copy()
    codes, scales = oracle.quantize_mx_rht(x, signs)
    want = indep.to_bf16_bits(indep.dequant_indep(1, codes, scales, 1.0))
    assert np.array_equal(oracle.fakequant_mx_rht(x, signs), want)


def test_constant_block_rotates_to_a_spike():
    # x = v * (column j of H D) makes H D x = 32 v e_j: one nonzero entry per block
    v = 3.0
    signs = 0x0F0F0F0F
    d = _signs_vec(signs)
    for j in (0, 7, 31):
        xv = v * d * H32[:, j]           # D H e_j (D and H symmetric, D^2 = I)
        y = oracle.rht32(indep.to_bf16_bits(xv.astype(np.float64)), signs)
        want = np.zeros(32, np.float32)
        want[j] = np.float32(32 * v) * np.float32(oracle.rht_norm())
        assert np.array_equal(y, want)
