"""Pins for the oracle's format codecs and rounding rules (CPU only).

Each test checks the oracle against a statement that does not reuse its code:
hand-written golden tables, torch's float8/bfloat16 conversions, brute-force
nearest-value and minimal-scale searches, and exact rational arithmetic.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from tests import indep

ALL_BF16 = np.arange(65536, dtype=np.uint32).astype(np.uint16)


def finite_bf16():
    v = indep.bf16_values(ALL_BF16)
    keep = np.isfinite(v)
    return ALL_BF16[keep], v[keep]


# ---------------------------------------------------------------- decoders

def test_e2m1_decode_matches_golden_grid():
    tab = indep.e2m1_table()
    for c in range(16):
        got = oracle.e2m1_value(c)
        assert got == tab[c] and np.signbit(got) == np.signbit(tab[c]), c
    # the magnitudes are exactly the grid {0, .5, 1, 1.5, 2, 3, 4, 6}
    assert sorted(set(abs(tab))) == [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]


def test_e4m3_decode_matches_torch_float8_e4m3fn():
    tab = indep.e4m3_table()
    for b in range(256):
        got = oracle.e4m3_value(b)
        if np.isnan(tab[b]):
            assert np.isnan(got), b
        else:
            assert got == tab[b] and np.signbit(got) == np.signbit(tab[b]), b
    assert oracle.e4m3_value(0x7E) == 448.0
    assert oracle.e4m3_value(0x01) == 2.0 ** -9


def test_e8m0_decode_matches_torch_float8_e8m0fnu():
    tab = indep.e8m0_table()
    for b in range(256):
        got = oracle.e8m0_value(b)
        if np.isnan(tab[b]):
            assert np.isnan(got), b
        else:
            assert got == tab[b], b


def test_bf16_decode_all_patterns():
    v = indep.bf16_values(ALL_BF16)
    for h in range(0, 65536, 7):
        got = oracle.bf16_value(h)
        if np.isnan(v[h]):
            assert np.isnan(got)
        else:
            assert got == v[h]


# ---------------------------------------------------------------- bf16 rounding

def _bf16_inputs():
    rng = np.random.default_rng(1)
    parts = [
        rng.standard_normal(200000) * np.exp2(rng.integers(-140, 130, 200000)),
        # exact ties and near ties around random bf16 values
        (indep.bf16_values(rng.integers(0, 0x7F80, 50000).astype(np.uint16)) *
         (1 + np.ldexp(1.0, -8) * rng.choice([1.0, 1.0 + 2 ** -30, 1.0 - 2 ** -30], 50000))),
        # subnormal range and overflow edge
        np.ldexp(rng.random(50000), -126) * rng.choice([-1, 1], 50000),
        np.array([3.3895313892515355e38, 3.3961775292304093e38, 3.4e38, 1e39, -1e39, 0.0, -0.0,
                  np.ldexp(1.0, -133), np.ldexp(1.0, -134), np.ldexp(1.5, -134), np.ldexp(1.0, -135),
                  np.ldexp(255.0, 120), np.ldexp(511.0, 119)]),
    ]
    return np.concatenate(parts)


def test_bf16_rounding_matches_torch_on_float32_inputs():
    """torch rounds float32 -> bfloat16 in one step (nearest, ties to even)."""
    with np.errstate(over="ignore"):
        v = np.float64(np.float32(_bf16_inputs()))  # exactly representable in float32
    v = v[np.isfinite(v)]
    got = oracle.bf16_from_double_array(v)
    want = torch.from_numpy(v.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    bad = np.nonzero(got != want)[0]
    assert v.size > 50000
    assert bad.size == 0, [(v[i], hex(got[i]), hex(want[i])) for i in bad[:5]]


def test_bf16_rounding_is_nearest_even_exact_rationals():
    """For inputs that are not float32-exact (where torch's float64 path
    rounds twice), check the defining property with exact rationals: no other
    bfloat16 value is nearer, and on a tie the chosen one has an even
    significand.  Neighbours are the adjacent bit patterns."""
    v = _bf16_inputs()
    with np.errstate(over="ignore"):
        inexact = np.float64(np.float32(v)) != v
    v = np.concatenate([v[inexact][::20], v[-13:]])
    got = oracle.bf16_from_double_array(v)
    maxf = Fraction(2) ** 128   # the value "one past" the largest finite bfloat16
    for x, h in zip(v, got):
        X = Fraction(float(x))
        mag = int(h) & 0x7FFF
        sgn = -1 if (int(h) & 0x8000) else 1
        if mag == 0x7F80:                            # overflow: |x| >= midpoint(max, 2^128)
            top = Fraction(oracle.bf16_value(0x7F7F))
            assert abs(X) >= (top + maxf) / 2, x
            continue
        chosen = Fraction(oracle.bf16_value(int(h)))
        d = abs(X - chosen)
        for nb in (mag - 1, mag + 1):
            if nb < 0 or nb >= 0x7F80:
                continue
            other = sgn * Fraction(oracle.bf16_value(nb))
            do = abs(X - other)
            assert d < do or (d == do and mag % 2 == 0), (x, hex(h))
        if mag == 0x7F7F:
            assert abs(X) < (Fraction(oracle.bf16_value(0x7F7F)) + maxf) / 2
    assert oracle.bf16_from_double(float("nan")) == 0x7FC0
    # hand-checked cases: exact midpoint below 2^128 overflows; just below it does not
    assert oracle.bf16_from_double(float(np.ldexp(511.0, 119))) == 0x7F80
    assert oracle.bf16_from_double(float(np.ldexp(511.0, 119) * (1 - 2 ** -40))) == 0x7F7F
    assert oracle.bf16_from_double(float(np.ldexp(1.0, -134))) == 0x0000   # tie -> even (zero)
    assert oracle.bf16_from_double(float(np.ldexp(3.0, -134))) == 0x0002   # tie -> even


# ---------------------------------------------------------------- E2M1 encode

def test_e2m1_tie_cases_golden():
    rows = []
    with open(indep.os.path.join(indep.GOLDEN, "e2m1_ties.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            r, c, v = line.split()
            rows.append((float(r), int(c), float(v)))
    assert len(rows) == 7
    for S in [1.0, 2.0 ** -20, 2.0 ** 30, 0.375, 448.0 * 2.0 ** -7, 1.125 * 3.0]:
        for r, c, v in rows:
            x = r * S
            assert oracle.e2m1_encode(x, S) == c, (r, S)
            assert oracle.e2m1_encode(-x, S) == 8 | c, (r, S)
            assert oracle.e2m1_value(c) == v


def _sweep(S):
    bits, v = finite_bf16()
    ax = np.abs(v)
    got = oracle.e2m1_encode_array(v, S)
    sign = np.signbit(v).astype(np.uint8) << 3
    # brute force where FP64 distances are exact; above that, everything saturates
    near = ax < S * 2.0 ** 40
    want = np.full(v.shape, 7, np.uint8)
    want[near] = indep.nearest_code_brute(ax[near], S)
    want |= sign
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(v[i], S, got[i], want[i]) for i in bad[:5]]


@pytest.mark.parametrize("e", [-127, -126, -120, -60, -9, -3, -1, 0, 1, 2, 7, 30, 100, 126, 127])
def test_e2m1_encode_exhaustive_bf16_mx_scales(e):
    """All 65,536 bf16 patterns against power-of-two (E8M0) scales."""
    _sweep(2.0 ** e)


@pytest.mark.parametrize("sbyte,g", [(0x01, 1.0), (0x07, 2.0 ** -3), (0x33, 1.0), (0x3B, 2.0 ** -20),
                                     (0x45, 2.0 ** 4), (0x7E, 1.0), (0x5D, 2.0 ** -126),
                                     (0x2A, 0.0123456789), (0x66, 3.14159)])
def test_e2m1_encode_exhaustive_bf16_nv_scales(sbyte, g):
    """All bf16 patterns against E4M3 x global scales (pow2 and arbitrary g)."""
    g = float(np.float32(g))
    S = indep.e4m3_table()[sbyte] * g
    _sweep(S)


def test_e2m1_encode_rational_sample():
    """Exact rational brute force on a random sample including near-ties."""
    rng = np.random.default_rng(7)
    e4 = indep.e4m3_table()
    for _ in range(3000):
        sb = int(rng.integers(1, 0x7F))
        g = float(np.float32(rng.choice([1.0, 2.0 ** int(rng.integers(-30, 30)), rng.random() * 3])))
        S = e4[sb] * g
        mid = rng.choice([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, rng.random() * 7])
        x = float(np.float64(np.float32(mid * S)))  # near (sometimes exactly at) a midpoint
        xb = indep.to_bf16_bits(np.array([x]))
        x = float(indep.bf16_values(xb)[0])
        want = indep.nearest_code_fraction(Fraction(x), Fraction(e4[sb]) * Fraction(g))
        assert oracle.e2m1_encode(x, S) & 7 == want, (x, S)


def test_e2m1_signed_zero_and_zero_scale():
    assert oracle.e2m1_encode(-0.0, 1.0) == 8
    assert oracle.e2m1_encode(-1e-30, 1.0) == 8
    assert oracle.e2m1_encode(0.0, 1.0) == 0
    assert oracle.e2m1_encode(-0.0, 0.0) == 8
    assert oracle.e2m1_encode(0.0, 0.0) == 0


# ---------------------------------------------------------------- scale rules

def test_mx_scale_is_minimal_power_of_two_all_bf16():
    """Brute force over all 255 E8M0 values for every positive finite bf16 amax."""
    bits, v = finite_bf16()
    amaxes = np.unique(np.abs(v))
    exps = np.arange(-127, 128)
    lim = 6.0 * np.exp2(exps.astype(np.float64))
    for a in amaxes:
        got = oracle.mx_scale_byte(float(a))
        ok = np.nonzero(a <= lim)[0]
        want = int(exps[ok[0]]) + 127
        assert got == want, (a, got, want)
        if a > 0:
            # the invariant amax/scale <= 6, and the next smaller scale breaks it
            s = indep.e8m0_table()[got]
            assert a <= 6 * s
            if got > 0:
                assert a > 6 * indep.e8m0_table()[got - 1]
    assert oracle.mx_scale_byte(float("nan")) == 0xFF
    assert oracle.mx_scale_byte(float("inf")) == 0xFF


@pytest.mark.parametrize("g", [1.0, 2.0 ** -12, 2.0 ** 9, 2.0 ** -126, 0.0123456789, 7.77e-5, 1234.5])
def test_nv_scale_is_minimal_e4m3_all_bf16(g):
    """Brute force over the 126 positive finite E4M3 values (torch's table)."""
    g = float(np.float32(g))
    tab = indep.e4m3_table()
    pos = [(tab[b], b) for b in range(1, 0x7F)]
    vals = np.array([p[0] for p in pos])
    bytes_ = np.array([p[1] for p in pos])
    assert np.all(np.diff(vals) > 0)
    bits, v = finite_bf16()
    amaxes = np.unique(np.abs(v))
    for a in amaxes:
        got = oracle.nv_scale_byte(float(a), g)
        if a == 0:
            assert got == 0
            continue
        ok = np.nonzero(a <= 6.0 * vals * g)[0]
        want = int(bytes_[ok[0]]) if ok.size else 0x7E
        assert got == want, (a, g, hex(got), hex(want))


def test_nv_global_scale_brute_force():
    bits, v = finite_bf16()
    amaxes = np.unique(np.abs(v))
    ks = np.arange(-126, 128)
    lim = 2688.0 * np.exp2(ks.astype(np.float64))
    for a in amaxes[::3]:
        got = oracle.nv_global_scale(float(a))
        if a == 0:
            assert got == 1.0
            continue
        want = 2.0 ** int(ks[np.nonzero(a <= lim)[0][0]])
        assert got == want, (a, got, want)
    # 2688 = 6 * 448 exactly on a power-of-two boundary: A = 2688 -> g = 1
    assert oracle.nv_global_scale(2688.0) == 1.0
    assert oracle.nv_global_scale(2688.0 * (1 + 2 ** -7)) == 2.0
    assert oracle.nv_global_scale(0.0) == 1.0
