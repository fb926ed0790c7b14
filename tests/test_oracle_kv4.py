"""Pins for the oracle's KV4 quantizer (E1M2 elements, NVFP4-style E4M3 block
and FP32 global scales, FP32 post-RoPE shift; CPU only)."""
import os

import numpy as np
import pytest

import oracle
from paper_2606_15682_amd import workloads as wl
from tests import indep

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def e1m2_golden():
    vals = np.zeros(16)
    for line in open(os.path.join(GOLDEN, "e1m2_grid.txt")):
        if line.startswith("#") or not line.strip():
            continue
        c, v = line.split()
        vals[int(c)] = float(v)
    return vals


def test_e1m2_decode_matches_golden_and_minifloat_formula():
    g = e1m2_golden()
    for c in range(16):
        s, e, m = c >> 3, (c >> 2) & 1, c & 3
        formula = (-1.0) ** s * ((m / 4.0) * 2.0 if e == 0 else (1 + m / 4.0) * 2.0)   # bias 0
        assert oracle.e1m2_value(c) == g[c] == formula or (g[c] == 0 and formula == 0)
        assert np.signbit(oracle.e1m2_value(c)) == bool(s)


def _nearest_even(a, S):
    grid = np.arange(8) * 0.5 * S
    d = np.abs(a - grid)
    best = d.min()
    hits = [i for i in range(8) if d[i] == best]
    ev = [i for i in hits if i % 2 == 0]
    return ev[0] if ev else hits[0]


def test_e1m2_encode_brute_force_including_ties():
    rng = np.random.default_rng(1)
    for S in (1.0, 0.375, 2.0 ** -20, 448.0 * 2.0 ** 7):
        vals = list(rng.uniform(0, 4.2, 400) * S) + [(0.25 + 0.5 * i) * S for i in range(7)]
        for v in vals:
            for sign in (1.0, -1.0):
                c = oracle.e1m2_encode(sign * v, S)
                assert (c & 7) == _nearest_even(v, S)
                assert (c >> 3) == (1 if sign < 0 else 0)


def test_global_scale_is_minimal_power_of_two():
    for a in (1e-30, 0.001, 1.0, 1568.0, 1568.0000001, 3.3e38, 5.0e-44):
        g = oracle.kv4_global_scale(a)
        k = int(np.round(np.log2(g)))
        assert a <= 1568.0 * g
        if k > -126:
            assert not (a <= 1568.0 * 2.0 ** (k - 1))
    assert oracle.kv4_global_scale(0.0) == 1.0


def test_block_scale_is_minimal_e4m3():
    tab = indep.e4m3_table()
    pos = sorted((tab[b], b) for b in range(1, 0x7F))
    rng = np.random.default_rng(2)
    for g in (1.0, 2.0 ** -9, 0.0123):
        for a in rng.uniform(0, 3.5 * 448 * g, 300):
            b = oracle.kv4_scale_byte(a, g)
            ok = [bb for v, bb in pos if a <= 3.5 * v * g]
            assert b == ok[0]


def _check_blocks(x, shift, g, codes, scales):
    d = indep.bf16_values(x).astype(np.float32)
    if shift is not None:
        d = (d - np.asarray(shift, np.float32)[None, :]).astype(np.float32)   # numpy FP32 subtraction
    d = d.astype(np.float64)
    c = indep.unpack_codes(codes)
    tab = indep.e4m3_table()
    for r in range(d.shape[0]):
        for b in range(d.shape[1] // 16):
            blk = d[r, 16 * b:16 * b + 16]
            sb = scales[r, b]
            if not np.all(np.isfinite(blk)):
                assert sb == 0x7F and np.all(c[r, 16 * b:16 * b + 16] == 0)
                continue
            a = np.max(np.abs(blk))
            if a == 0:
                assert sb == 0
                continue
            s = tab[sb]
            if a > 3.5 * 448.0 * g:
                assert sb == 0x7E                                      # caller's g too small: saturate
            else:
                assert a <= 3.5 * s * g                                # invariant
                prev = max([tab[bb] for bb in range(1, 0x7F) if tab[bb] < s], default=0.0)
                assert prev == 0.0 or not (a <= 3.5 * prev * g)        # minimal
            for j in range(16):
                cc = c[r, 16 * b + j]
                assert (cc & 7) == _nearest_even(abs(blk[j]), s * g)
                assert (cc >> 3) == (1 if np.signbit(blk[j]) else 0)


@pytest.mark.parametrize("with_shift", [False, True])
def test_quantize_blocks_with_and_without_shift(with_shift):
    x = wl.bf16_bits(wl.random_bf16(12, 128, 7, 1.0, "student_t")).copy()
    shift = np.random.default_rng(3).normal(0.0, 2.0, 128).astype(np.float32) if with_shift else None
    codes, scales, g = oracle.kv4_quantize(x, shift)
    d = indep.bf16_values(x).astype(np.float32)
    if shift is not None:
        d = d - shift[None, :]
    A = np.max(np.abs(d.astype(np.float64)))
    k = int(np.round(np.log2(g)))
    assert A <= 1568.0 * g and not (A <= 1568.0 * 2.0 ** (k - 1))
    _check_blocks(x, shift, g, codes, scales)


def test_given_scale_and_specials():
    x = np.zeros((4, 32), np.uint16)
    x[0, 3] = 0x7FC0                     # NaN -> NaN block
    x[1, :] = 0x8000                     # -0.0 everywhere: zero block, sign codes
    x[2, :16] = 0x4000                   # 2.0 with a caller's g too small -> 448, saturating
    x[3, 16] = 0x3F80
    codes, scales, g = oracle.kv4_quantize(x, None, g=2.0 ** -12)
    assert g == 2.0 ** -12
    assert scales[0, 0] == 0x7F and scales[1, 0] == 0 and scales[1, 1] == 0
    assert np.all(indep.unpack_codes(codes)[1] == 8)
    assert scales[2, 0] == 0x7E and np.all(indep.unpack_codes(codes)[2, :16] == 7)
    _check_blocks(x, None, g, codes, scales)


def test_fakequant_is_rounded_dequantization():
    x = wl.bf16_bits(wl.random_bf16(8, 64, 9, 1.0, "normal")).copy()
    shift = np.linspace(-1, 1, 64).astype(np.float32)
    codes, scales, g = oracle.kv4_quantize(x, shift)
    y, g2 = oracle.kv4_fakequant(x, shift)
    assert g2 == g
    c = indep.unpack_codes(codes)
    vals = e1m2_golden()[c] * np.repeat(indep.e4m3_table()[scales], 16, axis=1) * g
    assert np.array_equal(y, indep.to_bf16_bits(vals))
