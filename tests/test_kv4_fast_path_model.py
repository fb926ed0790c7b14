"""CPU model of the KV4 kernel's rounding fast path (no GPU, no oracle).

With a power-of-two global scale the E1M2 code magnitude of a shifted value
d is the integer nearest |d| / H (H = s*g/2, s the block's E4M3 scale), ties
to even, at most 7.  The kernel takes c = rint(d * r) with r the hardware
reciprocal of H (within one ulp of 1/H) and trusts it unless
|q - rint(q)| >= 0.5 - 2^-17, q = d * r in FP32.  This test replays that
arithmetic in numpy float32 for r = RN(1/H) and its two neighbours and checks
every trusted code against the exact rational rounding, on random values,
on the exact midpoints (k + 1/2) H and on their neighbours one to three ulps
away, for every E4M3 mantissa and a spread of exponents.  It also checks the
two facts the kernel relies on: a trusted c never exceeds 7 in magnitude when
|d| <= 7 H, and the sign of c is the sign of d (-0 for small negative d).
"""
from fractions import Fraction

import numpy as np

RISK = np.float32(0.5 - 2.0 ** -17)


def exact_code(d, H):
    """Nearest integer to |d| / H, ties to even, capped at 7 (exact rationals)."""
    q = abs(Fraction(float(d))) / Fraction(float(H))
    n = int(q)                       # floor for q >= 0
    rem = q - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return min(n, 7)


def fast_path(d, r):
    q = (d * r).astype(np.float32)
    c = np.rint(q).astype(np.float32)
    e = (q - c).astype(np.float32)
    trusted = np.abs(e) < RISK
    return c, trusted


def _values(H, rng, n_random=400):
    H32 = np.float32(H)
    rnd = (rng.uniform(-7.0, 7.0, n_random) * float(H)).astype(np.float32)
    rnd = rnd[np.abs(rnd) <= np.float32(7.0) * H32]
    mids = []
    for k in range(7):
        t = np.float32((k + 0.5) * float(H))
        assert float(t) == (k + 0.5) * float(H)          # midpoints are exact in FP32 (<= 8 bits)
        for j in range(-3, 4):
            v = t
            for _ in range(abs(j)):
                v = np.nextafter(v, np.float32(np.inf if j > 0 else -np.inf), dtype=np.float32)
            mids += [v, -v]
    extra = np.array([0.0, -0.0, float(H) * 2.0 ** -30, -float(H) * 2.0 ** -30, 7.0 * float(H), -7.0 * float(H)],
                     np.float32)
    return np.concatenate([rnd, np.array(mids, np.float32), extra])


def test_fast_path_codes_match_exact_rounding():
    rng = np.random.default_rng(2024)
    checked = trusted_total = 0
    for m in range(8, 16):
        for e in (-120, -60, -9, -3, 0, 5, 40, 100):
            H = np.float32(m / 8.0 * 2.0 ** e)
            d = _values(H, rng)
            r0 = np.float32(1.0) / H                      # RN(1/H)
            for r in (r0, np.nextafter(r0, np.float32(0)), np.nextafter(r0, np.float32(np.inf))):
                c, trusted = fast_path(d, np.float32(r))
                for di, ci, ti in zip(d, c, trusted):
                    checked += 1
                    if not ti:
                        continue
                    trusted_total += 1
                    want = exact_code(di, H)
                    assert abs(float(ci)) == want, (m, e, float(di), float(ci), want)
                    assert abs(float(ci)) <= 7.0
                    assert np.signbit(ci) == np.signbit(di), (float(di), float(ci))
    # the window rejects only values near a midpoint: most random values are trusted
    assert trusted_total > 0.8 * checked


def test_exact_midpoints_are_never_trusted():
    """Every exact tie (k + 1/2) H must take the exact path, whatever the
    reciprocal's last bit, since rint(q) alone cannot see which way to go."""
    for m in range(8, 16):
        for e in (-100, -7, 0, 3, 90):
            H = np.float32(m / 8.0 * 2.0 ** e)
            t = np.array([np.float32((k + 0.5) * float(H)) for k in range(7)], np.float32)
            r0 = np.float32(1.0) / H
            for r in (r0, np.nextafter(r0, np.float32(0)), np.nextafter(r0, np.float32(np.inf))):
                _, trusted = fast_path(np.concatenate([t, -t]), np.float32(r))
                assert not trusted.any(), (m, e)


def test_fake_quant_values_are_exact_bfloat16():
    """c * H for c in 0..7 has at most 7 significant bits and is normal (H >= 2^-126),
    so dropping the low 16 bits of its FP32 pattern gives it exactly."""
    for m in range(8, 16):
        for e in (-126, -50, 0, 100):
            H = np.float32(m / 8.0 * 2.0 ** e)
            for c in range(8):
                v = np.float32(c) * H
                assert float(v) == c * float(H)
                bits = np.array([v], np.float32).view(np.uint32)[0]
                assert bits & 0xFFFF == 0, (m, e, c)
