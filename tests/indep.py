"""Independent statements used to pin the oracle (test helpers only).

Nothing here calls the oracle's arithmetic: the E2M1 table comes from the
hand-written golden fixture, the FP8 scale tables from torch's own float8
dtypes, bfloat16 rounding from torch's float64 -> bfloat16 conversion, and
rounding decisions from brute-force nearest-value searches.
"""
from __future__ import annotations

import os
from fractions import Fraction

import numpy as np
import torch

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def e2m1_table() -> np.ndarray:
    """Value of each of the 16 E2M1 codes, from tests/golden/e2m1_grid.txt."""
    vals = np.zeros(16, np.float64)
    with open(os.path.join(GOLDEN, "e2m1_grid.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            c, v = line.split()
            vals[int(c)] = float(v)
    return vals


def e4m3_table() -> np.ndarray:
    """Value of each of the 256 E4M3FN bytes, decoded by torch."""
    return torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def e8m0_table() -> np.ndarray:
    """Value of each of the 256 E8M0 bytes, decoded by torch."""
    return torch.arange(256, dtype=torch.uint8).view(torch.float8_e8m0fnu).to(torch.float64).numpy()


def bf16_values(bits: np.ndarray) -> np.ndarray:
    """float64 values of bfloat16 bit patterns (via torch)."""
    t = torch.from_numpy(np.ascontiguousarray(bits, np.uint16).view(np.int16)).view(torch.bfloat16)
    return t.to(torch.float64).numpy()


def to_bf16_bits(v: np.ndarray) -> np.ndarray:
    """torch's round-to-nearest-even of float64 values to bfloat16, as bits."""
    t = torch.from_numpy(np.ascontiguousarray(v, np.float64)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


GRID = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def nearest_code_brute(ax: np.ndarray, S: float) -> np.ndarray:
    """Magnitude code (0..7) of the grid value v*S nearest to each |x|;
    on equal distance the even code wins.  Distances are exact in FP64 for
    |x| / S < 2^40 (callers keep to that range)."""
    cand = GRID[None, :] * S
    d = np.abs(ax[:, None] - cand)
    best = d.min(axis=1, keepdims=True)
    hit = d == best
    # prefer the even code among the nearest: first even hit, else first hit
    even = hit & (np.arange(8)[None, :] % 2 == 0)
    idx_even = np.where(even.any(axis=1), even.argmax(axis=1), -1)
    idx_any = hit.argmax(axis=1)
    return np.where(idx_even >= 0, idx_even, idx_any).astype(np.uint8)


def nearest_code_fraction(x: Fraction, S: Fraction) -> int:
    """Exact-rational brute force for one value."""
    ax = abs(x)
    ds = [abs(ax - Fraction(g).limit_denominator(4) * S) for g in GRID]
    best = min(ds)
    hits = [i for i, d in enumerate(ds) if d == best]
    ev = [i for i in hits if i % 2 == 0]
    return ev[0] if ev else hits[0]


def unpack_codes(codes: np.ndarray) -> np.ndarray:
    """[R, C/2] packed bytes -> [R, C] codes, element 2i from bits 3:0."""
    lo = codes & 0xF
    hi = codes >> 4
    out = np.empty((codes.shape[0], codes.shape[1] * 2), np.uint8)
    out[:, 0::2] = lo
    out[:, 1::2] = hi
    return out


def dequant_indep(fmt: int, codes: np.ndarray, scales: np.ndarray, g: float) -> np.ndarray:
    """Dequantized matrix from the golden E2M1 table and torch's FP8 tables."""
    B = 32 if fmt == 1 else 16
    c = unpack_codes(codes)
    v = e2m1_table()[c]
    st = (e8m0_table() if fmt == 1 else e4m3_table())[scales]
    S = np.repeat(st, B, axis=1)
    if fmt == 0:
        S = S * g
    return v * S


def gemm_error_metrics(got: np.ndarray, ref: np.ndarray, aref: np.ndarray) -> dict:
    """Error of a product against its FP64 reference, three ways: the largest
    |Y - Yref| / sum_k |A^ B^| (the scale FP32 accumulation error grows with),
    the largest elementwise relative error over entries with |Yref| >= 1e-2 of
    the rms of Yref, and the Frobenius relative error.  NaN references are left out."""
    ok = ~np.isnan(ref)
    got, ref, aref = got[ok].astype(np.float64), ref[ok], aref[ok]
    err = np.abs(got - ref)
    out = {"n": int(ok.sum()), "max_rel_sum": 0.0, "max_rel_elem": 0.0, "frob_rel": 0.0}
    if not ref.size:
        return out
    out["max_rel_sum"] = float(np.max(err / np.maximum(aref, 1e-300)))
    rms = float(np.sqrt(np.mean(ref * ref)))
    big = np.abs(ref) >= 1e-2 * rms
    if big.any():
        out["max_rel_elem"] = float(np.max(err[big] / np.abs(ref[big])))
    out["frob_rel"] = float(np.linalg.norm(got - ref) / max(float(np.linalg.norm(ref)), 1e-300))
    return out


def fp32_accumulation_bound(K: int) -> float:
    """A regression bound on max |Y - Yref| / sum_k |A^ B^| far tighter than the 1e-3
    contract: one FP32 rounding (2^-24 relative) per 16 elements of K, the finest
    matrix-instruction step the products use (the observed error is 0 on every
    workload: the sums fit FP32)."""
    return max(K / 16.0, 1.0) * 2.0 ** -24


def format_metrics(m: dict) -> str:
    return "n=%d max|err|/sum|ab|=%.3g max rel(|Yref|>=1e-2 rms)=%.3g frobenius rel=%.3g" % (
        m["n"], m["max_rel_sum"], m["max_rel_elem"], m["frob_rel"])


# ------------------------------------------------ exact block rotation (Python integers)

def _hadamard32() -> np.ndarray:
    import scipy.linalg
    return scipy.linalg.hadamard(32).astype(np.int64)


def rht_block_reference(x_bits: np.ndarray, signs: int):
    """(E8M0 byte, 32 codes) of the exactly rotated MXFP4 block y = H D x / sqrt(32),
    computed with Python integers and fractions: x * 2^133 is an integer for
    every bfloat16 value, the Hadamard matrix is scipy's, the E2M1 values
    (and so the midpoints and the largest value 6) come from the golden table,
    and |y| is compared with t * 2^e through y^2 = S^2 * 2^-266 / 32."""
    x_bits = np.asarray(x_bits, np.uint16).reshape(32)
    vals = bf16_values(x_bits)
    if not np.all(np.isfinite(vals)):
        return 0xFF, np.zeros(32, np.uint8)
    X = [int(Fraction(float(v)) * 2 ** 133) for v in vals]
    d = [-1 if (signs >> j) & 1 else 1 for j in range(32)]
    H = _hadamard32()
    S = [sum(int(H[i, j]) * d[j] * X[j] for j in range(32)) for i in range(32)]
    a2 = max(s * s for s in S)
    if a2 == 0:
        return 0, np.zeros(32, np.uint8)
    table = e2m1_table()
    pos = sorted(Fraction(float(v)) for v in table[:8])
    top = pos[-1]                                       # 6
    mids = [(pos[m] + pos[m + 1]) / 2 for m in range(7)]

    def above(s2, t, e):                                # |y| > t * 2^e, exactly
        return Fraction(s2, 32) > t * t * Fraction(2) ** (2 * e + 266)

    e = -127
    while e < 127 and above(a2, top, e):
        e += 1
    codes = np.zeros(32, np.uint8)
    for i, s in enumerate(S):
        m3 = sum(1 for t in mids if above(s * s, t, e))
        codes[i] = m3 | (8 if s < 0 else 0)
    return e + 127, codes


def rht_near_threshold_block(t: Fraction, e: int, above: bool, chunks: int, signs: int = 0,
                             big: Fraction | None = None) -> np.ndarray:
    """32 bfloat16 bit patterns whose rotated first value y_0 = sum_j d_j x_j / sqrt(32)
    lies just above (or below) t * 2^e: the pieces d_j x_j >= 0 (j < chunks) are
    consecutive 8-bit slices of the binary expansion of sqrt(32) * t * 2^e, cut after
    `chunks` slices (the last one rounded up for `above`), so a decision about y_0 hinges
    on bits about 8 * chunks below its leading one, far below FP64 precision.  Without
    `big`, S_0 is the largest |S_i| and sets the scale; with it, d_30 x_30 = big and
    d_31 x_31 = -big cancel in S_0 and give every odd S_i about 2 big, which then sets it."""
    from decimal import Decimal, getcontext
    getcontext().prec = 300
    target = Decimal(32).sqrt() * Decimal(t.numerator) / Decimal(t.denominator) * Decimal(2) ** e
    lead = 0
    while Decimal(2) ** (lead + 1) <= target:
        lead += 1
    while Decimal(2) ** lead > target:
        lead -= 1
    pieces = []
    rem = target
    chunks = min(chunks, (lead - 7 + 133) // 8 + 1)     # every slice a multiple of 2^-133
    for c in range(chunks):
        unit = Decimal(2) ** (lead - 7 - 8 * c)
        m = int(rem / unit)
        rem -= Decimal(m) * unit
        if c == chunks - 1 and above:
            m += 1
        assert 0 <= m <= 256
        pieces.append(Fraction(m) * Fraction(2) ** (lead - 7 - 8 * c))
    pieces += [Fraction(0)] * (32 - len(pieces))
    if big is not None:
        pieces[30], pieces[31] = big, -big
    vals = np.array([float(v) for v in pieces], np.float64)
    dv = np.array([-1.0 if (signs >> j) & 1 else 1.0 for j in range(32)])
    bits = to_bf16_bits(vals * dv)
    assert [Fraction(float(v)) for v in bf16_values(bits) * dv] == pieces, "a slice is not a bfloat16 value"
    return bits
