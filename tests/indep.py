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


def format_metrics(m: dict) -> str:
    return "n=%d max|err|/sum|ab|=%.3g max rel(|Yref|>=1e-2 rms)=%.3g frobenius rel=%.3g" % (
        m["n"], m["max_rel_sum"], m["max_rel_elem"], m["frob_rel"])
