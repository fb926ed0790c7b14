"""Oracle for the microscaled-FP4 linear layer -- TEST INFRASTRUCTURE ONLY.

A ctypes front end to ``reqat_oracle.c`` (plain single-threaded C, FP64,
exact decisions).  Only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import this package; the GPU library never does, and
this package imports nothing from it.

Formats and readings: see the header of ``reqat_oracle.c`` (ReQAT App. A,
Tab. mx_configs; the E2M1 layout of Sec. 1).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

FMT_NVFP4 = 0
FMT_MXFP4 = 1
BLOCK = {FMT_NVFP4: 16, FMT_MXFP4: 32}

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "reqat_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc -O2 (no OpenMP, no intrinsics)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        build(force=False)
        lib = ctypes.CDLL(_LIB)
        u8p = ctypes.POINTER(ctypes.c_uint8)
        u16p = ctypes.POINTER(ctypes.c_uint16)
        dp = ctypes.POINTER(ctypes.c_double)
        i64 = ctypes.c_int64
        i64p = ctypes.POINTER(ctypes.c_int64)
        sig = {
            "orc_e2m1_value": (ctypes.c_double, [ctypes.c_uint8]),
            "orc_e4m3_value": (ctypes.c_double, [ctypes.c_uint8]),
            "orc_e8m0_value": (ctypes.c_double, [ctypes.c_uint8]),
            "orc_bf16_value": (ctypes.c_double, [ctypes.c_uint16]),
            "orc_bf16_from_double": (ctypes.c_uint16, [ctypes.c_double]),
            "orc_mx_scale_byte": (ctypes.c_uint8, [ctypes.c_double]),
            "orc_nv_global_scale": (ctypes.c_float, [ctypes.c_double]),
            "orc_nv_scale_byte": (ctypes.c_uint8, [ctypes.c_double, ctypes.c_double]),
            "orc_e2m1_encode": (ctypes.c_uint8, [ctypes.c_double, ctypes.c_double]),
            "orc_tensor_amax": (ctypes.c_double, [u16p, i64, i64, i64]),
            "orc_quantize": (ctypes.c_int, [ctypes.c_int, u16p, i64, i64, i64, u8p, u8p, ctypes.c_double]),
            "orc_dequantize": (None, [ctypes.c_int, u8p, u8p, ctypes.c_double, i64, i64, dp]),
            "orc_fakequant": (ctypes.c_int, [ctypes.c_int, u16p, i64, i64, i64, u16p, i64,
                                             ctypes.c_double, u8p, u8p]),
            "orc_gemm_rows": (None, [ctypes.c_int, i64, i64, i64, u8p, u8p, ctypes.c_double,
                                     u8p, u8p, ctypes.c_double, i64, i64, dp]),
            "orc_gemm_points": (None, [ctypes.c_int, i64, u8p, u8p, ctypes.c_double,
                                       u8p, u8p, ctypes.c_double, i64p, i64p, i64, dp, dp]),
            "orc_e2m1_encode_array": (None, [dp, i64, ctypes.c_double, u8p]),
            "orc_bf16_from_double_array": (None, [dp, i64, u16p]),
            "orc_gemm_w4a16_points": (None, [i64, u16p, i64, u8p, u8p, i64p, i64p, i64, dp, dp]),
            "orc_e1m2_value": (ctypes.c_double, [ctypes.c_uint8]),
            "orc_e1m2_encode": (ctypes.c_uint8, [ctypes.c_double, ctypes.c_double]),
            "orc_kv4_global_scale": (ctypes.c_float, [ctypes.c_double]),
            "orc_kv4_scale_byte": (ctypes.c_uint8, [ctypes.c_double, ctypes.c_double]),
            "orc_kv4_amax": (ctypes.c_double, [u16p, i64, i64, i64, ctypes.POINTER(ctypes.c_float)]),
            "orc_kv4_quantize": (ctypes.c_int, [u16p, i64, i64, i64, ctypes.POINTER(ctypes.c_float),
                                                ctypes.c_double, u8p, u8p, u16p, i64]),
            "orc_quantize_mx_rht": (ctypes.c_int, [u16p, i64, i64, i64, ctypes.c_uint32, u8p, u8p]),
            "orc_fakequant_mx_rht": (ctypes.c_int, [u16p, i64, i64, i64, ctypes.c_uint32, u16p, i64]),
        }
        for name, (res, args) in sig.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
        return lib


def _p(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


# ----------------------------------------------------------------- scalars

def e2m1_value(code: int) -> float:
    return _load().orc_e2m1_value(code)


def e4m3_value(b: int) -> float:
    return _load().orc_e4m3_value(b)


def e8m0_value(b: int) -> float:
    return _load().orc_e8m0_value(b)


def bf16_value(h: int) -> float:
    return _load().orc_bf16_value(h)


def bf16_from_double(v: float) -> int:
    return _load().orc_bf16_from_double(v)


def mx_scale_byte(amax: float) -> int:
    return _load().orc_mx_scale_byte(amax)


def nv_global_scale(amax: float) -> float:
    return _load().orc_nv_global_scale(amax)


def nv_scale_byte(amax: float, g: float) -> int:
    return _load().orc_nv_scale_byte(amax, g)


def e2m1_encode(x: float, S: float) -> int:
    return _load().orc_e2m1_encode(x, S)


def e2m1_encode_array(x: np.ndarray, S: float) -> np.ndarray:
    """E2M1 codes (sign included) of each x[i] / S."""
    x = np.ascontiguousarray(x, np.float64)
    out = np.empty(x.shape, np.uint8)
    _load().orc_e2m1_encode_array(_p(x, ctypes.c_double), x.size, S, _p(out, ctypes.c_uint8))
    return out


def bf16_from_double_array(v: np.ndarray) -> np.ndarray:
    v = np.ascontiguousarray(v, np.float64)
    out = np.empty(v.shape, np.uint16)
    _load().orc_bf16_from_double_array(_p(v, ctypes.c_double), v.size, _p(out, ctypes.c_uint16))
    return out


# ----------------------------------------------------------------- tensors

def _as_u16(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x)
    if x.dtype != np.uint16:
        raise TypeError("oracle takes bfloat16 bit patterns as uint16")
    if x.ndim != 2:
        raise ValueError("2-D input expected")
    return x


def tensor_amax(x: np.ndarray) -> float:
    x = _as_u16(x)
    return _load().orc_tensor_amax(_p(x, ctypes.c_uint16), x.shape[0], x.shape[1], x.shape[1])


def global_scale(fmt: int, x: np.ndarray, given: float | None = None) -> float:
    """NVFP4: the given global scale, or the computed power of two.  MXFP4: 1."""
    if fmt == FMT_MXFP4:
        return 1.0
    if given is not None:
        return float(np.float32(given))
    return float(nv_global_scale(tensor_amax(x)))


def quantize(fmt: int, x: np.ndarray, g: float | None = None):
    """Return (codes uint8 [R, C/2], scales uint8 [R, C/B], g float)."""
    x = _as_u16(x)
    R, C = x.shape
    B = BLOCK[fmt]
    if C % B:
        raise ValueError("cols must be a multiple of the block size")
    g = global_scale(fmt, x, g)
    codes = np.zeros((R, C // 2), np.uint8)
    scales = np.zeros((R, C // B), np.uint8)
    rc = _load().orc_quantize(fmt, _p(x, ctypes.c_uint16), R, C, C,
                              _p(codes, ctypes.c_uint8), _p(scales, ctypes.c_uint8), g)
    assert rc == 0
    return codes, scales, g


def dequantize(fmt: int, codes: np.ndarray, scales: np.ndarray, g: float) -> np.ndarray:
    codes = np.ascontiguousarray(codes, np.uint8)
    scales = np.ascontiguousarray(scales, np.uint8)
    R, C = codes.shape[0], codes.shape[1] * 2
    out = np.empty((R, C), np.float64)
    _load().orc_dequantize(fmt, _p(codes, ctypes.c_uint8), _p(scales, ctypes.c_uint8), g, R, C,
                           _p(out, ctypes.c_double))
    return out


def fakequant(fmt: int, x: np.ndarray, g: float | None = None):
    """Return (y bfloat16 bits uint16 [R, C], g)."""
    x = _as_u16(x)
    R, C = x.shape
    B = BLOCK[fmt]
    g = global_scale(fmt, x, g)
    y = np.zeros((R, C), np.uint16)
    ct = np.zeros((R, C // 2), np.uint8)
    st = np.zeros((R, C // B), np.uint8)
    rc = _load().orc_fakequant(fmt, _p(x, ctypes.c_uint16), R, C, C, _p(y, ctypes.c_uint16), C, g,
                               _p(ct, ctypes.c_uint8), _p(st, ctypes.c_uint8))
    assert rc == 0
    return y, g


def gemm(fmt, a_codes, a_scales, ga, b_codes, b_scales, gb, rows=None) -> np.ndarray:
    """FP64 Y[m, n] = sum_k A^[m, k] B^[n, k] (rows = optional (m0, m1) slice)."""
    a_codes = np.ascontiguousarray(a_codes, np.uint8)
    b_codes = np.ascontiguousarray(b_codes, np.uint8)
    a_scales = np.ascontiguousarray(a_scales, np.uint8)
    b_scales = np.ascontiguousarray(b_scales, np.uint8)
    M, K = a_codes.shape[0], a_codes.shape[1] * 2
    N = b_codes.shape[0]
    m0, m1 = rows if rows is not None else (0, M)
    y = np.empty((m1 - m0, N), np.float64)
    _load().orc_gemm_rows(fmt, M, N, K, _p(a_codes, ctypes.c_uint8), _p(a_scales, ctypes.c_uint8), ga,
                          _p(b_codes, ctypes.c_uint8), _p(b_scales, ctypes.c_uint8), gb, m0, m1,
                          _p(y, ctypes.c_double))
    return y


def gemm_points(fmt, a_codes, a_scales, ga, b_codes, b_scales, gb, ms, ns):
    """FP64 Y at the (ms[i], ns[i]) pairs, and sum_k |A^ B^| at each."""
    a_codes = np.ascontiguousarray(a_codes, np.uint8)
    b_codes = np.ascontiguousarray(b_codes, np.uint8)
    a_scales = np.ascontiguousarray(a_scales, np.uint8)
    b_scales = np.ascontiguousarray(b_scales, np.uint8)
    ms = np.ascontiguousarray(ms, np.int64)
    ns = np.ascontiguousarray(ns, np.int64)
    K = a_codes.shape[1] * 2
    y = np.empty(len(ms), np.float64)
    ay = np.empty(len(ms), np.float64)
    _load().orc_gemm_points(fmt, K, _p(a_codes, ctypes.c_uint8), _p(a_scales, ctypes.c_uint8), ga,
                            _p(b_codes, ctypes.c_uint8), _p(b_scales, ctypes.c_uint8), gb,
                            _p(ms, ctypes.c_int64), _p(ns, ctypes.c_int64), len(ms),
                            _p(y, ctypes.c_double), _p(ay, ctypes.c_double))
    return y, ay


# ------------------------------------------------- block rotation (MXFP4)

def quantize_mx_rht(x: np.ndarray, signs: int):
    """MXFP4 codes and scales of the block-rotated rows: (codes [R, C/2], scales [R, C/32])."""
    x = _as_u16(x)
    R, C = x.shape
    if C % 32:
        raise ValueError("cols must be a multiple of 32")
    codes = np.zeros((R, C // 2), np.uint8)
    scales = np.zeros((R, C // 32), np.uint8)
    rc = _load().orc_quantize_mx_rht(_p(x, ctypes.c_uint16), R, C, C, ctypes.c_uint32(signs),
                                     _p(codes, ctypes.c_uint8), _p(scales, ctypes.c_uint8))
    assert rc == 0
    return codes, scales


def fakequant_mx_rht(x: np.ndarray, signs: int) -> np.ndarray:
    """bfloat16 bits of the dequantized rotated values (rotated basis), [R, C]."""
    x = _as_u16(x)
    R, C = x.shape
    y = np.zeros((R, C), np.uint16)
    rc = _load().orc_fakequant_mx_rht(_p(x, ctypes.c_uint16), R, C, C, ctypes.c_uint32(signs),
                                      _p(y, ctypes.c_uint16), C)
    assert rc == 0
    return y


# ------------------------------------------------------------------ W4A16

def gemm_w4a16_points(x: np.ndarray, w_codes: np.ndarray, w_scales: np.ndarray, ms, ns):
    """FP64 Y[m, n] = sum_k x[m, k] RN_bf16(w^[n, k]) at the (ms[i], ns[i]) pairs
    (x bfloat16 bits [M, K]; MXFP4 weights), and sum_k |x w^| at each."""
    x = _as_u16(x)
    w_codes = np.ascontiguousarray(w_codes, np.uint8)
    w_scales = np.ascontiguousarray(w_scales, np.uint8)
    ms = np.ascontiguousarray(ms, np.int64)
    ns = np.ascontiguousarray(ns, np.int64)
    K = x.shape[1]
    if w_codes.shape[1] * 2 != K or w_scales.shape[1] * 32 != K:
        raise ValueError("K mismatch")
    y = np.empty(len(ms), np.float64)
    ay = np.empty(len(ms), np.float64)
    _load().orc_gemm_w4a16_points(K, _p(x, ctypes.c_uint16), K, _p(w_codes, ctypes.c_uint8),
                                  _p(w_scales, ctypes.c_uint8), _p(ms, ctypes.c_int64),
                                  _p(ns, ctypes.c_int64), len(ms), _p(y, ctypes.c_double),
                                  _p(ay, ctypes.c_double))
    return y, ay


# ------------------------------------------------- KV4 (E1M2, post-RoPE shift)

def e1m2_value(code: int) -> float:
    return _load().orc_e1m2_value(code)


def e1m2_encode(v: float, S: float) -> int:
    return _load().orc_e1m2_encode(v, S)


def kv4_global_scale(amax: float) -> float:
    return _load().orc_kv4_global_scale(amax)


def kv4_scale_byte(amax: float, g: float) -> int:
    return _load().orc_kv4_scale_byte(amax, g)


def _shift_arg(shift, C):
    if shift is None:
        return None, None
    sh = np.ascontiguousarray(shift, np.float32).reshape(C)
    return sh, _p(sh, ctypes.c_float)


def kv4_global(x: np.ndarray, shift=None, g: float | None = None) -> float:
    """The given g (as FP32), or the computed power of two over the shifted values."""
    x = _as_u16(x)
    if g is not None:
        return float(np.float32(g))
    sh, shp = _shift_arg(shift, x.shape[1])
    amax = _load().orc_kv4_amax(_p(x, ctypes.c_uint16), x.shape[0], x.shape[1], x.shape[1], shp)
    return float(kv4_global_scale(amax))


def kv4_quantize(x: np.ndarray, shift=None, g: float | None = None):
    """KV4 codes [R, C/2], E4M3 scales [R, C/16] and g of the shifted rows x - shift."""
    x = _as_u16(x)
    R, C = x.shape
    if C % 16:
        raise ValueError("cols must be a multiple of 16")
    g = kv4_global(x, shift, g)
    sh, shp = _shift_arg(shift, C)
    codes = np.zeros((R, C // 2), np.uint8)
    scales = np.zeros((R, C // 16), np.uint8)
    rc = _load().orc_kv4_quantize(_p(x, ctypes.c_uint16), R, C, C, shp, g, _p(codes, ctypes.c_uint8),
                                  _p(scales, ctypes.c_uint8), None, 0)
    assert rc == 0
    return codes, scales, g


def kv4_fakequant(x: np.ndarray, shift=None, g: float | None = None):
    """bfloat16 bits of the dequantized shifted rows (shifted domain), and g."""
    x = _as_u16(x)
    R, C = x.shape
    g = kv4_global(x, shift, g)
    sh, shp = _shift_arg(shift, C)
    y = np.zeros((R, C), np.uint16)
    rc = _load().orc_kv4_quantize(_p(x, ctypes.c_uint16), R, C, C, shp, g, None, None,
                                  _p(y, ctypes.c_uint16), C)
    assert rc == 0
    return y, g


# ------------------------------------------------- SEM loss (QAT training side)

def sem_row_stats(logits_bits: np.ndarray, targets: np.ndarray):
    """Per token t (one row of bfloat16 logits over the vocabulary): the
    predictive entropy H_t = -sum_j p_j log p_j, the SFT term NLL_t =
    -log p_{y_t}, and log-sum-exp, with p = softmax(logits) (Sec. 4.2, the
    token-level entropy of Sec. 2 and the SFT objective), in FP64."""
    z = _bf16_rows_f64(logits_bits)
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    S = e.sum(axis=1, keepdims=True)
    logp = (z - m) - np.log(S)
    p = e / S
    H = -(p * logp).sum(axis=1)
    t = np.asarray(targets, np.int64)
    nll = -logp[np.arange(z.shape[0]), t]
    lse = (m + np.log(S))[:, 0]
    return H, nll, lse


def _bf16_rows_f64(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(bits, np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def sem_weights(H: np.ndarray, eps: float) -> np.ndarray:
    """Soft weights of SEM (Sec. 4.2): w_t = max(0, 1 - (H_t - H_min) / (tau - H_min + eps)),
    H_min the minibatch minimum and tau its 75th percentile (linear interpolation
    between order statistics at position 0.75 (T - 1))."""
    H = np.asarray(H, np.float64)
    hs = np.sort(H)
    q = 0.75 * (len(H) - 1)
    lo = int(np.floor(q))
    hi = min(lo + 1, len(H) - 1)
    tau = hs[lo] + (q - lo) * (hs[hi] - hs[lo])
    hmin = hs[0]
    return np.maximum(0.0, 1.0 - (H - hmin) / (tau - hmin + eps)), tau, hmin


def sem_loss(H, nll, lam: float, eps: float):
    """L_SEM = mean_t NLL_t + lam * (1/T) sum_t w_t H_t (Sec. 4.2).  Returns
    (L, L_SFT, L_ent, w)."""
    w, _, _ = sem_weights(H, eps)
    T = len(H)
    l_sft = float(np.sum(nll)) / T
    l_ent = float(np.sum(w * np.asarray(H, np.float64))) / T
    return l_sft + lam * l_ent, l_sft, l_ent, w


def sem_grad(logits_bits, targets, H, lse, w, lam: float, scale: float = 1.0):
    """dL/dlogits with the weights held fixed:
    (scale / T) * [(p - onehot(y)) - lam * w_t * p * (log p + H_t)]."""
    z = _bf16_rows_f64(logits_bits)
    T = z.shape[0]
    logp = z - np.asarray(lse, np.float64)[:, None]
    p = np.exp(logp)
    g = p.copy()
    g[np.arange(T), np.asarray(targets, np.int64)] -= 1.0
    g -= lam * np.asarray(w, np.float64)[:, None] * p * (logp + np.asarray(H, np.float64)[:, None])
    return g * (scale / T)
