"""ctypes binding of libreqat (C ABI in include/reqat.h).

Two layers:
  * ``reqat_quantize_fp4``, ``reqat_fakequant_fp4``, ``reqat_gemm_w4a4``, ... --
    the C entry points under the same names, taking raw device pointers
    (ints) and sizes; they return the C status code.
  * ``quantize``, ``fakequant``, ``gemm`` -- torch-tensor conveniences that
    allocate outputs with torch, pass ``data_ptr()`` and the current HIP
    stream, and raise ``ReqatError`` on a non-OK status.

Every step of the computation runs in the HIP library; this module only
marshals arguments.  It raises at load time when the library is missing.
"""
from __future__ import annotations

import ctypes
import os

import torch

NVFP4 = 0
MXFP4 = 1
BLOCK = {NVFP4: 16, MXFP4: 32}
DT_F32 = 0
DT_BF16 = 1
TS_COMPUTE = 0
TS_GIVEN = 1

STATUS = {0: "REQAT_OK", 1: "REQAT_E_NULL", 2: "REQAT_E_SHAPE", 3: "REQAT_E_ALIGN",
          4: "REQAT_E_ENUM", 5: "REQAT_E_UNSUPPORTED", 6: "REQAT_E_HIP", 7: "REQAT_E_TOO_LARGE"}
NOALLOC_SCRATCH_BYTES = 8 << 20          # REQAT_NOALLOC_SCRATCH_BYTES

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libreqat.so")

# every symbol include/reqat.h declares, with its ctypes signature
_VP = ctypes.c_void_p
_I64 = ctypes.c_int64
_INT = ctypes.c_int
SIGNATURES = {
    "reqat_quantize_fp4": (_INT, [_INT, _VP, _I64, _I64, _I64, _VP, _VP, _VP, _INT, _VP, _VP]),
    "reqat_fakequant_fp4": (_INT, [_INT, _VP, _I64, _I64, _I64, _VP, _I64, _VP, _INT, _VP, _VP]),
    "reqat_quantize_fakequant_fp4": (_INT, [_INT, _VP, _I64, _I64, _I64, _VP, _VP, _VP, _I64, _VP, _INT, _VP,
                                            _VP]),
    "reqat_gemm_w4a4": (_INT, [_INT, _I64, _I64, _I64, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _INT,
                               _I64, _VP]),
    "reqat_linear_w4a4": (_INT, [_INT, _I64, _I64, _I64, _VP, _I64, _VP, _INT, _VP, _VP, _VP, _VP,
                                 _INT, _I64, _VP, _VP]),
    "reqat_linear_workspace_bytes": (ctypes.c_size_t, [_INT, _I64, _I64]),
    "reqat_w4a4_packed_bytes": (ctypes.c_size_t, [_INT, _I64, _I64]),
    "reqat_pack_w4a4": (_INT, [_INT, _VP, _VP, _I64, _I64, _VP, _VP]),
    "reqat_gemm_w4a4_packed": (_INT, [_INT, _I64, _I64, _I64, _VP, _VP, _VP, _VP, _VP, _VP, _INT, _I64, _VP]),
    "reqat_linear_w4a4_packed": (_INT, [_INT, _I64, _I64, _I64, _VP, _I64, _VP, _INT, _VP, _VP, _VP, _INT, _I64,
                                        _VP, _VP]),
    "reqat_linear_w4a4_noalloc": (_INT, [_INT, _I64, _I64, _I64, _VP, _I64, _VP, _INT, _VP, _VP, _VP, _VP,
                                         _INT, _I64, _VP]),
    "reqat_sem_loss": (_INT, [_VP, _I64, _I64, _I64, _VP, ctypes.c_float, ctypes.c_float, _VP, _VP, _VP, _VP]),
    "reqat_sem_loss_backward": (_INT, [_VP, _I64, _I64, _I64, _VP, _VP, _VP, ctypes.c_float, ctypes.c_float,
                                       _VP, _INT, _I64, _VP]),
    "reqat_quantize_kv4": (_INT, [_VP, _I64, _I64, _I64, _VP, _VP, _VP, _VP, _INT, _VP, _VP]),
    "reqat_fakequant_kv4": (_INT, [_VP, _I64, _I64, _I64, _VP, _VP, _I64, _VP, _INT, _VP, _VP]),
    "reqat_gemm_w4a16": (_INT, [_I64, _I64, _I64, _VP, _I64, _VP, _VP, _VP, _INT, _I64, _VP, _VP]),
    "reqat_w4a16_workspace_bytes": (ctypes.c_size_t, [_I64, _I64, _I64]),
    "reqat_w4a16_packed_bytes": (ctypes.c_size_t, [_I64, _I64]),
    "reqat_pack_w4a16": (_INT, [_VP, _VP, _I64, _I64, _VP, _VP]),
    "reqat_gemm_w4a16_packed": (_INT, [_I64, _I64, _I64, _VP, _I64, _VP, _VP, _INT, _I64, _VP, _VP]),
    "reqat_quantize_mxfp4_rht": (_INT, [_VP, _I64, _I64, _I64, ctypes.c_uint32, _VP, _VP, _VP]),
    "reqat_fakequant_mxfp4_rht": (_INT, [_VP, _I64, _I64, _I64, ctypes.c_uint32, _VP, _I64, _VP]),
    "reqat_workspace_bytes": (ctypes.c_size_t, []),
    "reqat_status_str": (ctypes.c_char_p, [_INT]),
    "reqat_abi_version": (_INT, []),
}

_lib = None


class ReqatError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__("%s failed: %s" % (where, STATUS.get(status, status)))
        self.status = status


def load(path: str = LIB_PATH):
    """Load libreqat.so once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libreqat.so is not built (%s); run python -m paper_2606_15682_amd.build"
                           % path)
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


# ------------------------------------------------------------------ raw C entry points

def reqat_quantize_fp4(fmt, x, rows, cols, ldx, codes, scales, tensor_scale, ts, workspace, stream):
    return load().reqat_quantize_fp4(fmt, x, rows, cols, ldx, codes, scales, tensor_scale, ts,
                                     workspace, stream)


def reqat_fakequant_fp4(fmt, x, rows, cols, ldx, y, ldy, tensor_scale, ts, workspace, stream):
    return load().reqat_fakequant_fp4(fmt, x, rows, cols, ldx, y, ldy, tensor_scale, ts, workspace,
                                      stream)


def reqat_quantize_fakequant_fp4(fmt, x, rows, cols, ldx, codes, scales, y, ldy, tensor_scale, ts, workspace,
                                 stream):
    return load().reqat_quantize_fakequant_fp4(fmt, x, rows, cols, ldx, codes, scales, y, ldy, tensor_scale, ts,
                                               workspace, stream)


def reqat_gemm_w4a4(fmt, M, N, K, a_codes, a_scales, a_ts, b_codes, b_scales, b_ts, y, y_dtype,
                    ldy, stream):
    return load().reqat_gemm_w4a4(fmt, M, N, K, a_codes, a_scales, a_ts, b_codes, b_scales, b_ts, y,
                                  y_dtype, ldy, stream)


def reqat_linear_w4a4(fmt, M, N, K, x, ldx, x_ts, ts, w_codes, w_scales, w_ts, y, y_dtype, ldy,
                      workspace, stream):
    return load().reqat_linear_w4a4(fmt, M, N, K, x, ldx, x_ts, ts, w_codes, w_scales, w_ts, y,
                                    y_dtype, ldy, workspace, stream)


def reqat_sem_loss(logits, T, V, ld, targets, lam, eps, stats, weights, loss, stream):
    return load().reqat_sem_loss(logits, T, V, ld, targets, lam, eps, stats, weights, loss, stream)


def reqat_sem_loss_backward(logits, T, V, ld, targets, stats, weights, lam, scale, grad, grad_dtype, ldg, stream):
    return load().reqat_sem_loss_backward(logits, T, V, ld, targets, stats, weights, lam, scale, grad, grad_dtype,
                                          ldg, stream)


def reqat_quantize_kv4(x, rows, cols, ldx, shift, codes, scales, tensor_scale, ts, workspace, stream):
    return load().reqat_quantize_kv4(x, rows, cols, ldx, shift, codes, scales, tensor_scale, ts, workspace,
                                     stream)


def reqat_fakequant_kv4(x, rows, cols, ldx, shift, y, ldy, tensor_scale, ts, workspace, stream):
    return load().reqat_fakequant_kv4(x, rows, cols, ldx, shift, y, ldy, tensor_scale, ts, workspace, stream)


def reqat_gemm_w4a16(M, N, K, x, ldx, w_codes, w_scales, y, y_dtype, ldy, workspace, stream):
    return load().reqat_gemm_w4a16(M, N, K, x, ldx, w_codes, w_scales, y, y_dtype, ldy, workspace, stream)


def reqat_w4a16_workspace_bytes(M, N, K) -> int:
    return load().reqat_w4a16_workspace_bytes(M, N, K)


def reqat_w4a16_packed_bytes(N, K) -> int:
    return load().reqat_w4a16_packed_bytes(N, K)


def reqat_pack_w4a16(w_codes, w_scales, N, K, packed, stream):
    return load().reqat_pack_w4a16(w_codes, w_scales, N, K, packed, stream)


def reqat_gemm_w4a16_packed(M, N, K, x, ldx, packed, y, y_dtype, ldy, workspace, stream):
    return load().reqat_gemm_w4a16_packed(M, N, K, x, ldx, packed, y, y_dtype, ldy, workspace, stream)


def reqat_quantize_mxfp4_rht(x, rows, cols, ldx, signs, codes, scales, stream):
    return load().reqat_quantize_mxfp4_rht(x, rows, cols, ldx, signs, codes, scales, stream)


def reqat_fakequant_mxfp4_rht(x, rows, cols, ldx, signs, y, ldy, stream):
    return load().reqat_fakequant_mxfp4_rht(x, rows, cols, ldx, signs, y, ldy, stream)


def reqat_w4a4_packed_bytes(fmt, N, K) -> int:
    return load().reqat_w4a4_packed_bytes(fmt, N, K)


def reqat_pack_w4a4(fmt, w_codes, w_scales, N, K, packed, stream):
    return load().reqat_pack_w4a4(fmt, w_codes, w_scales, N, K, packed, stream)


def reqat_gemm_w4a4_packed(fmt, M, N, K, a_codes, a_scales, a_ts, packed, b_ts, y, y_dtype, ldy, stream):
    return load().reqat_gemm_w4a4_packed(fmt, M, N, K, a_codes, a_scales, a_ts, packed, b_ts, y, y_dtype, ldy,
                                         stream)


def reqat_linear_w4a4_packed(fmt, M, N, K, x, ldx, x_ts, ts, packed, w_ts, y, y_dtype, ldy, workspace, stream):
    return load().reqat_linear_w4a4_packed(fmt, M, N, K, x, ldx, x_ts, ts, packed, w_ts, y, y_dtype, ldy,
                                           workspace, stream)


def reqat_linear_workspace_bytes(fmt, M, K) -> int:
    return load().reqat_linear_workspace_bytes(fmt, M, K)


def reqat_linear_w4a4_noalloc(fmt, M, N, K, x, ldx, x_ts, ts, w_codes, w_scales, w_ts, y, y_dtype, ldy, stream):
    return load().reqat_linear_w4a4_noalloc(fmt, M, N, K, x, ldx, x_ts, ts, w_codes, w_scales, w_ts, y,
                                            y_dtype, ldy, stream)


def reqat_workspace_bytes() -> int:
    return load().reqat_workspace_bytes()


def reqat_status_str(s: int) -> str:
    return load().reqat_status_str(s).decode()


def reqat_abi_version() -> int:
    return load().reqat_abi_version()


# ------------------------------------------------------------------ torch conveniences

def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _check(st: int, where: str):
    if st != 0:
        raise ReqatError(st, where)


def _ptr(t):
    return None if t is None else t.data_ptr()


def _x2d(x: torch.Tensor):
    if not isinstance(x, torch.Tensor) or x.dtype != torch.bfloat16 or x.dim() != 2:
        raise TypeError("expected a 2-D bfloat16 tensor")
    if x.stride(1) != 1:
        raise ValueError("rows must be contiguous")
    return x.shape[0], x.shape[1], x.stride(0)


def _same_device(t, device, name):
    if t.device != device:
        raise ValueError("%s must be on %s" % (name, device))


def _require_cuda(t, name="x"):
    """Checked after every shape, dtype and size check, right before the C call."""
    if not t.is_cuda:
        raise TypeError("%s must be a CUDA (HIP) tensor" % name)


def _packed_u8(t, rows, cols, device, name):
    """A uint8 [rows, cols] tensor with dense rows (the C ABI takes no row stride for codes and scales)."""
    if not isinstance(t, torch.Tensor) or t.dtype != torch.uint8:
        raise TypeError("%s must be a uint8 tensor" % name)
    if tuple(t.shape) != (rows, cols):
        raise ValueError("%s must have shape (%d, %d), got %s" % (name, rows, cols, tuple(t.shape)))
    if rows > 1 and cols > 0 and t.stride(0) != cols or cols > 1 and t.stride(1) != 1:
        raise ValueError("%s must be contiguous" % name)
    _same_device(t, device, name)
    return t


def _out2d(t, rows, cols, dtype, device, name):
    """An output [rows, cols] of `dtype` with unit column stride; returns its row stride."""
    if not isinstance(t, torch.Tensor) or t.dtype != dtype:
        raise TypeError("%s must be a %s tensor" % (name, dtype))
    if t.dim() != 2 or tuple(t.shape) != (rows, cols):
        raise ValueError("%s must have shape (%d, %d), got %s" % (name, rows, cols, tuple(t.shape)))
    if cols > 1 and t.stride(1) != 1:
        raise ValueError("%s rows must be contiguous" % name)
    _same_device(t, device, name)
    return t.stride(0) if rows > 1 else max(cols, 1)


def _workspace_arg(ws, nbytes, device, name="ws"):
    if not isinstance(ws, torch.Tensor) or ws.dtype != torch.uint8 or not ws.is_contiguous():
        raise TypeError("%s must be a contiguous uint8 tensor" % name)
    if ws.numel() < nbytes:
        raise ValueError("%s holds %d bytes, %d needed" % (name, ws.numel(), nbytes))
    _same_device(ws, device, name)
    return ws


def _scale_arg(g, fmt, device, name):
    """The 1-element float32 device tensor of an NVFP4 global scale (MXFP4: None)."""
    if fmt == MXFP4:
        if g is not None:
            raise ValueError("MXFP4 has no global scale (%s must be None)" % name)
        return None
    if not isinstance(g, torch.Tensor) or g.dtype != torch.float32 or g.numel() < 1:
        raise TypeError("%s must be a float32 tensor holding the NVFP4 global scale" % name)
    _same_device(g, device, name)
    return g


def _fmt_arg(fmt):
    if fmt not in (NVFP4, MXFP4):
        raise ValueError("unknown format %r" % (fmt,))
    return fmt


_workspaces: dict = {}


def workspace(device) -> torch.Tensor:
    """A per-device workspace tensor (cached; calls on different streams must not share it)."""
    device = torch.device(device)
    key = (device.index if device.index is not None else torch.cuda.current_device())
    ws = _workspaces.get(key)
    if ws is None:
        ws = torch.empty(reqat_workspace_bytes(), dtype=torch.uint8, device=device)
        _workspaces[key] = ws
    return ws


def _gscale(fmt, x, tensor_scale, g_out=None):
    """(tensor_scale tensor or None, ts mode).  g_out: preallocated 1-element
    float32 tensor that receives the computed NVFP4 global scale."""
    if fmt == MXFP4:
        if tensor_scale is not None:
            raise ValueError("MXFP4 has no global scale")
        return None, TS_COMPUTE
    if tensor_scale is None:
        if g_out is not None:
            return _scale_arg(g_out, fmt, x.device, "g_out"), TS_COMPUTE
        return torch.empty(1, dtype=torch.float32, device=x.device), TS_COMPUTE
    if isinstance(tensor_scale, torch.Tensor):
        return _scale_arg(tensor_scale, fmt, x.device, "tensor_scale"), TS_GIVEN
    return torch.tensor([float(tensor_scale)], dtype=torch.float32, device=x.device), TS_GIVEN


def quantize(x: torch.Tensor, fmt: int = NVFP4, tensor_scale=None, out=None, g_out=None):
    """Quantize a 2-D bfloat16 CUDA tensor.  Returns (codes, scales, g) with g a
    1-element float32 tensor (NVFP4: computed unless given) or None (MXFP4)."""
    rows, cols, ldx = _x2d(x)
    B = BLOCK[_fmt_arg(fmt)]
    if cols % B:
        raise ValueError("cols must be a multiple of %d" % B)
    if out is not None:
        codes, scales = out
        _packed_u8(codes, rows, cols // 2, x.device, "codes")
        _packed_u8(scales, rows, cols // B, x.device, "scales")
    else:
        codes = torch.empty((rows, cols // 2), dtype=torch.uint8, device=x.device)
        scales = torch.empty((rows, cols // B), dtype=torch.uint8, device=x.device)
    g, ts = _gscale(fmt, x, tensor_scale, g_out)
    _require_cuda(x, 'x')
    ws = workspace(x.device)
    st = reqat_quantize_fp4(fmt, x.data_ptr(), rows, cols, ldx, codes.data_ptr(), scales.data_ptr(),
                            _ptr(g), ts, ws.data_ptr(), _stream(x.device))
    _check(st, "reqat_quantize_fp4")
    return codes, scales, g


def fakequant(x: torch.Tensor, fmt: int = NVFP4, tensor_scale=None, out=None, g_out=None):
    """Quantize-dequantize to bfloat16.  Returns (y, g)."""
    rows, cols, ldx = _x2d(x)
    _fmt_arg(fmt)
    y = out if out is not None else torch.empty((rows, cols), dtype=torch.bfloat16, device=x.device)
    ldy = _out2d(y, rows, cols, torch.bfloat16, x.device, "out")
    g, ts = _gscale(fmt, x, tensor_scale, g_out)
    _require_cuda(x, 'x')
    ws = workspace(x.device)
    st = reqat_fakequant_fp4(fmt, x.data_ptr(), rows, cols, ldx, y.data_ptr(), ldy, _ptr(g),
                             ts, ws.data_ptr(), _stream(x.device))
    _check(st, "reqat_fakequant_fp4")
    return y, g


def quantize_fakequant(x: torch.Tensor, fmt: int = NVFP4, tensor_scale=None, out=None, g_out=None):
    """Quantize and quantize-dequantize in one pass over x.  Returns
    (codes, scales, y, g): codes/scales as quantize(), y (bfloat16) as fakequant()."""
    rows, cols, ldx = _x2d(x)
    B = BLOCK[_fmt_arg(fmt)]
    if cols % B:
        raise ValueError("cols must be a multiple of %d" % B)
    if out is not None:
        codes, scales, y = out
        _packed_u8(codes, rows, cols // 2, x.device, "codes")
        _packed_u8(scales, rows, cols // B, x.device, "scales")
    else:
        codes = torch.empty((rows, cols // 2), dtype=torch.uint8, device=x.device)
        scales = torch.empty((rows, cols // B), dtype=torch.uint8, device=x.device)
        y = torch.empty((rows, cols), dtype=torch.bfloat16, device=x.device)
    ldy = _out2d(y, rows, cols, torch.bfloat16, x.device, "y")
    g, ts = _gscale(fmt, x, tensor_scale, g_out)
    _require_cuda(x, 'x')
    ws = workspace(x.device)
    st = reqat_quantize_fakequant_fp4(fmt, x.data_ptr(), rows, cols, ldx, codes.data_ptr(), scales.data_ptr(),
                                      y.data_ptr(), ldy, _ptr(g), ts, ws.data_ptr(), _stream(x.device))
    _check(st, "reqat_quantize_fakequant_fp4")
    return codes, scales, y, g


def quantize_rht(x: torch.Tensor, signs: int, out=None):
    """MXFP4 codes and scales of the block-rotated rows of x (randomized Hadamard
    of 32 with the given 32-bit sign draw).  Returns (codes, scales)."""
    rows, cols, ldx = _x2d(x)
    if cols % 32:
        raise ValueError("cols must be a multiple of 32")
    if out is not None:
        codes, scales = out
        _packed_u8(codes, rows, cols // 2, x.device, "codes")
        _packed_u8(scales, rows, cols // 32, x.device, "scales")
    else:
        codes = torch.empty((rows, cols // 2), dtype=torch.uint8, device=x.device)
        scales = torch.empty((rows, cols // 32), dtype=torch.uint8, device=x.device)
    _require_cuda(x, 'x')
    st = reqat_quantize_mxfp4_rht(x.data_ptr(), rows, cols, ldx, signs & 0xFFFFFFFF, codes.data_ptr(),
                                  scales.data_ptr(), _stream(x.device))
    _check(st, "reqat_quantize_mxfp4_rht")
    return codes, scales


def fakequant_rht(x: torch.Tensor, signs: int, out=None):
    """bfloat16 quantize-dequantize of the block-rotated rows (rotated basis)."""
    rows, cols, ldx = _x2d(x)
    y = out if out is not None else torch.empty((rows, cols), dtype=torch.bfloat16, device=x.device)
    ldy = _out2d(y, rows, cols, torch.bfloat16, x.device, "out")
    _require_cuda(x, 'x')
    st = reqat_fakequant_mxfp4_rht(x.data_ptr(), rows, cols, ldx, signs & 0xFFFFFFFF, y.data_ptr(),
                                   ldy, _stream(x.device))
    _check(st, "reqat_fakequant_mxfp4_rht")
    return y


def gemm(fmt, a_codes, a_scales, a_g, b_codes, b_scales, b_g, out_dtype=torch.float32, out=None):
    """Y[M, N] = A^ B^T with FP32 accumulation; Y float32 or bfloat16."""
    B = BLOCK[_fmt_arg(fmt)]
    dev = a_codes.device
    if a_codes.dim() != 2 or b_codes.dim() != 2:
        raise ValueError("codes must be 2-D")
    M, K = a_codes.shape[0], a_codes.shape[1] * 2
    N = b_codes.shape[0]
    if b_codes.shape[1] * 2 != K:
        raise ValueError("K mismatch")
    if K % 128:
        raise ValueError("K must be a multiple of 128")
    _packed_u8(a_codes, M, K // 2, dev, "a_codes")
    _packed_u8(a_scales, M, K // B, dev, "a_scales")
    _packed_u8(b_codes, N, K // 2, dev, "b_codes")
    _packed_u8(b_scales, N, K // B, dev, "b_scales")
    _scale_arg(a_g, fmt, dev, "a_g")
    _scale_arg(b_g, fmt, dev, "b_g")
    dt = _dtype_arg(out_dtype)
    y = out if out is not None else torch.empty((M, N), dtype=out_dtype, device=dev)
    ldy = _out2d(y, M, N, out_dtype, dev, "out")
    _require_cuda(a_codes, 'a_codes')
    st = reqat_gemm_w4a4(fmt, M, N, K, a_codes.data_ptr(), a_scales.data_ptr(), _ptr(a_g),
                         b_codes.data_ptr(), b_scales.data_ptr(), _ptr(b_g), y.data_ptr(), dt,
                         ldy, _stream(dev))
    _check(st, "reqat_gemm_w4a4")
    return y


def _dtype_arg(out_dtype):
    if out_dtype == torch.float32:
        return DT_F32
    if out_dtype == torch.bfloat16:
        return DT_BF16
    raise TypeError("out_dtype must be torch.float32 or torch.bfloat16")


def _shift_ptr(shift, cols, device):
    if shift is None:
        return None, None
    if shift.dtype != torch.float32 or shift.numel() != cols or not shift.is_contiguous() \
            or shift.device != device:
        raise ValueError("shift must be a contiguous float32 tensor of cols values on the same device")
    return shift, shift.data_ptr()


def quantize_kv4(x: torch.Tensor, shift=None, tensor_scale=None, out=None, g_out=None):
    """KV4 (E1M2 + E4M3 block scales of 16 + FP32 tensor scale) of x - shift.
    Returns (codes, scales, g)."""
    rows, cols, ldx = _x2d(x)
    if cols % 16:
        raise ValueError("cols must be a multiple of 16")
    if out is not None:
        codes, scales = out
        _packed_u8(codes, rows, cols // 2, x.device, "codes")
        _packed_u8(scales, rows, cols // 16, x.device, "scales")
    else:
        codes = torch.empty((rows, cols // 2), dtype=torch.uint8, device=x.device)
        scales = torch.empty((rows, cols // 16), dtype=torch.uint8, device=x.device)
    g, ts = _gscale(NVFP4, x, tensor_scale, g_out)
    _, sp = _shift_ptr(shift, cols, x.device)
    _require_cuda(x, 'x')
    st = reqat_quantize_kv4(x.data_ptr(), rows, cols, ldx, sp, codes.data_ptr(), scales.data_ptr(), _ptr(g), ts,
                            workspace(x.device).data_ptr(), _stream(x.device))
    _check(st, "reqat_quantize_kv4")
    return codes, scales, g


def fakequant_kv4(x: torch.Tensor, shift=None, tensor_scale=None, out=None, g_out=None):
    """bfloat16 quantize-dequantize of x - shift in KV4.  Returns (y, g)."""
    rows, cols, ldx = _x2d(x)
    y = out if out is not None else torch.empty((rows, cols), dtype=torch.bfloat16, device=x.device)
    ldy = _out2d(y, rows, cols, torch.bfloat16, x.device, "out")
    g, ts = _gscale(NVFP4, x, tensor_scale, g_out)
    _, sp = _shift_ptr(shift, cols, x.device)
    _require_cuda(x, 'x')
    st = reqat_fakequant_kv4(x.data_ptr(), rows, cols, ldx, sp, y.data_ptr(), ldy, _ptr(g), ts,
                             workspace(x.device).data_ptr(), _stream(x.device))
    _check(st, "reqat_fakequant_kv4")
    return y, g


def gemm_w4a16(x: torch.Tensor, w_codes, w_scales, out_dtype=torch.float32, out=None, ws=None):
    """Y = x . W^T with x bfloat16 [M, K] and MXFP4 weights (codes [N, K/2],
    scales [N, K/32]) dequantized to bfloat16; FP32 accumulation.
    ws: optional workspace tensor of reqat_w4a16_workspace_bytes(M, N, K) bytes."""
    M, K, ldx = _x2d(x)
    if w_codes.dim() != 2:
        raise ValueError("w_codes must be 2-D")
    N = w_codes.shape[0]
    if w_codes.shape[1] * 2 != K:
        raise ValueError("K mismatch")
    if K % 128:
        raise ValueError("K must be a multiple of 128")
    _packed_u8(w_codes, N, K // 2, x.device, "w_codes")
    _packed_u8(w_scales, N, K // 32, x.device, "w_scales")
    dt = _dtype_arg(out_dtype)
    y = out if out is not None else torch.empty((M, N), dtype=out_dtype, device=x.device)
    ldy = _out2d(y, M, N, out_dtype, x.device, "out")
    nbytes = reqat_w4a16_workspace_bytes(M, N, K)
    if ws is None and nbytes:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=x.device)
    if ws is not None:
        _workspace_arg(ws, nbytes, x.device)
    _require_cuda(x, 'x')
    st = reqat_gemm_w4a16(M, N, K, x.data_ptr(), ldx, w_codes.data_ptr(), w_scales.data_ptr(), y.data_ptr(),
                          dt, ldy, _ptr(ws), _stream(x.device))
    _check(st, "reqat_gemm_w4a16")
    return y


def pack_w4a16(w_codes, w_scales, out=None):
    """Packed weight image of MXFP4 weights (codes [N, K/2], scales [N, K/32])
    for gemm_w4a16_packed: a uint8 tensor of reqat_w4a16_packed_bytes(N, K)."""
    if w_codes.dim() != 2:
        raise ValueError("w_codes must be 2-D")
    N, K = w_codes.shape[0], w_codes.shape[1] * 2
    if K % 128:
        raise ValueError("K must be a multiple of 128")
    _packed_u8(w_codes, N, K // 2, w_codes.device, "w_codes")
    _packed_u8(w_scales, N, K // 32, w_codes.device, "w_scales")
    nbytes = reqat_w4a16_packed_bytes(N, K)
    packed = out if out is not None else torch.empty(max(nbytes, 16), dtype=torch.uint8, device=w_codes.device)
    if packed.dtype != torch.uint8 or not packed.is_contiguous() or packed.numel() < nbytes \
            or packed.device != w_codes.device:
        raise ValueError("out must be a contiguous uint8 tensor of at least %d bytes on the weights' device" % nbytes)
    _require_cuda(w_codes, "w_codes")
    st = reqat_pack_w4a16(w_codes.data_ptr(), w_scales.data_ptr(), N, K, packed.data_ptr(), _stream(w_codes.device))
    _check(st, "reqat_pack_w4a16")
    return packed


def gemm_w4a16_packed(x: torch.Tensor, packed, N, out_dtype=torch.float32, out=None, ws=None):
    """gemm_w4a16 on the packed image (pack_w4a16) of N x K weights: same result, bit for bit."""
    M, K, ldx = _x2d(x)
    if K % 128:
        raise ValueError("K must be a multiple of 128")
    nbytes_w = reqat_w4a16_packed_bytes(N, K)
    if packed.dtype != torch.uint8 or not packed.is_contiguous() or packed.numel() < nbytes_w \
            or packed.device != x.device:
        raise ValueError("packed must be the contiguous uint8 image of %d bytes on x's device" % nbytes_w)
    dt = _dtype_arg(out_dtype)
    y = out if out is not None else torch.empty((M, N), dtype=out_dtype, device=x.device)
    ldy = _out2d(y, M, N, out_dtype, x.device, "out")
    nbytes = reqat_w4a16_workspace_bytes(M, N, K)
    if ws is None and nbytes:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=x.device)
    if ws is not None:
        _workspace_arg(ws, nbytes, x.device)
    _require_cuda(x, 'x')
    st = reqat_gemm_w4a16_packed(M, N, K, x.data_ptr(), ldx, packed.data_ptr(), y.data_ptr(), dt, ldy, _ptr(ws),
                                 _stream(x.device))
    _check(st, "reqat_gemm_w4a16_packed")
    return y


def linear(x: torch.Tensor, fmt, w_codes, w_scales, w_g, x_tensor_scale=None, out_dtype=torch.bfloat16,
           out=None, g_out=None, ws=None):
    """Y = quantize(x) . W^T for already-quantized weights.  Returns (Y, g_x).
    ws: optional workspace tensor of reqat_linear_workspace_bytes(fmt, M, K) bytes."""
    M, K, ldx = _x2d(x)
    B = BLOCK[_fmt_arg(fmt)]
    if w_codes.dim() != 2:
        raise ValueError("w_codes must be 2-D")
    N = w_codes.shape[0]
    if w_codes.shape[1] * 2 != K:
        raise ValueError("K mismatch")
    if K % 128:
        raise ValueError("K must be a multiple of 128")
    _packed_u8(w_codes, N, K // 2, x.device, "w_codes")
    _packed_u8(w_scales, N, K // B, x.device, "w_scales")
    _scale_arg(w_g, fmt, x.device, "w_g")
    dt = _dtype_arg(out_dtype)
    y = out if out is not None else torch.empty((M, N), dtype=out_dtype, device=x.device)
    ldy = _out2d(y, M, N, out_dtype, x.device, "out")
    g, ts = _gscale(fmt, x, x_tensor_scale, g_out)
    nbytes = reqat_linear_workspace_bytes(fmt, M, K)
    if ws is None:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=x.device)
    _workspace_arg(ws, nbytes, x.device)
    _require_cuda(x, 'x')
    st = reqat_linear_w4a4(fmt, M, N, K, x.data_ptr(), ldx, _ptr(g), ts, w_codes.data_ptr(),
                           w_scales.data_ptr(), _ptr(w_g), y.data_ptr(), dt, ldy, ws.data_ptr(),
                           _stream(x.device))
    _check(st, "reqat_linear_w4a4")
    return y, g


def pack_w4a4(w_codes, w_scales, fmt, out=None):
    """Packed decode image of W4A4 weights (codes [N, K/2], scales [N, K/B]) for
    gemm_packed / linear_packed: a uint8 tensor of reqat_w4a4_packed_bytes(fmt, N, K)."""
    B = BLOCK[_fmt_arg(fmt)]
    if w_codes.dim() != 2:
        raise ValueError("w_codes must be 2-D")
    N, K = w_codes.shape[0], w_codes.shape[1] * 2
    if K % 128:
        raise ValueError("K must be a multiple of 128")
    _packed_u8(w_codes, N, K // 2, w_codes.device, "w_codes")
    _packed_u8(w_scales, N, K // B, w_codes.device, "w_scales")
    nbytes = reqat_w4a4_packed_bytes(fmt, N, K)
    packed = out if out is not None else torch.empty(max(nbytes, 16), dtype=torch.uint8, device=w_codes.device)
    _packed_image_arg(packed, nbytes, w_codes.device, "out")
    _require_cuda(w_codes, "w_codes")
    st = reqat_pack_w4a4(fmt, w_codes.data_ptr(), w_scales.data_ptr(), N, K, packed.data_ptr(),
                         _stream(w_codes.device))
    _check(st, "reqat_pack_w4a4")
    return packed


def _packed_image_arg(packed, nbytes, device, name):
    if not isinstance(packed, torch.Tensor) or packed.dtype != torch.uint8 or not packed.is_contiguous() \
            or packed.numel() < nbytes or packed.device != device:
        raise ValueError("%s must be a contiguous uint8 tensor of at least %d bytes on %s" % (name, nbytes, device))


def gemm_packed(fmt, a_codes, a_scales, a_g, packed, N, b_g, out_dtype=torch.float32, out=None):
    """gemm() for M <= 64 on the packed image (pack_w4a4) of N x K weights: same result, bit for bit."""
    B = BLOCK[_fmt_arg(fmt)]
    dev = a_codes.device
    if a_codes.dim() != 2:
        raise ValueError("codes must be 2-D")
    M, K = a_codes.shape[0], a_codes.shape[1] * 2
    if K % 128:
        raise ValueError("K must be a multiple of 128")
    if M > 64:
        raise ValueError("the packed image serves products with M <= 64")
    _packed_u8(a_codes, M, K // 2, dev, "a_codes")
    _packed_u8(a_scales, M, K // B, dev, "a_scales")
    _packed_image_arg(packed, reqat_w4a4_packed_bytes(fmt, N, K), dev, "packed")
    _scale_arg(a_g, fmt, dev, "a_g")
    _scale_arg(b_g, fmt, dev, "b_g")
    dt = _dtype_arg(out_dtype)
    y = out if out is not None else torch.empty((M, N), dtype=out_dtype, device=dev)
    ldy = _out2d(y, M, N, out_dtype, dev, "out")
    _require_cuda(a_codes, 'a_codes')
    st = reqat_gemm_w4a4_packed(fmt, M, N, K, a_codes.data_ptr(), a_scales.data_ptr(), _ptr(a_g), packed.data_ptr(),
                                _ptr(b_g), y.data_ptr(), dt, ldy, _stream(dev))
    _check(st, "reqat_gemm_w4a4_packed")
    return y


def linear_packed(x: torch.Tensor, fmt, packed, N, w_g, x_tensor_scale=None, out_dtype=torch.bfloat16,
                  out=None, g_out=None, ws=None):
    """linear() for M <= 64 on the packed image (pack_w4a4) of N x K weights.  Returns (Y, g_x)."""
    M, K, ldx = _x2d(x)
    _fmt_arg(fmt)
    if K % 128:
        raise ValueError("K must be a multiple of 128")
    if M > 64:
        raise ValueError("the packed image serves products with M <= 64")
    _packed_image_arg(packed, reqat_w4a4_packed_bytes(fmt, N, K), x.device, "packed")
    _scale_arg(w_g, fmt, x.device, "w_g")
    dt = _dtype_arg(out_dtype)
    y = out if out is not None else torch.empty((M, N), dtype=out_dtype, device=x.device)
    ldy = _out2d(y, M, N, out_dtype, x.device, "out")
    g, ts = _gscale(fmt, x, x_tensor_scale, g_out)
    nbytes = reqat_linear_workspace_bytes(fmt, M, K)
    if ws is None:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=x.device)
    _workspace_arg(ws, nbytes, x.device)
    _require_cuda(x, 'x')
    st = reqat_linear_w4a4_packed(fmt, M, N, K, x.data_ptr(), ldx, _ptr(g), ts, packed.data_ptr(), _ptr(w_g),
                                  y.data_ptr(), dt, ldy, ws.data_ptr(), _stream(x.device))
    _check(st, "reqat_linear_w4a4_packed")
    return y, g


def linear_workspace_views(ws: torch.Tensor, fmt, M: int, K: int):
    """(codes [M, K/2], scales [M, K/B]) views of the activation codes and scales
    that linear() leaves in its workspace: [4096 partial maxima | codes | scales | ...],
    each part on a 256-byte boundary."""
    B = BLOCK[_fmt_arg(fmt)]
    r256 = lambda n: (n + 255) // 256 * 256
    off = r256(4 * 4096)
    off2 = off + r256(M * (K // 2))
    codes = ws[off:off + M * (K // 2)].view(M, K // 2)
    scales = ws[off2:off2 + M * (K // B)].view(M, K // B)
    return codes, scales


# ------------------------------------------------------------------ QAT training side

def sem_loss(logits: torch.Tensor, targets: torch.Tensor, lam: float, eps: float = 1e-6):
    """SEM loss of bfloat16 logits [T, V] and int32 targets [T].  Returns
    (loss[4] = L, mean NLL, mean w H, tau; stats [T, 4]; weights [T])."""
    T, V, ld = _x2d(logits)
    if targets.dtype != torch.int32 or targets.numel() != T or not targets.is_contiguous():
        raise TypeError("targets must be a contiguous int32 tensor of T entries")
    stats = torch.empty((T, 4), dtype=torch.float32, device=logits.device)
    weights = torch.empty(T, dtype=torch.float32, device=logits.device)
    loss = torch.zeros(4, dtype=torch.float32, device=logits.device)
    _require_cuda(logits, 'logits')
    st = reqat_sem_loss(logits.data_ptr(), T, V, ld, targets.data_ptr(), lam, eps, stats.data_ptr(),
                        weights.data_ptr(), loss.data_ptr(), _stream(logits.device))
    _check(st, "reqat_sem_loss")
    return loss, stats, weights


def sem_loss_backward(logits, targets, stats, weights, lam: float, scale: float = 1.0, out_dtype=torch.bfloat16,
                      out=None):
    """dL/dlogits (weights held fixed) as out_dtype [T, V]."""
    T, V, ld = _x2d(logits)
    dt = _dtype_arg(out_dtype)
    if targets.dtype != torch.int32 or targets.numel() != T or not targets.is_contiguous():
        raise TypeError("targets must be a contiguous int32 tensor of T entries")
    for name, t, n in (("stats", stats, 4 * T), ("weights", weights, T)):
        if t.dtype != torch.float32 or t.numel() != n or not t.is_contiguous():
            raise TypeError("%s must be a contiguous float32 tensor of %d entries" % (name, n))
        _same_device(t, logits.device, name)
    g = out if out is not None else torch.empty((T, V), dtype=out_dtype, device=logits.device)
    ldg = _out2d(g, T, V, out_dtype, logits.device, "out")
    _require_cuda(logits, 'logits')
    st = reqat_sem_loss_backward(logits.data_ptr(), T, V, ld, targets.data_ptr(), stats.data_ptr(),
                                 weights.data_ptr(), lam, scale, g.data_ptr(), dt, ldg,
                                 _stream(logits.device))
    _check(st, "reqat_sem_loss_backward")
    return g


class FakeQuantSTE(torch.autograd.Function):
    """QAT forward = fake-quant (bfloat16 in, bfloat16 out); backward = the
    straight-through estimator.  Under the ceil scale rules no element clips,
    so the estimator is the identity on the incoming gradient."""

    @staticmethod
    def forward(ctx, x, fmt=NVFP4):
        y, _ = fakequant(x.contiguous(), fmt)
        return y

    @staticmethod
    def backward(ctx, gy):
        return gy, None


class SemLoss(torch.autograd.Function):
    """The SEM loss as an autograd function over bfloat16 logits."""

    @staticmethod
    def forward(ctx, logits, targets, lam, eps=1e-6):
        loss, stats, weights = sem_loss(logits, targets, lam, eps)
        ctx.save_for_backward(logits, targets, stats, weights)
        ctx.lam = lam
        return loss[0]

    @staticmethod
    def backward(ctx, g):
        logits, targets, stats, weights = ctx.saved_tensors
        grad = sem_loss_backward(logits, targets, stats, weights, ctx.lam, scale=float(g), out_dtype=logits.dtype)
        return grad, None, None, None
