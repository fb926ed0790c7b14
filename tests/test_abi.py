"""The C-ABI library loads, exports every symbol include/reqat.h declares, and
rejects bad arguments on the host before any HIP call (CPU only: no call here
reaches a kernel launch)."""
import os
import re
import subprocess

import pytest

from paper_2606_15682_amd import reqat

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "reqat.h")

NV, MX = reqat.NVFP4, reqat.MXFP4
P = 1 << 20          # a 16-byte aligned, never dereferenced fake pointer value
OK, E_NULL, E_SHAPE, E_ALIGN, E_ENUM, E_UNSUP = 0, 1, 2, 3, 4, 5


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(reqat_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(reqat.LIB_PATH):
        pytest.skip("libreqat.so not built")
    return reqat.load()


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("reqat_quantize_fp4", "reqat_fakequant_fp4", "reqat_gemm_w4a4",
              "reqat_quantize_mxfp4_rht", "reqat_fakequant_mxfp4_rht", "reqat_gemm_w4a16",
              "reqat_quantize_kv4", "reqat_fakequant_kv4", "reqat_sem_loss", "reqat_sem_loss_backward",
              "reqat_workspace_bytes", "reqat_status_str", "reqat_abi_version"):
        assert n in names
    assert set(names) == set(reqat.SIGNATURES), "binding and header disagree"


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", reqat.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s(\S+)", out))
    for n in declared_functions():
        assert n in exported, n
        assert hasattr(lib, n)


def test_library_imports_no_allocation_copy_or_sync(lib):
    """The library launches kernels and queries the device, nothing else: it
    allocates no memory, clears and copies none, and never synchronises (so
    callers may capture its calls in a graph and own every buffer)."""
    out = subprocess.run(["nm", "-D", "--undefined-only", reqat.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    imported = {s.split("@")[0] for s in re.findall(r"\sU\s(\S+)", out)}
    hip = {s for s in imported if s.lower().startswith(("hip", "__hip", "hsa"))}
    allowed = {"hipLaunchKernel", "hipFuncSetAttribute", "hipGetDevice", "hipDeviceGetAttribute", "hipGetSymbolAddress",
               "hipGetLastError", "__hipPushCallConfiguration", "__hipPopCallConfiguration",
               "__hipRegisterFatBinary", "__hipRegisterFunction", "__hipRegisterVar", "__hipUnregisterFatBinary"}
    assert hip <= allowed, sorted(hip - allowed)
    assert "hipLaunchKernel" in hip


def test_probe_library_is_separate_and_launch_only():
    """The rate probes (bench.py context) live in their own library:
    libreqat exports none of it, and it launches kernels and nothing else."""
    from paper_2606_15682_amd import build as pbuild
    if not os.path.exists(pbuild.PROBE_LIB):
        pytest.skip("libreqat_probe.so not built")
    nm = lambda *a: subprocess.run(["nm", "-D", *a], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s(\S+)", nm("--defined-only", pbuild.PROBE_LIB)))
    product = set(re.findall(r"\sT\s(\S+)", nm("--defined-only", reqat.LIB_PATH)))
    for name in ("reqat_probe_mfma", "reqat_probe_read"):
        assert name in exported
        assert name not in product
    imported = {x.split("@")[0] for x in re.findall(r"\sU\s(\S+)", nm("--undefined-only", pbuild.PROBE_LIB))}
    hip = {x for x in imported if x.lower().startswith(("hip", "__hip", "hsa"))}
    assert hip <= {"hipLaunchKernel", "hipGetLastError", "__hipPushCallConfiguration", "__hipPopCallConfiguration",
                   "__hipRegisterFatBinary", "__hipRegisterFunction", "__hipUnregisterFatBinary"}, sorted(hip)


def test_small_queries(lib):
    assert reqat.reqat_abi_version() == 11
    assert reqat.reqat_workspace_bytes() == 4 * 4096 + 2 * (1 << 19)   # partials + segment table
    for s in range(8):
        assert reqat.reqat_status_str(s).startswith(reqat.STATUS[s])
    assert "unknown" in reqat.reqat_status_str(99)


def q(fmt=NV, x=P, rows=4, cols=64, ldx=64, codes=P, scales=P, ts_ptr=P, ts=0, ws=P):
    return reqat.reqat_quantize_fp4(fmt, x, rows, cols, ldx, codes, scales, ts_ptr, ts, ws, None)


def fq(fmt=NV, x=P, rows=4, cols=64, ldx=64, y=P, ldy=64, ts_ptr=P, ts=0, ws=P):
    return reqat.reqat_fakequant_fp4(fmt, x, rows, cols, ldx, y, ldy, ts_ptr, ts, ws, None)


def qfq(fmt=NV, x=P, rows=4, cols=64, ldx=64, codes=P, scales=P, y=P + 4096, ldy=64, ts_ptr=P, ts=0, ws=P):
    return reqat.reqat_quantize_fakequant_fp4(fmt, x, rows, cols, ldx, codes, scales, y, ldy, ts_ptr, ts, ws,
                                              None)


def gm(fmt=NV, M=4, N=8, K=128, ac=P, as_=P, ag=P, bc=P, bs=P, bg=P, y=P, dt=0, ldy=8):
    return reqat.reqat_gemm_w4a4(fmt, M, N, K, ac, as_, ag, bc, bs, bg, y, dt, ldy, None)


def test_quantize_validation(lib):
    assert q(fmt=7) == E_ENUM
    assert q(ts=5) == E_ENUM
    assert q(rows=-1) == E_SHAPE
    assert q(cols=40) == E_SHAPE                 # not a multiple of 16
    assert q(fmt=MX, cols=48, ldx=48, ts_ptr=None) == E_SHAPE   # not a multiple of 32
    assert q(ldx=32) == E_SHAPE
    assert q(fmt=MX, ts_ptr=P) == E_UNSUP        # MXFP4 has no global scale
    assert q(ts_ptr=None) == E_NULL
    assert q(ws=None) == E_NULL                  # computed g needs the workspace
    assert q(x=None) == E_NULL
    assert q(codes=None) == E_NULL
    assert q(scales=None) == E_NULL
    assert q(x=P + 2) == E_ALIGN
    assert q(codes=P + 8) == E_ALIGN
    assert q(ldx=68) == E_ALIGN
    assert q(ts_ptr=P + 2) == E_ALIGN


def test_fakequant_validation(lib):
    assert fq(fmt=3) == E_ENUM
    assert fq(cols=24, ldx=24, ldy=24) == E_SHAPE
    assert fq(ldy=32) == E_SHAPE
    assert fq(y=None) == E_NULL
    assert fq(y=P + 4) == E_ALIGN
    assert fq(ldy=68) == E_ALIGN
    assert fq(fmt=MX) == E_UNSUP


def test_fakequant_in_place_rules(lib):
    # computed NVFP4 scale: the second pass re-reads x, so y must not overlap it
    assert fq(x=P, y=P) == E_UNSUP
    # partial overlaps are never allowed
    assert fq(fmt=MX, ts_ptr=None, x=P, y=P + 64) == E_UNSUP
    assert fq(ts=1, x=P, y=P + 64) == E_UNSUP
    assert fq(ts=1, x=P, y=P, ldx=64, ldy=72) == E_UNSUP


def test_quantize_fakequant_validation(lib):
    assert qfq(fmt=9) == E_ENUM
    assert qfq(ts=3) == E_ENUM
    assert qfq(cols=40, ldx=40, ldy=40) == E_SHAPE
    assert qfq(ldx=32) == E_SHAPE
    assert qfq(ldy=32) == E_SHAPE
    assert qfq(fmt=MX) == E_UNSUP                # MXFP4 has no global scale
    assert qfq(ws=None) == E_NULL
    assert qfq(codes=None) == E_NULL
    assert qfq(scales=None) == E_NULL
    assert qfq(y=None) == E_NULL
    assert qfq(x=P + 8) == E_ALIGN
    assert qfq(y=P + 4096 + 8) == E_ALIGN
    assert qfq(ldy=68) == E_ALIGN
    # y must not overlap x, in place included
    assert qfq(y=P) == E_UNSUP
    assert qfq(fmt=MX, ts_ptr=None, y=P + 256) == E_UNSUP
    assert qfq(ts=1, y=P + 496) == E_UNSUP       # x spans 4 rows * 64 * 2 = 512 bytes


def test_rotated_quantize_validation(lib):
    qr = lambda x=P, rows=4, cols=64, ldx=64, c=P, s=P: reqat.reqat_quantize_mxfp4_rht(
        x, rows, cols, ldx, 0x12345678, c, s, None)
    fr = lambda x=P, rows=4, cols=64, ldx=64, y=P, ldy=64: reqat.reqat_fakequant_mxfp4_rht(
        x, rows, cols, ldx, 0xFFFFFFFF, y, ldy, None)
    assert qr(rows=-1) == E_SHAPE
    assert qr(cols=48, ldx=48) == E_SHAPE        # blocks of 32
    assert qr(ldx=32) == E_SHAPE
    assert qr(x=None) == E_NULL and qr(c=None) == E_NULL and qr(s=None) == E_NULL
    assert qr(x=P + 2) == E_ALIGN and qr(c=P + 8) == E_ALIGN and qr(ldx=68) == E_ALIGN
    assert qr(rows=0, x=None, c=None, s=None) == 0                   # empty: no-op
    assert fr(ldy=32) == E_SHAPE
    assert fr(y=None) == E_NULL and fr(y=P + 4) == E_ALIGN and fr(ldy=68) == E_ALIGN


def test_w4a16_validation(lib):
    g16 = lambda M=4, N=8, K=128, x=P, ldx=128, wc=P, ws=P, y=P, dt=0, ldy=8, wk=None: reqat.reqat_gemm_w4a16(
        M, N, K, x, ldx, wc, ws, y, dt, ldy, wk, None)
    # K splits (FP32 partials): the fewest that give about two workgroups per CU,
    # spread evenly (80 weight tiles of 64 rows: 6 ways, 480 workgroups; 64 tiles:
    # 8 ways, 512), else enough for 1024 workgroups (10 tiles: 12 ways, the cap)
    assert reqat.reqat_w4a16_workspace_bytes(16, 5120, 27648) == 4 * 6 * 16 * 5120
    assert reqat.reqat_w4a16_workspace_bytes(32, 4096, 8192) == 4 * 8 * 32 * 4096
    assert reqat.reqat_w4a16_workspace_bytes(16, 640, 4096) == 4 * 12 * 16 * 640
    assert reqat.reqat_w4a16_workspace_bytes(16, 27648, 5120) == 0
    assert reqat.reqat_w4a16_workspace_bytes(4, 8, 128) == 0          # a single chunk: no split
    assert reqat.reqat_w4a16_workspace_bytes(4, 8, 100) == 0
    assert g16(M=16, N=5120, K=27648, ldx=27648, ldy=5120) == E_NULL  # needs the workspace
    assert g16(dt=5) == E_ENUM
    assert g16(M=-1) == E_SHAPE and g16(K=96, ldx=96) == E_SHAPE and g16(ldx=64) == E_SHAPE
    assert g16(ldy=4) == E_SHAPE
    assert g16(M=0, x=None, wc=None, ws=None, y=None) == 0 and g16(N=0, y=None) == 0
    assert g16(y=None) == E_NULL and g16(x=None) == E_NULL and g16(wc=None) == E_NULL and g16(ws=None) == E_NULL
    assert g16(x=P + 2) == E_ALIGN and g16(ldx=132) == E_ALIGN and g16(wc=P + 8) == E_ALIGN
    assert g16(ws=P + 2) == E_ALIGN and g16(ws=P + 1) == E_ALIGN
    assert g16(y=P + 2) == E_ALIGN and g16(y=P + 1, dt=1) == E_ALIGN


def test_w4a16_packed_validation(lib):
    """Packed weight image: size 1088 bytes per (16-row group, 128-element
    chunk), host-side argument checks of the pack and of the packed product."""
    assert reqat.reqat_w4a16_packed_bytes(5120, 27648) == 320 * 216 * 1088
    assert reqat.reqat_w4a16_packed_bytes(17, 256) == 2 * 2 * 1088        # a partial last group is padded
    assert reqat.reqat_w4a16_packed_bytes(16, 100) == 0 and reqat.reqat_w4a16_packed_bytes(-1, 128) == 0
    assert reqat.reqat_w4a16_packed_bytes(0, 128) == 0 and reqat.reqat_w4a16_packed_bytes(16, 0) == 0
    pk = lambda wc=P, ws=P, N=8, K=128, out=P: reqat.reqat_pack_w4a16(wc, ws, N, K, out, None)
    assert pk(K=96) == E_SHAPE and pk(N=-1) == E_SHAPE
    assert pk(N=0, wc=None, ws=None, out=None) == 0 and pk(K=0, wc=None, ws=None, out=None) == 0
    assert pk(wc=None) == E_NULL and pk(ws=None) == E_NULL and pk(out=None) == E_NULL
    assert pk(wc=P + 8) == E_ALIGN and pk(ws=P + 2) == E_ALIGN and pk(out=P + 4) == E_ALIGN
    # the image must not overlap the weights (8 x 128: 512 code bytes, 32 scale bytes, a 1088-byte image)
    far = P + (1 << 20)
    assert pk(wc=P, ws=far, out=P + 256) == E_UNSUP and pk(wc=far, ws=P + 1024, out=P) == E_UNSUP
    gp = lambda M=4, N=8, K=128, x=P, ldx=128, w=P, y=P, dt=0, ldy=8, wk=None: reqat.reqat_gemm_w4a16_packed(
        M, N, K, x, ldx, w, y, dt, ldy, wk, None)
    assert gp(M=16, N=5120, K=27648, ldx=27648, ldy=5120) == E_NULL  # needs the workspace
    assert gp(dt=5) == E_ENUM
    assert gp(M=-1) == E_SHAPE and gp(K=96, ldx=96) == E_SHAPE and gp(ldx=64) == E_SHAPE and gp(ldy=4) == E_SHAPE
    assert gp(M=0, x=None, w=None, y=None) == 0 and gp(N=0, y=None) == 0
    assert gp(y=None) == E_NULL and gp(x=None) == E_NULL and gp(w=None) == E_NULL
    assert gp(x=P + 2) == E_ALIGN and gp(ldx=132) == E_ALIGN and gp(w=P + 8) == E_ALIGN
    assert gp(y=P + 2) == E_ALIGN and gp(y=P + 1, dt=1) == E_ALIGN


def test_binding_w4a16_packed_checks(trapped):
    x5 = torch.zeros(16, 512, dtype=torch.bfloat16)
    mc, ms = _u8(5120, 256), _u8(5120, 16)
    nb = reqat.reqat_w4a16_packed_bytes(5120, 512)
    with pytest.raises(TypeError, match="CUDA"):
        reqat.pack_w4a16(mc, ms, out=_u8(nb))
    _raises_before_device(lambda: reqat.pack_w4a16(mc, ms, out=_u8(nb - 1)), match="out")
    _raises_before_device(lambda: reqat.pack_w4a16(mc, _u8(5120, 8)), match="w_scales")
    _raises_before_device(lambda: reqat.pack_w4a16(_u8(5120, 48), _u8(5120, 3)), match="multiple of 128")
    need16 = reqat.reqat_w4a16_workspace_bytes(16, 5120, 512)
    with pytest.raises(TypeError, match="CUDA"):
        reqat.gemm_w4a16_packed(x5, _u8(nb), 5120, ws=_u8(need16))
    _raises_before_device(lambda: reqat.gemm_w4a16_packed(x5, _u8(nb - 16), 5120), match="packed")
    _raises_before_device(lambda: reqat.gemm_w4a16_packed(x5, _u8(nb), 5120, ws=_u8(need16 - 4)), match="ws")
    _raises_before_device(lambda: reqat.gemm_w4a16_packed(x5, _u8(nb), 5120,
                                                          out=torch.zeros(16, 5120, dtype=torch.bfloat16)),
                          match="out")


def test_w4a4_packed_validation(lib):
    """Packed decode image: 2048 code bytes and 16 S scale bytes (S = 16 NVFP4,
    8 MXFP4) per (16-row group, 256-element chunk); host-side argument checks of
    the pack and of the packed product and linear layer (none reaches a launch)."""
    nb = lambda N, K, fmt=NV: reqat.reqat_w4a4_packed_bytes(fmt, N, K)
    assert nb(8960, 1536) == 560 * 6 * 2304 and nb(8960, 1536, MX) == 560 * 6 * 2176
    assert nb(17, 384) == 2 * 2 * 2304                  # partial last group, half last chunk: padded
    assert nb(16, 100) == 0 and nb(-1, 128) == 0 and nb(0, 128) == 0 and nb(16, 0) == 0 and nb(16, 128, 7) == 0
    pk = lambda fmt=NV, wc=P, ws=P, N=8, K=128, out=P: reqat.reqat_pack_w4a4(fmt, wc, ws, N, K, out, None)
    assert pk(fmt=7) == E_ENUM
    assert pk(K=96) == E_SHAPE and pk(N=-1) == E_SHAPE
    assert pk(N=0, wc=None, ws=None, out=None) == 0 and pk(K=0, wc=None, ws=None, out=None) == 0
    assert pk(wc=None) == E_NULL and pk(ws=None) == E_NULL and pk(out=None) == E_NULL
    assert pk(wc=P + 8) == E_ALIGN and pk(ws=P + 8) == E_ALIGN and pk(out=P + 4) == E_ALIGN
    # the image must not overlap the weights (NVFP4 8 x 128: 512 code bytes, 64 scale bytes, a 2304-byte image)
    far = P + (1 << 20)
    assert pk(wc=P, ws=far, out=P + 256) == E_UNSUP and pk(wc=far, ws=P + 1024, out=P) == E_UNSUP
    gp = lambda fmt=NV, M=4, N=8, K=128, a=P, sa=P, ag=P, w=P, bg=P, y=P, dt=0, ldy=8: \
        reqat.reqat_gemm_w4a4_packed(fmt, M, N, K, a, sa, ag, w, bg, y, dt, ldy, None)
    assert gp(fmt=7) == E_ENUM and gp(dt=5) == E_ENUM
    assert gp(M=-1) == E_SHAPE and gp(K=96) == E_SHAPE and gp(ldy=4) == E_SHAPE
    assert gp(M=65) == E_UNSUP and gp(fmt=MX) == E_UNSUP and gp(ag=None) == E_NULL and gp(bg=None) == E_NULL
    assert gp(M=0, a=None, sa=None, w=None, y=None) == 0 and gp(N=0, y=None) == 0
    assert gp(y=None) == E_NULL and gp(a=None) == E_NULL and gp(sa=None) == E_NULL and gp(w=None) == E_NULL
    assert gp(a=P + 8) == E_ALIGN and gp(sa=P + 8) == E_ALIGN and gp(w=P + 8) == E_ALIGN
    assert gp(y=P + 2) == E_ALIGN and gp(y=P + 1, dt=1) == E_ALIGN and gp(ag=P + 2) == E_ALIGN
    lp = lambda fmt=NV, M=4, N=8, K=128, x=P, ldx=128, xg=P, ts=1, w=P, wg=P, y=P, dt=0, ldy=8, wk=P: \
        reqat.reqat_linear_w4a4_packed(fmt, M, N, K, x, ldx, xg, ts, w, wg, y, dt, ldy, wk, None)
    assert lp(fmt=7) == E_ENUM and lp(ts=5) == E_ENUM and lp(dt=5) == E_ENUM
    assert lp(K=96, ldx=96) == E_SHAPE and lp(ldx=64) == E_SHAPE
    assert lp(M=65) == E_UNSUP and lp(fmt=MX) == E_UNSUP
    assert lp(wk=None) == E_NULL and lp(w=None) == E_NULL and lp(x=None) == E_NULL and lp(wg=None) == E_NULL
    assert lp(wk=P + 16) == E_ALIGN and lp(w=P + 8) == E_ALIGN and lp(x=P + 2) == E_ALIGN
    assert lp(M=0, x=None, w=None, y=None) == 0          # a given g: nothing to write, nothing launched


def test_binding_w4a4_packed_checks(trapped):
    mc, ms = _u8(8960, 768), _u8(8960, 96)
    nb = reqat.reqat_w4a4_packed_bytes(NV, 8960, 1536)
    with pytest.raises(TypeError, match="CUDA"):
        reqat.pack_w4a4(mc, ms, NV, out=_u8(nb))
    _raises_before_device(lambda: reqat.pack_w4a4(mc, ms, NV, out=_u8(nb - 1)), match="out")
    _raises_before_device(lambda: reqat.pack_w4a4(mc, _u8(8960, 48), NV), match="w_scales")
    _raises_before_device(lambda: reqat.pack_w4a4(mc, ms, 7), match="format")
    _raises_before_device(lambda: reqat.pack_w4a4(_u8(8960, 48), _u8(8960, 6), NV), match="multiple of 128")
    g = torch.ones(1, dtype=torch.float32)
    a, sa = _u8(16, 768), _u8(16, 96)
    with pytest.raises(TypeError, match="CUDA"):
        reqat.gemm_packed(NV, a, sa, g, _u8(nb), 8960, g.clone())
    _raises_before_device(lambda: reqat.gemm_packed(NV, a, sa, g, _u8(nb - 16), 8960, g.clone()), match="packed")
    _raises_before_device(lambda: reqat.gemm_packed(NV, _u8(65, 768), _u8(65, 96), g, _u8(nb), 8960, g.clone()),
                          match="M <= 64")
    _raises_before_device(lambda: reqat.gemm_packed(NV, a, _u8(16, 48), g, _u8(nb), 8960, g.clone()),
                          match="a_scales")
    _raises_before_device(lambda: reqat.gemm_packed(NV, a, sa, g, _u8(nb), 8960, g.clone(),
                                                    out=torch.zeros(16, 8960, dtype=torch.bfloat16)), match="out")
    x = torch.zeros(16, 1536, dtype=torch.bfloat16)
    ws = _u8(reqat.reqat_linear_workspace_bytes(NV, 16, 1536))
    with pytest.raises(TypeError, match="CUDA"):
        reqat.linear_packed(x, NV, _u8(nb), 8960, g, ws=ws)
    _raises_before_device(lambda: reqat.linear_packed(x, NV, _u8(nb - 16), 8960, g, ws=ws), match="packed")
    _raises_before_device(lambda: reqat.linear_packed(torch.zeros(65, 1536, dtype=torch.bfloat16), NV, _u8(nb),
                                                      8960, g, ws=ws), match="M <= 64")
    _raises_before_device(lambda: reqat.linear_packed(x, NV, _u8(nb), 8960, g, ws=ws[:-1]), match="ws")


def test_kv4_validation(lib):
    kq = lambda x=P, rows=4, cols=64, ldx=64, sh=None, c=P, s=P, ts_ptr=P, ts=0, ws=P: reqat.reqat_quantize_kv4(
        x, rows, cols, ldx, sh, c, s, ts_ptr, ts, ws, None)
    kf = lambda y=P, ldy=64, sh=P, ts=1: reqat.reqat_fakequant_kv4(P, 4, 64, 64, sh, y, ldy, P, ts, None, None)
    assert kq(ts=3) == E_ENUM
    assert kq(cols=40, ldx=40) == E_SHAPE and kq(ldx=32) == E_SHAPE
    assert kq(ts_ptr=None) == E_NULL and kq(ws=None) == E_NULL and kq(c=None) == E_NULL
    assert kq(sh=P + 4) == E_ALIGN and kq(x=P + 2) == E_ALIGN and kq(ldx=68) == E_ALIGN
    assert kf(ldy=32) == E_SHAPE and kf(y=None) == E_NULL and kf(sh=P + 8) == E_ALIGN
    # in place (y is x) only with a given g: a computed g's fix-up re-reads x
    kfw = lambda y=P, ts=0: reqat.reqat_fakequant_kv4(P, 4, 64, 64, None, y, 64, P, ts, P + 65536, None)
    assert kfw(y=P, ts=0) == E_UNSUP and kfw(y=P + 64, ts=1) == E_UNSUP


def test_sem_validation(lib):
    sl = lambda T=4, V=64, ld=64, lg=P, tg=P, st=P, w=P, loss=P: reqat.reqat_sem_loss(
        lg, T, V, ld, tg, 0.1, 1e-6, st, w, loss, None)
    sb = lambda T=4, V=64, ld=64, g=P, dt=1, ldg=64: reqat.reqat_sem_loss_backward(
        P, T, V, ld, P, P, P, 0.1, 1.0, g, dt, ldg, None)
    assert sl(T=-1) == E_SHAPE and sl(V=60, ld=60) == E_SHAPE and sl(ld=32) == E_SHAPE and sl(V=0) == E_SHAPE
    assert sl(loss=None) == E_NULL and sl(lg=None) == E_NULL and sl(tg=None) == E_NULL
    assert sl(lg=P + 2) == E_ALIGN and sl(ld=68) == E_ALIGN and sl(st=P + 2) == E_ALIGN
    assert sl(T=0, lg=None, tg=None, st=None, w=None) == 0
    assert sb(dt=7) == E_ENUM and sb(ldg=32) == E_SHAPE and sb(g=None) == E_NULL
    assert sb(g=P + 4) == E_ALIGN and sb(ldg=68) == E_ALIGN and sb(dt=0, ldg=66) == E_ALIGN


def test_gemm_validation(lib):
    assert gm(fmt=2) == E_ENUM
    assert gm(dt=9) == E_ENUM
    assert gm(M=-1) == E_SHAPE
    assert gm(K=64) == E_SHAPE                   # K % 128
    assert gm(ldy=4) == E_SHAPE
    assert gm(fmt=MX) == E_UNSUP                 # MXFP4 with tensor scales
    assert gm(ag=None) == E_NULL
    assert gm(y=None) == E_NULL
    assert gm(ac=None) == E_NULL
    assert gm(ac=P + 1) == E_ALIGN
    assert gm(y=P + 2) == E_ALIGN               # float32 output needs 4-byte alignment
    assert gm(y=P + 1, dt=1) == E_ALIGN         # bf16 output needs 2-byte alignment


def ln(fmt=NV, M=4, N=8, K=128, x=P, ldx=128, xg=P, ts=0, wc=P, ws_=P, wg=P, y=P, dt=0, ldy=8, ws=P):
    return reqat.reqat_linear_w4a4(fmt, M, N, K, x, ldx, xg, ts, wc, ws_, wg, y, dt, ldy, ws, None)


def test_linear_workspace_bytes(lib):
    # partials (1024 words) | codes M*K/2 | scales M*K/B, each rounded up to 256 bytes
    # NVFP4: partials, codes, scales, then one uint16 per 64 blocks of segment table
    assert reqat.reqat_linear_workspace_bytes(NV, 4, 128) == 16384 + 256 + 256 + 256
    assert reqat.reqat_linear_workspace_bytes(NV, 2048, 3584) == 16384 + 3670016 + 458752 + 7168 * 2
    assert reqat.reqat_linear_workspace_bytes(MX, 300, 1024) == 16384 + 153600 + 9728
    assert reqat.reqat_linear_workspace_bytes(NV, 4, 64) == 0      # K % 128
    assert reqat.reqat_linear_workspace_bytes(NV, -1, 128) == 0
    assert reqat.reqat_linear_workspace_bytes(7, 4, 128) == 0


def test_linear_validation(lib):
    assert ln(fmt=2) == E_ENUM
    assert ln(dt=9) == E_ENUM
    assert ln(ts=5) == E_ENUM
    assert ln(M=-1) == E_SHAPE
    assert ln(K=64, ldx=64) == E_SHAPE            # K % 128
    assert ln(ldx=64) == E_SHAPE                  # ldx < K
    assert ln(ldy=4) == E_SHAPE
    assert ln(fmt=MX) == E_UNSUP                  # MXFP4 with tensor scales
    assert ln(xg=None) == E_NULL
    assert ln(wg=None) == E_NULL
    assert ln(ws=None) == E_NULL
    assert ln(ws=P + 16) == E_ALIGN               # workspace 256-byte aligned
    assert ln(x=None) == E_NULL
    assert ln(y=None) == E_NULL
    assert ln(wc=None) == E_NULL
    assert ln(x=P + 2) == E_ALIGN
    assert ln(ldx=132) == E_ALIGN                 # ldx % 8
    assert ln(wc=P + 8) == E_ALIGN
    assert ln(y=P + 2) == E_ALIGN
    assert ln(xg=P + 2) == E_ALIGN
    # nothing to do: N == 0 with M > 0 enqueues nothing and returns OK
    assert ln(N=0, x=None, y=None) == OK


def test_binding_raises_when_library_missing(tmp_path):
    saved = reqat._lib
    reqat._lib = None
    try:
        with pytest.raises(RuntimeError, match="not built"):
            reqat.load(str(tmp_path / "missing.so"))
    finally:
        reqat._lib = saved


# ------------------------------------------------- binding-side buffer checks
# The C ABI takes no buffer sizes, so the torch binding is where an output,
# operand or workspace of the wrong shape, dtype or size is caught.  Every C
# entry point is replaced by a trap here: each bad call must raise before any
# of them is reached, and a well-formed call on CPU tensors gets as far as the
# final device check.

import torch  # noqa: E402


@pytest.fixture
def trapped(lib, monkeypatch):
    def trap(*a, **k):
        raise AssertionError("a C entry point was reached")
    for name in reqat.SIGNATURES:
        if name.endswith("_bytes") or name in ("reqat_status_str", "reqat_abi_version"):
            continue
        monkeypatch.setattr(reqat, name, trap)
    return reqat


def _u8(*shape):
    return torch.zeros(shape, dtype=torch.uint8)


def _gemm_args(fmt, M=8, N=16, K=256):
    B = reqat.BLOCK[fmt]
    g = torch.ones(1, dtype=torch.float32) if fmt == NV else None
    return [fmt, _u8(M, K // 2), _u8(M, K // B), g, _u8(N, K // 2), _u8(N, K // B),
            None if g is None else g.clone()]


def _raises_before_device(fn, exc=(ValueError, TypeError), match=None):
    with pytest.raises(exc) as ei:
        fn()
    assert "CUDA" not in str(ei.value), "the bad argument was not caught: %s" % ei.value
    if match:
        assert match in str(ei.value), str(ei.value)


@pytest.mark.parametrize("fmt", [NV, MX])
def test_binding_gemm_checks_operands_and_output(trapped, fmt):
    a = _gemm_args(fmt)
    with pytest.raises(TypeError, match="CUDA"):                    # well formed: only the device is wrong
        reqat.gemm(*a, out_dtype=torch.float32)
    # bfloat16 buffer for a float32 product (would be written 4 bytes per element)
    _raises_before_device(lambda: reqat.gemm(*a, out_dtype=torch.float32,
                                             out=torch.zeros(8, 16, dtype=torch.bfloat16)), match="out")
    _raises_before_device(lambda: reqat.gemm(*a, out=torch.zeros(8, 15)), match="out")
    _raises_before_device(lambda: reqat.gemm(*a, out_dtype=torch.float16))
    # the other format's scale layout (NVFP4 reads K/16 bytes per row)
    b = list(a)
    other = reqat.BLOCK[MX if fmt == NV else NV]
    b[2] = _u8(8, 256 // other)
    _raises_before_device(lambda: reqat.gemm(*b), match="a_scales")
    c = list(a)
    c[4] = _u8(16, 256)[:, ::2]                                        # strided codes rows
    _raises_before_device(lambda: reqat.gemm(*c), match="b_codes")
    d = list(a)
    d[3] = torch.ones(1, dtype=torch.float32) if fmt == MX else None   # a global scale where none is (not) allowed
    _raises_before_device(lambda: reqat.gemm(*d), match="a_g")
    e = list(a)
    e[1] = _u8(8, 64)                                                   # K = 128 against b's 256
    _raises_before_device(lambda: reqat.gemm(*e), match="K")


def test_binding_quantize_and_fakequant_check_outputs(trapped):
    x = torch.zeros(4, 64, dtype=torch.bfloat16)
    with pytest.raises(TypeError, match="CUDA"):
        reqat.quantize(x, NV, out=(_u8(4, 32), _u8(4, 4)))
    _raises_before_device(lambda: reqat.quantize(x, NV, out=(_u8(4, 32), _u8(4, 2))), match="scales")
    _raises_before_device(lambda: reqat.quantize(x, MX, out=(_u8(4, 16), _u8(4, 2))), match="codes")
    _raises_before_device(lambda: reqat.quantize(torch.zeros(4, 40, dtype=torch.bfloat16), MX))
    _raises_before_device(lambda: reqat.fakequant(x, NV, out=torch.zeros(4, 64)), match="out")
    _raises_before_device(lambda: reqat.fakequant(x, NV, out=torch.zeros(4, 32, dtype=torch.bfloat16)))
    _raises_before_device(lambda: reqat.quantize_fakequant(
        x, NV, out=(_u8(4, 32), _u8(4, 4), torch.zeros(4, 64, dtype=torch.float16))), match="y")
    _raises_before_device(lambda: reqat.quantize_rht(x, 1, out=(_u8(4, 32), _u8(4, 4))), match="scales")
    _raises_before_device(lambda: reqat.quantize(x, NV, g_out=torch.zeros(1, dtype=torch.float64)),
                          match="g_out")
    _raises_before_device(lambda: reqat.quantize(x, MX, tensor_scale=torch.ones(1)), match="MXFP4")


def test_binding_checks_workspace_sizes(trapped):
    x = torch.zeros(16, 256, dtype=torch.bfloat16)
    wc, ws_ = _u8(32, 128), _u8(32, 16)
    g = torch.ones(1, dtype=torch.float32)
    need = reqat.reqat_linear_workspace_bytes(NV, 16, 256)
    with pytest.raises(TypeError, match="CUDA"):
        reqat.linear(x, NV, wc, ws_, g, ws=_u8(need))
    _raises_before_device(lambda: reqat.linear(x, NV, wc, ws_, g, ws=_u8(need - 1)), match="ws")
    _raises_before_device(lambda: reqat.linear(x, NV, wc, ws_, g, ws=torch.zeros(need)), match="ws")
    _raises_before_device(lambda: reqat.linear(x, NV, wc, _u8(32, 8), g), match="w_scales")
    x5 = torch.zeros(16, 512, dtype=torch.bfloat16)
    mc, ms = _u8(5120, 256), _u8(5120, 16)
    need16 = reqat.reqat_w4a16_workspace_bytes(16, 5120, 512)      # K split in two (one pair of chunks each)
    assert need16 == 4 * 2 * 16 * 5120
    assert reqat.reqat_w4a16_workspace_bytes(16, 5120, 256) == 0     # a single pair of chunks: no split
    _raises_before_device(lambda: reqat.gemm_w4a16(x5, mc, ms, ws=_u8(need16 - 4)), match="ws")
    _raises_before_device(lambda: reqat.gemm_w4a16(x5, mc, _u8(5120, 32)), match="w_scales")
    _raises_before_device(lambda: reqat.gemm_w4a16(x5, mc, ms, out=torch.zeros(16, 5120, dtype=torch.bfloat16)),
                          match="out")


def lnn(fmt=NV, M=4, N=8, K=128, x=P, ldx=128, xg=P, ts=0, wc=P, ws_=P, wg=P, y=P, dt=0, ldy=8):
    return reqat.reqat_linear_w4a4_noalloc(fmt, M, N, K, x, ldx, xg, ts, wc, ws_, wg, y, dt, ldy, None)


def test_linear_noalloc_validation(lib):
    """The no-allocation linear call validates like reqat_linear_w4a4 and refuses
    inputs whose workspace would exceed its fixed scratch, before any HIP call."""
    assert lnn(fmt=2) == E_ENUM
    assert lnn(dt=9) == E_ENUM
    assert lnn(M=-1) == E_SHAPE
    assert lnn(K=64, ldx=64) == E_SHAPE
    assert lnn(fmt=MX) == E_UNSUP
    assert lnn(xg=None) == E_NULL
    assert lnn(x=None) == E_NULL
    assert lnn(x=P + 2) == E_ALIGN
    cap = reqat.NOALLOC_SCRATCH_BYTES
    for fmt, g in ((NV, P), (MX, None)):
        K = 5120
        M = 1
        while reqat.reqat_linear_workspace_bytes(fmt, M + 1, K) <= cap:
            M += 1
        assert reqat.reqat_linear_workspace_bytes(fmt, M, K) <= cap
        assert lnn(fmt=fmt, M=M + 1, K=K, ldx=K, xg=g, wg=g) == 7           # REQAT_E_TOO_LARGE
        assert lnn(fmt=fmt, M=1 << 20, K=K, ldx=K, xg=g, wg=g) == 7
    assert "no-allocation" in reqat.reqat_status_str(7)
