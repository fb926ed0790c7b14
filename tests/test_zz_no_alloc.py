"""GPU: the no-allocation linear entry point (fixed per-device scratch) against
reqat_linear_w4a4 with a caller workspace, through the C ABI: bit-identical
outputs and global scales on two calls in a row, the second with a smaller
input, for both formats (computed and given activation scales), plus the
refusal of an input beyond the scratch."""
import numpy as np
import pytest
import torch

from paper_2606_15682_amd import reqat
from paper_2606_15682_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _weights(fmt, N, K, seed):
    g = torch.Generator().manual_seed(seed)
    w = (torch.randn((N, K), generator=g) * 0.02).to(torch.bfloat16).to(DEV)
    wc, ws, wg = reqat.quantize(w, fmt)
    return wc, ws, wg


def _acts(M, K, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((M, K), generator=g)
    x[:, ::97] *= 20.0
    return x.to(torch.bfloat16).to(DEV)


def _run(noalloc, fmt, x, wc, ws, wg, N, dt, given):
    M, K = x.shape
    y = torch.full((M, N), float("nan"), dtype=dt, device=DEV)
    if fmt == reqat.NVFP4:
        xg = torch.tensor([0.0625], dtype=torch.float32, device=DEV) if given else \
            torch.full((1,), -1.0, dtype=torch.float32, device=DEV)
        ts = reqat.TS_GIVEN if given else reqat.TS_COMPUTE
    else:
        xg, ts = None, reqat.TS_COMPUTE
    ydt = reqat.DT_F32 if dt == torch.float32 else reqat.DT_BF16
    stream = torch.cuda.current_stream().cuda_stream
    ptr = lambda t: None if t is None else t.data_ptr()
    if noalloc:
        st = reqat.reqat_linear_w4a4_noalloc(fmt, M, N, K, x.data_ptr(), x.stride(0), ptr(xg), ts, wc.data_ptr(),
                                             ws.data_ptr(), ptr(wg), y.data_ptr(), ydt, y.stride(0), stream)
    else:
        wsp = torch.empty(reqat.reqat_linear_workspace_bytes(fmt, M, K), dtype=torch.uint8, device=DEV)
        st = reqat.reqat_linear_w4a4(fmt, M, N, K, x.data_ptr(), x.stride(0), ptr(xg), ts, wc.data_ptr(),
                                     ws.data_ptr(), ptr(wg), y.data_ptr(), ydt, y.stride(0), wsp.data_ptr(), stream)
    assert st == 0, reqat.STATUS.get(st, st)
    torch.cuda.synchronize()
    return y.cpu(), (None if xg is None else float(xg.cpu()[0]))


@pytest.mark.parametrize("fmt", [reqat.NVFP4, reqat.MXFP4])
@pytest.mark.parametrize("given", [False, True])
def test_noalloc_linear_matches_workspace_linear(fmt, given):
    if fmt == reqat.MXFP4 and given:
        pytest.skip("MXFP4 has no activation global scale")
    N, K = 1536, 5120
    wc, ws, wg = _weights(fmt, N, K, 3)
    # first a prefill-sized call (2048 x 5120: 5.9 MB of the 8 MB scratch), then a smaller decode-sized one
    for M, seed, dt in ((2048, 11, torch.float32), (16, 12, torch.bfloat16), (300, 13, torch.float32)):
        print("noalloc linear fmt=%d given=%s M=%d" % (fmt, given, M), flush=True)
        x = _acts(M, K, seed)
        y0, g0 = _run(False, fmt, x, wc, ws, wg, N, dt, given)
        y1, g1 = _run(True, fmt, x, wc, ws, wg, N, dt, given)
        assert not torch.isnan(y0).any()
        assert torch.equal(y0.view(torch.int16) if dt == torch.bfloat16 else y0.view(torch.int32),
                           y1.view(torch.int16) if dt == torch.bfloat16 else y1.view(torch.int32))
        assert g0 == g1


def test_noalloc_linear_refuses_beyond_scratch():
    fmt, K, N = reqat.NVFP4, 5120, 256
    M = 4096                                           # 11.8 MB of workspace > 8 MB
    assert reqat.reqat_linear_workspace_bytes(fmt, M, K) > reqat.NOALLOC_SCRATCH_BYTES
    x = _acts(M, K, 5)
    wc, ws, wg = _weights(fmt, N, K, 6)
    y = torch.zeros((M, N), dtype=torch.float32, device=DEV)
    xg = torch.zeros(1, dtype=torch.float32, device=DEV)
    st = reqat.reqat_linear_w4a4_noalloc(fmt, M, N, K, x.data_ptr(), K, xg.data_ptr(), reqat.TS_COMPUTE,
                                         wc.data_ptr(), ws.data_ptr(), wg.data_ptr(), y.data_ptr(), reqat.DT_F32,
                                         N, torch.cuda.current_stream().cuda_stream)
    assert st == 7
    torch.cuda.synchronize()
    assert torch.all(y == 0).item() and float(xg.cpu()[0]) == 0.0      # nothing was enqueued
