"""The matrix-core rate probe that bench.py reports as context
(libreqat_probe.so, not the product path) runs the MFMAs it claims: on
all-ones operands every accumulator element gains K per instruction."""
import ctypes

import pytest
import torch

from paper_2606_15682_amd import build as pbuild

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kind,byte_pattern,k", [(0, 0x22, 64),        # E2M1 1.0 in both nibbles, K = 64
                                                 (1, 0x3C00, 16)])      # FP16 1.0, K = 16
def test_probe_counts_its_mfmas(kind, byte_pattern, k):
    lib = ctypes.CDLL(pbuild.PROBE_LIB)
    lib.reqat_probe_mfma.restype = ctypes.c_int
    lib.reqat_probe_mfma.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                     ctypes.c_void_p]
    dev = torch.device("cuda:0")
    if kind == 0:
        ops = torch.full((8192,), byte_pattern, dtype=torch.uint8, device=dev)
    else:
        ops = torch.full((4096,), byte_pattern, dtype=torch.int16, device=dev).view(torch.uint8)
    blocks, iters = 8, 10
    out = torch.full((blocks * 256,), float("nan"), dtype=torch.float32, device=dev)
    rc = lib.reqat_probe_mfma(kind, ops.data_ptr(), out.data_ptr(), blocks, iters,
                              torch.cuda.current_stream(dev).cuda_stream)
    assert rc == 0
    torch.cuda.synchronize()
    # each lane sums its 16 accumulators x 16 registers, each iters * k
    assert torch.all(out == 16 * 16 * iters * k), out[:4]
    assert lib.reqat_probe_mfma(2, ops.data_ptr(), out.data_ptr(), blocks, iters, None) == 1
