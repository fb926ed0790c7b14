"""The rate probes that bench.py reports as context (libreqat_probe.so, not
the product path) do the work they claim: the matrix-core loop runs its
MFMAs (on all-ones operands every accumulator element gains K per
instruction), and the read stream reads every word once (the XOR of its
per-thread folds is the XOR of the buffer)."""
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


@pytest.mark.parametrize("nbytes,blocks", [(1 << 20, 64), (16 * 1000003, 256), (16, 4)])
def test_read_probe_reads_every_word(nbytes, blocks):
    import numpy as np
    lib = ctypes.CDLL(pbuild.PROBE_LIB)
    lib.reqat_probe_read.restype = ctypes.c_int
    lib.reqat_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    dev = torch.device("cuda:0")
    words = np.random.default_rng(nbytes).integers(0, 2 ** 32, nbytes // 4, dtype=np.uint32)
    buf = torch.from_numpy(words.view(np.int32)).to(dev)
    out = torch.full((blocks * 256,), -1, dtype=torch.int32, device=dev)
    assert lib.reqat_probe_read(buf.data_ptr(), nbytes, out.data_ptr(), blocks,
                                torch.cuda.current_stream(dev).cuda_stream) == 0
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(words)
    assert lib.reqat_probe_read(buf.data_ptr(), nbytes - 4, out.data_ptr(), blocks, None) == 1   # not 16-byte whole
