"""Seeded synthetic inputs for the microscaled-FP4 linear layer.

This module draws random bfloat16 matrices and nothing else: it holds none of
the quantization or GEMM arithmetic, so both the GPU path and the CPU oracle
can be fed from it without sharing any of the method's code.

The shapes stand in for the linear layers of the distilled Qwen-family
reasoning models the paper quantizes (R1-Qwen 1.5B/7B/14B/32B; the main model
R1-Qwen-14B has hidden size 5120 and MLP width 13824), and the value
distributions follow its description of activations: Gaussian bulk with a
small number of extreme outlier channels, and heavy tails for the MLP
down-projection input (App. C.2, Fig. mxfp4_activation).  Weights are
Gaussian with standard deviation 0.02.

Recipe (every workload):
  rng = numpy Generator(PCG64(seed)), seed = 20260000 + 10 * config + stream,
  stream 0 = X, 1 = W, 2 = outlier channel indices.  Values are sampled in
  float32 (Student-t in float64 chunks), outlier channels (chosen without
  replacement) are multiplied by 20, and the result is rounded once to
  bfloat16 (round to nearest even, via torch).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

NVFP4 = "nvfp4"
MXFP4 = "mxfp4"


@dataclass(frozen=True)
class Workload:
    index: int          # 1-based workload number
    name: str
    fmt: str            # "nvfp4" | "mxfp4"
    M: int              # activation rows (tokens)
    N: int              # weight rows (output features)
    K: int              # reduction dimension
    x_dist: str         # "normal" | "normal_outliers" | "student_t"
    n_outliers: int     # outlier channels in X (multiplied by 20)
    w_std: float        # weight standard deviation
    kind: str = "w4a4"  # "w4a4" (both operands FP4) | "w4a16" (FP4 weights, bfloat16 activations)
    #                     | "sem" (loss head) | "kv4" (KV-cache keys)

    @property
    def flops(self) -> int:
        return 2 * self.M * self.N * self.K


WORKLOADS = {
    1: Workload(1, "tiny NVFP4 linear 16x256x256", NVFP4, 16, 256, 256, "normal", 0, 1.0),
    2: Workload(2, "decode NVFP4 up-proj 1.5B-like 16x8960x1536", NVFP4, 16, 8960, 1536,
                "normal_outliers", 4, 0.02),
    3: Workload(3, "prefill NVFP4 QKV 7B-like 2048x4608x3584", NVFP4, 2048, 4608, 3584,
                "normal_outliers", 36, 0.02),
    4: Workload(4, "prefill NVFP4 gate/up 14B-like 4096x27648x5120", NVFP4, 4096, 27648, 5120,
                "normal_outliers", 51, 0.02),
    5: Workload(5, "MXFP4 down-proj 32B-like 8192x5120x27648", MXFP4, 8192, 5120, 27648,
                "student_t", 0, 0.02),
    # MXFP4 W4A16 decode (weights FP4, activations bfloat16)
    6: Workload(6, "W4A16 decode MXFP4 down-proj 32B-like 16x5120x27648", MXFP4, 16, 5120, 27648,
                "student_t", 0, 0.02, "w4a16"),
    7: Workload(7, "W4A16 decode MXFP4 gate/up 14B-like 16x27648x5120", MXFP4, 16, 27648, 5120,
                "normal_outliers", 51, 0.02, "w4a16"),
    # SEM loss head of QAT: M tokens x N vocabulary logits (Qwen-family vocabulary)
    8: Workload(8, "SEM loss head 4096 tokens x 152064 vocabulary", NVFP4, 4096, 152064, 0,
                "normal", 0, 3.0, "sem"),
    # the 14B-like gate/up shape of workload 4 in MXFP4 (E8M0 scales feed the FP4 matrix cores directly)
    10: Workload(10, "MXFP4 gate/up 14B-like 4096x27648x5120", MXFP4, 4096, 27648, 5120,
                 "normal_outliers", 51, 0.02),
    # KV4 cache: post-RoPE keys of one 14B-like layer (8 KV heads x 128 channels) over a
    # 32768-token prefill, M tokens x K channels
    9: Workload(9, "KV4 keys 14B-like 32768 tokens x 1024 channels", NVFP4, 32768, 0, 1024,
                "normal_offsets", 0, 0.0, "kv4"),
}


def make_logits(w: Workload, rows: int | None = None):
    """Logits [M, N] (bfloat16, CPU) ~ N(0, w_std) and int32 targets [M], seeded."""
    M = w.M if rows is None else rows
    rng = np.random.Generator(np.random.PCG64(_seed(w.index, 0)))
    z = np.empty((M, w.N), np.float32)
    for r0 in range(0, M, 256):
        r1 = min(M, r0 + 256)
        z[r0:r1] = rng.standard_normal((r1 - r0, w.N), dtype=np.float32) * np.float32(w.w_std)
    trng = np.random.Generator(np.random.PCG64(_seed(w.index, 1)))
    t = trng.integers(0, w.N, w.M, dtype=np.int64)[:M].astype(np.int32)
    return _to_bf16(z), torch.from_numpy(t)


def make_keys(w: Workload, rows: int | None = None):
    """Keys [M, K] (bfloat16, CPU) and the channel shift [K] (float32) that a
    calibration would supply: per-channel offsets mu_c ~ N(0, 2) added to a
    N(0, 1) bulk, and mu itself as the shift.  Seeded; stream 0 = bulk,
    stream 1 = offsets."""
    M = w.M if rows is None else rows
    rng = np.random.Generator(np.random.PCG64(_seed(w.index, 0)))
    a = rng.standard_normal((M, w.K), dtype=np.float32)
    orng = np.random.Generator(np.random.PCG64(_seed(w.index, 1)))
    mu = (orng.standard_normal(w.K, dtype=np.float32) * np.float32(2.0)).astype(np.float32)
    a += mu[None, :]
    return _to_bf16(a), torch.from_numpy(mu)


def _seed(index: int, stream: int) -> int:
    return 20260000 + 10 * index + stream


def _to_bf16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)


def _student_t(rng: np.random.Generator, rows: int, cols: int, nu: float = 4.0) -> np.ndarray:
    out = np.empty((rows, cols), np.float32)
    chunk = max(1, (1 << 22) // cols)
    for r0 in range(0, rows, chunk):
        r1 = min(rows, r0 + chunk)
        out[r0:r1] = rng.standard_t(nu, size=(r1 - r0, cols))
    return out


def make_x(w: Workload, rows: int | None = None) -> torch.Tensor:
    """Activation X [M, K] as a CPU bfloat16 tensor (first `rows` rows only if given)."""
    M = w.M if rows is None else rows
    rng = np.random.Generator(np.random.PCG64(_seed(w.index, 0)))
    if w.x_dist == "student_t":
        a = _student_t(rng, M, w.K)
    else:
        a = rng.standard_normal((M, w.K), dtype=np.float32)
    if w.n_outliers:
        orng = np.random.Generator(np.random.PCG64(_seed(w.index, 2)))
        idx = orng.choice(w.K, w.n_outliers, replace=False)
        a[:, idx] *= np.float32(20.0)
    return _to_bf16(a)


def make_w(w: Workload, rows: int | None = None) -> torch.Tensor:
    """Weight W [N, K] as a CPU bfloat16 tensor (first `rows` rows only if given)."""
    N = w.N if rows is None else rows
    rng = np.random.Generator(np.random.PCG64(_seed(w.index, 1)))
    a = rng.standard_normal((N, w.K), dtype=np.float32)
    a *= np.float32(w.w_std)
    return _to_bf16(a)


def random_bf16(rows: int, cols: int, seed: int, std: float = 1.0, dist: str = "normal") -> torch.Tensor:
    """Generic seeded bfloat16 matrix for tests (normal or Student-t)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if dist == "student_t":
        a = _student_t(rng, rows, cols)
    else:
        a = rng.standard_normal((rows, cols), dtype=np.float32)
    a *= np.float32(std)
    return _to_bf16(a)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """The uint16 bit patterns of a CPU bfloat16 tensor (zero-copy view)."""
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def from_bits(bits: np.ndarray) -> torch.Tensor:
    """A CPU bfloat16 tensor with the given uint16 bit patterns."""
    return torch.from_numpy(np.ascontiguousarray(bits, np.uint16).view(np.int16)).view(torch.bfloat16)
