"""Build libreqat.so (HIP, gfx950) in-tree with hipcc, and libreqat_probe.so,
the matrix-core rate probe that bench.py reports as context (not the product).

    python -m paper_2606_15682_amd.build          # or: python paper_2606_15682_amd/build.py
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libreqat.so")
SOURCES = ["api.hip", "quantize.hip", "gemm.hip", "gemm_skinny.hip", "gemm_tile256.hip", "gemm_w4a16.hip", "kv4.hip", "sem.hip"]
PROBE_LIB = os.path.join(HERE, "libreqat_probe.so")
PROBE_SOURCE = "probe_mfma.hip"

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-ffp-contract=off",
    # no packed-FP32 instructions anywhere in the library
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libreqat)")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed: %s" % " ".join(cmd[-3:]))
    # keep warnings visible, minus hipcc's host-pass note about the device-only feature flag
    noise = ("packed-fp32-ops", "is not a recognized feature")
    for line in (res.stdout + res.stderr).splitlines():
        if line.strip() and not any(n in line for n in noise):
            sys.stderr.write(line + "\n")


def build(verbose: bool = False) -> str:
    """Compile every HIP source (in parallel, one object each) and link LIB, and
    build PROBE_LIB; always recompiles."""
    from concurrent.futures import ThreadPoolExecutor

    cc = hipcc()
    tag = "%d" % os.getpid()
    objs = [os.path.join(CSRC, s[:-4] + ".%s.o" % tag) for s in SOURCES]
    flags = [f for f in HIPCC_FLAGS if f != "-shared"]
    jobs = [[cc, *flags, "-c", os.path.join(CSRC, s), "-o", o] for s, o in zip(SOURCES, objs)]
    tmp = LIB + ".tmp" + tag
    ptmp = PROBE_LIB + ".tmp" + tag
    jobs.append([cc, *HIPCC_FLAGS, os.path.join(CSRC, PROBE_SOURCE), "-o", ptmp])
    workers = max(1, min(len(jobs), len(os.sched_getaffinity(0)), 8))
    try:
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(lambda c: _run(c, verbose), jobs))
        _run([cc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
        os.replace(tmp, LIB)
        os.replace(ptmp, PROBE_LIB)
    finally:
        for o in objs + [tmp, ptmp]:
            if os.path.exists(o):
                os.remove(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
