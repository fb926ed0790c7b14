"""CPU builds under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU):
the oracle, driven through every entry point on inputs with special values,
and the C ABI's host-side argument validation, driven through every rejection
path before any HIP call.  Sanitizers apply to host code only (each hipcc
-fsanitize flag is preceded by -Xarch_host; device code is never instrumented)."""
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
SAN_ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, "%s\n%s%s" % (" ".join(cmd), r.stdout[-3000:], r.stderr[-3000:])
    return r


def test_oracle_under_asan_ubsan(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_driver")
    _run(["gcc", "-O1", "-g", "-std=c99", "-ffp-contract=off", "-fsanitize=address,undefined",
          "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", os.path.join(HERE, "oracle_driver.c"),
          os.path.join(ROOT, "oracle", "reqat_oracle.c"), "-lm", "-o", exe])
    r = _run([exe], env=SAN_ENV)
    assert "oracle driver ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr


def test_abi_validation_under_asan_ubsan(tmp_path):
    hipcc = "/opt/rocm/bin/hipcc"
    clang = "/opt/rocm/llvm/bin/clang"
    if not (os.path.exists(hipcc) and os.path.exists(clang)):
        pytest.skip("ROCm compilers not found")
    from paper_2606_15682_amd import build as libbuild
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = [f for f in libbuild.HIPCC_FLAGS if f not in ("-shared", "-O3")] + ["-O1", "-g"] + san
    objs = [str(tmp_path / (s[:-4] + ".o")) for s in libbuild.SOURCES]
    jobs = [[hipcc, *flags, "-c", os.path.join(libbuild.CSRC, s), "-o", o] for s, o in zip(libbuild.SOURCES, objs)]
    with ThreadPoolExecutor(min(8, len(jobs))) as ex:
        list(ex.map(_run, jobs))
    lib = str(tmp_path / "libreqat_san.so")
    _run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *san, "-o", lib, *objs])
    exe = str(tmp_path / "abi_driver")
    _run([clang, "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          os.path.join(HERE, "abi_driver.c"), lib, "-Wl,-rpath," + str(tmp_path),
          "-Wl,-rpath,/opt/rocm/lib", "-o", exe])
    r = _run([exe], env=SAN_ENV)
    assert "abi driver ok" in r.stdout, r.stdout
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr, r.stderr[-3000:]
