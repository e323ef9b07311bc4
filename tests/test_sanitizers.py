"""The library's host code and the C oracle under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU (no GPU): tests/sanitize/host_check.cpp
drives the host-side C ABI (descriptor checks, packing, folding, planning for
many layer shapes, stack validation) against a build of libifq whose host code
is instrumented (device code is built as usual); tests/sanitize/oracle_check.c
drives every oracle entry point. Any sanitizer report fails the test."""
import os
import shutil
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1911_08076_amd", "csrc")
HERE = os.path.join(ROOT, "tests", "sanitize")
HIPCC = "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang++"

ENV = dict(os.environ, UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
           OMP_NUM_THREADS="2")


def _sources():
    import sys
    sys.path.insert(0, ROOT)
    from paper_1911_08076_amd.build import SOURCES
    return SOURCES


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    return r.returncode, r.stdout + r.stderr


def _clean(out):
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]


@pytest.mark.skipif(not shutil.which("gcc"), reason="gcc not found")
def test_oracle_under_asan_ubsan():
    with tempfile.TemporaryDirectory() as tmp:
        exe = os.path.join(tmp, "oracle_check")
        rc, out = _run(["gcc", "-O1", "-g", "-fsanitize=address,undefined",
                        "-fno-omit-frame-pointer", "-fopenmp", "-o", exe,
                        os.path.join(HERE, "oracle_check.c"),
                        os.path.join(ROOT, "oracle", "ifq_oracle.c"), "-lm"])
        assert rc == 0, out
        rc, out = _run([exe], env=dict(ENV, ASAN_OPTIONS="detect_leaks=1"))
        _clean(out)
        assert rc == 0 and "oracle checks passed" in out, out


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)),
                    reason="ROCm toolchain not found")
def test_library_host_code_under_asan_ubsan():
    # device code is compiled as in the product build; only the host side of
    # every translation unit is instrumented
    flags = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
             "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include"), "-I", CSRC,
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-omit-frame-pointer"]
    with tempfile.TemporaryDirectory() as tmp:
        srcs = [os.path.join(CSRC, s) for s in _sources()] + [os.path.join(HERE, "host_check.cpp")]

        def one(src):
            obj = os.path.join(tmp, os.path.splitext(os.path.basename(src))[0] + ".o")
            rc, out = _run(flags + ["-c", src, "-o", obj])
            return obj, rc, out

        with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
            built = list(ex.map(one, srcs))
        for obj, rc, out in built:
            assert rc == 0, out
        exe = os.path.join(tmp, "host_check")
        rc, out = _run([CLANG, "-fsanitize=address,undefined", "-o", exe] +
                       [b[0] for b in built] +
                       ["-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"])
        assert rc == 0, out
        # the HIP runtime keeps allocations to the end of the process
        rc, out = _run([exe], env=dict(ENV, ASAN_OPTIONS="detect_leaks=0"))
        _clean(out)
        assert rc == 0 and "host checks passed" in out, out
