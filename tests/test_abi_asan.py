"""The C ABI's host code under AddressSanitizer (CPU only): the library is rebuilt with its host
code instrumented (device code as usual) and tests/test_abi.py runs against that build in a
child process with the sanitizer runtime preloaded.  Argument validation, size queries, the
workspace layout arithmetic and the error strings must run clean."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

from paper_2609_37001_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OUT = os.path.join(ROOT, "_build", "asan")


def asan_runtime():
    cands = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    return cands[0] if cands else None


@pytest.mark.skipif(asan_runtime() is None or shutil.which(build.hipcc()) is None,
                    reason="no clang AddressSanitizer runtime in this image")
def test_abi_under_address_sanitizer():
    os.makedirs(OUT, exist_ok=True)
    lib = os.path.join(OUT, "libpsa.so")
    flags = [f for f in build.compile_flags() if f != "-O3"] + ["-O1", "-g"]
    # host code only: each sanitizer flag goes to the host compilation
    flags += "-Xarch_host -fsanitize=address -Xarch_host -fno-omit-frame-pointer".split()
    cmd = [build.hipcc()] + flags + ["-shared"] + [os.path.join(build.CSRC, s) for s in build.SOURCES] + ["-o", lib]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    env = dict(os.environ, LD_PRELOAD=asan_runtime(), ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               PSA_LIBRARY=lib)
    run = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_abi.py")],
                         capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)
    out = run.stdout + run.stderr
    assert "AddressSanitizer" not in out, out[-4000:]
    assert run.returncode == 0, out[-4000:]
    assert " passed" in out
