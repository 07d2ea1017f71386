"""Build libpsa.so (HIP, gfx950) in-tree with hipcc.

Usage: python -m paper_2609_37001_amd.build [-v]
"""
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libpsa.so")
SOURCES = ("psa_api.hip", "psa_kernels.hip")
ARCH = "gfx950"


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def compile_flags():
    return ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
            # keep hipcc from forming packed fp32 VALU instructions
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            # MFMA accumulators in VGPRs: the per-wave state fits in 256 VGPRs, and the AGPR form
            # makes the allocator shuttle softmax inputs between register files
            "-mllvm", "-amdgpu-mfma-vgpr-form=1",
            "-Wno-unused-result", "-I", INCLUDE, "-I", CSRC]


def build(verbose=False):
    """Compile every HIP source into paper_2609_37001_amd/libpsa.so; returns the path."""
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc()] + compile_flags() + ["-shared"] + [os.path.join(CSRC, s) for s in SOURCES] + ["-o", tmp]
    if verbose:
        print(" ".join(cmd))
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(line for line in (res.stdout + res.stderr).splitlines()
                     if "packed-fp32-ops" not in line)
    if res.returncode != 0:
        if os.path.exists(tmp):
            os.remove(tmp)
        raise RuntimeError("hipcc failed:\n" + msgs)
    if verbose and msgs.strip():
        print(msgs)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
