"""Builds libctc.so (the C ABI of include/ctc.h) for gfx950 with hipcc.

Every HIP source is compiled with packed-FP32 instruction selection turned
off; the host runtime and the kernels link into one shared library that
stays in this directory (no install step).
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SO = os.path.join(HERE, "libctc.so")
SOURCES = [os.path.join(HERE, "csrc", "ctc_api.cpp"),
           os.path.join(HERE, "csrc", "kernels.hip")]
ARCH = "gfx950"


def hipcc():
    p = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    return p if os.path.exists(p) else "hipcc"


def build(verbose=False):
    tmp = "%s.tmp%d" % (SO, os.getpid())
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-mcode-object-version=5",
           "-O3", "-std=c++17", "-fPIC",
           "-shared", "-Wall", "-Wno-unused-function",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-o", tmp] + SOURCES
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines()
            if "packed-fp32-ops" not in ln]
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs))
    os.replace(tmp, SO)
    return SO


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(SO)
