"""Compiles the HIP library libbigcn.so in place for gfx950."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libbigcn.so")
SOURCES = [os.path.join(HERE, "csrc", f)
           for f in ("bigcn_kernels.hip", "bigcn_api.hip", "bigcn_backward.hip")]

# -packed-fp32-ops keeps the compiler from emitting packed fp32 VALU ops in
# the device code.  hipcc hands -Xclang options to the host pass as well,
# where the x86 back end prints that it does not know the feature and
# ignores it; the driver cannot forward a -Xclang pair to the device pass
# alone (-Xarch_device takes options without arguments), and a per-function
# target attribute would keep header device functions from inlining.
HIPCC_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
               "-Wall", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-I", os.path.join(ROOT, "include")]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc()] + HIPCC_FLAGS + SOURCES + ["-o", tmp]
    if verbose:
        print(" ".join(cmd))
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + res.stdout + res.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
