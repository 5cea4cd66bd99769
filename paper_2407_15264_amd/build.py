"""Build the gfx950 HIP library (liblsmgnn.so) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB_PATH = os.path.join(PKG, "liblsmgnn.so")
SOURCES = [os.path.join(PKG, "csrc", f) for f in ("gather_kernels.hip", "runtime.hip", "pagerank.hip", "sampler.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# packed-FP32 instructions are disabled: the library's only float math is the
# float64 static-score pass, and the option keeps the compiler from ever
# emitting them.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(PKG, "csrc")]


def build_hip(verbose: bool = False) -> str:
    tmp = LIB_PATH + ".tmp"
    cmd = [HIPCC, *FLAGS, *SOURCES, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + r.stdout + r.stderr)
    if verbose:
        print(" ".join(cmd))
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build_hip(verbose=True))
