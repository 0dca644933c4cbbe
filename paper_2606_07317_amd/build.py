"""Build libgbla.so (the HIP kernels and the C ABI) in-tree for gfx950."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libgbla.so")
SOURCES = [os.path.join(CSRC, "gbla_kernels.hip"), os.path.join(CSRC, "gbla_stream.hip"),
           os.path.join(CSRC, "gbla_state128.hip"),
           os.path.join(CSRC, "gbla_backward.hip"), os.path.join(CSRC, "gbla_layer.hip"),
           os.path.join(CSRC, "gbla_plan.cpp"), os.path.join(CSRC, "gbla_ext_plan.cpp"),
           os.path.join(CSRC, "gbla_api.cpp"), os.path.join(CSRC, "gbla_ceiling.hip"),
           os.path.join(CSRC, "gbla_noalloc.hip")]

# Packed fp32 VALU ops are switched off for all device code; hipcc's host
# pass warns that it does not know the feature, which is harmless.
HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build(out: str = LIB, extra_flags=(), verbose: bool = False) -> str:
    """Compile every source into one shared library; always rebuilds."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *HIPCC_FLAGS, *extra_flags, "-I", INCLUDE, "-I", CSRC, *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed to build %s" % out)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
