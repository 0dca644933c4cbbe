"""Build libgbla.so (the HIP kernels and the C ABI) in-tree for gfx950."""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libgbla.so")
SOURCES = [os.path.join(CSRC, "gbla_kernels.hip"), os.path.join(CSRC, "gbla_stream.hip"),
           os.path.join(CSRC, "gbla_state64.hip"), os.path.join(CSRC, "gbla_state128.hip"),
           os.path.join(CSRC, "gbla_backward.hip"), os.path.join(CSRC, "gbla_layer.hip"),
           os.path.join(CSRC, "gbla_plan.cpp"), os.path.join(CSRC, "gbla_ext_plan.cpp"),
           os.path.join(CSRC, "gbla_api.cpp"), os.path.join(CSRC, "gbla_ceiling.hip"),
           os.path.join(CSRC, "gbla_noalloc.hip")]

# Packed fp32 VALU ops are switched off for all device code; hipcc's host
# pass warns that it does not know the feature, which is harmless.
HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(" ".join(cmd) + "\n" + res.stdout + res.stderr)
        raise RuntimeError("hipcc failed: %s" % cmd[-1])
    return res


def build(out: str = LIB, extra_flags=(), verbose: bool = False, jobs: int = 0) -> str:
    """Compile every source (in parallel, one object each) and link one shared
    library; always rebuilds."""
    tmpdir = tempfile.mkdtemp(prefix="gbla_build_")
    try:
        objs, cmds = [], []
        for src in SOURCES:
            obj = os.path.join(tmpdir, os.path.basename(src) + ".o")
            objs.append(obj)
            cmds.append([hipcc(), *HIPCC_FLAGS, *extra_flags, "-I", INCLUDE, "-I", CSRC, "-c", src,
                         "-o", obj])
        if verbose:
            for c in cmds:
                print(" ".join(c), flush=True)
        workers = jobs or min(len(cmds), max(1, (os.cpu_count() or 2)))
        with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as pool:
            list(pool.map(_run, cmds))
        tmp = out + ".tmp%d" % os.getpid()
        _run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
        os.replace(tmp, out)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
