"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

Two builds, both with ``-fsanitize=address,undefined -fno-sanitize-recover``:

* the library's host side (shape validation, plans, workspace layouts and the
  argument checks of every C entry point; ``gbla_plan.cpp``,
  ``gbla_ext_plan.cpp``, ``gbla_api.cpp``) linked into
  ``tests/sanitize/host_plans.cpp``, a driver that stubs out the kernel
  launchers and walks the edge shapes: head_dim 32/64/128 and invalid ones,
  every conv width, the largest dense extents, empty and one-token ragged
  batches, fp32 inputs, each flag, and the layer shapes;
* the fp64 oracle, on which the pin suites run in a child process with the
  ASan runtime preloaded.

A planted heap overrun in a copy of the oracle checks that the sanitizer is
armed (a run that reported nothing would otherwise prove nothing).
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_07317_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
ENV_SAN = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0", "UBSAN_OPTIONS": "print_stacktrace=1"}


def _libasan():
    if shutil.which("gcc") is None or shutil.which("g++") is None:
        return None
    p = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


LIBASAN = _libasan()
pytestmark = pytest.mark.skipif(LIBASAN is None, reason="gcc with libasan is not installed")


def _env(**extra):
    env = dict(os.environ)
    env.update(ENV_SAN)
    env.update(extra)
    return env


def test_host_plans_and_entry_checks_are_clean(tmp_path):
    exe = str(tmp_path / "host_plans")
    subprocess.run(
        ["g++", "-std=c++17", "-g", "-O1", *SAN, "-D__HIP_PLATFORM_AMD__",
         "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
         os.path.join(ROOT, "tests", "sanitize", "host_plans.cpp"),
         os.path.join(CSRC, "gbla_plan.cpp"), os.path.join(CSRC, "gbla_ext_plan.cpp"),
         os.path.join(CSRC, "gbla_api.cpp"), "-o", exe],
        check=True)
    run = subprocess.run([exe], capture_output=True, text=True, env=_env(), timeout=300)
    assert run.returncode == 0, run.stderr[-4000:]
    assert "host plans ok" in run.stdout
    assert "runtime error" not in run.stderr


def _build_oracle(src, out):
    import oracle
    # -O1 keeps the reports readable; OpenMP stays on so the threaded loops are covered too
    return oracle.build(force=True, out=out, src=src, extra_flags=["-g", "-O1", *SAN])


def test_oracle_pin_suites_under_asan_ubsan(tmp_path):
    lib = _build_oracle(os.path.join(ROOT, "oracle", "gbla_oracle.c"), str(tmp_path / "liboracle_san.so"))
    tests = [os.path.join(ROOT, "tests", t) for t in
             ("test_oracle_pins.py", "test_backward_oracle.py", "test_layer_oracle.py", "test_inputs.py")]
    run = subprocess.run(
        [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu", *tests],
        capture_output=True, text=True, cwd=ROOT, timeout=900,
        env=_env(GBLA_ORACLE_LIB=lib, LD_PRELOAD=LIBASAN))
    out = run.stdout + run.stderr
    assert run.returncode == 0, out[-4000:]
    assert "passed" in run.stdout
    assert "AddressSanitizer" not in out and "runtime error" not in out


def test_sanitizer_reports_a_planted_overrun(tmp_path):
    text = open(os.path.join(ROOT, "oracle", "gbla_oracle.c")).read()
    old = "for (int64_t j = 0; j < L; ++j) g[j] /= denom;"
    assert text.count(old) == 1
    src = tmp_path / "overrun.c"
    src.write_text(text.replace(old, "for (int64_t j = 0; j <= L; ++j) g[j] /= denom;"))
    lib = _build_oracle(str(src), str(tmp_path / "liboracle_overrun.so"))
    code = ("import oracle\n"
            "from paper_2606_07317_amd import inputs as gin\n"
            "w = gin.WORKLOADS['tiny_f32'].with_(heads=1, seqlen=8)\n"
            "oracle.load().forward_inputs(gin.make_inputs(w))\n")
    run = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, cwd=ROOT,
                         timeout=300, env=_env(GBLA_ORACLE_LIB=lib, LD_PRELOAD=LIBASAN))
    assert run.returncode != 0
    assert "heap-buffer-overflow" in run.stderr
