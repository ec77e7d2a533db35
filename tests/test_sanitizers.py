"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Two drivers are built in a temporary directory and run:

* the trusted-side verifier (``verifier.cpp``, plain host C++), with g++
  sanitizers and leak detection, through its float32 / float64
  recomputations (ragged float32 and bfloat16 layers, several thread counts)
  and every path of the verification step;
* the GPU library's host-side planners (workspace layouts, split plans, tail
  splits, norm-form choice, argument checks) of every source, compiled with
  hipcc for gfx950 with the sanitizers on the host code only, queried over
  the benchmark workloads, WRN-16-4's convolutions, more layers than one
  launch takes, degenerate and ragged shapes. No kernel is launched.
"""

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")
CSRC = os.path.join(ROOT, "paper_2609_20532_amd", "csrc")
HERE = os.path.join(ROOT, "tests", "sanitize")
ROCM = "/opt/rocm"

sys.path.insert(0, ROOT)


def _run(cmd, env=None, timeout=600):
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                         env=env, timeout=timeout)
    assert res.returncode == 0, f"{' '.join(cmd[:3])} ... failed:\n{res.stdout[-4000:]}"
    return res.stdout


def _san_env():
    env = dict(os.environ)
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    return env


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_verifier_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "verifier_driver")
    _run(["g++", "-O1", "-g", "-std=c++17", "-pthread", "-fno-omit-frame-pointer",
          "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-I", INCLUDE,
          os.path.join(HERE, "verifier_driver.cpp"), os.path.join(CSRC, "verifier.cpp"), "-o", exe])
    env = _san_env()
    env["ASAN_OPTIONS"] = "detect_leaks=1"
    out = _run([exe], env=env)
    assert "verifier driver ok" in out


@pytest.mark.skipif(not os.path.exists(os.path.join(ROCM, "bin", "hipcc")), reason="needs hipcc")
def test_planners_under_asan_and_ubsan(tmp_path):
    from paper_2609_20532_amd import build as B
    clang = os.path.join(ROCM, "llvm", "bin", "clang++")
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-omit-frame-pointer"]

    def compile_one(src):
        obj = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
        _run([B.hipcc_path(), f"--offload-arch={B.ARCH}", "-O1", "-g", "-std=c++17",
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
              "-Wno-unused-command-line-argument", *host_san, "-I", INCLUDE, "-I", CSRC,
              "-c", os.path.join(CSRC, src), "-o", obj])
        return obj

    with ThreadPoolExecutor(max_workers=min(8, len(B.SOURCES))) as ex:
        objs = list(ex.map(compile_one, B.SOURCES))
    drv = str(tmp_path / "planner_driver.o")
    _run([clang, "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined",
          "-fno-omit-frame-pointer", "-I", INCLUDE, "-c", os.path.join(HERE, "planner_driver.cpp"),
          "-o", drv])
    exe = str(tmp_path / "planner_driver")
    _run([clang, "-fsanitize=address,undefined", drv, *objs, f"-L{ROCM}/lib", "-lamdhip64",
          f"-Wl,-rpath,{ROCM}/lib", "-o", exe])
    env = _san_env()
    env["ASAN_OPTIONS"] = "detect_leaks=0"   # the HIP runtime's own allocations
    out = _run([exe], env=env, timeout=300)
    assert "planner driver ok" in out
