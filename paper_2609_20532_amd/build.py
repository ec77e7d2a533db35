"""Build the gfx950 HIP library ``libdpsgd.so`` and the CPU verifier library
``libdpsgd_verifier.so`` in-tree.

Usage: ``python -m paper_2609_20532_amd.build`` (or ``build()`` from Python).
Every HIP source is compiled for gfx950 only. Packed fp32 instructions are
switched off for the device code (``-packed-fp32-ops``): the compiler would
otherwise fuse pairs of float operations into ``v_pk_*_f32`` forms. The
verifier is plain host C++ (g++, x86-64-v3), with no GPU runtime.
"""

from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libdpsgd.so")
VERIFIER_LIB = os.path.join(PKG, "libdpsgd_verifier.so")
VERIFIER_SOURCES = ["verifier.cpp"]
OBJ_DIR = os.path.join(PKG, "_build")
SOURCES = ["api.hip", "noise.hip", "norms.hip", "ghost.hip", "gram32.hip", "gemm.hip", "gemm_tr.hip", "gemm_wide.hip",
           "skinny.hip"]
ARCH = "gfx950"


def hipcc_path() -> str:
    p = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(p):
        raise RuntimeError("hipcc not found; the ROCm toolchain is required to build libdpsgd")
    return p


def common_flags() -> list[str]:
    return [
        f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wno-unused-command-line-argument",
        "-I", INCLUDE, "-I", CSRC,
    ]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(OBJ_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc_path(), *common_flags(), "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(line for line in res.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in line)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{out}")
    if verbose and out.strip():
        print(out)
    return obj


def build_verifier(verbose: bool = False) -> str:
    """Compile the host-only verifier into ``libdpsgd_verifier.so``."""
    cxx = shutil.which("g++") or shutil.which("c++")
    if not cxx:
        raise RuntimeError("no C++ compiler found for the verifier library")
    tmp = VERIFIER_LIB + ".tmp"
    cmd = [cxx, "-O3", "-march=x86-64-v3", "-std=c++17", "-fPIC", "-shared", "-pthread",
           "-Wall", "-Wextra", "-I", INCLUDE,
           *[os.path.join(CSRC, s) for s in VERIFIER_SOURCES], "-o", tmp]
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"verifier build failed:\n{res.stdout}")
    if verbose and res.stdout.strip():
        print(res.stdout)
    os.replace(tmp, VERIFIER_LIB)
    return VERIFIER_LIB


def build(verbose: bool = False) -> str:
    """Compile every HIP source and link ``libdpsgd.so`` (and build the verifier
    library); returns the path of ``libdpsgd.so``."""
    os.makedirs(OBJ_DIR, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES) + 1) as ex:
        ver = ex.submit(build_verifier, verbose)
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
        ver.result()
    tmp = LIB + ".tmp"
    cmd = [hipcc_path(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    path = build(verbose="-v" in sys.argv)
    print(path)
