"""Build the native libraries in-tree.

* ``libapex.so``       every entry point of include/apex.h: HIP kernels for gfx950 plus
                       the host code around them (hipcc).
* ``libapex_plan.so``  the host-only part (cache plan, expert packing, errors), built
                       with g++ so that it loads and runs on machines without a GPU.

Usage: ``python -m paper_2608_11688_amd.build`` (or ``__graft_entry__.build()``).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libapex.so")
PLAN_LIB = os.path.join(PKG, "libapex_plan.so")

HIP_SOURCES = ["errors.cpp", "residency.cpp", "pack_fp8.cpp", "pack_mxfp4.cpp", "pack_fp32.cpp",
               "decode.cpp", "route_gate.hip", "moe_ffn.cpp", "ffn_b1.hip", "ffn_b1_e4m3.hip",
               "ffn_b1_mxfp4.hip", "ffn_b1_fp32.hip", "ffn_gemm.hip", "ffn_noalloc.hip",
               "attention.hip", "prefetch.hip", "util.hip"]
HOST_SOURCES = ["errors.cpp", "residency.cpp", "pack_fp8.cpp", "pack_mxfp4.cpp", "pack_fp32.cpp"]

HIPCC_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
               # keep the compiler from forming packed fp32 instructions
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               # load the first kernel arguments into SGPRs at dispatch (gfx950 kernarg
               # preload; the code object keeps a fallback that loads them itself), so a
               # kernel's prologue does not wait on several rounds of argument loads
               "-mllvm", "-amdgpu-kernarg-preload-count=16",
               "-Wall", "-Wno-unused-result"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout)
        raise RuntimeError(f"build failed: {' '.join(cmd[:3])} ... (exit {r.returncode})")
    return r.stdout


def _hipcc():
    return os.environ.get("HIPCC") or shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


def build_hip(verbose=False):
    hipcc = _hipcc()
    with tempfile.TemporaryDirectory(dir=PKG, prefix="_build") as tmp:
        objs, procs = [], []
        for src in HIP_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            lang = ["-x", "hip"] if src.endswith(".hip") else []
            cmd = [hipcc, *HIPCC_FLAGS, "-I", INCLUDE, "-I", CSRC, *lang, "-c",
                   os.path.join(CSRC, src), "-o", obj]
            procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                stderr=subprocess.STDOUT, text=True)))
            objs.append(obj)
        failed = []
        for cmd, p in procs:
            out, _ = p.communicate()
            if verbose and out:
                sys.stderr.write(out)
            if p.returncode != 0:
                sys.stderr.write(out)
                failed.append(cmd[-3])
        if failed:
            raise RuntimeError(f"hipcc failed on {failed}")
        tmp_lib = LIB + ".tmp"
        _run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp_lib])
        os.replace(tmp_lib, LIB)
    return LIB


def build_plan():
    cxx = shutil.which("g++") or "g++"
    tmp_lib = PLAN_LIB + ".tmp"
    _run([cxx, "-O2", "-std=c++17", "-fPIC", "-shared", "-Wall", "-D__HIP_PLATFORM_AMD__",
          "-I", INCLUDE, "-I", CSRC, "-I", "/opt/rocm/include",
          *[os.path.join(CSRC, s) for s in HOST_SOURCES], "-o", tmp_lib])
    os.replace(tmp_lib, PLAN_LIB)
    return PLAN_LIB


def build(verbose=False):
    build_plan()
    build_hip(verbose)


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(LIB)
    print(PLAN_LIB)
