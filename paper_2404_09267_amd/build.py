"""Build libtg.so in-tree: the host planner with g++, the kernels with hipcc for gfx950.

    python -m paper_2404_09267_amd.build              # the library the binding loads
    python -m paper_2404_09267_amd.build --sanitize   # host code under ASan + UBSan

Objects go to _build/ at the repository root; the shared library lands next to this
file, where the ctypes binding looks for it. With --sanitize the host-only sources
(planner, invoker, normalisation constants) are compiled with
-fsanitize=address,undefined (every undefined-behaviour report fatal) into
_build/sanitize/libtg.so; the HIP sources are built as usual (no GPU code is ever
instrumented). Load that library with GCC's ASan runtime preloaded
(tests/sanitize_host.py does).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libtg.so")
PROBE_LIB = os.path.join(PKG, "libtg_probe.so")  # the benchmark's streaming probe only
PROBE_SOURCES = ["probe.hip"]
ARCH = "gfx950"

HOST_SOURCES = ["plan.cpp", "norm.cpp", "invoker.cpp"]
HIP_SOURCES = ["stitch.hip", "unstitch.hip", "partition.hip", "merge.hip", "gmm.hip", "rois.hip",
               "upload.hip"]

# Packed FP32 instructions are kept out of every kernel; scalar code is all we need.
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE,
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wall", "-Wno-unused-command-line-argument"]
# Sources whose binary32 results decide integers (foreground flags, suppression, box
# assignment): every operation rounded on its own, no multiply-add fusion. The rounded
# intrinsics (__fmul_rn and the like) are plain operators in the clang headers, so only
# the command-line switch reaches them.
EXACT_FP32 = {"unstitch.hip", "merge.hip", "gmm.hip"}
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-I", INCLUDE, "-Wall", "-Wextra"]
SANITIZE_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                  "-fno-omit-frame-pointer", "-g"]
SANITIZE_LIB = os.path.join(BUILD, "sanitize", "libtg.so")


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found; the HIP library cannot be built")


def _run(cmd):
    print("+", " ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose_isa: bool = False, sanitize: bool = False) -> str:
    out_dir = os.path.join(BUILD, "sanitize") if sanitize else BUILD
    os.makedirs(out_dir, exist_ok=True)
    objs = []
    for src in HOST_SOURCES:
        obj = os.path.join(out_dir, src + ".o")
        _run(["g++", *HOST_FLAGS, *(SANITIZE_FLAGS if sanitize else []), "-c",
              os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    cc = hipcc()
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        if not sanitize or not os.path.exists(obj):
            extra = ["-save-temps=obj"] if verbose_isa else []
            if src in EXACT_FP32:
                extra.append("-ffp-contract=off")
            _run([cc, *HIP_FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    if sanitize:
        # the GCC sanitizer runtimes the host objects were built against
        rt = [subprocess.run(["gcc", f"-print-file-name={n}"], check=True, capture_output=True,
                             text=True).stdout.strip() for n in ("libasan.so", "libubsan.so")]
        tmp = SANITIZE_LIB + ".tmp"
        _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs, *rt])
        os.replace(tmp, SANITIZE_LIB)
        return SANITIZE_LIB
    tmp = LIB + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    probe_objs = []
    for src in PROBE_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        _run([cc, *HIP_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
        probe_objs.append(obj)
    tmp = PROBE_LIB + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *probe_objs])
    os.replace(tmp, PROBE_LIB)
    return LIB


if __name__ == "__main__":
    build(verbose_isa="--isa" in sys.argv, sanitize="--sanitize" in sys.argv)
