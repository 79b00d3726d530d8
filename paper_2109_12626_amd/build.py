"""Builds libdpar.so in place: HIP kernels for gfx950 with hipcc, host C++
with g++, linked by hipcc.  ``python -m paper_2109_12626_amd.build``."""

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libdpar.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
ARCH = "gfx950"

HIP_FLAGS = [
    "-O3", "-fPIC", "-std=c++17", f"--offload-arch={ARCH}",
    "-fno-fast-math", "-ffp-contract=off",
    # keep fp32 arithmetic on the scalar (non-packed) VALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]
HOST_FLAGS = ["-O2", "-fPIC", "-std=c++17", "-Wall", "-Wextra",
              "-Wno-unused-parameter", "-D__HIP_PLATFORM_AMD__"]


def _run(cmd):
    print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose=True, out=None, defines=(), host_sanitize=False):
    """Compiles libdpar.so (or ``out``); ``defines`` are extra -D flags for
    kernel experiments.  ``host_sanitize``: the host C++ (plan.cpp, api.cpp
    and the host side of the launches) built with AddressSanitizer and
    UndefinedBehaviorSanitizer, for CPU runs of the no-device entry points
    (needs ``out``; load it with libasan and libubsan preloaded)."""
    if host_sanitize and out is None:
        raise ValueError("a sanitized build needs its own output path")
    build_dir = BUILD if out is None else os.path.dirname(out) + "/_obj"
    os.makedirs(build_dir, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC,
           "-I", os.path.join(ROCM, "include")]
    hipcc = os.path.join(ROCM, "bin", "hipcc")
    objs = []
    san = ["-fsanitize=address,undefined", "-g"] if host_sanitize else []
    for src in ("plan.cpp", "api.cpp"):
        obj = os.path.join(build_dir, src + ".o")
        _run(["g++"] + HOST_FLAGS + san + inc +
             ["-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    obj = os.path.join(build_dir, "kernels.hip.o")
    _run([hipcc] + HIP_FLAGS + [f"-D{d}" for d in defines] + inc
         + ["-c", os.path.join(CSRC, "kernels.hip"), "-o", obj])
    objs.append(obj)
    lib = LIB if out is None else out
    tmp = lib + ".tmp"
    link_san = (["-Xarch_host", "-fsanitize=address",
                 "-Xarch_host", "-fsanitize=undefined"] if host_sanitize else [])
    _run([hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}"] + link_san
         + ["-o", tmp] + objs + ["-Wl,-soname,libdpar.so"])
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    build()
    sys.exit(0)
