"""Build the native parts of the package in-tree.

- ``libsynth.so``: the seeded input generator (gcc, OpenMP).
- ``librc.so``: the C-ABI library (host C++ compiled by hipcc, linked with
  the HIP runtime and hipRTC).  The gfx950 kernels are HIP sources embedded
  into the library as string literals and compiled per schedule by hipRTC at
  plan creation (cached on disk as code objects).
- ``precompile(...)``: compile a list of schedules' kernels ahead of time for
  gfx950 (no GPU needed), filling the code-object cache.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")


def gen_kernel_sources() -> str:
    out = os.path.join(CSRC, "kernels_src.inc")
    parts = ["// Generated from csrc/kernels/*.hip by build.py; do not edit.\n"]
    for path in sorted(glob.glob(os.path.join(CSRC, "kernels", "*.hip"))):
        name = os.path.splitext(os.path.basename(path))[0]
        text = open(path).read()
        assert ')RCK"' not in text
        parts.append(f'static const char SRC_{name}[] = R"RCK({text})RCK";\n')
    new = "".join(parts)
    if not os.path.exists(out) or open(out).read() != new:
        with open(out, "w") as f:
            f.write(new)
    return out


def build_static_object(verbose: bool = False) -> str:
    """rc_static.hip holds a file-scope device array (the no-allocation
    launch's workspace), so hipcc compiles it for gfx950 and the host."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    obj = os.path.join(HERE, "rc_static.o")
    cmd = [os.path.join(rocm, "bin", "hipcc"), "-c", "-fPIC", "-O2", "-std=c++17",
           "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, os.path.join(CSRC, "rc_static.hip"),
           "-o", obj]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    return obj


def build_lib(verbose: bool = False) -> str:
    gen_kernel_sources()
    lib = os.path.join(HERE, "librc.so")
    srcs = [os.path.join(CSRC, f) for f in ("rc_core.cpp", "rc_plan.cpp", "rc_search.cpp")]
    obj = build_static_object(verbose)
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    # Host C++: the operator kernels are compiled for gfx950 by hipRTC per
    # schedule; rc_static.o carries the static workspace array.
    cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-Wall", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-I", os.path.join(rocm, "include"),
           *srcs, obj, "-o", lib + ".tmp", "-L", os.path.join(rocm, "lib"),
           "-Wl,-rpath," + os.path.join(rocm, "lib"), "-lamdhip64", "-lhiprtc", "-ldl",
           "-lpthread"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(lib + ".tmp", lib)
    return lib


def build_synth() -> str:
    from . import inputs
    return inputs.build_synth()


def build_all(verbose: bool = False) -> None:
    build_synth()
    build_lib(verbose)


if __name__ == "__main__":
    sys.path.insert(0, ROOT)
    build_all(verbose=True)
