"""Build libfate.so (HIP kernels for gfx950 + host packer + C ABI) in-tree.

``python -m paper_2605_07238_amd.build`` compiles the library next to this
file with hipcc.  Packed fp32 instructions are disabled for the device code
(``-target-feature -packed-fp32-ops``); the host pass may warn that it does
not know that feature.
"""

from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libfate.so")
SOURCES = [os.path.join(CSRC, "fate_host.cpp"), os.path.join(CSRC, "fate_kernels.hip"),
           os.path.join(CSRC, "fate_commit.hip"), os.path.join(CSRC, "fate_plan.hip"),
           os.path.join(CSRC, "fate_sim.cpp"), os.path.join(CSRC, "fate_simdev.hip")]
ARCH = os.environ.get("FATE_OFFLOAD_ARCH", "gfx950")


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.sep not in cand or os.path.exists(cand)):
            return cand
    return "hipcc"


COMMON = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# The kernels never produce NaN (inputs are validated finite; +inf is only a
# sentinel), so min/max need no NaN quieting.  Host validation relies on
# isfinite() and is compiled without this flag.
KERNEL_FLAGS = ["-fno-honor-nans"]


def commands(out: str = LIB, objdir: str = None) -> list:
    objdir = objdir or os.path.join(HERE, "_build")
    host_o = os.path.join(objdir, "fate_host.o")
    kern_o = os.path.join(objdir, "fate_kernels.o")
    commit_o = os.path.join(objdir, "fate_commit.o")
    plan_o = os.path.join(objdir, "fate_plan.o")
    sim_o = os.path.join(objdir, "fate_sim.o")
    simdev_o = os.path.join(objdir, "fate_simdev.o")
    inc = ["-I", INCLUDE, "-I", CSRC]
    return [
        [hipcc(), *COMMON, *inc, "-c", SOURCES[0], "-o", host_o],
        [hipcc(), *COMMON, *KERNEL_FLAGS, *inc, "-c", SOURCES[1], "-o", kern_o],
        [hipcc(), *COMMON, *KERNEL_FLAGS, *inc, "-c", SOURCES[2], "-o", commit_o],
        [hipcc(), *COMMON, *KERNEL_FLAGS, *inc, "-c", SOURCES[3], "-o", plan_o],
        [hipcc(), *COMMON, *inc, "-c", SOURCES[4], "-o", sim_o],
        [hipcc(), *COMMON, *KERNEL_FLAGS, *inc, "-c", SOURCES[5], "-o", simdev_o],
        [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", host_o, kern_o, commit_o, plan_o, sim_o, simdev_o,
         "-o", out, "-lpthread"],
    ]


def build(verbose: bool = False) -> str:
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    tmp = LIB + ".tmp%d" % os.getpid()
    for cmd in commands(tmp, objdir):
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


SAN_DIR = os.path.join(HERE, "_build_san")
SAN_LIB = os.path.join(SAN_DIR, "libfate_san.so")


def build_sanitized(verbose: bool = False) -> str:
    """The library with its host code (packer, layouts, plan execution)
    built with clang's AddressSanitizer and UndefinedBehaviorSanitizer, for
    CPU test runs with the runtime preloaded; the device code is built as
    usual (no sanitizer reaches the GPU code)."""
    os.makedirs(SAN_DIR, exist_ok=True)
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host",
           "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]
    inc = ["-I", INCLUDE, "-I", CSRC]
    objs = []
    for src in SOURCES:
        obj = os.path.join(SAN_DIR, os.path.basename(src) + ".o")
        host_only = src.endswith(".cpp")
        cmd = [hipcc(), *COMMON, *([] if host_only else KERNEL_FLAGS), *(san if host_only else []), *inc, "-c", src,
               "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        objs.append(obj)
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-shared-libasan", "-Xarch_host", "-fsanitize=address",
           "-Xarch_host", "-fsanitize=undefined", *objs, "-o", SAN_LIB, "-lpthread"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return SAN_LIB


if __name__ == "__main__":
    if "--sanitize" in sys.argv:
        print(build_sanitized(verbose=True))
    else:
        build(verbose=True)
        print(LIB)
    sys.exit(0)
