"""Build libflowpool.so for gfx950 with hipcc, in-tree next to this file."""

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libflowpool.so")
SOURCES = [os.path.join(HERE, "csrc", f) for f in ("pool.hip", "kernels.hip", "schedule.cpp", "allocate.cpp")]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-result",
    # keep the compiler from emitting packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # the pack kernel's eleven leading scalar arguments arrive preloaded in
    # scalar registers (the hardware fills them at wave launch)
    "-mllvm", "-amdgpu-kernarg-preload-count=11",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build(verbose: bool = False) -> str:
    """Compile the library (always, even if a built copy exists)."""
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(HERE, "csrc"), *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed with status {r.returncode}")
    os.replace(tmp, LIB)
    return LIB


DRIVER_SRC = os.path.join(ROOT, "tests", "c_abi", "pack_driver.c")
DRIVER = os.path.join(ROOT, "tests", "c_abi", "pack_driver")


def build_driver(verbose: bool = False) -> str:
    """Compile the plain-C test driver of the C ABI (host code only, gcc),
    linked against the in-tree library and the HIP runtime."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    tmp = DRIVER + ".tmp"
    # The HIP runtime header, included by plain C through gcc rather than
    # hipcc, needs its platform macro defined by the compiler line; the
    # driver itself has one code path.
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(rocm, "include"),
           DRIVER_SRC, "-o", tmp, "-L", HERE, "-lflowpool", "-L", os.path.join(rocm, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2606_23087_amd", "-Wl,-rpath," + os.path.join(rocm, "lib")]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"gcc failed with status {r.returncode}")
    os.replace(tmp, DRIVER)
    return DRIVER


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_driver(verbose=True))
