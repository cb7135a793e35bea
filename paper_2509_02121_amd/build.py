"""Build libhalo_attn.so (gfx950) in-tree with hipcc.

    python -m paper_2509_02121_amd.build          # or build() from Python

The planner is plain host C++ (g++); the kernels and run-time entry points
are HIP compiled for gfx950 only. Every build recompiles from source.
"""

import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libhalo_attn.so"
LIB_PATH = os.path.join(PKG, LIB_NAME)
# Context microbenchmarks (measurement only), a library of their own.
PROBE_LIB_PATH = os.path.join(PKG, "libhalo_probe.so")
DRIVER_SRC = os.path.join(ROOT, "tests", "abi_driver", "decode.cpp")
DRIVER_BIN = os.path.join(ROOT, "tests", "abi_driver", "decode")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 VALU forms stay off: the kernels are written for scalar fp32
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # no kernel tests for NaN: masked scores are replaced by selects, tail V
    # slots by bit masks, and the gather copies integers, so max reductions
    # can skip the NaN-quieting operand canonicalization
    "-fno-honor-nans",
    "-Wall", "-Wno-unused-function",
]


def _run(cmd):
    print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)


def build(verbose=True):
    """Compile every source and link the shared library next to this file."""
    tmp = tempfile.mkdtemp(prefix="halo_build_")
    try:
        plan_o = os.path.join(tmp, "halo_plan.o")
        forest_o = os.path.join(tmp, "halo_forest.o")
        kern_o = os.path.join(tmp, "halo_kernels.o")
        pages_o = os.path.join(tmp, "halo_pages.o")
        probe_o = os.path.join(tmp, "halo_probe.o")
        procs = [
            subprocess.Popen(["g++", "-std=c++17", "-O2", "-fPIC", "-Wall", "-Wextra",
                              "-I", INCLUDE, "-c", os.path.join(CSRC, "halo_plan.cpp"), "-o", plan_o]),
            subprocess.Popen(["g++", "-std=c++17", "-O2", "-fPIC", "-Wall", "-Wextra",
                              "-I", INCLUDE, "-c", os.path.join(CSRC, "halo_forest.cpp"), "-o", forest_o]),
            subprocess.Popen([HIPCC] + HIP_FLAGS + ["-I", INCLUDE, "-c",
                                                   os.path.join(CSRC, "halo_kernels.hip"), "-o", kern_o]),
            subprocess.Popen([HIPCC] + HIP_FLAGS + ["-I", INCLUDE, "-c",
                                                   os.path.join(CSRC, "halo_pages.hip"), "-o", pages_o]),
            subprocess.Popen([HIPCC] + HIP_FLAGS + ["-I", INCLUDE, "-c",
                                                   os.path.join(CSRC, "halo_probe.hip"), "-o", probe_o]),
        ]
        rcs = [p.wait() for p in procs]
        if any(rcs):
            raise RuntimeError(f"compilation failed (exit codes {rcs})")
        out_tmp = LIB_PATH + ".tmp"
        _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", plan_o, forest_o, kern_o, pages_o, "-o", out_tmp])
        os.replace(out_tmp, LIB_PATH)
        probe_tmp = PROBE_LIB_PATH + ".tmp"
        _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", probe_o, "-o", probe_tmp])
        os.replace(probe_tmp, PROBE_LIB_PATH)
        # the C-ABI driver of the tests (host code against the built library)
        _run(["g++", "-std=c++17", "-O2", "-Wall", "-D__HIP_PLATFORM_AMD__", "-I", INCLUDE,
              "-I", "/opt/rocm/include", DRIVER_SRC, "-o", DRIVER_BIN, "-L", PKG, "-lhalo_attn",
              "-L", "/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,$ORIGIN/../../paper_2509_02121_amd",
              "-Wl,-rpath,/opt/rocm/lib"])
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return LIB_PATH


if __name__ == "__main__":
    sys.exit(0 if build() else 1)
