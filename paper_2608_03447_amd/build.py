"""Build ``libasd.so`` (the C-ABI verifier library) for gfx950 with hipcc.

The library is built in-tree next to this file.  Every HIP source is compiled
with packed FP32 instructions disabled and without FMA contraction, so the
binary32/binary64 operations of the verifier are exactly the ones written.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIBRARY = os.path.join(HERE, "libasd.so")
SOURCES = [os.path.join(CSRC, "asd_api.cpp"), os.path.join(CSRC, "asd_kernels.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-I" + os.path.join(ROOT, "include"),
]


def build_library(verbose: bool = False, output: str = LIBRARY, extra_flags=()) -> str:
    cmd = [HIPCC, *HIP_FLAGS, *extra_flags, "-shared", *SOURCES, "-o", output + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(output + ".tmp", output)
    return output


if __name__ == "__main__":
    print(build_library(verbose=True))
