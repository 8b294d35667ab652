"""Build ``libasd.so`` (the C-ABI verifier library) for gfx950 with hipcc.

The library is built in-tree next to this file.  Every HIP source is compiled
with packed FP32 instructions disabled and without FMA contraction, so the
binary32/binary64 operations of the verifier are exactly the ones written.

The build embeds a hash of the sources it compiled in ``asd_version()``; the
binding refuses a library whose hash differs from the sources beside it, so a
stale build is never tested, benchmarked or smoke-checked by mistake.
"""
import hashlib
import os
import re
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIBRARY = os.path.join(HERE, "libasd.so")
SOURCES = [os.path.join(CSRC, "asd_api.cpp"), os.path.join(CSRC, "asd_kernels.hip")]
# Every file whose code goes into the library (sources and headers).
HASHED_SOURCES = [os.path.join(CSRC, "asd_kernels.hip"), os.path.join(CSRC, "asd_plan.h"),
                  os.path.join(CSRC, "asd_api.cpp"), os.path.join(ROOT, "include", "asd.h")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-I" + os.path.join(ROOT, "include"),
]


def source_hash(paths=None) -> str:
    """SHA-256 (first 16 hex digits) of the library's sources with comments and
    whitespace removed: an edit to a comment keeps the hash, any code edit
    changes it."""
    h = hashlib.sha256()
    for p in (HASHED_SOURCES if paths is None else paths):
        with open(p) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def build_library(verbose: bool = False, output: str = LIBRARY, extra_flags=()) -> str:
    tag = '-DASD_SOURCE_HASH="%s"' % source_hash()
    cmd = [HIPCC, *HIP_FLAGS, tag, *extra_flags, "-shared", *SOURCES, "-o", output + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(output + ".tmp", output)
    return output


if __name__ == "__main__":
    print(build_library(verbose=True))
