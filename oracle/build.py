"""Build the CPU oracle (plain C, gcc) into ``oracle/liboracle.so``.

Test infrastructure: the oracle is compiled without fast-math or FMA
contraction so that every binary32/binary64 operation it states is the one
executed.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "asd_oracle.c")
LIBRARY = os.path.join(HERE, "liboracle.so")


def build_oracle(verbose: bool = False) -> str:
    cmd = [
        "gcc", "-std=c99", "-O2", "-fPIC", "-shared",
        "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
        SOURCE, "-o", LIBRARY + ".tmp", "-lm",
    ]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIBRARY + ".tmp", LIBRARY)
    return LIBRARY


if __name__ == "__main__":
    print(build_oracle(verbose=True))
