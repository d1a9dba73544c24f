"""Compile the float64 C oracle with gcc (test infrastructure only)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "crf_oracle.c")
LIB = os.path.join(HERE, "libcrforacle.so")


def build(force: bool = True) -> str:
    """Build ``libcrforacle.so`` next to the source and return its path.

    ``-ffp-contract=off`` keeps every multiply and add a separately rounded
    IEEE operation, so the CKY chart is bit-reproducible.
    """
    if not force and os.path.exists(LIB) and os.path.getmtime(LIB) >= os.path.getmtime(SRC):
        return LIB
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-Wextra", "-o", tmp, SRC, "-lm", "-lpthread"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
