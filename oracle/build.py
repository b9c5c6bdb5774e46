"""Builds the oracle's shared library with the host C compiler.

TEST INFRASTRUCTURE ONLY: the oracle is the slow CPU reference that the test
suite, the smoke check and the benchmark's CPU-baseline leg compare against.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "lethe_oracle.c")
LIB = os.path.join(HERE, "liblethe_oracle.so")


def build(force: bool = True) -> str:
    """Compile ``lethe_oracle.c`` into ``liblethe_oracle.so`` (fp-contract off,
    no fast-math, so every operation rounds as written)."""
    if not force and os.path.exists(LIB) and os.path.getmtime(LIB) >= os.path.getmtime(SRC):
        return LIB
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-o", tmp, SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
