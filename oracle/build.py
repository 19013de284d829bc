"""Compile the C oracle into ``oracle/libqmlp_oracle.so`` with gcc.

No FMA contraction and no fast-math, so every fp64 operation is one IEEE
rounding.  Building the checker is not using it: the top-level ``build()`` entry point
compiles it alongside the HIP library.
"""
import os
import subprocess
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))


def build() -> str:
    src = os.path.join(_HERE, "qmlp_oracle.c")
    out = os.path.join(_HERE, "libqmlp_oracle.so")
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-o", tmp, src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(), file=sys.stderr)
