"""Build the reference oracle (test infrastructure) into oracle/libnfo.so.

Plain g++, single-threaded code, no contraction of multiply-adds, no fast-math.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libnfo.so")


def build(out=LIB, src=None, extra=()):
    """Compile the oracle; `src` and `extra` let a test build a variant copy."""
    src = src or os.path.join(HERE, "nfo.cpp")
    inc = os.path.dirname(os.path.abspath(src))
    cmd = ["g++", "-std=c++14", "-O2", "-fPIC", "-shared", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-Wextra", "-I", inc, src, "-o", out + ".tmp",
           *extra]
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build())
