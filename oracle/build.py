"""Compile the fp64 CPU oracle (test infrastructure) into ``oracle/libspc_oracle.so``.

Plain C11 + OpenMP, built with the host gcc.  ``extra`` flags may add host
sanitizers, e.g. ``["-fsanitize=address,undefined"]`` for a debug build.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libspc_oracle.so")
SRC = os.path.join(HERE, "spc_oracle.c")


def build(out=LIB, extra=()):
    cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-fopenmp", "-Wall", "-Wextra",
           "-Werror", *extra, SRC, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build())
