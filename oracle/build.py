"""Build step for the CPU oracle (test infrastructure): compiles
``sbvr_oracle.c`` with gcc into ``oracle/_build/libsbvr_oracle.so``.

Strict IEEE binary64: no fast-math, no floating-point contraction."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "sbvr_oracle.c")


def library_path() -> str:
    return os.path.join(HERE, "_build", "libsbvr_oracle.so")


def build() -> str:
    out = library_path()
    os.makedirs(os.path.dirname(out), exist_ok=True)
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-D_POSIX_C_SOURCE=200809L",
           "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra", "-Werror",
           SRC, "-o", tmp, "-lm", "-lpthread"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build())
