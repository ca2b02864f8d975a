"""Build the CPU oracle's shared library with gcc (test infrastructure only)."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "tq_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

# -ffp-contract=off: the quantizer's multiply must round on its own (no fused
# multiply-add); no -ffast-math anywhere.
# -fopenmp: orc_gemv's row loop may run on several threads (whole rows per thread, the
# same arithmetic per row).
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
          "-Wall", "-Wextra", "-Werror"]


def build(src: str = SRC, out: str = LIB, werror: bool = True) -> str:
    flags = CFLAGS if werror else [f for f in CFLAGS if f != "-Werror"]
    cmd = ["gcc", *flags, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(*sys.argv[1:]))
