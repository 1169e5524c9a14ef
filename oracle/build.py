"""Build the CPU oracle into ``oracle/liboracle.so`` with gcc.

Test infrastructure only (see ``oracle.c``). Plain C99, OpenMP, -O2 and no
fast-math flags, so double-precision arithmetic follows IEEE 754 in program
order.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "oracle.c")           # decode attention
SOURCES = [SOURCE, os.path.join(HERE, "append.c")]  # + KV append / E4M3 quantise-on-write
LIBRARY = os.path.join(HERE, "liboracle.so")

CFLAGS = ["-std=c99", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fPIC",
          "-shared", "-fopenmp", "-Wall", "-Wextra"]


# The host sanitizers, for a separate build of the oracle run under AddressSanitizer and
# UndefinedBehaviorSanitizer by the sanitizer test.
SANITIZE_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]


def build(sources: str | list[str] | None = None, output: str = LIBRARY,
          extra: list[str] | None = None) -> str:
    """Compile ``sources`` (default: every oracle source) into the shared library
    ``output`` and return its path."""
    if sources is None:
        sources = SOURCES
    elif isinstance(sources, str):
        sources = [sources]
    tmp = output + ".tmp%d" % os.getpid()
    cmd = ["gcc", *CFLAGS, *(extra or []), *sources, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, output)
    return output


if __name__ == "__main__":
    print(build(sys.argv[1:] or None))
