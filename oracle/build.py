"""Build the fp64 oracle shared library (test infrastructure only).

``python -m oracle.build`` (or ``build()``) compiles ``oracle.c`` with the host
C compiler into ``oracle/liboracle.so``.  No GPU code is involved; no fast-math
flags are used, so every floating-point operation is the plain IEEE double one
the source spells out.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False, src: str = None, out: str = None, extra_flags=()) -> str:
    """extra_flags: more compiler flags (the sanitizer test builds an
    AddressSanitizer + UndefinedBehaviorSanitizer copy with them)."""
    src = src or os.path.join(HERE, "oracle.c")
    out = out or LIB
    tmp = out + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-fno-fast-math", "-ffp-contract=off", *extra_flags, "-o", tmp, src, "-lpthread", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
